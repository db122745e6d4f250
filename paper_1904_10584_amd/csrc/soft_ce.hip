// Sparse soft-target cross-entropy (student-teacher training against the
// teacher's k-best posteriors), HBM-bound.
//
// One wave per frame row: the row of logits is read once with 16-byte loads
// issued back to back and kept in registers (up to 8192 classes), max and
// sum-of-exponentials are
// wave reductions, the k teacher logits are read with wave-uniform loads, and
// the gradient row  s (M softmax(z) - scatter(p))  is written once.  The
// teacher terms reach the lanes that hold their classes through a small LDS
// scratch per wave (one 256-class chunk at a time).  Row losses
// are summed per block in a fixed order, then over blocks by a single block,
// so the loss is deterministic.
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int ROWS_PER_BLOCK = 4;  // one per wave

template <typename DT> __device__ __forceinline__ void store4(DT* p, float4 v);
template <> __device__ __forceinline__ void store4<float>(float* p, float4 v) {
  *reinterpret_cast<float4*>(p) = v;
}
template <> __device__ __forceinline__ void store4<bf16_t>(bf16_t* p, float4 v) {
  uint2 w;
  w.x = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
  w.y = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = w;
}

template <int NCH, typename DT>
__global__ __launch_bounds__(256) void soft_ce_rows(
    int64_t N, int C, int K, const float* __restrict__ z, const int32_t* __restrict__ idx,
    const float* __restrict__ prob, const uint8_t* __restrict__ mask,
    const float* __restrict__ scale_dev, float scale_host, DT* __restrict__ dz,
    float* __restrict__ partials) {
  __shared__ float wl[ROWS_PER_BLOCK];
  __shared__ __align__(16) float corr[ROWS_PER_BLOCK][256];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t f = (int64_t)blockIdx.x * ROWS_PER_BLOCK + wave;
  float row_loss = 0.f;

  if (f < N) {
    const float* zr = z + f * C;
    DT* dr = dz + f * C;
    // with a mask, the row's mask byte first: a masked row's logits are
    // never read (without one, no dependent load precedes the row)
    const float m = mask ? (mask[f] != 0 ? 1.f : 0.f) : 1.f;
    // the row, 16-byte loads issued back to back (a lane past C re-reads
    // the row's start; its values are replaced below), so that the row
    // costs one memory latency, not one per chunk
    float4 v[NCH];
    if (m != 0.f) {
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = i * 256 + lane * 4;
        v[i] = *reinterpret_cast<const float4*>(zr + (c < C ? c : 0));
      }
    }
    // teacher entries: lane j holds entry j (K <= 64 per pass)
    const int32_t* ir = idx + f * K;
    const float* pr = prob + f * K;
    int tc = -1;
    float tp = 0.f;
    if (lane < K) {
      tc = ir[lane];
      tp = pr[lane];
    }
    const float s = m * (scale_dev ? *scale_dev : scale_host);
    if (s == 0.f) {
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = i * 256 + lane * 4;
        if (c < C) store4<DT>(dr + c, make_float4(0.f, 0.f, 0.f, 0.f));
      }
    } else {
      // each entry's own logit (a lane's slot past K, an empty slot or an
      // out-of-range index reads the row's first logit and is dropped);
      // issued before the reductions below, which hide its latency
      const bool tok = tc >= 0 && tc < C;
      float tz = zr[tok ? tc : 0];
      asm volatile("" ::: "memory");  // keep the load here, ahead of its use
      if (!tok) { tc = -1; tp = 0.f; }
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        if (i * 256 + lane * 4 >= C) v[i] = make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        mx = fmaxf(mx, fmaxf(fmaxf(v[i].x, v[i].y), fmaxf(v[i].z, v[i].w)));
      }
      mx = wave_max(mx);
      // e = exp(z - max) kept in place of the row (0 past C)
      float se = 0.f;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        v[i].x = __expf(v[i].x - mx);
        v[i].y = __expf(v[i].y - mx);
        v[i].z = __expf(v[i].z - mx);
        v[i].w = __expf(v[i].w - mx);
        se += (v[i].x + v[i].y) + (v[i].z + v[i].w);
      }
      se = wave_sum(se);
      const float lse = mx + __logf(se);

      float mass = tp, lf = tc >= 0 ? -tp * (tz - lse) : 0.f;
      for (int j0 = 64; j0 < K; j0 += 64) {  // more than 64 entries per frame
        const int j = j0 + lane;
        if (j < K) {
          const int c = ir[j];
          if (c >= 0 && c < C) {
            mass += pr[j];
            lf -= pr[j] * (zr[c] - lse);
          }
        }
      }
      mass = wave_sum(mass);
      lf = wave_sum(lf);
      // s M softmax(z) = e (s M / sum e)
      const float sm = s * mass / se;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        v[i].x *= sm;
        v[i].y *= sm;
        v[i].z *= sm;
        v[i].w *= sm;
      }
      // Entries 0-63 (one per lane): s p_j comes off the slot of class c_j
      // through a 1 KiB LDS scratch of the wave, one 256-class chunk at a
      // time: zeroed, each entry lane adds its term at its class (an LDS
      // atomic add, so that repeated classes sum), every lane reads its four
      // slots back.  A wave's LDS operations run in order, so no barrier is
      // needed; the chunks' operations issue back to back.
      {
        float* cw = corr[wave];
        const float dj = tc >= 0 ? s * tp : 0.f;
        const int tch = tc >= 0 ? tc >> 8 : -1, tslot = tc & 255;
        float4 cv[NCH];
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
          reinterpret_cast<float4*>(cw)[lane] = make_float4(0.f, 0.f, 0.f, 0.f);
          __builtin_amdgcn_wave_barrier();
          if (tch == i) atomicAdd(cw + tslot, dj);
          __builtin_amdgcn_wave_barrier();
          cv[i] = reinterpret_cast<const float4*>(cw)[lane];
          __builtin_amdgcn_wave_barrier();
        }
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
          v[i].x -= cv[i].x;
          v[i].y -= cv[i].y;
          v[i].z -= cv[i].z;
          v[i].w -= cv[i].w;
        }
      }
      // entries past the 64th (K > 64), one at a time
      for (int jj = 64; jj < K; ++jj) {
        int c = ir[jj];
        const float p = pr[jj];
        if (c >= C) c = -1;
        if (c < 0) continue;
        const int owner = (c & 255) >> 2, cc = c & 3;
        const float d = lane == owner ? s * p : 0.f;
        // v[c / 256] component cc -= d, the chunk chosen with uniform tests
        // on its group of four, then within the group (an index into the
        // register array computed at run time would put it in scratch)
        const int ci = c >> 8;
#pragma unroll
        for (int g = 0; g < (NCH + 3) / 4; ++g) {
          if (g == (ci >> 2)) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if (4 * g + k < NCH && k == (ci & 3)) {
                v[4 * g + k].x -= cc == 0 ? d : 0.f;
                v[4 * g + k].y -= cc == 1 ? d : 0.f;
                v[4 * g + k].z -= cc == 2 ? d : 0.f;
                v[4 * g + k].w -= cc == 3 ? d : 0.f;
              }
            }
          }
        }
      }
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = i * 256 + lane * 4;
        if (c < C) store4<DT>(dr + c, v[i]);
      }
      row_loss = s * lf;
    }
  }
  if (lane == 0) wl[wave] = row_loss;
  __syncthreads();
  if (threadIdx.x == 0) partials[blockIdx.x] = ((wl[0] + wl[1]) + wl[2]) + wl[3];
}

// Fixed-order sum of the per-block losses: thread x adds elements x, x + 256,
// ... in that order, then a tree over the threads.  The loads of a batch of
// 16 are issued before its adds, so that a thread waits for memory once per
// batch rather than once per element.
__global__ __launch_bounds__(256) void sum_partials(const float* __restrict__ partials, int64_t n,
                                                    float* __restrict__ out) {
  __shared__ float red[256];
  float acc = 0.f;
  for (int64_t b = 0; b < n; b += 16 * 256) {
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int64_t i = b + (int64_t)k * 256 + threadIdx.x;
      v[k] = i < n ? partials[i] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (b + (int64_t)k * 256 + threadIdx.x < n) acc += v[k];
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

// 1 / (number of rows with a nonzero mask), 0 if there are none.
__global__ __launch_bounds__(256) void mask_scale(const uint8_t* __restrict__ mask, int64_t n,
                                                  float* __restrict__ out) {
  __shared__ int64_t red[256];
  int64_t cnt = 0;
  for (int64_t i = threadIdx.x; i < n; i += 256) cnt += mask[i] != 0;
  red[threadIdx.x] = cnt;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0] > 0 ? 1.0f / (float)red[0] : 0.f;
}

template <int NCH, typename DT>
void launch_rows(const SoftCeArgs& a, const float* scale_dev, float scale_host, hipStream_t s) {
  const int64_t blocks = (a.N + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK;
  hipLaunchKernelGGL((soft_ce_rows<NCH, DT>), dim3((unsigned)blocks), dim3(256), 0, s, a.N, a.C,
                     a.K, a.z, a.idx, a.prob, a.mask, scale_dev, scale_host,
                     static_cast<DT*>(a.dz), a.ws_partials);
}

template <typename DT>
hipError_t dispatch_rows(const SoftCeArgs& a, const float* sd, float sh, hipStream_t s) {
  const int nch = (a.C + 255) / 256;
  if (nch <= 2) launch_rows<2, DT>(a, sd, sh, s);
  else if (nch <= 4) launch_rows<4, DT>(a, sd, sh, s);
  else if (nch <= 8) launch_rows<8, DT>(a, sd, sh, s);
  else if (nch <= 12) launch_rows<12, DT>(a, sd, sh, s);
  else if (nch <= 16) launch_rows<16, DT>(a, sd, sh, s);
  else if (nch <= 24) launch_rows<24, DT>(a, sd, sh, s);
  else if (nch <= 32) launch_rows<32, DT>(a, sd, sh, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

int64_t soft_ce_partials(int64_t N) { return (N + ROWS_PER_BLOCK - 1) / ROWS_PER_BLOCK; }

hipError_t soft_ce(const SoftCeArgs& a, hipStream_t s) {
  const float* sd = nullptr;
  float sh = 1.f;
  if (a.reduction == 0) {  // mean over valid rows
    if (a.mask) {
      hipLaunchKernelGGL(mask_scale, dim3(1), dim3(256), 0, s, a.mask, a.N, a.ws_scale);
      sd = a.ws_scale;
    } else {
      sh = a.N > 0 ? 1.0f / (float)a.N : 0.f;
    }
  }
  hipError_t e = hipSuccess;
  if (a.N > 0) {
    e = a.dz_bf16 ? dispatch_rows<bf16_t>(a, sd, sh, s) : dispatch_rows<float>(a, sd, sh, s);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(sum_partials, dim3(1), dim3(256), 0, s, a.ws_partials, a.n_partials, a.loss);
  return hipGetLastError();
}

}  // namespace am
