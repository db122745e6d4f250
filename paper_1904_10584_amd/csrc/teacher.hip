// Teacher target generation (§V-A, §V-C): the pieces the bidirectional
// teacher adds to the student's kernels, and the k-best logits.
//
// gather_rows: copies the packed rows of a batch, optionally reversing each
// sequence in time (row (t, b) takes row (len_b - 1 - t, b)), into a column
// range of another matrix.  The teacher's backward direction runs the
// student's forward recurrence on the time-reversed input projections and
// writes its hidden states back in time order next to the forward
// direction's.  One thread per 16-byte chunk; a row's frame index comes from
// a binary search in the packed row offsets.
//
// topk_rows: the k largest logits of each row in descending order (equal
// values by ascending index, NaN after every number), one wave per row with
// the row held in registers as order-preserving integer keys.  Each lane
// finds its best two entries in one pass; each of the k rounds takes the
// wave-wide best of the lanes' current entries, and the lane that held it
// moves to its next: the second from the pass, then each time a scan for
// its best entry below the one taken.
//
// kbest_posterior_rows: the posterior rebuilt from k stored logits with the
// missing ones at -infinity, i.e. the softmax over the k values (fp32).
#include <cmath>

#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

// Device copies of a batch's schedule: offs[t] = sum_b min(len_b, t) for
// t = 0..T, and the lengths.
__global__ __launch_bounds__(256) void schedule_tables_kernel(SchedTables a) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t <= a.T) {
    int64_t o = 0;
    for (int b = 0; b < a.B; ++b) o += a.len[b] < t ? a.len[b] : t;
    a.offs[t] = o;
  }
  if (t < a.B) a.lens[t] = a.len[t];
}

template <typename T>
__global__ __launch_bounds__(256) void gather_rows_kernel(GatherRows a) {
  constexpr int EPC = 16 / sizeof(T);
  const int cpr = a.width / EPC;
  const int64_t total = a.N * cpr;
  const T* __restrict__ src = static_cast<const T*>(a.src);
  T* __restrict__ dst = static_cast<T*>(a.dst);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / cpr;
    const int c = (int)(e % cpr);
    int64_t sr = r;
    if (a.reverse) {
      // frame t of row r: the last t with offs[t] <= r
      int lo = 0, hi = a.T - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.offs[mid] <= r) lo = mid; else hi = mid - 1;
      }
      const int b = (int)(r - a.offs[lo]);
      sr = a.offs[a.lens[b] - 1 - lo] + b;
    }
    const uint4 v = *reinterpret_cast<const uint4*>(src + sr * a.src_ld + c * EPC);
    *reinterpret_cast<uint4*>(dst + r * a.dst_ld + a.dst_col + c * EPC) = v;
  }
}

// Order-preserving key of a logit: larger values get larger keys, -0 and +0
// the same key, NaN key 1 (below every number), and 0 marks an entry already
// taken.  A wave-wide candidate is (key << 32) | ~index, so equal keys rank
// the lower index first.
__device__ __forceinline__ uint32_t logit_key(float f) {
  if (f != f) return 1u;
  uint32_t u = __float_as_uint(f == 0.f ? 0.f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int CPL, bool VEC>
__global__ __launch_bounds__(256) void topk_rows_kernel(int64_t N, int C, int K,
                                                        const float* __restrict__ z,
                                                        int32_t* __restrict__ idx,
                                                        float* __restrict__ val) {
  static_assert(CPL % 4 == 0, "registers in fours");
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const float* zr = z + row * C;
  // register q holds class cls(q): with VEC (C % 4 == 0) four consecutive
  // classes per 16-byte load, else one class per 64-lane stride
  auto cls = [&](int q) {
    return VEC ? 4 * lane + 256 * (q >> 2) + (q & 3) : lane + 64 * q;
  };
  uint32_t key[CPL];
#pragma unroll
  for (int q4 = 0; q4 < CPL / 4; ++q4) {
    if (VEC) {
      const int c = 4 * lane + 256 * q4;
      const float4 f = c < C ? *reinterpret_cast<const float4*>(zr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      key[4 * q4 + 0] = c < C ? logit_key(f.x) : 0u;
      key[4 * q4 + 1] = c < C ? logit_key(f.y) : 0u;
      key[4 * q4 + 2] = c < C ? logit_key(f.z) : 0u;
      key[4 * q4 + 3] = c < C ? logit_key(f.w) : 0u;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int c = cls(4 * q4 + e);
        key[4 * q4 + e] = c < C ? logit_key(zr[c]) : 0u;
      }
    }
  }
  // candidate of register q: (key << 32) | ~class, unique per class, larger
  // = earlier in the output; 0 for no class
  auto cand = [&](int q) -> uint64_t {
    return key[q] ? ((uint64_t)key[q] << 32) | (uint32_t)~(uint32_t)cls(q) : 0ull;
  };
  // this lane's best two candidates, from one pass over its registers
  uint64_t b0 = 0ull, b1 = 0ull;
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const uint64_t v = cand(q);
    const bool g0 = v > b0, g1 = v > b1;
    b1 = g0 ? b0 : (g1 ? v : b1);
    b0 = g0 ? v : b0;
  }
  bool second = true;  // b1 still holds this lane's next candidate
  int mine = -1;       // lane j keeps the class of round j
  for (int j = 0; j < K; ++j) {
    uint64_t best = b0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const uint64_t other = __shfl_xor(best, o, 64);
      best = other > best ? other : best;
    }
    if (best == 0ull) continue;  // fewer than K entries: -1 below
    if (lane == j) mine = (int)~(uint32_t)best;
    if (b0 == best) {  // the lane that held it takes its next candidate
      if (second) {
        b0 = b1;
        second = false;
      } else {  // the best of its candidates below the one taken
        uint64_t m = 0ull;
#pragma unroll
        for (int q = 0; q < CPL; ++q) {
          const uint64_t v = cand(q);
          m = (v < best && v > m) ? v : m;
        }
        b0 = m;
      }
    }
  }
  // the k results, one lane each (values reloaded from the row: exact,
  // signed zeros and NaN payloads included)
  if (lane < K) {
    idx[row * K + lane] = mine;
    val[row * K + lane] = mine >= 0 ? zr[mine] : -INFINITY;
  }
}

__global__ __launch_bounds__(256) void kbest_posterior_rows(int64_t N, int K,
                                                            const float* __restrict__ val,
                                                            float* __restrict__ prob) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= N) return;
  const float* v = val + row * K;
  float m = -INFINITY;
  for (int j = 0; j < K; ++j) m = fmaxf(m, v[j]);
  float s = 0.f;
  for (int j = 0; j < K; ++j) s += expf(v[j] - m);
  for (int j = 0; j < K; ++j) prob[row * K + j] = expf(v[j] - m) / s;
}

}  // namespace

hipError_t schedule_tables(const SchedTables& a, hipStream_t s) {
  const int n = (a.T + 1 > a.B ? a.T + 1 : a.B);
  hipLaunchKernelGGL(schedule_tables_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t gather_rows(const GatherRows& a, bool bf16, hipStream_t s) {
  const int epc = bf16 ? 8 : 4;
  const int64_t total = a.N * (a.width / epc);
  if (total == 0) return hipSuccess;
  const int64_t want = (total + 255) / 256;
  const unsigned grid = (unsigned)(want < 65536 ? want : 65536);
  if (bf16)
    hipLaunchKernelGGL(gather_rows_kernel<bf16_t>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(gather_rows_kernel<float>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

#define AM_TOPK_CASE(CPL_)                                                                    \
  if (cpl <= CPL_) {                                                                          \
    if (vec)                                                                                  \
      hipLaunchKernelGGL((topk_rows_kernel<CPL_, true>), dim3((unsigned)((N + 3) / 4)),        \
                         dim3(256), 0, s, N, C, K, z, idx, val);                               \
    else                                                                                      \
      hipLaunchKernelGGL((topk_rows_kernel<CPL_, false>), dim3((unsigned)((N + 3) / 4)),       \
                         dim3(256), 0, s, N, C, K, z, idx, val);                               \
    return hipGetLastError();                                                                 \
  }

hipError_t topk_rows(int64_t N, int C, int K, const float* z, int32_t* idx, float* val,
                     hipStream_t s) {
  if (N == 0 || K == 0) return hipSuccess;
  const int cpl = (C + 63) / 64;
  // 16-byte row loads need every row start 16-byte aligned
  const bool vec = C % 4 == 0 && (reinterpret_cast<uintptr_t>(z) & 15) == 0;
  AM_TOPK_CASE(16) AM_TOPK_CASE(32) AM_TOPK_CASE(48) AM_TOPK_CASE(64) AM_TOPK_CASE(96)
  AM_TOPK_CASE(128)
  return hipErrorInvalidValue;
}

hipError_t kbest_posteriors(int64_t N, int K, const float* val, float* prob, hipStream_t s) {
  if (N == 0 || K == 0) return hipSuccess;
  hipLaunchKernelGGL(kbest_posterior_rows, dim3((unsigned)((N + 255) / 256)), dim3(256), 0, s, N,
                     K, val, prob);
  return hipGetLastError();
}

}  // namespace am
