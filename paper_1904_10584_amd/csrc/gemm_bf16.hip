// bf16 MFMA GEMM for gfx950: the batched products of the training step.
//   forward projections  P = X Wx^T + b,  Z = H Wo^T + bo      (A, B k-major)
//   data gradients       dH = dZ Wo,  dX = dA Wx              (B n-major)
//   weight gradients     [dWx | dWh] = dA^T [X | Hs],  dWo = dZ^T H
//                                                  (A m-major, B n-major)
// Each operand tile is copied to LDS in its global layout with 16-byte
// loads and stores; no operand is transposed in registers:
//   * a k-major tile is [rows][64 k] (128 B per row); the fragment of a
//     16x16x32 MFMA (8 consecutive k of one row per lane) is one 16-byte LDS
//     read;
//   * an m/n-major tile is [64 k][rows]; the fragment is read with two
//     gfx950 transposing LDS reads (ds_read_b64_tr_b16).  Within each group
//     of 16 lanes, lane i receives element i % 4 of the 4-element pieces
//     addressed by lanes 4q + i / 4 (q = 0..3); so when lane j of the group
//     addresses k-row k0 + j / 4 at column c0 + 4 (j % 4), lane i receives
//     column c0 + i at k-rows k0 .. k0 + 3.
// Both layouts XOR-swizzle their 16-byte chunks so that the fragment reads
// and the tile stores are free of LDS bank conflicts.
// One 256-thread workgroup computes a 128x128 tile (four waves of 64x64 as
// 4x4 MFMA tiles); the global loads of k-tile t+2 are in flight while tile t
// is multiplied (two register stages, two LDS stages).
// Workgroups are dispatched to the 8 XCDs round-robin; the tile order gives
// each XCD a contiguous range of tiles, so tiles that share operand rows
// share an L2.
// Weight gradients split K over workgroups (fp32 partial tiles, summed in
// split order by splitk_reduce in gemm.hip) and, for an m-major A, also
// produce the row sums of A over each split (the bias gradient).
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int TB = 128;   // tile rows and columns
constexpr int BK = 64;    // k per tile
constexpr int NT = 256;   // threads per workgroup
constexpr int NX = 8;     // XCDs

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// Element offset of chunk c (8 bf16) of row r in a k-major tile.
__device__ __forceinline__ int kofs(int r, int c) { return r * BK + ((c ^ (r & 7)) << 3); }
// Element offset of chunk c of k-row k in an m/n-major tile of TB columns.
__device__ __forceinline__ int mofs(int k, int c) { return k * TB + ((c ^ ((k & 3) << 1)) << 3); }

// One operand: rows (of the tile dimension) below `split` come from p0, the
// others from p1 at row - split.
struct Op {
  const bf16_t* p0; int64_t ld0;
  const bf16_t* p1; int64_t ld1;
  int split;
};

// Global -> register stage of one operand tile: 4 chunks per thread.
template <bool KMAJOR, bool SUM> struct Stage {
  uint4 v[4];
  __device__ __forceinline__ void load(const Op& o, int row0, int nrows, int k0, int kend) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int idx = threadIdx.x + NT * j;
      int r, k;
      if (KMAJOR) { r = idx >> 3; k = k0 + ((idx & 7) << 3); }
      else { r = (idx & 15) << 3; k = k0 + (idx >> 4); }
      const int gr = row0 + r;
      const bool sec = gr >= o.split;
      const bf16_t* p = sec ? o.p1 : o.p0;
      const int64_t ld = sec ? o.ld1 : o.ld0;
      const int rr = sec ? gr - o.split : gr;
      const bool ok = gr < nrows && k < kend;
      const int64_t off = KMAJOR ? (int64_t)rr * ld + k : (int64_t)k * ld + rr;
      v[j] = ok ? *reinterpret_cast<const uint4*>(p + off) : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(bf16_t* lds) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int idx = threadIdx.x + NT * j;
      const int o = KMAJOR ? kofs(idx >> 3, idx & 7) : mofs(idx >> 4, idx & 15);
      *reinterpret_cast<uint4*>(lds + o) = v[j];
    }
  }
  // m-major only: this thread's 8 rows summed over its 4 k-rows of the tile.
  __device__ __forceinline__ void accumulate(float* rs) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        rs[2 * e] += __uint_as_float(w[e] << 16);
        rs[2 * e + 1] += __uint_as_float(w[e] & 0xFFFF0000u);
      }
    }
  }
};

// Fragment of rows/columns r0 .. r0+15, k-step ks of the tile.
template <bool KMAJOR>
__device__ __forceinline__ Frag<bf16_t> frag(const bf16_t* lds, int r0, int ks, int lane) {
  Frag<bf16_t> f;
  if (KMAJOR) {
    f.v = *reinterpret_cast<const uint4*>(lds + kofs(r0 + (lane & 15), ks * 4 + (lane >> 4)));
  } else {
    const int j = lane & 15;
    const int k = ks * 32 + (lane >> 4) * 8 + (j >> 2);
    const int col = r0 + ((j & 3) << 2);
    const int c = col >> 3, half = (col & 7);
    const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s_t*)(lds + mofs(k, c) + half));
    const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s_t*)(lds + mofs(k + 4, c) + half));
    f.v = make_uint4((uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16),
                     (uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16),
                     (uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16),
                     (uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16));
  }
  return f;
}

template <typename OutT> struct Out {
  OutT* c0; int64_t ld0;
  OutT* c1; int64_t ld1;
  int split;
  int64_t zstride;  // elements between the outputs of consecutive k-splits
};

// ROWSUM: A is m-major; the workgroups of the first column of tiles write
// the row sums of A over their split's k-range to rowsum[z * M + m].
template <bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM>
__global__ __launch_bounds__(NT, 2) void gemm_bf16_kernel(
    Op A, Op B, Out<OutT> C, const bf16_t* __restrict__ bias, float* __restrict__ rowsum,
    int M, int N, int K, int kps, int tm, int tn, int S) {
  __shared__ __align__(16) bf16_t smem[2][2][TB * BK];  // [stage][A|B]

  // XCD-contiguous tile order: workgroup b runs on XCD b % 8.
  const int G = tm * tn * S;
  const int b = blockIdx.x, x = b % NX, q = G / NX, rem = G % NX;
  const int T = x * q + min(x, rem) + b / NX;
  const int z = T / (tm * tn), t2 = T % (tm * tn);
  const int m0 = (t2 / tn) * TB, n0 = (t2 % tn) * TB;
  const int kbeg = z * kps, kend = min(K, kbeg + kps);
  const bool do_sum = ROWSUM && n0 == 0;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float rs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};

  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  Stage<AK, ROWSUM> sa[2];
  Stage<BKM, false> sb[2];
  if (nk > 0) {
    sa[0].load(A, m0, M, kbeg, kend);
    sb[0].load(B, n0, N, kbeg, kend);
  }
  if (nk > 1) {
    sa[1].load(A, m0, M, kbeg + BK, kend);
    sb[1].load(B, n0, N, kbeg + BK, kend);
  }
  if (nk > 0) {
    if (do_sum) sa[0].accumulate(rs);
    sa[0].store(smem[0][0]);
    sb[0].store(smem[0][1]);
  }
  __syncthreads();

  // Two k-tiles per pass so that the register stages are indexed statically.
  for (int kt = 0; kt < nk; kt += 2) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int t = kt + u;
      if (t >= nk) break;
      // stage u is free (stored at the previous tile): fetch tile t + 2
      if (t + 2 < nk) {
        sa[u].load(A, m0, M, kbeg + (t + 2) * BK, kend);
        sb[u].load(B, n0, N, kbeg + (t + 2) * BK, kend);
      }
      const bf16_t* la = smem[u][0];
      const bf16_t* lb = smem[u][1];
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
        Frag<bf16_t> af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = frag<AK>(la, wm + 16 * i, ks, lane);
#pragma unroll
        for (int j = 0; j < 4; ++j) bf[j] = frag<BKM>(lb, wn + 16 * j, ks, lane);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) mma_16x16x32(acc[i][j], af[i], bf[j]);
      }
      // tile t + 1 (register stage 1 - u) goes to LDS stage 1 - u
      if (t + 1 < nk) {
        if (do_sum) sa[1 - u].accumulate(rs);
        sa[1 - u].store(smem[1 - u][0]);
        sb[1 - u].store(smem[1 - u][1]);
      }
      __syncthreads();
    }
  }

  if (do_sum) {  // LDS is free after the loop's final barrier
    float* red = reinterpret_cast<float*>(&smem[0][0][0]);  // [16][TB]
    const int c = threadIdx.x & 15, kr = threadIdx.x >> 4;
#pragma unroll
    for (int e = 0; e < 8; ++e) red[kr * TB + c * 8 + e] = rs[e];
    __syncthreads();
    if (threadIdx.x < TB && m0 + (int)threadIdx.x < M) {
      float s = 0.f;
#pragma unroll
      for (int r = 0; r < 16; ++r) s += red[r * TB + threadIdx.x];
      rowsum[(int64_t)z * M + m0 + threadIdx.x] = s;
    }
  }

#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = n0 + wn + j * 16 + mfma_col(lane);
    if (col >= N) continue;
    const float bv = BIAS ? bf16_to_f32(bias[col]) : 0.f;
    const bool sec = col >= C.split;
    OutT* cb = (sec ? C.c1 : C.c0) + (int64_t)z * C.zstride;
    const int64_t ldc = sec ? C.ld1 : C.ld0;
    const int cc = sec ? col - C.split : col;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + i * 16 + mfma_row(lane, r);
        if (row < M) cb[(int64_t)row * ldc + cc] = from_f32<OutT>(acc[i][j][r] + bv);
      }
  }
}

template <bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM>
void launch(const GemmArgs& g, Out<OutT> dst, float* rowsum, int S, int kps, hipStream_t s) {
  const bf16_t* a = static_cast<const bf16_t*>(g.A);
  const bf16_t* b = static_cast<const bf16_t*>(g.B);
  const bf16_t* b2 = g.B2 ? static_cast<const bf16_t*>(g.B2) : b;
  Op A{a, g.lda, a, g.lda, 1 << 30};
  Op B{b, g.ldb, b2, g.B2 ? g.ldb2 : g.ldb, g.B2 ? g.n_split : (1 << 30)};
  const int tm = (g.M + TB - 1) / TB, tn = (g.N + TB - 1) / TB;
  hipLaunchKernelGGL((gemm_bf16_kernel<AK, BKM, OutT, BIAS, ROWSUM>), dim3(tm * tn * S), dim3(NT),
                     0, s, A, B, dst, static_cast<const bf16_t*>(g.bias), rowsum, g.M, g.N, g.K,
                     kps, tm, tn, S);
}

template <typename OutT> Out<OutT> direct_out(const GemmArgs& g) {
  Out<OutT> d;
  d.c0 = static_cast<OutT*>(g.C);
  d.ld0 = g.ldc;
  d.c1 = static_cast<OutT*>(g.C2 ? g.C2 : g.C);
  d.ld1 = g.C2 ? g.ldc2 : g.ldc;
  d.split = g.C2 ? g.n_split : (1 << 30);
  d.zstride = 0;
  return d;
}

}  // namespace

hipError_t gemm_bf16(const GemmArgs& g, hipStream_t s) {
  if (g.a_kmajor && g.b_kmajor) {  // forward projections
    if (g.c_f32) {
      if (g.bias) launch<true, true, float, true, false>(g, direct_out<float>(g), nullptr, 1, g.K, s);
      else launch<true, true, float, false, false>(g, direct_out<float>(g), nullptr, 1, g.K, s);
    } else {
      if (g.bias) launch<true, true, bf16_t, true, false>(g, direct_out<bf16_t>(g), nullptr, 1, g.K, s);
      else launch<true, true, bf16_t, false, false>(g, direct_out<bf16_t>(g), nullptr, 1, g.K, s);
    }
    return hipGetLastError();
  }
  if (g.a_kmajor && !g.b_kmajor && !g.bias && !g.rowsum) {  // data gradients
    if (g.c_f32) launch<true, false, float, false, false>(g, direct_out<float>(g), nullptr, 1, g.K, s);
    else launch<true, false, bf16_t, false, false>(g, direct_out<bf16_t>(g), nullptr, 1, g.K, s);
    return hipGetLastError();
  }
  if (!g.a_kmajor && !g.b_kmajor && !g.bias && g.c_f32) {  // weight gradients
    const int tiles = ((g.N + TB - 1) / TB) * ((g.M + TB - 1) / TB);
    const int ktiles = (g.K + BK - 1) / BK;
    int S = 1;
    if (g.ws) {
      S = (512 + tiles - 1) / tiles;
      S = S > 8 ? 8 : S;
      while (S > 1 && ktiles / S < 8) --S;  // keep at least 8 k-tiles per split
      while (S > 1 && (int64_t)S * g.M * g.N + (int64_t)S * g.M > g.ws_floats) --S;
    }
    if (S == 1) {
      if (g.rowsum) launch<false, false, float, false, true>(g, direct_out<float>(g), g.rowsum, 1, g.K, s);
      else launch<false, false, float, false, false>(g, direct_out<float>(g), nullptr, 1, g.K, s);
      return hipGetLastError();
    }
    const int kps = ((ktiles + S - 1) / S) * BK;
    float* part = g.ws;
    float* rs_part = g.ws + (int64_t)S * g.M * g.N;
    Out<float> d{part, g.N, part, g.N, 1 << 30, (int64_t)g.M * g.N};  // one slice per split
    if (g.rowsum) launch<false, false, float, false, true>(g, d, rs_part, S, kps, s);
    else launch<false, false, float, false, false>(g, d, nullptr, S, kps, s);
    return splitk_reduce_launch(part, S, g, rs_part, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace am
