// fp32 MFMA GEMM family (the fp32 model path; bf16 products are in
// gemm_bf16.hip):
//   forward projections  P = X Wx^T + b,  Z = H Wo^T + bo      (NT, bias)
//   data gradients       dH = dZ Wo,  dX = dA Wx              (NN)
//   weight gradients     [dWx | dWh] = dA^T [X | Hs],  dWo = dZ^T H   (TN)
// One 256-thread workgroup computes a 128x128 tile; its four waves each own a
// 64x64 quadrant as 4x4 MFMA 16x16 tiles (8 x 16x16x4 fp32 per 32-wide
// k-step).  Operands are staged in LDS as [row][k] with a 16-byte pad per
// row.  A k-major operand is copied with 16-byte loads; an m/n-major one (the
// TN and NN cases) is loaded as 4(k) x 4(m) blocks that each thread
// transposes in registers, so every LDS tile is k-contiguous.  Global loads
// for tile k+1 are issued before the MFMAs of tile k (double-buffered LDS,
// one barrier per k-tile).
//
// Weight gradients reduce over all frames into a small output, so they split
// K over workgroups: each split writes an fp32 partial tile to the workspace
// and splitk_reduce adds the partials in split order (deterministic; no
// atomics).  The same pass yields the bias gradient: while loading the A tile
// (dA or dZ, m-major) each thread keeps the sums of its 4 rows over its
// k-rows, and the first column of tiles writes them.  The B operand of the TN
// product may come from two matrices side by side (X and the shifted hidden
// states), so dWx and dWh are one launch.
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int TB = 128;   // tile rows and columns
constexpr int NT = 256;   // threads per workgroup

template <typename T> struct KT;
template <> struct KT<float>  { static constexpr int BK = 32, VEC = 4; };

template <typename T> struct Tile {
  static constexpr int BK = KT<T>::BK;
  static constexpr int VEC = KT<T>::VEC;
  static constexpr int LDK = BK + VEC;               // padded row, elements
  static constexpr int STAGE = 2 * TB * LDK;         // A + B tiles, elements
};

// Source of one operand: rows (of the tile dimension) below `split` come
// from p0, the others from p1 at row - split.
template <typename T> struct Src {
  const T* p0; int64_t ld0;
  const T* p1; int64_t ld1;
  int split;
};

// Operand loader: 4 x 16 bytes of staging registers per thread.
template <typename T, bool KMAJOR> struct Loader;

// k-major: rows of the operand are contiguous in k.
template <typename T> struct Loader<T, true> {
  uint4 reg[4];
  __device__ void load(const Src<T>& s, int row0, int nrows, int k0, int kend) {
    constexpr int CPR = Tile<T>::BK / Tile<T>::VEC;  // 16-byte chunks per row = 8
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = threadIdx.x + NT * j;
      int row = c / CPR, kc = c % CPR;
      int grow = row0 + row, gk = k0 + kc * Tile<T>::VEC;
      if (grow < nrows && gk < kend)
        reg[j] = *reinterpret_cast<const uint4*>(s.p0 + (int64_t)grow * s.ld0 + gk);
      else
        reg[j] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ void store(T* lds) {
    constexpr int CPR = Tile<T>::BK / Tile<T>::VEC;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = threadIdx.x + NT * j;
      int row = c / CPR, kc = c % CPR;
      *reinterpret_cast<uint4*>(lds + row * Tile<T>::LDK + kc * Tile<T>::VEC) = reg[j];
    }
  }
  __device__ void rowsum_init() {}
  __device__ float rowsum(int) const { return 0.f; }
};

// m/n-major, fp32: 4 k-rows x 4 rows-of-the-tile per thread.
template <> struct Loader<float, false> {
  uint4 reg[4];
  float rs[4];
  __device__ void rowsum_init() { rs[0] = rs[1] = rs[2] = rs[3] = 0.f; }
  __device__ float rowsum(int q) const { return rs[q]; }
  template <bool SUM = false>
  __device__ void load(const Src<float>& s, int row0, int nrows, int k0, int kend) {
    const int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
    const int m = row0 + mb * 4;
    const bool second = m >= s.split;
    const float* base = second ? s.p1 : s.p0;
    const int64_t ld = second ? s.ld1 : s.ld0;
    const int mm = second ? m - s.split : m;
    float4 in[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int k = k0 + kb * 4 + r;
      if (k < kend && m < nrows)
        in[r] = *reinterpret_cast<const float4*>(base + (int64_t)k * ld + mm);
      else
        in[r] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    if (SUM) {
      rs[0] += ((in[0].x + in[1].x) + in[2].x) + in[3].x;
      rs[1] += ((in[0].y + in[1].y) + in[2].y) + in[3].y;
      rs[2] += ((in[0].z + in[1].z) + in[2].z) + in[3].z;
      rs[3] += ((in[0].w + in[1].w) + in[2].w) + in[3].w;
    }
    reg[0] = make_uint4(__float_as_uint(in[0].x), __float_as_uint(in[1].x), __float_as_uint(in[2].x), __float_as_uint(in[3].x));
    reg[1] = make_uint4(__float_as_uint(in[0].y), __float_as_uint(in[1].y), __float_as_uint(in[2].y), __float_as_uint(in[3].y));
    reg[2] = make_uint4(__float_as_uint(in[0].z), __float_as_uint(in[1].z), __float_as_uint(in[2].z), __float_as_uint(in[3].z));
    reg[3] = make_uint4(__float_as_uint(in[0].w), __float_as_uint(in[1].w), __float_as_uint(in[2].w), __float_as_uint(in[3].w));
  }
  __device__ void store(float* lds) {
    int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(lds + (mb * 4 + q) * Tile<float>::LDK + kb * 4) = reg[q];
  }
};

template <typename T, bool KMAJOR, bool SUM>
__device__ __forceinline__ void load_op(Loader<T, KMAJOR>& l, const Src<T>& s, int row0, int nrows,
                                        int k0, int kend) {
  if constexpr (KMAJOR) l.load(s, row0, nrows, k0, kend);
  else l.template load<SUM>(s, row0, nrows, k0, kend);
}

// Epilogue destination: columns below `split` go to c0, the others to c1.
template <typename OutT> struct Dst {
  OutT* c0; int64_t ld0;
  OutT* c1; int64_t ld1;
  int split;
  int64_t zstride;  // elements between the outputs of consecutive k-splits
};

// ROWSUM: the A operand is m-major and row sums of A over this split's
// k-range are written by the workgroups of the first column of tiles to
// rowsum[blockIdx.z * M + m].  Partial results (split-K) use c0 = the
// split's slice of the workspace with ld0 = N and split = N.
template <typename T, bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM>
__global__ __launch_bounds__(NT, 2) void gemm_kernel(
    Src<T> A, Src<T> B, Dst<OutT> C, const T* __restrict__ bias, float* __restrict__ rowsum,
    int M, int N, int K, int kps) {
  using TL = Tile<T>;
  __shared__ __align__(16) T smem[2 * TL::STAGE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * TB, n0 = blockIdx.x * TB;
  const int kbeg = blockIdx.z * kps;
  const int kend = min(K, kbeg + kps);
  const bool do_sum = ROWSUM && blockIdx.x == 0;

  Loader<T, AK> la;
  Loader<T, BKM> lb;
  la.rowsum_init();
  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = kend > kbeg ? (kend - kbeg + TL::BK - 1) / TL::BK : 0;
  if (do_sum) load_op<T, AK, true>(la, A, m0, M, kbeg, kend);
  else load_op<T, AK, false>(la, A, m0, M, kbeg, kend);
  load_op<T, BKM, false>(lb, B, n0, N, kbeg, kend);
  la.store(smem);
  lb.store(smem + TB * TL::LDK);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    T* cur = smem + (kt & 1) * TL::STAGE;
    const bool more = kt + 1 < nk;
    if (more) {
      const int k1 = kbeg + (kt + 1) * TL::BK;
      if (do_sum) load_op<T, AK, true>(la, A, m0, M, k1, kend);
      else load_op<T, AK, false>(la, A, m0, M, k1, kend);
      load_op<T, BKM, false>(lb, B, n0, N, k1, kend);
    }
    const T* sa = cur;
    const T* sb = cur + TB * TL::LDK;
#pragma unroll
    for (int ks = 0; ks < TL::BK / 32; ++ks) {
      const int koff = ks * 32 + (lane >> 4) * 8;
      Frag<T> af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = frag_load<T>(sa + (wm * 64 + i * 16 + (lane & 15)) * TL::LDK + koff);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = frag_load<T>(sb + (wn * 64 + j * 16 + (lane & 15)) * TL::LDK + koff);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) mma_16x16x32(acc[i][j], af[i], bfr[j]);
    }
    if (more) {
      T* nxt = smem + ((kt + 1) & 1) * TL::STAGE;
      la.store(nxt);
      lb.store(nxt + TB * TL::LDK);
    }
    __syncthreads();
  }

  if (do_sum) {  // smem is free after the final barrier of the loop
    float* rs = reinterpret_cast<float*>(smem);  // [8][128]
    const int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
#pragma unroll
    for (int q = 0; q < 4; ++q) rs[kb * TB + mb * 4 + q] = la.rowsum(q);
    __syncthreads();
    if (threadIdx.x < TB && m0 + (int)threadIdx.x < M) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < 8; ++k) s += rs[k * TB + threadIdx.x];
      rowsum[(int64_t)blockIdx.z * M + m0 + threadIdx.x] = s;
    }
  }

#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = n0 + wn * 64 + j * 16 + mfma_col(lane);
    if (col >= N) continue;
    const float bv = BIAS ? to_f32<T>(bias[col]) : 0.f;
    const bool second = col >= C.split;
    OutT* cbase = (second ? C.c1 : C.c0) + (int64_t)blockIdx.z * C.zstride;
    const int64_t ldc = second ? C.ld1 : C.ld0;
    const int ccol = second ? col - C.split : col;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 64 + i * 16 + mfma_row(lane, r);
        if (row < M) cbase[(int64_t)row * ldc + ccol] = from_f32<OutT>(acc[i][j][r] + bv);
      }
    }
  }
}

// Sum of the split-K partials in split order, routed to the two destinations,
// and of the partial row sums.
// V4: every destination row chunk is 16-byte aligned (pointers, pitches
// and the column split multiples of 4 floats), so the sum leaves as one
// 16-byte store instead of four 4-byte ones.
template <bool V4>
__global__ __launch_bounds__(256) void splitk_reduce(const float* __restrict__ part, int S, int M,
                                                     int N, float* __restrict__ c0, int64_t ld0,
                                                     float* __restrict__ c1, int64_t ld1, int split,
                                                     const float* __restrict__ rs_part,
                                                     float* __restrict__ rowsum) {
  const int64_t MN = (int64_t)M * N;
  const int64_t nq = MN / 4;  // N % 4 == 0
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < nq) {
    const float4* p = reinterpret_cast<const float4*>(part) + i;
    float4 s = p[0];
    for (int k = 1; k < S; ++k) {
      const float4 v = p[k * nq];
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    const int64_t e = i * 4;
    const int m = (int)(e / N), n = (int)(e % N);
    float* dst = n >= split ? c1 + (int64_t)m * ld1 + (n - split) : c0 + (int64_t)m * ld0 + n;
    if constexpr (V4) {
      *reinterpret_cast<float4*>(dst) = s;
    } else {
      dst[0] = s.x; dst[1] = s.y; dst[2] = s.z; dst[3] = s.w;
    }
  } else if (rowsum && i - nq < M) {
    const int64_t m = i - nq;
    float s = rs_part[m];
    for (int k = 1; k < S; ++k) s += rs_part[(int64_t)k * M + m];
    rowsum[m] = s;
  }
}

template <typename T, bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM>
void launch(const GemmArgs& g, Dst<OutT> dst, float* rowsum, int S, int kps, hipStream_t s) {
  Src<T> A{static_cast<const T*>(g.A), g.lda, static_cast<const T*>(g.A), g.lda, 1 << 30};
  Src<T> B{static_cast<const T*>(g.B), g.ldb,
           static_cast<const T*>(g.B2 ? g.B2 : g.B), g.B2 ? g.ldb2 : g.ldb,
           g.B2 ? g.n_split : (1 << 30)};
  dim3 grid((g.N + TB - 1) / TB, (g.M + TB - 1) / TB, S);
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, OutT, BIAS, ROWSUM>), grid, dim3(NT), 0, s, A, B,
                     dst, static_cast<const T*>(g.bias), rowsum, g.M, g.N, g.K, kps);
}

template <typename T, typename OutT>
Dst<OutT> direct_dst(const GemmArgs& g) {
  Dst<OutT> d;
  d.c0 = static_cast<OutT*>(g.C);
  d.ld0 = g.ldc;
  d.c1 = static_cast<OutT*>(g.C2 ? g.C2 : g.C);
  d.ld1 = g.C2 ? g.ldc2 : g.ldc;
  d.split = g.C2 ? g.n_split : (1 << 30);
  d.zstride = 0;
  return d;
}

template <typename T>
hipError_t dispatch(const GemmArgs& g, hipStream_t s) {
  if (g.a_kmajor && g.b_kmajor) {           // NT: forward projections
    if (g.c_f32) {
      if (g.bias) launch<T, true, true, float, true, false>(g, direct_dst<T, float>(g), nullptr, 1, g.K, s);
      else launch<T, true, true, float, false, false>(g, direct_dst<T, float>(g), nullptr, 1, g.K, s);
    } else {
      if (g.bias) launch<T, true, true, T, true, false>(g, direct_dst<T, T>(g), nullptr, 1, g.K, s);
      else launch<T, true, true, T, false, false>(g, direct_dst<T, T>(g), nullptr, 1, g.K, s);
    }
    return hipGetLastError();
  }
  if (g.a_kmajor && !g.b_kmajor && !g.bias && !g.rowsum) {  // NN: data gradients
    if (g.c_f32) launch<T, true, false, float, false, false>(g, direct_dst<T, float>(g), nullptr, 1, g.K, s);
    else launch<T, true, false, T, false, false>(g, direct_dst<T, T>(g), nullptr, 1, g.K, s);
    return hipGetLastError();
  }
  if (!g.a_kmajor && !g.b_kmajor && !g.bias && g.c_f32) {  // TN: weight gradients
    const int tiles = ((g.N + TB - 1) / TB) * ((g.M + TB - 1) / TB);
    const int BK = Tile<T>::BK;
    const int ktiles = (g.K + BK - 1) / BK;
    int S = 1;
    if (g.ws) {
      S = (512 + tiles - 1) / tiles;
      S = S > 8 ? 8 : S;
      while (S > 1 && ktiles / S < 8) --S;  // keep at least 8 k-tiles per split
      while (S > 1 && (int64_t)S * g.M * g.N + (int64_t)S * g.M > g.ws_floats) --S;
    }
    if (S == 1) {
      if (g.rowsum) launch<T, false, false, float, false, true>(g, direct_dst<T, float>(g), g.rowsum, 1, g.K, s);
      else launch<T, false, false, float, false, false>(g, direct_dst<T, float>(g), nullptr, 1, g.K, s);
      return hipGetLastError();
    }
    const int kps = ((ktiles + S - 1) / S) * BK;
    float* part = g.ws;
    float* rs_part = g.ws + (int64_t)S * g.M * g.N;
    Dst<float> d{part, g.N, part, g.N, 1 << 30, (int64_t)g.M * g.N};  // one slice per split
    if (g.rowsum) launch<T, false, false, float, false, true>(g, d, rs_part, S, kps, s);
    else launch<T, false, false, float, false, false>(g, d, nullptr, S, kps, s);
    return splitk_reduce_launch(part, S, g, rs_part, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t splitk_reduce_launch(const float* part, int S, const GemmArgs& g, const float* rs_part,
                                hipStream_t s) {
  const int64_t nq = (int64_t)g.M * g.N / 4;
  const int64_t threads = nq + (g.rowsum ? g.M : 0);
  float* c0 = static_cast<float*>(g.C);
  float* c1 = static_cast<float*>(g.C2 ? g.C2 : g.C);
  const int64_t ld1 = g.C2 ? g.ldc2 : g.ldc;
  const int split = g.C2 ? g.n_split : (1 << 30);
  const bool v4 = (reinterpret_cast<uintptr_t>(c0) | reinterpret_cast<uintptr_t>(c1)) % 16 == 0 &&
                  g.ldc % 4 == 0 && ld1 % 4 == 0 && split % 4 == 0;
  if (v4)
    hipLaunchKernelGGL(splitk_reduce<true>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                       part, S, g.M, g.N, c0, g.ldc, c1, ld1, split, rs_part, g.rowsum);
  else
    hipLaunchKernelGGL(splitk_reduce<false>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s,
                       part, S, g.M, g.N, c0, g.ldc, c1, ld1, split, rs_part, g.rowsum);
  return hipGetLastError();
}

hipError_t gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  return g.bf16 ? gemm_bf16(g, s) : dispatch<float>(g, s);
}

}  // namespace am
