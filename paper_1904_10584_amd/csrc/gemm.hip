// MFMA GEMM family for the batched products of the training step:
//   forward projections  P = X Wx^T + b,  Z = H Wo^T + bo      (NT, bias)
//   data gradients       dH = dZ Wo,  dX = dA Wx              (NN)
//   weight gradients     dW = dA^T X,  dWo = dZ^T H           (TN, K = frames)
// One 256-thread workgroup computes a 128x128 tile; its four waves each own a
// 64x64 quadrant as 4x4 MFMA 16x16 tiles (16x16x32 bf16, or 8 x 16x16x4
// fp32 per 32-wide k-step).  Operands are staged in LDS as [row][k] with a
// 16-byte pad per row.  A k-major operand is copied with 16-byte loads; an
// m/n-major one (the TN and NN cases) is loaded as 8(k) x 4(m) blocks that
// each thread transposes in registers, so every LDS tile is k-contiguous and
// the fragment reads are single 16-byte LDS loads.  Global loads for tile
// k+1 are issued before the MFMAs of tile k (double-buffered LDS, one
// barrier per k-tile).  Reductions are never split across workgroups, so
// results are deterministic.
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int TB = 128;   // tile rows and columns
constexpr int NT = 256;   // threads per workgroup

template <typename T> struct KT;
template <> struct KT<bf16_t> { static constexpr int BK = 64, VEC = 8; };
template <> struct KT<float>  { static constexpr int BK = 32, VEC = 4; };

template <typename T> struct Tile {
  static constexpr int BK = KT<T>::BK;
  static constexpr int VEC = KT<T>::VEC;
  static constexpr int LDK = BK + VEC;               // padded row, elements
  static constexpr int STAGE = 2 * TB * LDK;         // A + B tiles, elements
};

// Operand loader: 4 x 16 bytes of staging registers per thread.
template <typename T, bool KMAJOR> struct Loader;

// k-major: rows of the operand are contiguous in k.
template <typename T> struct Loader<T, true> {
  uint4 reg[4];
  __device__ void load(const T* __restrict__ base, int64_t ld, int row0, int nrows, int k0, int K) {
    constexpr int CPR = Tile<T>::BK / Tile<T>::VEC;  // 16-byte chunks per row = 8
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      int c = threadIdx.x + NT * j;
      int row = c / CPR, kc = c % CPR;
      int grow = row0 + row, gk = k0 + kc * Tile<T>::VEC;
      if (grow < nrows && gk < K)
        reg[j] = *reinterpret_cast<const uint4*>(base + (int64_t)grow * ld + gk);
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
};

// m/n-major, bf16: thread (kb, mb) loads 8 k-rows x 4 rows-of-the-tile and
// transposes them into 4 k-octets.
template <> struct Loader<bf16_t, false> {
  uint4 reg[4];
  __device__ void load(const bf16_t* __restrict__ base, int64_t ld, int row0, int nrows, int k0, int K) {
    int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
    int m = row0 + mb * 4;
    uint2 in[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      int k = k0 + kb * 8 + r;
      if (k < K && m < nrows)
        in[r] = *reinterpret_cast<const uint2*>(base + (int64_t)k * ld + m);
      else
        in[r] = make_uint2(0, 0);
    }
    // element q of row r: q=0 low half of .x, 1 high half of .x, 2/3 in .y
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint32_t w[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        uint32_t d = (q < 2) ? in[r].x : in[r].y;
        w[r] = (q & 1) ? (d >> 16) : (d & 0xFFFFu);
      }
      reg[q] = make_uint4(w[0] | (w[1] << 16), w[2] | (w[3] << 16),
                          w[4] | (w[5] << 16), w[6] | (w[7] << 16));
    }
  }
  __device__ void store(bf16_t* lds) {
    int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<uint4*>(lds + (mb * 4 + q) * Tile<bf16_t>::LDK + kb * 8) = reg[q];
  }
};

// m/n-major, fp32: 4 k-rows x 4 rows-of-the-tile per thread.
template <> struct Loader<float, false> {
  uint4 reg[4];
  __device__ void load(const float* __restrict__ base, int64_t ld, int row0, int nrows, int k0, int K) {
    int kb = threadIdx.x >> 5, mb = threadIdx.x & 31;
    int m = row0 + mb * 4;
    float4 in[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int k = k0 + kb * 4 + r;
      if (k < K && m < nrows)
        in[r] = *reinterpret_cast<const float4*>(base + (int64_t)k * ld + m);
      else
        in[r] = make_float4(0.f, 0.f, 0.f, 0.f);
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

template <typename T, bool AK, bool BKM, typename OutT, bool BIAS>
__global__ __launch_bounds__(NT, 2) void gemm_kernel(
    const T* __restrict__ A, int64_t lda, const T* __restrict__ B, int64_t ldb,
    OutT* __restrict__ C, int64_t ldc, const T* __restrict__ bias, int M, int N, int K) {
  using TL = Tile<T>;
  __shared__ __align__(16) T smem[2 * TL::STAGE];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int m0 = blockIdx.y * TB, n0 = blockIdx.x * TB;

  Loader<T, AK> la;
  Loader<T, BKM> lb;
  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  const int nk = (K + TL::BK - 1) / TL::BK;
  la.load(A, lda, m0, M, 0, K);
  lb.load(B, ldb, n0, N, 0, K);
  la.store(smem);
  lb.store(smem + TB * TL::LDK);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    T* cur = smem + (kt & 1) * TL::STAGE;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(A, lda, m0, M, (kt + 1) * TL::BK, K);
      lb.load(B, ldb, n0, N, (kt + 1) * TL::BK, K);
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

#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = n0 + wn * 64 + j * 16 + mfma_col(lane);
    if (col >= N) continue;
    const float bv = BIAS ? to_f32<T>(bias[col]) : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm * 64 + i * 16 + mfma_row(lane, r);
        if (row < M) C[(int64_t)row * ldc + col] = from_f32<OutT>(acc[i][j][r] + bv);
      }
    }
  }
}

template <typename T, bool AK, bool BKM, typename OutT, bool BIAS>
hipError_t run(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + TB - 1) / TB, (g.M + TB - 1) / TB);
  hipLaunchKernelGGL((gemm_kernel<T, AK, BKM, OutT, BIAS>), grid, dim3(NT), 0, s,
                     static_cast<const T*>(g.A), g.lda, static_cast<const T*>(g.B), g.ldb,
                     static_cast<OutT*>(g.C), g.ldc, static_cast<const T*>(g.bias), g.M, g.N, g.K);
  return hipGetLastError();
}

template <typename T>
hipError_t dispatch(const GemmArgs& g, hipStream_t s) {
  // The combinations the training step uses.
  if (g.a_kmajor && g.b_kmajor) {           // NT: forward projections
    if (g.c_f32)
      return g.bias ? run<T, true, true, float, true>(g, s) : run<T, true, true, float, false>(g, s);
    return g.bias ? run<T, true, true, T, true>(g, s) : run<T, true, true, T, false>(g, s);
  }
  if (g.a_kmajor && !g.b_kmajor && !g.bias) {  // NN: data gradients
    return g.c_f32 ? run<T, true, false, float, false>(g, s) : run<T, true, false, T, false>(g, s);
  }
  if (!g.a_kmajor && !g.b_kmajor && !g.bias && g.c_f32)  // TN: weight gradients
    return run<T, false, false, float, false>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t gemm(const GemmArgs& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0) return hipSuccess;
  return g.bf16 ? dispatch<bf16_t>(g, s) : dispatch<float>(g, s);
}

}  // namespace am
