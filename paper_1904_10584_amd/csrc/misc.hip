// Elementwise and data-movement kernels of the training step: the SGD update
// with its bf16 copy, fp32 -> bf16 casts, the recurrent-weight transpose used
// by BPTT, bias-gradient column sums and the final-state gather.
#include <cstdlib>

#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

// (sgd_one, the step of one element, is in am_device.h: the fused decode +
// SGD of gtc.hip applies the same arithmetic.)

template <bool ALIGNED, bool BF16>
__global__ __launch_bounds__(256) void sgd_kernel(int64_t n, float* __restrict__ master,
                                                  bf16_t* __restrict__ wb,
                                                  const float* __restrict__ u, float lr) {
  const double lr64 = (double)lr;
  const int64_t stride = (int64_t)gridDim.x * 256 * 4;
  for (int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; e < n; e += stride) {
    if (ALIGNED && e + 3 < n) {
      float4 w = *reinterpret_cast<const float4*>(master + e);
      const float4 g = *reinterpret_cast<const float4*>(u + e);
      w.x = sgd_one(w.x, g.x, lr64);
      w.y = sgd_one(w.y, g.y, lr64);
      w.z = sgd_one(w.z, g.z, lr64);
      w.w = sgd_one(w.w, g.w, lr64);
      *reinterpret_cast<float4*>(master + e) = w;
      if (BF16) {
        uint2 b;
        b.x = (uint32_t)f32_to_bf16(w.x) | ((uint32_t)f32_to_bf16(w.y) << 16);
        b.y = (uint32_t)f32_to_bf16(w.z) | ((uint32_t)f32_to_bf16(w.w) << 16);
        *reinterpret_cast<uint2*>(wb + e) = b;
      }
    } else {
      for (int64_t i = e; i < e + 4 && i < n; ++i) {
        const float w = sgd_one(master[i], u[i], lr64);
        master[i] = w;
        if (BF16) wb[i] = f32_to_bf16(w);
      }
    }
  }
}

template <bool ALIGNED>
__global__ __launch_bounds__(256) void cast_kernel(int64_t n, const float* __restrict__ src,
                                                   bf16_t* __restrict__ dst) {
  const int64_t stride = (int64_t)gridDim.x * 256 * 4;
  for (int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; e < n; e += stride) {
    if (ALIGNED && e + 3 < n) {
      const float4 v = *reinterpret_cast<const float4*>(src + e);
      uint2 b;
      b.x = (uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16);
      b.y = (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16);
      *reinterpret_cast<uint2*>(dst + e) = b;
    } else {
      for (int64_t i = e; i < e + 4 && i < n; ++i) dst[i] = f32_to_bf16(src[i]);
    }
  }
}

// Zero n0 floats at d0, then n1 at d1 (one launch for two ranges).
__global__ __launch_bounds__(256) void fill_zero_kernel(int64_t n0, float* __restrict__ d0, int64_t n1,
                                                        float* __restrict__ d1) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n0 + n1; i += (int64_t)gridDim.x * 256) {
    if (i < n0) d0[i] = 0.f;
    else d1[i - n0] = 0.f;
  }
}

// dst[0..n) = +0.0 if *flag is nonzero; otherwise nothing (one workgroup:
// the cheap case is the common one).
__global__ __launch_bounds__(256) void zero_if_set_kernel(const int* __restrict__ flag, int64_t n,
                                                          float* __restrict__ dst) {
  if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) return;
  for (int64_t i = threadIdx.x; i < n; i += 256) dst[i] = 0.f;
}

template <typename T>
__global__ __launch_bounds__(256) void convert_kernel(int64_t n, const float* __restrict__ src,
                                                      T* __restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = from_f32<T>(src[i]);
}

// 64x64 tiles through LDS; 256 threads, each moves 16 elements.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ src,
                                                        T* __restrict__ dst, int rows, int cols) {
  __shared__ T tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    if (r < rows && c < cols) tile[i][tx] = src[(int64_t)r * cols + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (r < rows && c < cols) dst[(int64_t)c * rows + r] = tile[tx][i];
  }
}

// bf16 with both dimensions multiples of 8 and 16-byte aligned rows: 64 x 64
// tiles moved as 16-byte chunks (eight elements) on both sides, transposed
// through LDS.  Thread (column, row chunk) gathers eight rows of one column.
// The chunks of tile row i sit XOR-permuted by (i / 8) % 8, so the eight
// rows 8 apart that the lanes of one read touch fall in different banks.
// Several matrices of one shape in one launch: blockIdx.z picks the pair.
__global__ __launch_bounds__(256) void transpose_bf16_x8(TransposeBatch tb, int rows, int cols) {
  const bf16_t* __restrict__ src = static_cast<const bf16_t*>(tb.src[blockIdx.z]);
  bf16_t* __restrict__ dst = static_cast<bf16_t*>(tb.dst[blockIdx.z]);
  __shared__ __align__(16) bf16_t tile[64 * 64];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  auto at = [](int i, int j) { return i * 64 + (((j >> 3) ^ ((i >> 3) & 7)) << 3) + (j & 7); };
  // 64 rows x 8 chunks: thread t loads chunks t and t + 256
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int e = threadIdx.x + 256 * h, i = e >> 3, ch = e & 7;
    const int r = r0 + i, c = c0 + ch * 8;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (r < rows && c < cols) v = *reinterpret_cast<const uint4*>(src + (int64_t)r * cols + c);
    *reinterpret_cast<uint4*>(&tile[at(i, ch * 8)]) = v;
  }
  __syncthreads();
  // 64 columns x 8 row chunks: thread t writes chunks t and t + 256
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int e = threadIdx.x + 256 * h, j = e >> 3, rc = e & 7;
    const int c = c0 + j, r = r0 + rc * 8;
    if (c < cols && r < rows) {
      uint32_t w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k)
        w[k] = (uint32_t)tile[at(rc * 8 + 2 * k, j)] | ((uint32_t)tile[at(rc * 8 + 2 * k + 1, j)] << 16);
      *reinterpret_cast<uint4*>(dst + (int64_t)c * rows + r) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

// Partial column sums over a chunk of rows; partial[chunk][c].
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial(const T* __restrict__ in, int64_t rows,
                                                      int cols, int64_t rows_per_chunk,
                                                      float* __restrict__ partial) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per_chunk;
  const int64_t r1 = r0 + rows_per_chunk < rows ? r0 + rows_per_chunk : rows;
  float acc = 0.f;
  for (int64_t r = r0; r < r1; ++r) acc += to_f32<T>(in[r * cols + c]);
  partial[(int64_t)blockIdx.y * cols + c] = acc;
}

__global__ __launch_bounds__(256) void colsum_final(const float* __restrict__ partial, int chunks,
                                                    int cols, float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= cols) return;
  float acc = 0.f;
  for (int k = 0; k < chunks; ++k) acc += partial[(int64_t)k * cols + c];
  out[c] = acc;
}

template <typename T>
__global__ __launch_bounds__(256) void gather_state_kernel(GatherState a, int b0) {
  const int bi = blockIdx.x;
  const int b = b0 + bi;
  const int row = a.rows[bi];
  const int H = a.hidden;
  const T* Hr = static_cast<const T*>(a.Hrows);
  for (int j = threadIdx.x; j < H; j += 256) {
    float h, c;
    if (row >= 0) {
      h = to_f32<T>(Hr[(int64_t)row * H + j]);
      c = a.Crows[(int64_t)row * H + j];
    } else {
      h = a.h0 ? a.h0[(int64_t)b * H + j] : 0.f;
      c = a.c0 ? a.c0[(int64_t)b * H + j] : 0.f;
    }
    if (a.hT) a.hT[(int64_t)b * H + j] = h;
    if (a.cT) a.cT[(int64_t)b * H + j] = c;
  }
}

inline unsigned grid_for(int64_t n, int64_t per_block) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g > 65536) g = 65536;
  return (unsigned)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t sgd_apply_f32(int64_t n, float* master, uint16_t* w_bf16, const float* u, float lr,
                         hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool al = ((reinterpret_cast<uintptr_t>(master) | reinterpret_cast<uintptr_t>(u)) & 15) == 0 &&
                  (reinterpret_cast<uintptr_t>(w_bf16) & 7) == 0;
  const unsigned g = grid_for(n, 1024);
  if (w_bf16) {
    if (al) hipLaunchKernelGGL((sgd_kernel<true, true>), dim3(g), dim3(256), 0, s, n, master, w_bf16, u, lr);
    else hipLaunchKernelGGL((sgd_kernel<false, true>), dim3(g), dim3(256), 0, s, n, master, w_bf16, u, lr);
  } else {
    if (al) hipLaunchKernelGGL((sgd_kernel<true, false>), dim3(g), dim3(256), 0, s, n, master, nullptr, u, lr);
    else hipLaunchKernelGGL((sgd_kernel<false, false>), dim3(g), dim3(256), 0, s, n, master, nullptr, u, lr);
  }
  return hipGetLastError();
}

hipError_t cast_f32_bf16(int64_t n, const float* src, uint16_t* dst, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const bool al = (reinterpret_cast<uintptr_t>(src) & 15) == 0 && (reinterpret_cast<uintptr_t>(dst) & 7) == 0;
  const unsigned g = grid_for(n, 1024);
  if (al) hipLaunchKernelGGL(cast_kernel<true>, dim3(g), dim3(256), 0, s, n, src, dst);
  else hipLaunchKernelGGL(cast_kernel<false>, dim3(g), dim3(256), 0, s, n, src, dst);
  return hipGetLastError();
}

hipError_t convert_rows(const float* src, void* dst, int64_t count, bool bf16, hipStream_t s) {
  if (count <= 0) return hipSuccess;
  const unsigned g = grid_for(count, 256);
  if (bf16) hipLaunchKernelGGL(convert_kernel<bf16_t>, dim3(g), dim3(256), 0, s, count, src, (bf16_t*)dst);
  else hipLaunchKernelGGL(convert_kernel<float>, dim3(g), dim3(256), 0, s, count, src, (float*)dst);
  return hipGetLastError();
}

hipError_t fill_zero(float* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  return fill_zero2(dst, n, nullptr, 0, s);
}

hipError_t fill_zero2(float* d0, int64_t n0, float* d1, int64_t n1, hipStream_t s) {
  if (n0 + n1 == 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(grid_for(n0 + n1, 256)), dim3(256), 0, s, n0, d0, n1, d1);
  return hipGetLastError();
}

hipError_t zero_if_set(const int* flag, float* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_if_set_kernel, dim3(1), dim3(256), 0, s, flag, n, dst);
  return hipGetLastError();
}

hipError_t transpose(const void* src, void* dst, int rows, int cols, bool bf16, hipStream_t s) {
  dim3 grid((cols + 63) / 64, (rows + 63) / 64);
  const bool x8 = rows % 8 == 0 && cols % 8 == 0 &&
                  ((reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst)) & 15) == 0;
  if (bf16 && x8) {
    TransposeBatch tb{};
    tb.src[0] = src;
    tb.dst[0] = dst;
    hipLaunchKernelGGL(transpose_bf16_x8, grid, dim3(256), 0, s, tb, rows, cols);
  }
  else if (bf16) hipLaunchKernelGGL(transpose_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)src, (bf16_t*)dst, rows, cols);
  else hipLaunchKernelGGL(transpose_kernel<float>, grid, dim3(256), 0, s, (const float*)src, (float*)dst, rows, cols);
  return hipGetLastError();
}

hipError_t transpose_bf16_batch(const TransposeBatch& tb, int n, int rows, int cols, hipStream_t s) {
  if (n <= 0 || n > TransposeBatch::MAX || rows % 8 != 0 || cols % 8 != 0) return hipErrorInvalidValue;
  for (int i = 0; i < n; ++i)
    if (((reinterpret_cast<uintptr_t>(tb.src[i]) | reinterpret_cast<uintptr_t>(tb.dst[i])) & 15) != 0)
      return hipErrorInvalidValue;
  hipLaunchKernelGGL(transpose_bf16_x8, dim3((cols + 63) / 64, (rows + 63) / 64, n), dim3(256), 0, s,
                     tb, rows, cols);
  return hipGetLastError();
}

hipError_t colsum(const void* in, int64_t rows, int cols, bool bf16, float* out, float* ws_partial,
                  int n_chunks, hipStream_t s) {
  const int64_t rpc = rows > 0 ? (rows + n_chunks - 1) / n_chunks : 1;
  dim3 grid((cols + 255) / 256, n_chunks);
  if (bf16) hipLaunchKernelGGL(colsum_partial<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)in, rows, cols, rpc, ws_partial);
  else hipLaunchKernelGGL(colsum_partial<float>, grid, dim3(256), 0, s, (const float*)in, rows, cols, rpc, ws_partial);
  hipLaunchKernelGGL(colsum_final, dim3((cols + 255) / 256), dim3(256), 0, s, ws_partial, n_chunks, cols, out);
  return hipGetLastError();
}

hipError_t gather_state(const GatherState& a, int b0, int nb, hipStream_t s) {
  if (nb <= 0) return hipSuccess;
  if (a.h_bf16) hipLaunchKernelGGL(gather_state_kernel<bf16_t>, dim3(nb), dim3(256), 0, s, a, b0);
  else hipLaunchKernelGGL(gather_state_kernel<float>, dim3(nb), dim3(256), 0, s, a, b0);
  return hipGetLastError();
}

hipError_t resident_launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds,
                           hipStream_t s) {
  static const bool cooperative = [] {
    const char* v = getenv("AM_COOPERATIVE");
    return v && v[0] == '1';
  }();
  if (cooperative) return hipLaunchCooperativeKernel(fn, grid, block, args, (unsigned)lds, s);
  return hipLaunchKernel(fn, grid, block, args, lds, s);
}

}  // namespace am
