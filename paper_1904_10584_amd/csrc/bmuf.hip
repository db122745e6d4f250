// BMUF-NBM global step (blockwise model update filtering with Nesterov block
// momentum, §VI-B eqs. (2)-(5)), one HBM-bound pass over the flat model:
//   Wbar  = (sum of the `count` addends) / workers       (2)
//   G     = Wbar - W_g                                   (3)
//   Delta = eta Delta + zeta G                           (4)
//   W_g   = W_g + Delta + eta_next Delta                 (5)
// and, optionally, the restart copy of the local model (fp32 and bf16).
// Each element is evaluated in fp64 from its fp32 inputs, in the order
// written, with no fused multiply-add, and each output is rounded once to
// fp32, so the result is bit-identical to the element-wise definition.
// Every thread reads all inputs of its elements before writing any output,
// so outputs may alias inputs of the same index (in-place W_g and Delta, or
// the local model written over one of the addends).
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

struct BmufOne {
  float w, d;
};

__device__ __forceinline__ BmufOne bmuf_one(double s, float wg, float d0, double workers,
                                            double eta, double eta_next, double zeta) {
#pragma clang fp contract(off)
  const double wbar = s / workers;
  const double g = wbar - (double)wg;
  const double d = eta * (double)d0 + zeta * g;
  const double w = ((double)wg + d) + eta_next * d;
  return BmufOne{(float)w, (float)d};
}

template <bool ALIGNED>
__global__ __launch_bounds__(256) void bmuf_kernel(int64_t n, int count, double workers,
                                                   const float* models,
                                                   int64_t stride, float* wg, float* delta,
                                                   double eta, double eta_next, double zeta,
                                                   float* local, bf16_t* local_bf16) {
#pragma clang fp contract(off)
  const int64_t step = (int64_t)gridDim.x * 256 * 4;
  for (int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4; e < n; e += step) {
    if (ALIGNED && e + 3 < n) {
      double s[4] = {0.0, 0.0, 0.0, 0.0};
      for (int i = 0; i < count; ++i) {
        const float4 m = *reinterpret_cast<const float4*>(models + (int64_t)i * stride + e);
        s[0] = s[0] + (double)m.x;
        s[1] = s[1] + (double)m.y;
        s[2] = s[2] + (double)m.z;
        s[3] = s[3] + (double)m.w;
      }
      const float4 w4 = *reinterpret_cast<const float4*>(wg + e);
      const float4 d4 = *reinterpret_cast<const float4*>(delta + e);
      const BmufOne r0 = bmuf_one(s[0], w4.x, d4.x, workers, eta, eta_next, zeta);
      const BmufOne r1 = bmuf_one(s[1], w4.y, d4.y, workers, eta, eta_next, zeta);
      const BmufOne r2 = bmuf_one(s[2], w4.z, d4.z, workers, eta, eta_next, zeta);
      const BmufOne r3 = bmuf_one(s[3], w4.w, d4.w, workers, eta, eta_next, zeta);
      const float4 nw = make_float4(r0.w, r1.w, r2.w, r3.w);
      *reinterpret_cast<float4*>(wg + e) = nw;
      *reinterpret_cast<float4*>(delta + e) = make_float4(r0.d, r1.d, r2.d, r3.d);
      if (local) *reinterpret_cast<float4*>(local + e) = nw;
      if (local_bf16) {
        uint2 b;
        b.x = (uint32_t)f32_to_bf16(nw.x) | ((uint32_t)f32_to_bf16(nw.y) << 16);
        b.y = (uint32_t)f32_to_bf16(nw.z) | ((uint32_t)f32_to_bf16(nw.w) << 16);
        *reinterpret_cast<uint2*>(local_bf16 + e) = b;
      }
    } else {
      for (int64_t j = e; j < e + 4 && j < n; ++j) {
        double s = 0.0;
        for (int i = 0; i < count; ++i) s = s + (double)models[(int64_t)i * stride + j];
        const BmufOne r = bmuf_one(s, wg[j], delta[j], workers, eta, eta_next, zeta);
        wg[j] = r.w;
        delta[j] = r.d;
        if (local) local[j] = r.w;
        if (local_bf16) local_bf16[j] = f32_to_bf16(r.w);
      }
    }
  }
}

}  // namespace

hipError_t bmuf_update(int64_t n, int count, int workers, const float* models, int64_t stride,
                       float* wg, float* delta, float eta, float eta_next, float zeta,
                       float* local, uint16_t* local_bf16, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const uintptr_t bits = reinterpret_cast<uintptr_t>(models) | reinterpret_cast<uintptr_t>(wg) |
                         reinterpret_cast<uintptr_t>(delta) | reinterpret_cast<uintptr_t>(local);
  const bool aligned = (bits & 15) == 0 && (reinterpret_cast<uintptr_t>(local_bf16) & 7) == 0 &&
                       (count == 1 || stride % 4 == 0);
  const int64_t quads = (n + 3) / 4;
  const int64_t want = (quads + 255) / 256;
  const unsigned blocks = (unsigned)(want < 8192 ? want : 8192);
  if (aligned)
    hipLaunchKernelGGL(bmuf_kernel<true>, dim3(blocks), dim3(256), 0, s, n, count, (double)workers,
                       models, stride, wg, delta, (double)eta, (double)eta_next, (double)zeta,
                       local, local_bf16);
  else
    hipLaunchKernelGGL(bmuf_kernel<false>, dim3(blocks), dim3(256), 0, s, n, count,
                       (double)workers, models, stride, wg, delta, (double)eta, (double)eta_next,
                       (double)zeta, local, local_bf16);
  return hipGetLastError();
}

}  // namespace am
