// The student's input frames and delayed targets (§II-B).
//
// lfr_features: for each utterance, raw frames (10 ms, raw_dim values each,
// utterances one after another) are stacked `stack` at a time at a `skip`
// advance from a frame offset, the causal mean of the stacked frames so far
// is subtracted, and the result is normalised by global per-dimension mean
// and standard deviation.  Output rows follow the model's packed time-major
// layout (frame (t, b) is row off_t + b), so utterances are given longest
// (in stacked frames) first.  One workgroup per utterance, one thread per
// stacked dimension walking the frames in order with the running sum in
// fp64; each value is evaluated in fp64 in the order of the definition with
// no fused multiply-add and rounded once to the output type, so the output is
// bit-identical to the element-wise definition.  Loads of the next 32 frames
// are kept in flight ahead of the running sum.
//
// delay_targets: the targets of the packed rows shifted by `delay` frames
// within each sequence (the model's look-ahead): row (t, b) takes the target
// of row (t - delay, b); rows with t < delay get idx -1, prob 0, mask 0.
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

// fp64 result -> output type, rounded once to fp32 (then to bf16 for a bf16
// model, round to nearest even).
template <typename T> __device__ __forceinline__ T from_f64(double v);
template <> __device__ __forceinline__ float from_f64<float>(double v) { return (float)v; }
template <> __device__ __forceinline__ bf16_t from_f64<bf16_t>(double v) { return f32_to_bf16((float)v); }

// Sum of one value per thread over a 256-thread workgroup (all threads get
// it).  `red` is 4 LDS slots; the call contains two barriers.
__device__ __forceinline__ int64_t block_sum(int64_t v, int64_t* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();  // earlier readers of red are done
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

template <typename OutT>
__global__ __launch_bounds__(256) void lfr_features_kernel(LfrArgs a) {
#pragma clang fp contract(off)
  const int b = blockIdx.x;
  const int D = a.stack * a.raw_dim;
  __shared__ uint16_t T_len[1024];
  __shared__ int64_t red[4];
  int64_t r0 = 0;  // raw frames of the utterances before this one
  for (int i = threadIdx.x; i < a.B; i += blockDim.x) {
    const int U = a.U[i];
    const int T = (U - a.offset - a.stack) / a.skip + 1;
    T_len[i] = (uint16_t)(U - a.offset - a.stack >= 0 ? T : 0);
    if (i < b) r0 += U;
  }
  r0 = block_sum(r0, red);  // its barriers also publish T_len
  const int Tb = T_len[b];
  const float* __restrict__ raw = a.raw + r0 * a.raw_dim;
  OutT* __restrict__ x = static_cast<OutT*>(a.x);
  for (int j = threadIdx.x; j < D; j += blockDim.x) {
    const int k = j / a.raw_dim, d = j % a.raw_dim;
    const double mean = (double)a.mean[j], sd = (double)a.std[j];
    double run = 0.0;
    int64_t off = 0;  // packed offset of frame t
    int nb = a.B;     // sequences longer than t
    constexpr int AH = 32;  // frames whose loads are in flight (one utterance per
                            // workgroup: fewer would leave HBM latency exposed)
    float ahead[AH];
#pragma unroll
    for (int q = 0; q < AH; ++q)
      ahead[q] = q < Tb ? raw[(int64_t)(a.offset + a.skip * q + k) * a.raw_dim + d] : 0.f;
    for (int t0 = 0; t0 < Tb; t0 += AH) {
#pragma unroll
      for (int q = 0; q < AH; ++q) {
        const int t = t0 + q;
        if (t >= Tb) break;
        const double y = (double)ahead[q];
        const int tn = t + AH;
        ahead[q] = tn < Tb ? raw[(int64_t)(a.offset + a.skip * tn + k) * a.raw_dim + d] : 0.f;
        run = run + y;
        const double z = y - run / (double)(t + 1);
        const double v = (z - mean) / sd;
        while (nb > 0 && T_len[nb - 1] <= t) --nb;
        x[(off + b) * D + j] = from_f64<OutT>(v);
        off += nb;
      }
    }
  }
}

__global__ __launch_bounds__(256) void delay_targets_kernel(DelayArgs a) {
  const int t = blockIdx.x;
  __shared__ int64_t red[4];
  // packed offsets of frames t and t - delay (off_t = sum of min(len_b, t))
  // and the sequences active at t
  const int ts = t >= a.delay ? t - a.delay : 0;
  int64_t o = 0, os = 0, c = 0;
  for (int b = threadIdx.x; b < a.B; b += blockDim.x) {
    const int len = a.len[b];
    o += len < t ? len : t;
    os += len < ts ? len : ts;
    c += len > t;
  }
  const int64_t s_off = block_sum(o, red);
  const int64_t s_src = block_sum(os, red);
  const int nb = (int)block_sum(c, red);
  const bool has = t >= a.delay;
  for (int e = threadIdx.x; e < nb * a.K; e += blockDim.x) {
    const int b = e / a.K, q = e % a.K;
    const int64_t dst = (s_off + b) * a.K + q;
    if (has) {
      const int64_t src = (s_src + b) * a.K + q;
      a.idx_out[dst] = a.idx[src];
      a.prob_out[dst] = a.prob[src];
    } else {
      a.idx_out[dst] = -1;
      a.prob_out[dst] = 0.f;
    }
  }
  for (int b = threadIdx.x; b < nb; b += blockDim.x) a.mask_out[s_off + b] = has ? 1 : 0;
}

}  // namespace

hipError_t lfr_features(const LfrArgs& a, bool bf16, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(lfr_features_kernel<bf16_t>, dim3(a.B), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(lfr_features_kernel<float>, dim3(a.B), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t delay_targets(const DelayArgs& a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  hipLaunchKernelGGL(delay_targets_kernel, dim3(a.T), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace am
