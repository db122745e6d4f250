// Device-side helpers shared by the gfx950 kernels of the training step.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace am {

typedef uint16_t bf16_t;  // bf16 storage: upper half of an IEEE binary32
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// fp32 -> bf16, round to nearest even; NaN becomes the quiet NaN 0x7FC0.
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)0x7FC0;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// Activation storage type <-> fp32.
template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t v) { return bf16_to_f32(v); }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float v) { return f32_to_bf16(v); }

// Saved gate activations of a row: unit j's four gates (i, f, g, o) sit
// together at 4j .. 4j+3, so one cell's gates move as one 8-byte (bf16) or
// 16-byte (fp32) access.
__device__ __forceinline__ uint2 pack_gates(float i, float f, float g, float o) {
  return make_uint2((uint32_t)f32_to_bf16(i) | ((uint32_t)f32_to_bf16(f) << 16),
                    (uint32_t)f32_to_bf16(g) | ((uint32_t)f32_to_bf16(o) << 16));
}
__device__ __forceinline__ void store_gates(bf16_t* grow, int j, uint2 packed) {
  *reinterpret_cast<uint2*>(grow + 4 * j) = packed;
}
__device__ __forceinline__ void store_gates(bf16_t* grow, int j, float i, float f, float g, float o) {
  store_gates(grow, j, pack_gates(i, f, g, o));
}
__device__ __forceinline__ void store_gates(float* grow, int j, float i, float f, float g, float o) {
  *reinterpret_cast<float4*>(grow + 4 * j) = make_float4(i, f, g, o);
}
__device__ __forceinline__ void load_gates(const bf16_t* grow, int j, bf16_t (&v)[4]) {
  const uint2 u = *reinterpret_cast<const uint2*>(grow + 4 * j);
  v[0] = (bf16_t)(u.x & 0xFFFFu); v[1] = (bf16_t)(u.x >> 16);
  v[2] = (bf16_t)(u.y & 0xFFFFu); v[3] = (bf16_t)(u.y >> 16);
}
__device__ __forceinline__ void load_gates(const float* grow, int j, float (&v)[4]) {
  const float4 u = *reinterpret_cast<const float4*>(grow + 4 * j);
  v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
}

// One MFMA operand fragment: 8 consecutive k-elements of one row (A) or one
// column (B) of a 16x16 output tile.  Lane l serves row/column l % 16 and
// the k-octet l / 16 of a 32-wide k-step.  The same k-octet mapping is used
// for both operands, so the product is independent of how the hardware
// orders k inside an instruction.
template <typename T> struct Frag;
template <> struct Frag<bf16_t> { uint4 v; };
template <> struct Frag<float> { float4 lo, hi; };

template <typename T> __device__ __forceinline__ Frag<T> frag_zero();
template <> __device__ __forceinline__ Frag<bf16_t> frag_zero<bf16_t>() {
  Frag<bf16_t> f; f.v = make_uint4(0, 0, 0, 0); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_zero<float>() {
  Frag<float> f; f.lo = make_float4(0.f, 0.f, 0.f, 0.f); f.hi = f.lo; return f;
}

// 8 elements starting at p (16-byte aligned for bf16, 32-byte for fp32).
template <typename T> __device__ __forceinline__ Frag<T> frag_load(const T* p);
template <> __device__ __forceinline__ Frag<bf16_t> frag_load<bf16_t>(const bf16_t* p) {
  Frag<bf16_t> f; f.v = *reinterpret_cast<const uint4*>(p); return f;
}
template <> __device__ __forceinline__ Frag<float> frag_load<float>(const float* p) {
  Frag<float> f;
  f.lo = reinterpret_cast<const float4*>(p)[0];
  f.hi = reinterpret_cast<const float4*>(p)[1];
  return f;
}

// acc(16x16) += A(16x32) * B(32x16).
__device__ __forceinline__ void mma_16x16x32(f32x4_t& acc, const Frag<bf16_t>& a,
                                             const Frag<bf16_t>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a.v),
                                                __builtin_bit_cast(bf16x8_t, b.v), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma_16x16x32(f32x4_t& acc, const Frag<float>& a,
                                             const Frag<float>& b) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, acc, 0, 0, 0);
}

// Output tile layout of a 16x16 MFMA: lane l holds rows 4*(l/16)+r, r=0..3,
// of column l%16.
__device__ __forceinline__ int mfma_row(int lane, int r) { return 4 * (lane >> 4) + r; }
__device__ __forceinline__ int mfma_col(int lane) { return lane & 15; }

// Logistic sigmoid and tanh from their definitions with the hardware
// exponential and reciprocal (about 1e-7 absolute error):
//   sigm(x) = 1 / (1 + e^-x),   tanh(x) = 2 sigm(2x) - 1.
// Both saturate correctly: e^-x overflows to +inf and its reciprocal is 0.
__device__ __forceinline__ float sigm(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}
__device__ __forceinline__ float tanh_f(float x) { return 2.0f * sigm(2.0f * x) - 1.0f; }

// One LSTM cell step of one unit (bf16 per-step paths) from its gate
// pre-activations (i, f, g, o) and c_{t-1}: the gates, c_t and h_t.  The
// products are rounded separately (no multiply-add contraction), so every
// kernel that calls this gets the same bits from the same inputs.
struct CellStep {
  float gi, gf, gg, go, c, h;
};
__device__ __forceinline__ CellStep lstm_cell_step(float a0, float a1, float a2, float a3,
                                                   float cprev) {
#pragma clang fp contract(off)
  CellStep r;
  r.gi = sigm(a0);
  r.gf = sigm(a1);
  r.gg = tanh_f(a2);
  r.go = sigm(a3);
  const float keep = r.gf * cprev;
  const float add = r.gi * r.gg;
  r.c = keep + add;
  r.h = r.go * tanh_f(r.c);
  return r;
}

// SGD step of one element: w <- fl32(w - lr * u) evaluated in fp64 (lr * u
// of two fp32 values is exact in fp64, so a fused or an unfused evaluation
// rounds identically); the bf16 copy is the round-to-nearest-even image of
// the new fp32 value.
__device__ __forceinline__ float sgd_one(float w, float u, double lr) {
  return (float)((double)w - lr * (double)u);
}

// Byte address of an LDS object (for instructions that take it in M0).
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// 16 bytes per lane from global memory straight to LDS at lds_base + 16 *
// lane (global_load_lds_dwordx4; lds_base is wave-uniform).  On gfx950 this
// moves about 2.5x the bytes per CU per clock of loads into VGPRs.  The load
// is counted by vmcnt and is invisible to the compiler's wait insertion, so
// the caller waits explicitly (wait_vm) before the data is read, with
// counts that leave the later stages' loads in flight.  M0 is a reserved
// register, which the compiler does not allocate; in the compiled kernels
// of this library no instruction but these loads reads it (no dynamically
// indexed register arrays, no LDS parameter loads), so the clobber only
// documents the write and its warning is silenced.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* src, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(lds_base) : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(N), other counters untouched.
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// The same wait as an opaque instruction, for counts that include loads the
// compiler issued itself: it neither drops nor merges the wait (its own
// bookkeeping may find such a count already met), and it still places its
// own waits before the first use of each of those loads.
template <int N> __device__ __forceinline__ void wait_vm_asm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// wait_vm_asm<n> for a count n that is a constant once the caller's loops
// are unrolled (the chain folds to one instruction); a count above N, or
// one left unresolved, waits for every load (vmcnt 0).
template <int N> __device__ __forceinline__ void wait_vm_n(int n) {
  if constexpr (N == 0) {
    wait_vm_asm<0>();
  } else {
    if (n == N) wait_vm_asm<N>();
    else wait_vm_n<N - 1>(n);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace am
