// One time step of one LSTM layer, forward and backward, with the recurrent
// product fused to the cell arithmetic.
//
// Work split (both directions): a 256-thread workgroup owns 16 hidden units
// j0..j0+15 and 64 consecutive active sequences of the step.  The recurrent
// product's k-range is split across the four waves (k-steps w, w+4, ...), so
// each wave streams a disjoint quarter of the operands straight from global
// memory into MFMA fragments; the four partial tiles are summed in LDS in a
// fixed order (deterministic), and each wave then finishes 16 of the 64 rows.
// In the 16x16 MFMA output layout a lane holds one unit for four rows; the
// forward product keeps the four gate tiles (i, f, g, o) of the same units
// side by side, so every lane has all four gate pre-activations of its
// (row, unit) pairs in registers and the cell update needs no exchange.
//
// Forward  (per active row b, unit j):
//   a = P[b] + h_{t-1}[b] Wh^T;  i,f,o = sigm, g = tanh;  c = f c_{t-1} + i g;
//   h = o tanh(c).  Stores h_t, c_t, the gate activations and a copy of h_{t-1}.
// Backward (reverse time):
//   dh = dH_above + dA_{t+1} Wh (rows still active at t+1);
//   do = dh tanh c;  dc = dh o (1 - tanh^2 c) + dc_{t+1};
//   di = dc g, dg = dc i, df = dc c_{t-1};  dc_t = dc f;
//   dA = [di i(1-i), df f(1-f), dg (1-g^2), do o(1-o)].
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int UNITS = 16;  // hidden units per workgroup
constexpr int ROWS = 64;   // active sequences per workgroup

template <typename T>
__global__ __launch_bounds__(256) void lstm_fwd_step_kernel(
    const T* __restrict__ P, const T* __restrict__ Wh, const T* __restrict__ hprev,
    const float* __restrict__ cprev, T* __restrict__ Hout, T* __restrict__ Hs,
    float* __restrict__ Cout, T* __restrict__ G, int nb, int H) {
  __shared__ f32x4_t red[4][4][4][64];  // [wave][row tile][gate][lane], 64 KB

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j0 = blockIdx.x * UNITS;
  const int b0 = blockIdx.y * ROWS;
  const int ksteps = (H + 31) / 32;
  const int koct = (lane >> 4) * 8;

  f32x4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[i][g] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // operands of the cell update (independent of the product); rows past the
  // active ones read a valid row (clamped) and are never stored
  const int j = j0 + mfma_col(lane);
  const int G4 = 4 * H;
  T pin[4][4], hp[4];
  float cpv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = min(b0 + wave * 16 + mfma_row(lane, r), nb - 1);
    const T* prow = P + (int64_t)row * G4;
#pragma unroll
    for (int g = 0; g < 4; ++g) pin[r][g] = prow[g * H + j];
    cpv[r] = cprev ? cprev[(int64_t)row * H + j] : 0.f;
    hp[r] = hprev ? hprev[(int64_t)row * H + j] : from_f32<T>(0.f);
  }

  if (hprev) {
    for (int ks = wave; ks < ksteps; ks += 4) {
      const int k = ks * 32 + koct;
      const bool kin = k < H;
      const int kc = kin ? k : 0;
      // Clamped, unmasked A loads: an output row depends only on its own A
      // row and rows past the active ones are not stored.  Only a ragged
      // k-tail (H % 32 != 0) zeroes the B fragments past H.
      Frag<T> a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = min(b0 + i * 16 + (lane & 15), nb - 1);
        a[i] = frag_load<T>(hprev + (int64_t)row * H + kc);
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int wrow = g * H + j0 + (lane & 15);
        b[g] = frag_load<T>(Wh + (int64_t)wrow * H + kc);
      }
      if (H % 32 != 0) {
#pragma unroll
        for (int g = 0; g < 4; ++g)
          if (!kin) b[g] = frag_zero<T>();
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) mma_16x16x32(acc[i][g], a[i], b[g]);
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int g = 0; g < 4; ++g) red[wave][i][g][lane] = acc[i][g];
  __syncthreads();

  f32x4_t s[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    s[g] = red[0][wave][g][lane];
    s[g] += red[1][wave][g][lane];
    s[g] += red[2][wave][g][lane];
    s[g] += red[3][wave][g][lane];
  }

#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = b0 + wave * 16 + mfma_row(lane, r);
    if (row >= nb) continue;
    const float ai = s[0][r] + to_f32<T>(pin[r][0]);
    const float af = s[1][r] + to_f32<T>(pin[r][1]);
    const float ag = s[2][r] + to_f32<T>(pin[r][2]);
    const float ao = s[3][r] + to_f32<T>(pin[r][3]);
    const float gi = sigm(ai), gf = sigm(af), gg = tanh_f(ag), go = sigm(ao);
    const float c = gf * cpv[r] + gi * gg;
    const float h = go * tanh_f(c);
    const int64_t o = (int64_t)row * H + j;
    Cout[o] = c;
    Hout[o] = from_f32<T>(h);
    Hs[o] = hp[r];
    store_gates(G + (int64_t)row * G4, j, gi, gf, gg, go);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void lstm_bwd_step_kernel(
    const T* __restrict__ dAnext, int nbn, const T* __restrict__ WhT,
    const T* __restrict__ dHa, const T* __restrict__ G, const float* __restrict__ C,
    const float* __restrict__ Cprev, float* __restrict__ dc, T* __restrict__ dA, int nb, int H) {
  __shared__ f32x4_t red[4][4][64];  // [wave][row tile][lane], 16 KB

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j0 = blockIdx.x * UNITS;
  const int b0 = blockIdx.y * ROWS;
  const int G4 = 4 * H;
  const int ksteps = G4 / 32;  // 4H is a multiple of 32 when H % 8 == 0
  const int koct = (lane >> 4) * 8;

  f32x4_t acc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  // operands of the cell backward (independent of the product); rows past
  // the active ones read a valid row (clamped) and are never stored
  const int j = j0 + mfma_col(lane);
  T gv[4][4], dhv[4];
  float cv[4], cpv[4], dcv[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row0 = b0 + wave * 16 + mfma_row(lane, r);
    const int row = min(row0, nb - 1);
    const int64_t o = (int64_t)row * H + j;
    load_gates(G + (int64_t)row * G4, j, gv[r]);
    cv[r] = C[o];
    cpv[r] = Cprev ? Cprev[o] : 0.f;
    dcv[r] = dc[o];  // used only where the sequence continues to t+1
    dhv[r] = dHa[o];
    (void)row0;
  }

  if (dAnext && b0 < nbn) {
    for (int ks = wave; ks < ksteps; ks += 4) {
      const int k = ks * 32 + koct;
      // clamped, unmasked loads; rows without a step t+1 are zeroed below
      Frag<T> a[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = min(b0 + i * 16 + (lane & 15), nbn - 1);
        a[i] = frag_load<T>(dAnext + (int64_t)row * G4 + k);
      }
      const Frag<T> b = frag_load<T>(WhT + (int64_t)(j0 + (lane & 15)) * G4 + k);
#pragma unroll
      for (int i = 0; i < 4; ++i) mma_16x16x32(acc[i], a[i], b);
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
  __syncthreads();
  f32x4_t s = red[0][wave][lane];
  s += red[1][wave][lane];
  s += red[2][wave][lane];
  s += red[3][wave][lane];

#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = b0 + wave * 16 + mfma_row(lane, r);
    if (row >= nb) continue;
    const int64_t o = (int64_t)row * H + j;
    const float gi = to_f32<T>(gv[r][0]), gf = to_f32<T>(gv[r][1]);
    const float gg = to_f32<T>(gv[r][2]), go = to_f32<T>(gv[r][3]);
    const bool cont = row < nbn;  // the sequence continues to step t+1
    const float dh = to_f32<T>(dhv[r]) + (cont ? s[r] : 0.f);
    const float tc = tanh_f(cv[r]);
    const float d_o = dh * tc;
    const float dcell = dh * go * (1.f - tc * tc) + (cont ? dcv[r] : 0.f);
    const float d_i = dcell * gg, d_g = dcell * gi, d_f = dcell * cpv[r];
    dc[o] = dcell * gf;
    T* arow = dA + (int64_t)row * G4;
    arow[j] = from_f32<T>(d_i * gi * (1.f - gi));
    arow[H + j] = from_f32<T>(d_f * gf * (1.f - gf));
    arow[2 * H + j] = from_f32<T>(d_g * (1.f - gg * gg));
    arow[3 * H + j] = from_f32<T>(d_o * go * (1.f - go));
  }
}

// The cell of one step on its own (bf16 activations), after the recurrent
// product of the step ran as a batched product into pre [nb][4H] fp32 (or
// pre == null: a zero h_{t-1}).  One thread per (row, unit), consecutive
// threads consecutive units.
__global__ __launch_bounds__(256) void lstm_cell_fwd_kernel(
    const float* __restrict__ pre, const bf16_t* __restrict__ P, const bf16_t* __restrict__ hprev,
    const float* __restrict__ cprev, bf16_t* __restrict__ Hout, bf16_t* __restrict__ Hs,
    float* __restrict__ Cout, bf16_t* __restrict__ G, int nb, int H) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)nb * H) return;
  const int64_t row = e / H;
  const int j = (int)(e - row * H);
  const int64_t G4 = 4 * (int64_t)H, pr = row * G4;
  float a[4];
#pragma unroll
  for (int g = 0; g < 4; ++g)
    a[g] = (pre ? pre[pr + g * H + j] : 0.f) + bf16_to_f32(P[pr + g * H + j]);
  const CellStep cs = lstm_cell_step(a[0], a[1], a[2], a[3], cprev ? cprev[e] : 0.f);
  Cout[e] = cs.c;
  Hout[e] = f32_to_bf16(cs.h);
  Hs[e] = hprev ? hprev[e] : (bf16_t)0;
  store_gates(G + pr, j, cs.gi, cs.gf, cs.gg, cs.go);
}

// The cell backward of one step: dh = dHa + dhrec (rows < nbn; dhrec holds
// the `splits` k-split partials [splits][nbn][H] fp32 of the batched product
// dA_{t+1} Wh, summed in split order), dc carried in dc.
__global__ __launch_bounds__(256) void lstm_cell_bwd_kernel(
    const float* __restrict__ dhrec, int splits, int nbn, const bf16_t* __restrict__ dHa,
    const bf16_t* __restrict__ G, const float* __restrict__ C, const float* __restrict__ Cprev,
    float* __restrict__ dc, bf16_t* __restrict__ dA, int nb, int H) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= (int64_t)nb * H) return;
  const int64_t row = e / H;
  const int j = (int)(e - row * H);
  const int64_t G4 = 4 * (int64_t)H;
  bf16_t gv[4];
  load_gates(G + row * G4, j, gv);
  const float gi = bf16_to_f32(gv[0]), gf = bf16_to_f32(gv[1]);
  const float gg = bf16_to_f32(gv[2]), go = bf16_to_f32(gv[3]);
  const bool cont = row < nbn;  // the sequence continues to step t+1
  float rec = 0.f;
  if (cont)
    for (int z = 0; z < splits; ++z) rec += dhrec[(int64_t)z * nbn * H + e];
  const float dh = bf16_to_f32(dHa[e]) + rec;
  const float tc = tanh_f(C[e]);
  const float d_o = dh * tc;
  const float dcell = dh * go * (1.f - tc * tc) + (cont ? dc[e] : 0.f);
  const float d_i = dcell * gg, d_g = dcell * gi, d_f = dcell * (Cprev ? Cprev[e] : 0.f);
  dc[e] = dcell * gf;
  bf16_t* arow = dA + row * G4;
  arow[j] = f32_to_bf16(d_i * gi * (1.f - gi));
  arow[H + j] = f32_to_bf16(d_f * gf * (1.f - gf));
  arow[2 * H + j] = f32_to_bf16(d_g * (1.f - gg * gg));
  arow[3 * H + j] = f32_to_bf16(d_o * go * (1.f - go));
}

// The same for four consecutive cells of one row per thread (H % 4 == 0):
// 16-byte loads of the partials and states, two of the 32 bytes of gates,
// 8-byte stores of each gate's dA.  Per cell the arithmetic is that of
// lstm_cell_bwd_kernel, in the same order, so the results are the same bits
// (at one cell per thread the B = 512, H = 1536 launch moved about 3.8 TB/s;
// this form took the wide model's backward class from 9.9-10.0 to 9.3-9.4 ms
// per training step).
__global__ __launch_bounds__(256) void lstm_cell_bwd4_kernel(
    const float* __restrict__ dhrec, int splits, int nbn, const bf16_t* __restrict__ dHa,
    const bf16_t* __restrict__ G, const float* __restrict__ C, const float* __restrict__ Cprev,
    float* __restrict__ dc, bf16_t* __restrict__ dA, int nb, int H) {
  const int64_t e0 = 4 * ((int64_t)blockIdx.x * 256 + threadIdx.x);
  if (e0 >= (int64_t)nb * H) return;
  const int64_t row = e0 / H;
  const int j0 = (int)(e0 - row * H);
  const int64_t G4 = 4 * (int64_t)H;
  const uint4 ga = *reinterpret_cast<const uint4*>(G + row * G4 + 4 * j0);
  const uint4 gb = *reinterpret_cast<const uint4*>(G + row * G4 + 4 * j0 + 8);
  const uint32_t gw[8] = {ga.x, ga.y, ga.z, ga.w, gb.x, gb.y, gb.z, gb.w};
  const bool cont = row < nbn;
  float rec[4] = {0.f, 0.f, 0.f, 0.f};
  if (cont)
    for (int z = 0; z < splits; ++z) {
      const float4 p = *reinterpret_cast<const float4*>(dhrec + (int64_t)z * nbn * H + e0);
      rec[0] += p.x; rec[1] += p.y; rec[2] += p.z; rec[3] += p.w;
    }
  const uint2 dh2 = *reinterpret_cast<const uint2*>(dHa + e0);
  const uint32_t dhw[2] = {dh2.x, dh2.y};
  const float4 c4 = *reinterpret_cast<const float4*>(C + e0);
  const float4 cp4 = Cprev ? *reinterpret_cast<const float4*>(Cprev + e0) : make_float4(0.f, 0.f, 0.f, 0.f);
  const float4 dc4 = cont ? *reinterpret_cast<const float4*>(dc + e0) : make_float4(0.f, 0.f, 0.f, 0.f);
  const float cv[4] = {c4.x, c4.y, c4.z, c4.w}, cpv[4] = {cp4.x, cp4.y, cp4.z, cp4.w};
  const float dcv[4] = {dc4.x, dc4.y, dc4.z, dc4.w};
  float dco[4];
  uint32_t a_i[2], a_f[2], a_g[2], a_o[2];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t w0 = gw[2 * k], w1 = gw[2 * k + 1];
    const float gi = bf16_to_f32((bf16_t)(w0 & 0xFFFFu)), gf = bf16_to_f32((bf16_t)(w0 >> 16));
    const float gg = bf16_to_f32((bf16_t)(w1 & 0xFFFFu)), go = bf16_to_f32((bf16_t)(w1 >> 16));
    const float dh = bf16_to_f32((bf16_t)((dhw[k >> 1] >> (16 * (k & 1))) & 0xFFFFu)) + rec[k];
    const float tc = tanh_f(cv[k]);
    const float d_o = dh * tc;
    const float dcell = dh * go * (1.f - tc * tc) + (cont ? dcv[k] : 0.f);
    const float d_i = dcell * gg, d_g = dcell * gi, d_f = dcell * cpv[k];
    dco[k] = dcell * gf;
    const uint32_t sh = 16 * (k & 1);
    const uint32_t vi = (uint32_t)f32_to_bf16(d_i * gi * (1.f - gi)) << sh;
    const uint32_t vf = (uint32_t)f32_to_bf16(d_f * gf * (1.f - gf)) << sh;
    const uint32_t vg = (uint32_t)f32_to_bf16(d_g * (1.f - gg * gg)) << sh;
    const uint32_t vo = (uint32_t)f32_to_bf16(d_o * go * (1.f - go)) << sh;
    if ((k & 1) == 0) {
      a_i[k >> 1] = vi; a_f[k >> 1] = vf; a_g[k >> 1] = vg; a_o[k >> 1] = vo;
    } else {
      a_i[k >> 1] |= vi; a_f[k >> 1] |= vf; a_g[k >> 1] |= vg; a_o[k >> 1] |= vo;
    }
  }
  *reinterpret_cast<float4*>(dc + e0) = make_float4(dco[0], dco[1], dco[2], dco[3]);
  bf16_t* arow = dA + row * G4 + j0;
  *reinterpret_cast<uint2*>(arow) = make_uint2(a_i[0], a_i[1]);
  *reinterpret_cast<uint2*>(arow + H) = make_uint2(a_f[0], a_f[1]);
  *reinterpret_cast<uint2*>(arow + 2 * H) = make_uint2(a_g[0], a_g[1]);
  *reinterpret_cast<uint2*>(arow + 3 * H) = make_uint2(a_o[0], a_o[1]);
}

}  // namespace

hipError_t lstm_cell_fwd(const float* pre, const LstmFwdStep& a, hipStream_t s) {
  if (a.nb <= 0) return hipSuccess;
  const int64_t cells = (int64_t)a.nb * a.hidden;
  hipLaunchKernelGGL(lstm_cell_fwd_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s,
                     pre, (const bf16_t*)a.P, (const bf16_t*)a.hprev, a.cprev, (bf16_t*)a.H,
                     (bf16_t*)a.Hs, a.C, (bf16_t*)a.G, a.nb, a.hidden);
  return hipGetLastError();
}

hipError_t lstm_cell_bwd(const float* dhrec, int splits, const LstmBwdStep& a, hipStream_t s) {
  if (a.nb <= 0) return hipSuccess;
  const int64_t cells = (int64_t)a.nb * a.hidden;
  if (a.hidden % 4 == 0) {
    hipLaunchKernelGGL(lstm_cell_bwd4_kernel, dim3((unsigned)((cells / 4 + 255) / 256)), dim3(256), 0, s,
                       dhrec, dhrec ? splits : 0, a.nbn, (const bf16_t*)a.dHa, (const bf16_t*)a.G, a.C,
                       a.Cprev, a.dc, (bf16_t*)a.dA, a.nb, a.hidden);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(lstm_cell_bwd_kernel, dim3((unsigned)((cells + 255) / 256)), dim3(256), 0, s,
                     dhrec, dhrec ? splits : 0, a.nbn, (const bf16_t*)a.dHa, (const bf16_t*)a.G, a.C, a.Cprev, a.dc,
                     (bf16_t*)a.dA, a.nb, a.hidden);
  return hipGetLastError();
}

hipError_t lstm_fwd_step(const LstmFwdStep& a, hipStream_t s) {
  if (a.nb <= 0) return hipSuccess;
  dim3 grid(a.hidden / UNITS, (a.nb + ROWS - 1) / ROWS);
  if (a.bf16)
    hipLaunchKernelGGL(lstm_fwd_step_kernel<bf16_t>, grid, dim3(256), 0, s,
                       (const bf16_t*)a.P, (const bf16_t*)a.Wh, (const bf16_t*)a.hprev, a.cprev,
                       (bf16_t*)a.H, (bf16_t*)a.Hs, a.C, (bf16_t*)a.G, a.nb, a.hidden);
  else
    hipLaunchKernelGGL(lstm_fwd_step_kernel<float>, grid, dim3(256), 0, s,
                       (const float*)a.P, (const float*)a.Wh, (const float*)a.hprev, a.cprev,
                       (float*)a.H, (float*)a.Hs, a.C, (float*)a.G, a.nb, a.hidden);
  return hipGetLastError();
}

hipError_t lstm_bwd_step(const LstmBwdStep& a, hipStream_t s) {
  if (a.nb <= 0) return hipSuccess;
  dim3 grid(a.hidden / UNITS, (a.nb + ROWS - 1) / ROWS);
  if (a.bf16)
    hipLaunchKernelGGL(lstm_bwd_step_kernel<bf16_t>, grid, dim3(256), 0, s,
                       (const bf16_t*)a.dAnext, a.nbn, (const bf16_t*)a.WhT, (const bf16_t*)a.dHa,
                       (const bf16_t*)a.G, a.C, a.Cprev, a.dc, (bf16_t*)a.dA, a.nb, a.hidden);
  else
    hipLaunchKernelGGL(lstm_bwd_step_kernel<float>, grid, dim3(256), 0, s,
                       (const float*)a.dAnext, a.nbn, (const float*)a.WhT, (const float*)a.dHa,
                       (const float*)a.G, a.C, a.Cprev, a.dc, (float*)a.dA, a.nb, a.hidden);
  return hipGetLastError();
}

}  // namespace am
