// Persistent LSTM layer kernels: one launch, whose grid fits on the device at
// once, runs every time step of one layer, forward or backward.
//
// Work split as in the single-step kernels: a workgroup owns 16 hidden units
// and 64 sequences, and its four waves split the recurrent product's k-range
// (k-steps w, w+4, ...).  What changes is what stays on chip across steps:
//   * each wave's slice of the recurrent weights is held in registers as
//     MFMA B fragments for the whole layer (read once, not once per step);
//   * the cell state c and the previous h (forward), and the carried dc
//     (backward), of each lane's (row, unit) pairs stay in registers;
//   * operands that do not depend on the recurrence (input projection, saved
//     gates, cell states, gradient from above) are loaded before the barrier.
// Step barrier: the workgroups that share a block of 64 sequences need each
// other's h_{t-1} (dA_{t+1} backward).  After its stores a workgroup makes
// them visible at device scope and increments that block's counter; before
// reading, it waits until the counter reaches (number of unit slices) x
// (steps the block has done).  The wait is bounded: past ~0.5 s it records an
// error flag and carries on, so every wave always reaches the end of the
// kernel.  The grid is sized to fit on the device (occupancy x CUs), so on
// an otherwise idle device all workgroups are resident (see resident_launch).
#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int UNITS = 16;
constexpr int ROWS = 64;
constexpr unsigned SPIN_LIMIT = 1u << 22;

// One thread waits; its device-scope acquire invalidates the CU's and the
// XCD's caches, which serves every wave of the workgroup after the barrier.
__device__ __forceinline__ void wait_counter(unsigned* cnt, unsigned target, int* err) {
  if (threadIdx.x == 0) {
    unsigned spins = 0;
    while (__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++spins > SPIN_LIMIT) {
        __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

// Each wave's stores complete (workgroup-scope release inside the barrier);
// then one thread writes the XCD's cache back (device-scope release) and
// publishes the step.
__device__ __forceinline__ void signal_counter(unsigned* cnt) {
  __builtin_amdgcn_s_waitcnt(0);  // this wave's stores have reached the L2
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// B_t (active sequences at step t) from B_{t-1} or from B_{t+1}; lengths
// are sorted non-increasing.
__device__ __forceinline__ int active_down(const PersistSchedule& ps, int nb, int t) {
  if (!ps.varlen) return ps.B;
  while (nb > 0 && (int)ps.lens[nb - 1] <= t) --nb;  // from B_{t-1} (>= B_t)
  return nb;
}
__device__ __forceinline__ int active_up(const PersistSchedule& ps, int nb, int t) {
  if (!ps.varlen) return ps.B;
  while (nb < ps.B && (int)ps.lens[nb] > t) ++nb;     // from B_{t+1} (<= B_t)
  return nb;
}

// ----------------------------------------------------------------- forward --

template <typename T, int KPW>
__global__ __launch_bounds__(256, 1) void lstm_fwd_persist(PersistFwd a, PersistSchedule ps) {
  // each wave's k-slices of Wh for the 4 gates of the 16 units, as MFMA B
  // fragments, resident for the whole layer: [wave][k-step][gate][lane]
  __shared__ Frag<T> wl[4][KPW][4][64];
  // partial sums a wave hands to the owners of the other row tiles:
  // [writer][slot][gate][lane], slot = tile index with the writer's own skipped
  __shared__ f32x4_t red[4][3][4][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = a.hidden, G4 = 4 * H;
  const int j0 = blockIdx.x * UNITS, b0 = blockIdx.y * ROWS;
  const int ksteps = (H + 31) / 32;
  const int koct = (lane >> 4) * 8;
  const T* __restrict__ P = static_cast<const T*>(a.P);
  const T* __restrict__ Wh = static_cast<const T*>(a.Wh);
  const T* __restrict__ h0 = static_cast<const T*>(a.h0);
  T* __restrict__ Hb = static_cast<T*>(a.H);
  T* __restrict__ Hs = static_cast<T*>(a.Hs);
  T* __restrict__ Gb = static_cast<T*>(a.G);
  unsigned* cnt = a.counters + blockIdx.y;
  const unsigned nunits = gridDim.x;

#pragma unroll
  for (int s = 0; s < KPW; ++s) {
    const int ks = wave + 4 * s;
    const int k = ks * 32 + koct;
#pragma unroll
    for (int g = 0; g < 4; ++g)
      wl[wave][s][g][lane] = (ks < ksteps && k < H)
                                 ? frag_load<T>(Wh + (int64_t)(g * H + j0 + (lane & 15)) * H + k)
                                 : frag_zero<T>();
  }

  // per-lane state of its (row, unit) pairs: rows b0 + 16 wave + 4(lane/16) + r
  const int j = j0 + mfma_col(lane);
  float c_reg[4];
  T h_reg[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int b = b0 + wave * 16 + mfma_row(lane, r);
    const bool ok = b < ps.B;
    c_reg[r] = ok ? a.c0[(int64_t)b * H + j] : 0.f;
    h_reg[r] = (ok && h0) ? h0[(int64_t)b * H + j] : from_f32<T>(0.f);
  }
  __syncthreads();

  int nb = ps.B, off = 0, off_prev = 0;
  for (int t = 0; t < ps.T; ++t) {
    nb = active_down(ps, nb, t);
    if (b0 >= nb) break;  // this block of sequences has ended for good

    // input projection of this step for the lane's pairs (no barrier needed);
    // rows past the active ones read a valid row and are never used
    T pin[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int b = min(b0 + wave * 16 + mfma_row(lane, r), nb - 1);
      const T* prow = P + (int64_t)(off + b) * G4;
#pragma unroll
      for (int g = 0; g < 4; ++g) pin[r][g] = prow[g * H + j];
    }

    f32x4_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) acc[i][g] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const T* hprev = h0;
    if (t > 0) {
      wait_counter(cnt, nunits * (unsigned)t, a.err);
      hprev = Hb + (int64_t)off_prev * H;
    }
    if (hprev) {
      // All A fragments are requested before the first product.  Addresses
      // are clamped (always valid) and what they return is not masked (a
      // select on a loaded value would serialise the loads): an output row
      // depends only on its own A row, rows past the active ones are never
      // stored, and past the end of k the B fragments are zero.
      Frag<T> af[KPW][4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const T* hrow = hprev + (int64_t)min(b0 + i * 16 + (lane & 15), nb - 1) * H + koct;
#pragma unroll
        for (int s = 0; s < KPW; ++s) {
          const int ks = wave + 4 * s;
          af[s][i] = frag_load<T>(hrow + ((ks < ksteps && ks * 32 + koct < H) ? ks * 32 : 0));
        }
      }
      __builtin_amdgcn_sched_barrier(0);  // keep every load ahead of the products
#pragma unroll
      for (int s = 0; s < KPW; ++s)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const Frag<T> bf = wl[wave][s][g][lane];
#pragma unroll
          for (int i = 0; i < 4; ++i) mma_16x16x32(acc[i][g], af[s][i], bf);
        }
    }

    // cross-wave sum in a fixed order: wave w owns row tile w
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i != wave) {
#pragma unroll
        for (int g = 0; g < 4; ++g) red[wave][i < wave ? i : i - 1][g][lane] = acc[i][g];
      }
    f32x4_t own[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (i == wave) {
#pragma unroll
        for (int g = 0; g < 4; ++g) own[g] = acc[i][g];
      }
    __syncthreads();
    f32x4_t sum[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      sum[g] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int v = 0; v < 4; ++v)
        sum[g] += v == wave ? own[g] : red[v][wave < v ? wave : wave - 1][g][lane];
    }

#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int b = b0 + wave * 16 + mfma_row(lane, r);
      if (b >= nb) continue;
      const float gi = sigm(sum[0][r] + to_f32<T>(pin[r][0]));
      const float gf = sigm(sum[1][r] + to_f32<T>(pin[r][1]));
      const float gg = tanh_f(sum[2][r] + to_f32<T>(pin[r][2]));
      const float go = sigm(sum[3][r] + to_f32<T>(pin[r][3]));
      const float c = gf * c_reg[r] + gi * gg;
      const T h = from_f32<T>(go * tanh_f(c));
      const int64_t o = (int64_t)(off + b) * H + j;
      a.C[o] = c;
      Hb[o] = h;
      Hs[o] = h_reg[r];
      store_gates(Gb + (int64_t)(off + b) * G4, j, gi, gf, gg, go);
      c_reg[r] = c;
      h_reg[r] = h;
    }
    // the barrier inside also keeps the next step's LDS writes after this
    // step's LDS reads
    signal_counter(cnt);
    off_prev = off;
    off += nb;
  }
}

// ---------------------------------------------------------------- backward --

// Backward: the recurrent product reduces over 4H, so per step a workgroup
// streams 64 rows x 4H of dA_{t+1}.  It runs 8 waves that split that k-range
// (k-steps w, w+8, ...), each with all of its A fragments in flight at once;
// the W_h^T fragments stay in LDS.  For the cell backward wave w takes row
// tile w % 4 and, of each lane's 4 rows, the pair w / 4.
template <typename T, int KPW>
__global__ __launch_bounds__(512, 1) void lstm_bwd_persist(PersistBwd a, PersistSchedule ps) {
  __shared__ Frag<T> wl[8][KPW][64];   // W_h^T fragments [wave][k-step][lane]
  __shared__ f32x4_t red[8][4][64];    // partial sums [wave][row tile][lane], 32 KB
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = a.hidden, G4 = 4 * H;
  const int j0 = blockIdx.x * UNITS, b0 = blockIdx.y * ROWS;
  const int ksteps = G4 / 32;
  const int koct = (lane >> 4) * 8;
  const T* __restrict__ Wh = static_cast<const T*>(a.Wh);
  const T* __restrict__ dHa = static_cast<const T*>(a.dHa);
  const T* __restrict__ Gb = static_cast<const T*>(a.G);
  T* __restrict__ dA = static_cast<T*>(a.dA);
  unsigned* cnt = a.counters + blockIdx.y;
  const unsigned nunits = gridDim.x;

  // B fragment of k-step ks: W_h^T[j][k .. k+7] = W_h[k .. k+7][j], j = j0 + lane%16
#pragma unroll
  for (int s = 0; s < KPW; ++s) {
    const int ks = wave + 8 * s;
    const int k = ks * 32 + koct;
    T v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      v[e] = ks < ksteps ? Wh[(int64_t)(k + e) * H + j0 + (lane & 15)] : from_f32<T>(0.f);
    Frag<T> f;
    memcpy(&f, v, sizeof f);
    wl[wave][s][lane] = f;
  }

  const int tile = wave & 3, rpair = wave >> 2;  // this wave's rows in the cell backward
  const int j = j0 + mfma_col(lane);
  float dc_reg[2] = {0.f, 0.f};
  __syncthreads();

  // schedule at the last step: B_{T-1} and its row offset N - B_{T-1}
  int nb = ps.T > 0 ? active_up(ps, 0, ps.T - 1) : 0;
  int off = ps.N - nb;
  int nb_next = 0, off_next = 0;  // step t+1
  unsigned done = 0;              // steps this block of sequences has finished
  for (int t = ps.T - 1; t >= 0; --t) {
    if (t < ps.T - 1) {
      nb_next = nb;
      off_next = off;
      nb = active_up(ps, nb_next, t);
      off = off_next - nb;
    }
    if (b0 >= nb) continue;  // no sequence of this block reaches step t
    const int nb_prev = t > 0 ? active_up(ps, nb, t - 1) : 0;
    const int off_prev = off - nb_prev;

    // operands that do not depend on other workgroups; rows past the active
    // ones read a valid row (clamped) and are never used
    T gi[2], gf[2], gg[2], go[2], dh[2];
    float cc[2], cp[2];
    const float* cprev_rows = t > 0 ? a.C + (int64_t)off_prev * H : a.c0;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int b = min(b0 + tile * 16 + mfma_row(lane, 2 * rpair + q), nb - 1);
      const int64_t o = (int64_t)(off + b) * H + j;
      T gq[4];
      load_gates(Gb + (int64_t)(off + b) * G4, j, gq);
      gi[q] = gq[0];
      gf[q] = gq[1];
      gg[q] = gq[2];
      go[q] = gq[3];
      cc[q] = a.C[o];
      cp[q] = cprev_rows[(int64_t)b * H + j];
      dh[q] = dHa[o];
    }

    f32x4_t acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (b0 < nb_next) {  // some sequence of the block continues to step t+1
      wait_counter(cnt, nunits * done, a.err);
      const T* dAn = dA + (int64_t)off_next * G4;
      // clamped, unmasked loads (see the forward kernel), in phases of at
      // most 6 k-steps whose loads are all in flight together; rows without
      // a step t+1 are zeroed after the reduction
      const T* arow[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        arow[i] = dAn + (int64_t)min(b0 + i * 16 + (lane & 15), nb_next - 1) * G4 + koct;
      constexpr int PH = KPW > 6 ? 6 : KPW;
#pragma unroll
      for (int s0 = 0; s0 < KPW; s0 += PH) {
        Frag<T> af[PH][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int s = 0; s < PH; ++s) {
            const int ks = wave + 8 * (s0 + s);
            af[s][i] = frag_load<T>(arow[i] + (s0 + s < KPW && ks < ksteps ? ks * 32 : 0));
          }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int s = 0; s < PH; ++s) {
          if (s0 + s >= KPW) break;
          const Frag<T> bf = wl[wave][s0 + s][lane];
#pragma unroll
          for (int i = 0; i < 4; ++i) mma_16x16x32(acc[i], af[s][i], bf);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][i][lane] = acc[i];
    __syncthreads();
    f32x4_t rec = red[0][tile][lane];
#pragma unroll
    for (int v = 1; v < 8; ++v) rec += red[v][tile][lane];

#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int r = 2 * rpair + q;
      const int b = b0 + tile * 16 + mfma_row(lane, r);
      if (b >= nb) continue;
      const bool cont = b < nb_next;  // the sequence continues to step t+1
      const float dcn = cont ? dc_reg[q] : 0.f;
      const float vi = to_f32<T>(gi[q]), vf = to_f32<T>(gf[q]);
      const float vg = to_f32<T>(gg[q]), vo = to_f32<T>(go[q]);
      const float dhh = to_f32<T>(dh[q]) + (cont ? rec[r] : 0.f);
      const float tc = tanh_f(cc[q]);
      const float d_o = dhh * tc;
      const float dcell = dhh * vo * (1.f - tc * tc) + dcn;
      const float d_i = dcell * vg, d_g = dcell * vi, d_f = dcell * cp[q];
      dc_reg[q] = dcell * vf;
      T* arow = dA + (int64_t)(off + b) * G4;
      arow[j] = from_f32<T>(d_i * vi * (1.f - vi));
      arow[H + j] = from_f32<T>(d_f * vf * (1.f - vf));
      arow[2 * H + j] = from_f32<T>(d_g * (1.f - vg * vg));
      arow[3 * H + j] = from_f32<T>(d_o * vo * (1.f - vo));
    }
    signal_counter(cnt);  // its barrier also orders this step's LDS reads
    ++done;
  }
}

// ------------------------------------------------------------------ launch --

struct Occ {
  int cus = 0;
};

bool fits(const void* fn, int blocks, int threads = 256) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
  int per = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, threads, 0) != hipSuccess) return false;
  return per > 0 && blocks <= per * cus;
}

template <typename K>
hipError_t coop(K kernel, dim3 grid, void** args, hipStream_t s, bool* used, int threads = 256) {
  if (!fits(reinterpret_cast<const void*>(kernel), (int)(grid.x * grid.y), threads)) {
    *used = false;
    return hipSuccess;
  }
  *used = true;
  return resident_launch(reinterpret_cast<const void*>(kernel), grid, dim3(threads), args, 0, s);
}

template <typename T>
hipError_t fwd_dispatch(PersistFwd& a, PersistSchedule& ps, hipStream_t s, bool* used) {
  const int kpw = ((a.hidden + 31) / 32 + 3) / 4;
  dim3 grid(a.hidden / UNITS, (ps.B + ROWS - 1) / ROWS);
  void* args[] = {&a, &ps};
  constexpr int MAXK = sizeof(T) == 2 ? 6 : 2;  // B fragments held in registers
  if (kpw > MAXK) { *used = false; return hipSuccess; }
  switch (kpw) {
    case 1: return coop(lstm_fwd_persist<T, 1>, grid, args, s, used);
    case 2: return coop(lstm_fwd_persist<T, 2>, grid, args, s, used);
    case 3: return coop(lstm_fwd_persist<T, sizeof(T) == 2 ? 3 : 2>, grid, args, s, used);
    case 4: return coop(lstm_fwd_persist<T, sizeof(T) == 2 ? 4 : 2>, grid, args, s, used);
    case 5: return coop(lstm_fwd_persist<T, sizeof(T) == 2 ? 5 : 2>, grid, args, s, used);
    default: return coop(lstm_fwd_persist<T, sizeof(T) == 2 ? 6 : 2>, grid, args, s, used);
  }
}

template <typename T>
hipError_t bwd_dispatch(PersistBwd& a, PersistSchedule& ps, hipStream_t s, bool* used) {
  const int kpw = (4 * a.hidden / 32 + 7) / 8;
  dim3 grid(a.hidden / UNITS, (ps.B + ROWS - 1) / ROWS);
  void* args[] = {&a, &ps};
  constexpr int MAXK = sizeof(T) == 2 ? 12 : 3;
  if (kpw > MAXK) { *used = false; return hipSuccess; }
  if (kpw <= 1) return coop(lstm_bwd_persist<T, 1>, grid, args, s, used, 512);
  if (kpw <= 2) return coop(lstm_bwd_persist<T, 2>, grid, args, s, used, 512);
  if (kpw <= 3) return coop(lstm_bwd_persist<T, 3>, grid, args, s, used, 512);
  if (kpw <= 6) return coop(lstm_bwd_persist<T, sizeof(T) == 2 ? 6 : 3>, grid, args, s, used, 512);
  return coop(lstm_bwd_persist<T, sizeof(T) == 2 ? 12 : 3>, grid, args, s, used, 512);
}

}  // namespace

bool lstm_persistent_fits(bool forward, int hidden, int B, bool bf16, int T) {
  if (B > 1024 || T > 65535 || hidden % UNITS) return false;
  const int blocks = (hidden / UNITS) * ((B + ROWS - 1) / ROWS);
  if (forward) {
    const int kpw = ((hidden + 31) / 32 + 3) / 4;
    if (kpw > (bf16 ? 6 : 2)) return false;
    return bf16 ? fits(reinterpret_cast<const void*>(lstm_fwd_persist<bf16_t, 6>), blocks)
                : fits(reinterpret_cast<const void*>(lstm_fwd_persist<float, 2>), blocks);
  }
  const int kpw = (4 * hidden / 32 + 7) / 8;
  if (kpw > (bf16 ? 12 : 3)) return false;
  return bf16 ? fits(reinterpret_cast<const void*>(lstm_bwd_persist<bf16_t, 12>), blocks, 512)
              : fits(reinterpret_cast<const void*>(lstm_bwd_persist<float, 3>), blocks, 512);
}

hipError_t lstm_fwd_persistent(PersistFwd a, PersistSchedule ps, bool bf16, hipStream_t s, bool* used) {
  return bf16 ? fwd_dispatch<bf16_t>(a, ps, s, used) : fwd_dispatch<float>(a, ps, s, used);
}

hipError_t lstm_bwd_persistent(PersistBwd a, PersistSchedule ps, bool bf16, hipStream_t s, bool* used) {
  return bf16 ? bwd_dispatch<bf16_t>(a, ps, s, used) : bwd_dispatch<float>(a, ps, s, used);
}

}  // namespace am
