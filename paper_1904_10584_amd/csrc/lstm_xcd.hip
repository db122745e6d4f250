// XCD-local persistent LSTM layer kernels.
//
// The recurrence exchanges h_{t-1} (dA_{t+1} backward) between the
// workgroups that share a block of sequences at every step.  MI355X has 8
// XCDs, each with its own L2; an exchange through device memory pays a
// write-back of the producer's L2, an invalidation of the consumer's, and
// memory latency on every step.  Here the sequences are split into blocks,
// one or two per XCD, and the workgroups of a block all run on that XCD, so
// the exchange and the step barrier stay inside one L2:
//   * with m workgroups per block, workgroup i serves block i % 8 + 8 (i / 8m)
//     and unit slice (i / 8) % m (workgroups are dispatched to XCDs
//     round-robin); at start every workgroup records its XCC id and, unless
//     every block really is on one XCD, the kernel falls back to
//     device-scope release/acquire for its whole run;
//   * the step barrier is one 128-byte flag line per block: every member
//     stores its count of completed steps in its own word once its stores
//     of the step have completed, and one wave polls the line; within one
//     XCD both stay in its L2 (a store that the L1 passes through, polled
//     with non-temporal loads, which the L1 does not serve from a kept
//     line), a block spanning XCDs uses device-scope accesses and fences;
//   * every exchanged row is written once and read only after it was written,
//     so no consumer's L1 can hold a stale copy.
// A workgroup owns U hidden units (U % 4 == 0) of one block of RB sequences
// (RB = 16 or 32).  The forward product keeps the workgroup's 4U columns of
// W_h resident in registers in unit-major, gate-minor order, so a 16-column
// MFMA tile holds 4 units x 4 gates; reading the partial tiles back from
// LDS in 4x4-quad-transposed order then gives each lane all four gate
// pre-activations of one (sequence, unit).  The backward product keeps the
// U columns of W_h in registers too.
#include <cstdlib>

#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int NX = 8;                    // XCDs
constexpr unsigned SPIN_LIMIT = 1u << 22;

__device__ __forceinline__ unsigned xcc_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xfu;
}

// One-time check that the workgroups of this block share one XCD: each
// publishes its XCD (+1; the launch's sync slot starts zeroed) in its word
// of the block's line, and one wave waits for all members and compares.
// Only the block's members take part, with plain device-scope loads and
// stores: no read-modify-write, no cache write-back or invalidation.  Every
// member of a block returns the same answer; y.fenced forces the fenced
// exchange regardless (so that tests can run it).
__device__ bool check_local(const XcdSync& y, int blk, int us, int members, int* bad_sh) {
  unsigned* line = reinterpret_cast<unsigned*>(y.xcc) + blk * 32;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    if (lane == 0) __hip_atomic_store(line + us, xcc_id() + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    unsigned v = 0, spins = 0;
    for (;;) {
      v = lane < members ? __hip_atomic_load(line + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 1u;
      if (__all(v != 0)) break;
      if (++spins > SPIN_LIMIT) {
        if (lane == 0) __hip_atomic_store(y.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    const unsigned first = __shfl(v, 0, 64);
    const bool bad = __any(lane < members && v != first);
    if (lane == 0) *bad_sh = bad || y.fenced ? 1 : 0;
  }
  __syncthreads();
  return *bad_sh == 0;
}

// One poll of a flag word from the XCD's L2: a non-temporal load, which
// does not keep the line in the CU's L1 (an agent-coherent load, sc1, goes
// past the L2 to memory).
__device__ __forceinline__ unsigned poll_l2(const unsigned* p) {
  unsigned v;
  asm volatile("global_load_dword %0, %1, off nt\n\ts_waitcnt vmcnt(0)" : "=v"(v) : "v"(p) : "memory");
  return v;
}

// This workgroup's stores of the step have completed: publish its count of
// completed steps in its own word of the block's flag line (one 128-byte
// line of 32 words, word us for member us).  The store reaches the XCD's L2
// after the data stores it follows have completed there, so a poller that
// sees the count then reads the data from L2.  When a block spans XCDs the
// store is device-scope (it goes on to memory) after a release fence (a
// write-back of this XCD's L2); within one XCD the word stays in the L2,
// where the polls read it (a device-scope access would go past the L2 to
// memory: 1.5-3 % slower recurrences).
// Separate words need no atomic read-modify-write, which the L2 would
// serialise over the block's members.
__device__ __forceinline__ void xsignal(const XcdSync& y, bool local, int blk, int us,
                                        unsigned count) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    if (local) {
      __hip_atomic_store(y.flags + blk * 32 + us, count, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    } else {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      __hip_atomic_store(y.flags + blk * 32 + us, count, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Wait until every member of the block has published a count >= target.
// Wave `poller` polls: lane m < members reads member m's word (one request
// for the line; from the XCD's L2 with a non-temporal load, or with a
// device-scope load when the block spans XCDs) and the wave votes.  The other workgroups' exchanged rows are then read from
// the shared L2 (local) or after an acquire that invalidates this CU's
// caches (block spans XCDs).  Each poll waits for every load its wave has
// in flight, so the poller should be a wave with none outstanding.
__device__ __forceinline__ void xwait(const XcdSync& y, bool local, int blk, int members,
                                      unsigned target, int poller = 0) {
  if ((int)(threadIdx.x >> 6) == poller) {
    const int lane = threadIdx.x & 63;
    const unsigned* line = y.flags + blk * 32;
    unsigned spins = 0;
    for (;;) {
      const unsigned v = lane >= members ? target
                         : local ? poll_l2(line + lane)
                                 : __hip_atomic_load(line + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (__all(v >= target)) break;
      if (++spins > SPIN_LIMIT) {
        if (lane == 0) __hip_atomic_store(y.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (!local) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

// Block of sequences served by this workgroup: workgroup i runs on XCD
// i % 8 and serves block i % 8 + 8 (i / 8 / members), so with two blocks per
// XCD both of them sit on the XCD of their workgroups.
__device__ __forceinline__ int xcd_block(int members) {
  return (int)(blockIdx.x % NX) + NX * (int)(blockIdx.x / NX / members);
}

__device__ __forceinline__ int active_down(const PersistSchedule& ps, int nb, int t) {
  if (!ps.varlen) return ps.B;
  while (nb > 0 && (int)ps.lens[nb - 1] <= t) --nb;
  return nb;
}
__device__ __forceinline__ int active_up(const PersistSchedule& ps, int nb, int t) {
  if (!ps.varlen) return ps.B;
  while (nb < ps.B && (int)ps.lens[nb] > t) ++nb;
  return nb;
}

// ----------------------------------------------------------------- forward --
// Eight waves, two per SIMD (a single wave can issue independent MFMAs at
// about 87 % of the peak, but not also cover its own LDS and memory waits).
// Tile group g = wave % 4 owns the output tiles t = g + 4 ts
// (row tile t % MT, column tile t / MT; all tiles of a group share row tile
// g % MT); k-half kh = wave / 4 multiplies k-steps [kh KS/2, (kh+1) KS/2).
// The W_h fragments of a wave's tiles and k-steps stay in its registers for
// the whole launch.  Each step wave 0 polls the step barrier and waves 1-7
// copy the block's rows of h_{t-1} to LDS with direct loads (whole 128-byte
// lines), laid out line-major
// [H/64 lines][RB rows][128 B] with the 16-byte chunks of a row XOR-swizzled
// by row, and read back as MFMA fragments.  The two k-halves of a group
// publish their partial tiles to LDS: the k-half-0 wave finishes the first
// ceil(TPW/2) tiles, the k-half-1 wave the rest.  A step is signalled as soon
// as its h stores (the only exchanged data) are complete; the cell state,
// gate and h_{t-1} copies are stored after the signal.
template <int MT, int KS, int TPW, bool STG>
__global__ __launch_bounds__(512, 1) void lstm_fwd_xcd(PersistFwd a, PersistSchedule ps, XcdSync y) {
  constexpr int RB = 16 * MT;             // sequences per block
  constexpr int KH = KS / 2;              // k-steps per wave
  constexpr int FIN = (TPW + 1) / 2;      // tiles finished by the k-half-0 wave
  constexpr int HS_BYTES = RB * KS * 64;  // the block's h rows: RB x H bf16
  static_assert(KS % 2 == 0, "H must be a multiple of 64");
  extern __shared__ __align__(16) unsigned char lds[];
  bf16_t* hl = reinterpret_cast<bf16_t*>(lds);
  f32x4_t* red = reinterpret_cast<f32x4_t*>(lds + HS_BYTES);  // [8][TPW][64]
  // STG (U % 8 == 0): the block's cell states, h_{t-1} copies and gates of
  // the step, staged as rows of the unit slice (strides padded by 16 bytes,
  // which spreads a write's 16 rows over the LDS banks) and written out by
  // waves 1-7 after the signal as 16-byte row chunks: about 100 cache lines
  // per step instead of 16 per store instruction (768).
  unsigned char* stC = lds + HS_BYTES + 8 * TPW * 64 * 16;
  __shared__ int bad_sh;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = wave & 3, kh = wave >> 2;
  const int H = KS * 32, G4 = 4 * H, U = y.units;
  const int ntiles = MT * (U / 4);
  const int members = H / U;
  const int blk = xcd_block(members), us = (blockIdx.x / NX) % members;
  const int b0 = blk * RB, j0 = us * U;
  const int mw = g % MT;
  const int CSB = U * 4 + 16, HSB = U * 2 + 16, GSB = U * 8 + 16;  // staged row strides
  unsigned char* stH = stC + RB * CSB;
  unsigned char* stG = stH + RB * HSB;
  const bf16_t* __restrict__ P = static_cast<const bf16_t*>(a.P);
  const bf16_t* __restrict__ Wh = static_cast<const bf16_t*>(a.Wh);
  const bf16_t* __restrict__ h0 = static_cast<const bf16_t*>(a.h0);
  bf16_t* __restrict__ Hb = static_cast<bf16_t*>(a.H);
  bf16_t* __restrict__ Hs = static_cast<bf16_t*>(a.Hs);
  bf16_t* __restrict__ Gb = static_cast<bf16_t*>(a.G);

  // resident weights: column c of tile n is unit j0 + 4n + c/4, gate c%4
  Frag<bf16_t> wf[TPW][KH];
#pragma unroll
  for (int ts = 0; ts < TPW; ++ts) {
    const int t = g + 4 * ts;
    const int n = (t < ntiles ? t : 0) / MT;
    const int c = lane & 15;
    const int row = (c & 3) * H + j0 + 4 * n + (c >> 2);
#pragma unroll
    for (int s = 0; s < KH; ++s)
      wf[ts][s] = frag_load<bf16_t>(Wh + (int64_t)row * H + (kh * KH + s) * 32 + (lane >> 4) * 8);
  }
  const bool local = check_local(y, blk, us, members, &bad_sh);

  // The tiles this wave finishes ("own slots" o < FIN): tile index
  // ts = o (k-half 0) or FIN + o (k-half 1).  The lane's cells in tile t:
  // row mw*16 + 4(lane/16) + lane%4 of the block, unit j0 + 4(t/MT) + (lane%16)/4.
  const int qrow = mw * 16 + 4 * (lane >> 4) + (lane & 3);
  auto slot_ts = [&](int o) { return kh == 0 ? o : FIN + o; };
  auto slot_ok = [&](int o) { return slot_ts(o) < TPW && g + 4 * slot_ts(o) < ntiles; };
  auto unit = [&](int o) {
    const int t = g + 4 * slot_ts(o);
    return j0 + 4 * ((t < ntiles ? t : 0) / MT) + ((lane & 15) >> 2);
  };
  float c_reg[FIN];
  bf16_t h_reg[FIN];
#pragma unroll
  for (int o = 0; o < FIN; ++o) {
    const int b = min(b0 + qrow, ps.B - 1), j = unit(o);
    c_reg[o] = a.c0[(int64_t)b * H + j];
    h_reg[o] = h0 ? h0[(int64_t)b * H + j] : (bf16_t)0;
  }

  // The polling wave (wave 0) copies no h rows and issues no stores between
  // the signal and its next poll: a wave's memory counter retires in order,
  // so stores issued before the poll would hold up the poll's loads.  With
  // STG the staged rows are written out by waves 1-7; without, wave 0 stores
  // its cells' cell state, gates and h_{t-1} one step late, right after its
  // next poll, from dc / dg / dh (row drow, or -1).
  float dc[FIN];
  uint2 dg[FIN];
  bf16_t dh[FIN];
  int drow = -1;
  auto post_stores = [&](int row, const float* cv, const uint2* gv, const bf16_t* hv) {
#pragma unroll
    for (int o = 0; o < FIN; ++o) {
      if (!slot_ok(o)) continue;
      const int j = unit(o);
      const int64_t ofs = (int64_t)row * H + j;
      a.C[ofs] = cv[o];
      Hs[ofs] = hv[o];
      store_gates(Gb + (int64_t)row * G4, j, gv[o]);
    }
  };
  // every load so far (weights, state) is complete here, so the compiler
  // keeps no waits for them inside the loop
  wait_vm<0>();
  int nb = ps.B, off = 0, off_prev = 0;
  for (int t = 0; t < ps.T; ++t) {
    nb = active_down(ps, nb, t);
    if (b0 >= nb) break;  // this block of sequences has ended for good

    // Input projections of this lane's cells (independent of the exchange;
    // clamped, unmasked loads so that they issue back to back).  Waves 1-7
    // issue them before the exchange, so that they have the poll's time to
    // arrive; the polling wave issues its own after the poll, which would
    // otherwise wait for them (its memory counter retires in order).
    bf16_t pin[FIN][4];
    auto load_pin = [&]() {
      const bf16_t* prow = P + (int64_t)(off + min(b0 + qrow, nb - 1)) * G4;
#pragma unroll
      for (int o = 0; o < FIN; ++o)
#pragma unroll
        for (int q = 0; q < 4; ++q) pin[o][q] = prow[q * H + unit(o)];
    };
    if (wave != 0) load_pin();

    f32x4_t acc[TPW];
#pragma unroll
    for (int ts = 0; ts < TPW; ++ts) acc[ts] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const bf16_t* hsrc = h0;
    if (t > 0) {
      xwait(y, local, blk, members, (unsigned)t);
      hsrc = Hb + (int64_t)off_prev * H;
    }
    if (wave == 0 && drow >= 0) {
      post_stores(drow, dc, dg, dh);
      drow = -1;
    }
    if (wave == 0) load_pin();
    if (hsrc) {
      // the block's rows of h_{t-1} (inactive rows read an active one) to
      // LDS, by waves 1-7
      constexpr int RG = RB / 8, NQ = (KS / 2) * RG;
      if (wave > 0) {
        for (int q = wave - 1; q < NQ; q += 7) {
          const int line = q / RG, rg = q % RG;
          const int r = rg * 8 + (lane >> 3);
          const int chunk = line * 8 + ((lane & 7) ^ (r & 7));
          dma16(hsrc + (int64_t)min(b0 + r, nb - 1) * H + chunk * 8,
                __builtin_amdgcn_readfirstlane(lds_address(hl + (line * RB + rg * 8) * 64)));
        }
        wait_vm<0>();
      }
      __syncthreads();
      // A fragments in batches of up to four, each batch read before its
      // MFMAs (the resident weights leave room for four in registers)
      constexpr int AB = KH > 4 ? 4 : KH;
      const int r = mw * 16 + (lane & 15);
#pragma unroll
      for (int s0 = 0; s0 < KH; s0 += AB) {
        Frag<bf16_t> af[AB];
#pragma unroll
        for (int s = 0; s < AB; ++s) {
          const int c = (kh * KH + s0 + s) * 4 + (lane >> 4);
          af[s] = *reinterpret_cast<const Frag<bf16_t>*>(
              hl + ((c >> 3) * RB + r) * 64 + (((c & 7) ^ (r & 7)) << 3));
        }
        __builtin_amdgcn_sched_barrier(0);
        // unconditional: a tile past the last holds tile 0's weights and its
        // result is never used (a guard here would branch around each MFMA)
#pragma unroll
        for (int s = 0; s < AB; ++s)
#pragma unroll
          for (int ts = 0; ts < TPW; ++ts) mma_16x16x32(acc[ts], af[s], wf[ts][s0 + s]);
      }
    }

    // both k-halves publish all their partial tiles; each lane then reads
    // the two partials of its cells straight in transposed order (4x4 quads:
    // lane l takes, for row 4(l/16) + l%4, the 4 gates of its unit from
    // lanes (l & ~3) + q).  Selecting among the accumulators by the runtime
    // k-half instead would index them dynamically: compare/select chains.
#pragma unroll
    for (int ts = 0; ts < TPW; ++ts) red[(wave * TPW + ts) * 64 + lane] = acc[ts];
    __syncthreads();
    float gate[FIN][4];
#pragma unroll
    for (int o = 0; o < FIN; ++o) {
      const int ts = slot_ts(o) % TPW;
      const float* p0 = reinterpret_cast<const float*>(red + (g * TPW + ts) * 64 + (lane & ~3));
      const float* p1 = reinterpret_cast<const float*>(red + ((g + 4) * TPW + ts) * 64 + (lane & ~3));
#pragma unroll
      for (int q = 0; q < 4; ++q) gate[o][q] = p0[4 * q + (lane & 3)] + p1[4 * q + (lane & 3)];
    }

    const int b = b0 + qrow;
    const bool row_ok = b < nb;
    float cnew[FIN];
    bf16_t hprev[FIN];
#pragma unroll
    for (int o = 0; o < FIN; ++o) {
      hprev[o] = h_reg[o];
      gate[o][0] = sigm(gate[o][0] + bf16_to_f32(pin[o][0]));
      gate[o][1] = sigm(gate[o][1] + bf16_to_f32(pin[o][1]));
      gate[o][2] = tanh_f(gate[o][2] + bf16_to_f32(pin[o][2]));
      gate[o][3] = sigm(gate[o][3] + bf16_to_f32(pin[o][3]));
      cnew[o] = gate[o][1] * c_reg[o] + gate[o][0] * gate[o][2];
      const bf16_t h = f32_to_bf16(gate[o][3] * tanh_f(cnew[o]));
      if (row_ok && slot_ok(o)) {
        Hb[(int64_t)(off + b) * H + unit(o)] = h;
        c_reg[o] = cnew[o];
        h_reg[o] = h;
        if constexpr (STG) {
          const int u = unit(o) - j0;
          *reinterpret_cast<float*>(stC + qrow * CSB + 4 * u) = cnew[o];
          *reinterpret_cast<bf16_t*>(stH + qrow * HSB + 2 * u) = hprev[o];
          *reinterpret_cast<uint2*>(stG + qrow * GSB + 8 * u) =
              pack_gates(gate[o][0], gate[o][1], gate[o][2], gate[o][3]);
        }
      }
    }
    xsignal(y, local, blk, us, (unsigned)(t + 1));  // h stores complete; its barrier also orders the LDS reuse
    // stores only the backward pass reads
    if constexpr (STG) {
      // 16-byte chunks of the staged rows: C, then Hs, then G; chunk e of a
      // section with cpr chunks per row is row e / cpr (by a multiply: e is
      // small), chunk e % cpr
      if (wave > 0) {
        const int cC = U / 4, cH = U / 8, cG = U / 2;
        const int nC = RB * cC, nH = RB * cH, nG = RB * cG;
        auto divr = [](int e, int d) { return (int)(((unsigned)e * ((65536u + d - 1) / d)) >> 16); };
        for (int e = threadIdx.x - 64; e < nC + nH + nG; e += 448) {
          int r, c;
          const unsigned char* src;
          void* dst;
          if (e < nC) {
            r = divr(e, cC); c = e - r * cC;
            src = stC + r * CSB + 16 * c;
            dst = a.C + (int64_t)(off + b0 + r) * H + j0 + 4 * c;
          } else if (e < nC + nH) {
            const int f = e - nC;
            r = divr(f, cH); c = f - r * cH;
            src = stH + r * HSB + 16 * c;
            dst = Hs + (int64_t)(off + b0 + r) * H + j0 + 8 * c;
          } else {
            const int f = e - nC - nH;
            r = divr(f, cG); c = f - r * cG;
            src = stG + r * GSB + 16 * c;
            dst = Gb + (int64_t)(off + b0 + r) * G4 + 4 * j0 + 8 * c;
          }
          if (b0 + r < nb) *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
        }
      }
    } else {
    uint2 gp[FIN];
#pragma unroll
    for (int o = 0; o < FIN; ++o) gp[o] = pack_gates(gate[o][0], gate[o][1], gate[o][2], gate[o][3]);
    if (wave != 0) {
      if (row_ok) post_stores(off + b, cnew, gp, hprev);
    } else if (row_ok) {
#pragma unroll
      for (int o = 0; o < FIN; ++o) {
        dc[o] = cnew[o];
        dg[o] = gp[o];
        dh[o] = hprev[o];
      }
      drow = off + b;
    }
    }
    off_prev = off;
    off += nb;
  }
  if (wave == 0 && drow >= 0) post_stores(drow, dc, dg, dh);
}

// ---------------------------------------------------------------- backward --
// dh_rec[rows][units] = dA_{t+1}[rows][4H] W_h[4H][units]: output tiles of
// 16 units (the last one partly empty).  Eight waves split the 4H-long k
// range: wave w multiplies k-steps [w KW, (w+1) KW) and keeps the W_h^T
// fragments of those k-steps, for every unit tile, in registers.  Each wave
// fetches its k-slice of the block's dA_{t+1} rows itself, with direct loads
// into private LDS buffers in chunks of CH k-steps, so it waits only on its
// own loads: one buffer per chunk where the LDS holds them all (16-row
// blocks: three chunks, 96 KiB over the eight waves), else two used in turn.
// The eight partial products are summed in a fixed order through LDS; the
// cell backward (dc carried in registers) is spread over the first seven
// waves in items of one row per lane, an equal number per SIMD, while the
// last wave polls the step barrier.
constexpr int bwd_chunk_buffers(int MT, int KW) {
  const int ch = KW >= 4 ? 4 : KW, nch = KW / ch;
  const int fit = 160 * 1024 / (8 * 16 * MT * ch * 64);  // buffer sets the LDS holds
  return nch < fit ? nch : (fit < 2 ? fit : 2);
}
template <int MT, int NTU, int KW>
__global__ __launch_bounds__(512, 1) void lstm_bwd_xcd(PersistBwd a, PersistSchedule ps, XcdSync y) {
  constexpr int RB = 16 * MT;                 // sequences per block
  constexpr int CH = KW >= 4 ? 4 : KW;        // k-steps per chunk
  constexpr int NCH = KW / CH;                // chunks per step
  constexpr int NB = bwd_chunk_buffers(MT, KW);  // chunk buffers per wave
  constexpr int CPR = CH * 4;                 // 16-byte pieces per chunk row
  constexpr int SW = (CPR < 8 ? CPR : 8) - 1; // swizzle mask
  constexpr int CHB = RB * CH * 64;           // bytes per chunk
  constexpr int IPC = CHB / 1024;             // direct loads per chunk
  static_assert(KW % CH == 0 && IPC >= 1, "chunking");
  static_assert(NB >= 1 && NB <= NCH, "chunk buffers");
  static_assert(MT * NTU * 4 <= 32, "cell items: at most 8 per SIMD");
  extern __shared__ __align__(16) unsigned char lds[];
  bf16_t* buf = reinterpret_cast<bf16_t*>(lds + (threadIdx.x >> 6) * NB * CHB);
  f32x4_t* red = reinterpret_cast<f32x4_t*>(lds);  // [8][MT][NTU][64], after the products
  __shared__ int bad_sh;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = a.hidden, G4 = 4 * H, U = y.units;
  const int members = H / U;
  const int blk = xcd_block(members), us = (blockIdx.x / NX) % members;
  const int b0 = blk * RB, j0 = us * U;
  const bf16_t* __restrict__ WhT = static_cast<const bf16_t*>(a.WhT);
  const bf16_t* __restrict__ dHa = static_cast<const bf16_t*>(a.dHa);
  const bf16_t* __restrict__ Gb = static_cast<const bf16_t*>(a.G);
  bf16_t* __restrict__ dA = static_cast<bf16_t*>(a.dA);

  // resident W_h^T fragments (8 consecutive k of one unit: one 16-byte load
  // of the transposed W_h): k-step wave KW + s, unit tile n, lane column
  // c -> unit j0 + 16n + min(c, vc_n - 1) (vc_n = valid columns of tile n)
  Frag<bf16_t> wb[KW][NTU];
#pragma unroll
  for (int n = 0; n < NTU; ++n) {
    const int unit = j0 + 16 * n + min(lane & 15, min(16, U - 16 * n) - 1);
#pragma unroll
    for (int s = 0; s < KW; ++s)
      wb[s][n] = frag_load<bf16_t>(WhT + (int64_t)unit * G4 + (wave * KW + s) * 32 + (lane >> 4) * 8);
  }
  const bool local = check_local(y, blk, us, members, &bad_sh);

  // Cell work: items p = (row tile m, unit tile n, quad row r), MT NTU 4 of
  // them; item p covers, per lane, unit 16n + lane%16 and row
  // 16m + 4(lane/16) + r.  The last wave polls the barrier and takes none;
  // a wave's items run as one dependent chain (the phase is bound by its
  // latency, not by the SIMD's issue rate), so no wave takes more than
  // IPS = ceil(NI / 7): waves 0-3 (one per SIMD) IPS each, waves 4-6 the
  // rest, evenly (12 items: 2, 2, 2, 2 and 2, 1, 1).
  constexpr int NI = MT * NTU * 4, IPS = (NI + 6) / 7;
  constexpr int FIRST = NI < 4 * IPS ? NI : 4 * IPS, REST = NI - FIRST;
  const int wv = __builtin_amdgcn_readfirstlane(wave);  // (scalar: the item indices are wave-uniform)
  int i_lo, i_hi;
  if (wv < 4) {
    i_lo = min(NI, wv * IPS);
    i_hi = min(FIRST, i_lo + IPS);
  } else if (wv < 7) {
    const int w = wv - 4;
    i_lo = FIRST + w * (REST / 3) + min(w, REST % 3);
    i_hi = i_lo + REST / 3 + (w < REST % 3 ? 1 : 0);
  } else {
    i_lo = i_hi = NI;
  }
  const int nitems = i_hi - i_lo;  // at most IPS
  auto item_m = [&](int k) { return (i_lo + k) / (NTU * 4); };
  auto item_n = [&](int k) { return ((i_lo + k) / 4) % NTU; };
  auto item_r = [&](int k) { return (i_lo + k) % 4; };
  auto item_u = [&](int k) { return 16 * item_n(k) + (lane & 15); };  // unit within the slice
  auto item_j = [&](int k) { return j0 + (item_u(k) < U ? item_u(k) : 0); };
  auto item_row = [&](int k) { return item_m(k) * 16 + mfma_row(lane, item_r(k)); };
  float dc_reg[IPS];
#pragma unroll
  for (int k = 0; k < IPS; ++k) dc_reg[k] = 0.f;

  int nb = ps.T > 0 ? active_up(ps, 0, ps.T - 1) : 0;
  int off = ps.N - nb;
  int nb_next = 0, off_next = 0;
  unsigned done = 0;
  for (int t = ps.T - 1; t >= 0; --t) {
    if (t < ps.T - 1) {
      nb_next = nb;
      off_next = off;
      nb = active_up(ps, nb_next, t);
      off = off_next - nb;
    }
    if (b0 >= nb) continue;
    const int nb_prev = t > 0 ? active_up(ps, nb, t - 1) : 0;
    const int off_prev = off - nb_prev;

    // This wave's cell inputs (independent of the exchange), issued after
    // the first NB chunks' direct loads so that the chunk waits can leave
    // them in flight: NL loads (one instruction each), the same number in
    // every wave (clamped addresses for items past the wave's last), which
    // the wait counts below assume.  Issued before the exchange instead, they would sit ahead of
    // the chunks in the in-order memory counter and hold up the product.
    bf16_t gv[IPS][4], dhv[IPS];
    float cv[IPS], cpv[IPS];
    constexpr int NL = 4 * IPS;  // gates (8 bytes), c_t, c_{t-1}, dh_t per item
    auto load_cell = [&]() {
      const float* cprev_rows = t > 0 ? a.C + (int64_t)off_prev * H : a.c0;
#pragma unroll
      for (int k = 0; k < IPS; ++k) {
        const int b = min(b0 + item_row(k), nb - 1), j = item_j(k);
        const int64_t o = (int64_t)(off + b) * H + j;
        load_gates(Gb + (int64_t)(off + b) * G4, j, gv[k]);
        cv[k] = a.C[o];
        cpv[k] = cprev_rows[(int64_t)b * H + j];
        dhv[k] = dHa[o];
      }
    };

    f32x4_t acc[MT][NTU];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < NTU; ++n) acc[m][n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (b0 < nb_next) {
      // polled from the last wave, which has no cell work and no loads in flight
      xwait(y, local, blk, members, done, 7);
      const bf16_t* dAn = dA + (int64_t)off_next * G4 + wave * KW * 32;
      // chunk c of this wave's k-slice into buffer bi: RB rows x CH k-steps;
      // instruction i covers rows i*(64/CPR) .., 16-byte pieces swizzled by row
      auto issue = [&](int c, int bi) {
#pragma unroll
        for (int i = 0; i < IPC; ++i) {
          const int row = i * (64 / CPR) + lane / CPR;
          const int piece = (lane % CPR) ^ (row & SW);
          dma16(dAn + (int64_t)min(b0 + row, nb_next - 1) * G4 + c * CH * 32 + piece * 8,
                __builtin_amdgcn_readfirstlane(lds_address(buf + bi * (CHB / 2) + i * 512)));
        }
      };
      // the first NB chunks at once (every chunk where the buffers allow:
      // one memory latency per step rather than one per buffer round), then
      // the cell inputs; chunk c + NB goes into chunk c's buffer once c has
      // been read
#pragma unroll
      for (int c = 0; c < NB; ++c) issue(c, c);
      load_cell();
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        // in flight behind chunk c at its wait: the chunks issued after it
        // (up to c + NB - 1) and, while c is one of the first NB, the cell
        // loads
        wait_vm_n<40>(((c + NB < NCH ? c + NB : NCH) - c - 1) * IPC + (c < NB ? NL : 0));
        const bf16_t* bb = buf + (c % NB) * (CHB / 2);
#pragma unroll
        for (int ks = 0; ks < CH; ++ks) {
          Frag<bf16_t> af[MT];
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const int row = m * 16 + (lane & 15), piece = ks * 4 + (lane >> 4);
            af[m] = *reinterpret_cast<const Frag<bf16_t>*>(bb + row * CH * 32 + ((piece ^ (row & SW)) << 3));
          }
#pragma unroll
          for (int n = 0; n < NTU; ++n)
#pragma unroll
            for (int m = 0; m < MT; ++m) mma_16x16x32(acc[m][n], af[m], wb[c * CH + ks][n]);
        }
        if (c + NB < NCH) {
          __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this buffer's reads are done
          issue(c + NB, c % NB);
        }
      }
    } else {
      load_cell();
    }
    // fixed-order sum of the eight partial products
    __syncthreads();
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
      for (int n = 0; n < NTU; ++n) red[((wave * MT + m) * NTU + n) * 64 + lane] = acc[m][n];
    __syncthreads();

#pragma unroll
    for (int k = 0; k < IPS; ++k) {
      if (k >= nitems) break;  // (wave-uniform)
      // the eight partial products of this item's cell, in wave order
      const int m = item_m(k), n = item_n(k), r = item_r(k);
      float rec = 0.f;
#pragma unroll
      for (int w = 0; w < 8; ++w) rec += reinterpret_cast<const float*>(red + ((w * MT + m) * NTU + n) * 64 + lane)[r];
      const int b = b0 + item_row(k), j = item_j(k);
      if (item_u(k) >= U || b >= nb) continue;
      const bool cont = b < nb_next;
      const float vi = bf16_to_f32(gv[k][0]), vf = bf16_to_f32(gv[k][1]);
      const float vg = bf16_to_f32(gv[k][2]), vo = bf16_to_f32(gv[k][3]);
      const float dhh = bf16_to_f32(dhv[k]) + (cont ? rec : 0.f);
      const float tc = tanh_f(cv[k]);
      const float d_o = dhh * tc;
      const float dcell = dhh * vo * (1.f - tc * tc) + (cont ? dc_reg[k] : 0.f);
      const float d_i = dcell * vg, d_g = dcell * vi, d_f = dcell * cpv[k];
      dc_reg[k] = dcell * vf;
      bf16_t* arow = dA + (int64_t)(off + b) * G4;
      arow[j] = f32_to_bf16(d_i * vi * (1.f - vi));
      arow[H + j] = f32_to_bf16(d_f * vf * (1.f - vf));
      arow[2 * H + j] = f32_to_bf16(d_g * (1.f - vg * vg));
      arow[3 * H + j] = f32_to_bf16(d_o * vo * (1.f - vo));
    }
    ++done;
    xsignal(y, local, blk, us, done);  // its barrier also orders the LDS reuse
  }
}

// ------------------------------------------------------------------ launch --

// Units per workgroup: the least multiple of 4 dividing H with at most
// `members` workgroups per block.
int xcd_units(int H, int members) {
  for (int U = 4; U <= H; U += 4)
    if (H % U == 0 && H / U <= members) return U;
  return 0;
}

bool fits(const void* fn, int blocks, int threads, size_t lds) {
  int dev = 0, cus = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return false;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, fn, threads, lds) != hipSuccess) return false;
  return per > 0 && blocks <= per * cus;
}

template <typename K>
hipError_t coop(K kernel, int blocks, int threads, size_t lds, void** args, hipStream_t s,
                bool* used) {
  const void* fn = reinterpret_cast<const void*>(kernel);
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess ||
      !fits(fn, blocks, threads, lds)) {
    (void)hipGetLastError();
    *used = false;
    return hipSuccess;
  }
  *used = true;
  return resident_launch(fn, dim3(blocks), dim3(threads), args, lds, s);
}

// Shapes covered: bf16 (the resident slices are sized for it), B <= 256,
// hidden sizes with H % 64 == 0 and the resident weight slices within the
// register budget.  Blocks hold RB = 16 MT sequences; BPX blocks share an
// XCD, each served by 32 / BPX workgroups.  B > 128 takes blocks of 16, two
// per XCD (AM_XCD_BLOCKS=1 in the environment selects blocks of 32, one per
// XCD): per step each workgroup then reads half as many exchanged bytes
// (16 rows instead of 32) for twice as many units, and the backward's unit
// tiles are full (48 units = 3 x 16 instead of 24 = 16 + 8).
struct XShape {
  int MT, BPX, KS, U, NT, TPW, NTU, KW;
  bool ok;
};

XShape xshape(int H, int B) {
  XShape x{};
  x.ok = false;
  if (H % 64 != 0 || B > 256 || B < 1) return x;
  const char* e = getenv("AM_XCD_BLOCKS");
  const bool one = e && e[0] == '1' && e[1] == 0;
  x.MT = B > 128 && one ? 2 : 1;
  x.BPX = B > 128 && !one ? 2 : 1;
  x.KS = H / 32;
  x.U = xcd_units(H, 32 / x.BPX);
  if (x.U == 0) return x;
  x.NT = x.U / 4;
  x.TPW = (x.MT * x.NT + 3) / 4;
  x.NTU = (x.U + 15) / 16;
  x.KW = 4 * H / 32 / 8;  // backward k-steps per wave (eight waves)
  // resident weight fragments per wave (4 VGPRs each): forward TPW x KS/2,
  // backward KW x NTU
  x.ok = x.TPW * x.KS / 2 <= 36 && x.KW * x.NTU <= 36 && x.TPW <= 3 && x.NTU <= 3;
  return x;
}

}  // namespace

#define AM_FWD_CASE(MT_, KS_, TPW_, STG_)                                                \
  if (x.MT == MT_ && x.KS == KS_ && x.TPW == TPW_ && (x.U % 8 == 0) == STG_)             \
    return coop(lstm_fwd_xcd<MT_, KS_, TPW_, STG_>, blocks, 512, lds, args, s, used);

// AM_XCD_FENCED=1 in the environment: exchange with fences (as a block that
// spans XCDs does) even when every block sits on one XCD.
bool fenced_forced() {
  const char* e = getenv("AM_XCD_FENCED");
  return e && e[0] == '1' && e[1] == 0;
}

hipError_t lstm_fwd_xcd_launch(PersistFwd a, PersistSchedule ps, XcdSync y, hipStream_t s, bool* used) {
  *used = false;
  const XShape x = xshape(a.hidden, ps.B);
  if (!x.ok) return hipSuccess;
  y.units = x.U;
  y.fenced = fenced_forced() ? 1 : 0;
  const int blocks = NX * x.BPX * (a.hidden / x.U);
  // h rows, partial tiles, and (U % 8 == 0) the staged rows of C, Hs and G
  const size_t lds = (size_t)16 * x.MT * x.KS * 64 + 8 * x.TPW * 64 * 16 +
                     (x.U % 8 == 0 ? (size_t)16 * x.MT * (14 * x.U + 48) : 0);
  void* args[] = {&a, &ps, &y};
  // instantiated shapes: H = 768 (B <= 128, B <= 256 in blocks of 16 or 32),
  // H = 64, 128
  AM_FWD_CASE(1, 24, 3, true) AM_FWD_CASE(2, 24, 3, true) AM_FWD_CASE(1, 24, 2, true)
  AM_FWD_CASE(2, 2, 1, false) AM_FWD_CASE(1, 2, 1, false)
  AM_FWD_CASE(2, 4, 1, false) AM_FWD_CASE(1, 4, 1, false)
  AM_FWD_CASE(2, 4, 1, true) AM_FWD_CASE(1, 4, 1, true)
  return hipSuccess;
}

#define AM_BWD_CASE(MT_, NTU_, KW_)                                                       \
  if (x.MT == MT_ && x.NTU == NTU_ && x.KW == KW_)                                       \
    return coop(lstm_bwd_xcd<MT_, NTU_, KW_>, blocks, 512, lds, args, s, used);

hipError_t lstm_bwd_xcd_launch(PersistBwd a, PersistSchedule ps, XcdSync y, hipStream_t s, bool* used) {
  *used = false;
  const XShape x = xshape(a.hidden, ps.B);
  if (!x.ok) return hipSuccess;
  y.units = x.U;
  y.fenced = fenced_forced() ? 1 : 0;
  const int blocks = NX * x.BPX * (a.hidden / x.U);
  // the waves' private chunk buffers, or the partial products if larger
  const int ch = x.KW >= 4 ? 4 : x.KW;
  const size_t chunks = (size_t)8 * bwd_chunk_buffers(x.MT, x.KW) * 16 * x.MT * ch * 64;
  const size_t red = (size_t)8 * x.MT * x.NTU * 64 * 16;
  const size_t lds = chunks > red ? chunks : red;
  void* args[] = {&a, &ps, &y};
  AM_BWD_CASE(1, 3, 12) AM_BWD_CASE(2, 2, 12) AM_BWD_CASE(1, 2, 12)
  AM_BWD_CASE(2, 1, 1) AM_BWD_CASE(1, 1, 1)
  AM_BWD_CASE(2, 1, 2) AM_BWD_CASE(1, 1, 2)
  return hipSuccess;
}

bool lstm_xcd_instantiated(bool forward, int hidden, int B) {
  const XShape x = xshape(hidden, B);
  if (!x.ok) return false;
  if (forward)
    return (x.KS == 24 && ((x.MT == 2 && x.TPW == 3) || (x.MT == 1 && (x.TPW == 2 || x.TPW == 3)))) ||
           ((x.KS == 2 || x.KS == 4) && x.TPW == 1);
  return (x.KW == 12 && (x.NTU == 2 || (x.MT == 1 && x.NTU == 3))) ||
         ((x.KW == 1 || x.KW == 2) && x.NTU == 1);
}

}  // namespace am
