// bf16 MFMA GEMM for gfx950: the batched products of the training step.
//   forward projections  P = X Wx^T + b,  Z = H Wo^T + bo      (A, B k-major)
//   data gradients       dH = dZ Wo,  dX = dA Wx              (B n-major)
//   weight gradients     [dWx | dWh] = dA^T [X | Hs],  dWo = dZ^T H
//                                                  (A m-major, B n-major)
// Design, from measurements on MI355X:
//   * operand tiles go from global memory straight to LDS (global_load_lds,
//     16 bytes per lane), which moves about 2.5x the bytes per CU per clock
//     of loads into VGPRs; fed through VGPRs, a GEMM tops out near a
//     quarter of the MFMA peak;
//   * a workgroup is eight waves (two per SIMD, one workgroup per CU): a
//     single wave issues independent MFMAs at about 87 % of the peak, but
//     four waves with 128 x 128 tiles each ran 25-40 % slower than eight,
//     also with the next k-step's fragments double-buffered in registers:
//     one wave per SIMD does not cover its own LDS waits and address work;
//   * a 256 x BN tile (BN = 256, or 192 where that fills the CUs) with waves
//     of 128 x BN/4 reads 384 bytes or less of LDS per MFMA; products of at
//     most 2048 rows take 128 x 128, 64 x 192 or 64 x 64 tiles, whichever
//     fills the CUs best, and one LSTM step's recurrent product can carry
//     the cell in its epilogue (CELL).
// Tiles keep their global layout in LDS:
//   * a k-major tile is [rows][64 k] (128 B per row); the fragment of a
//     16x16x32 MFMA (8 consecutive k of one row per lane) is one 16-byte LDS
//     read;
//   * an m/n-major tile is [64 k][rows]; the fragment is read with two
//     transposing LDS reads (ds_read_b64_tr_b16).  Within each group of 16
//     lanes, lane i receives element i % 4 of the 4-element pieces addressed
//     by lanes 4q + i / 4 (q = 0..3); so when lane j of the group addresses
//     k-row k0 + j / 4 at column c0 + 4 (j % 4), lane i receives column
//     c0 + i at k-rows k0 .. k0 + 3.
// Both layouts XOR-swizzle their 16-byte chunks (the direct-load lane that
// fills a slot fetches the chunk that belongs there), and an m/n-major row
// of more than 8 chunks also rotates them by 8 in the k-rows with bit 3 set:
// the two 16-lane groups served together by a transposing read address
// k-rows 8 apart, which the XOR alone puts on the same banks (the rotation
// took the weight gradients' bank-conflict cycles from 15.7 % to 5.3 %).
// This keeps the fragment reads nearly free of LDS bank conflicts and each
// 128-byte line of a tile row in one load instruction.  Chunks outside the
// operand are read from a zero vector.  The loads of k-tile t + NS - 1 are
// in flight while tile t is multiplied (NS LDS stages, explicit vmcnt waits,
// one barrier per k-tile).  Workgroups are dispatched to the 8 XCDs round-robin; the tile
// order gives each XCD a contiguous range of tiles, so tiles that share
// operand rows share an L2.  Weight gradients split K over workgroups (fp32
// partial tiles, summed in split order by splitk_reduce in gemm.hip); for an
// m-major A the first column of tiles also forms the row sums of A (the bias
// gradient) with one more MFMA per row tile against a fragment of ones.
#include <cstdlib>
#include <type_traits>

#include "am_device.h"
#include "am_internal.h"

namespace am {
namespace {

constexpr int BK = 64;    // k per tile
constexpr int BM0 = 256;  // tile rows (192 for some weight-gradient shapes)
constexpr int NT = 512;   // threads per workgroup (8 waves: 2 x 4)
constexpr int NW = 8;
constexpr int NX = 8;     // XCDs

__device__ uint4 g_zero[1];  // 16 zero bytes (the source of out-of-range chunks)

template <int BN, int BM> struct Cfg {
  static constexpr int WM = BM / 2;            // wave tile rows
  static constexpr int WN = BN / 4;            // wave tile columns
  static constexpr int MI = WM / 16;           // 8 or 6
  static constexpr int NJ = WN / 16;           // 4 or 3
  static constexpr int A_BYTES = BM * BK * 2;
  static constexpr int B_BYTES = BN * BK * 2;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  // LDS stages: 3 (2 for the largest tiles); small tiles, whose k-tiles
  // are short next to a memory round trip, keep up to 8 in flight
  static constexpr int NS = STAGE <= 32 * 1024 ? (8 * STAGE <= 150 * 1024 ? 8 : 150 * 1024 / STAGE)
                                               : (3 * STAGE <= 150 * 1024 ? 3 : 2);
  static constexpr int LDS = NS * STAGE;
  static constexpr int A_IPW = A_BYTES / 1024 / NW;  // direct loads per wave per tile
  static constexpr int B_IPW = B_BYTES / 1024 / NW;
  static constexpr int IPW = A_IPW + B_IPW;
  static_assert(A_BYTES % (1024 * NW) == 0 && B_BYTES % (1024 * NW) == 0, "tile split");
};

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// (a, b) -> packed bf16 pair, a in the low half (hardware conversion).
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;

// Element offset of chunk c (8 bf16) of row r in a k-major tile.
__device__ __forceinline__ int kofs(int r, int c) { return r * BK + ((c ^ (r & 7)) << 3); }
// Slot of chunk c in k-row k of an m/n-major tile of R columns: XOR with
// 2 (k % 4), then, where a row holds more than 8 chunks, rotated by 8 for
// the k-rows with bit 3 set.
template <int R> __device__ __forceinline__ int mslot(int k, int c) {
  constexpr int NC = R / 8;
  int x = c ^ ((k & 3) << 1);
  if (NC > 8 && (k & 8)) { x += 8; if (x >= NC) x -= NC; }
  return x;
}
// Chunk held by slot s of k-row k (the inverse of mslot).
template <int R> __device__ __forceinline__ int mchunk(int k, int s) {
  constexpr int NC = R / 8;
  if (NC > 8 && (k & 8)) { s -= 8; if (s < 0) s += NC; }
  return s ^ ((k & 3) << 1);
}
// Element offset of chunk c of k-row k in an m/n-major tile of R columns.
template <int R> __device__ __forceinline__ int mofs(int k, int c) {
  return k * R + (mslot<R>(k, c) << 3);
}

// Workgroup barrier without a memory fence (a fence would wait for every
// load in flight, including the later tiles' direct loads).  The empty asm
// statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void tile_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// One operand: rows (of the tile dimension) below `split` come from p0, the
// others from p1 at row - split.
struct Op {
  const bf16_t* p0; int64_t ld0;
  const bf16_t* p1; int64_t ld1;
  int split;
};

// Arguments of the LSTM cell epilogue (CELL kernels): the rows of step t.
struct CellArgs {
  const bf16_t* P;      // [nb][4H] input projection + bias
  const bf16_t* hprev;  // [nb][H] h_{t-1}
  const float* cprev;   // [nb][H] c_{t-1}, or null
  bf16_t* H;            // [nb][H] h_t
  bf16_t* Hs;           // [nb][H] copy of h_{t-1}
  float* C;             // [nb][H] c_t
  bf16_t* G;            // [nb][H][4] gates
  int hidden;
};

__device__ __forceinline__ const bf16_t* op_ptr(const Op& o, int row, int k, bool kmajor) {
  const bool sec = row >= o.split;
  const bf16_t* p = sec ? o.p1 : o.p0;
  const int64_t ld = sec ? o.ld1 : o.ld0;
  const int r = sec ? row - o.split : row;
  return kmajor ? p + (int64_t)r * ld + k : p + (int64_t)k * ld + r;
}

// Direct loads of one R-row operand tile: R * BK * 2 bytes in R / 8 loads of
// 1 KiB, R / 8 / NW per wave.  A k-major load fetches 8 rows x 8 chunks; an
// m/n-major load k-rows of R / 8 chunks laid end to end.  A load whose row
// is outside the operand, or whose k index has passed kend, reads the zero
// vector.  Two ways to address them:
//   * DirectLoader works out each address at the issue;
//   * TileLoader works them out once per workgroup: load j of this wave
//     keeps its source pointer and k index, and each issue advances both by
//     one k-tile (a load is issued once per k-tile, in k-tile order).  Used
//     where both operands are m/n-major (the weight gradients: 7 % faster);
//     on the other products the extra live registers cost more than the
//     address arithmetic they save.
template <bool KMAJOR, int R, int NL, bool GI = false>
struct DirectLoader {
  Op o;
  int row0, nrows, gh;

  __device__ __forceinline__ void init(const Op& o_, int row0_, int nrows_, int, int, int,
                                       int gh_ = 0) {
    o = o_;
    row0 = row0_;
    nrows = nrows_;
    gh = gh_;
  }
  __device__ __forceinline__ void issue(int j, int k0, int kend, const bf16_t* lds, int wave,
                                        int lane) {
    const int q = wave + NW * j;
    int row, k;
    if (KMAJOR) {
      const int r = 8 * q + (lane >> 3);
      row = row0 + r;
      k = k0 + (((lane & 7) ^ (r & 7)) << 3);
    } else {
      constexpr int CPR = R / 8;
      const int e = q * 64 + lane;  // chunk index in the tile
      const int kr = e / CPR;
      k = k0 + kr;
      row = row0 + (mchunk<R>(kr, e % CPR) << 3);
    }
    const bool ok = row < nrows && k < kend;
    // gate-interleaved: tile row 4u + g is operand row g * gh + u
    const int mrow = GI ? (row & 3) * gh + (row >> 2) : row;
    const void* src = ok ? (const void*)op_ptr(o, mrow, k, KMAJOR) : (const void*)g_zero;
    dma16(src, __builtin_amdgcn_readfirstlane(lds_address(lds + q * 512)));
  }
};

template <bool KMAJOR, int R, int NL>
struct TileLoader {
  static constexpr int L = NL > 0 ? NL : 1;
  const bf16_t* p[L];
  int kk[L];
  int inc[L];  // elements per k-tile (m-major: BK rows of the lane's source)

  __device__ __forceinline__ void init(const Op& o, int row0, int nrows, int k0, int wave,
                                       int lane) {
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int q = wave + NW * j;
      int row, k;
      if (KMAJOR) {
        const int r = 8 * q + (lane >> 3);
        row = row0 + r;
        k = k0 + (((lane & 7) ^ (r & 7)) << 3);
      } else {
        constexpr int CPR = R / 8;
        const int e = q * 64 + lane;
        const int kr = e / CPR;
        k = k0 + kr;
        row = row0 + (mchunk<R>(kr, e % CPR) << 3);
      }
      const bool sec = row >= o.split;
      const bf16_t* base = sec ? o.p1 : o.p0;
      const int64_t ld = sec ? o.ld1 : o.ld0;
      const int r = sec ? row - o.split : row;
      const bool in = row < nrows;
      p[j] = in ? (KMAJOR ? base + (int64_t)r * ld + k : base + (int64_t)k * ld + r) : base;
      kk[j] = in ? k : (1 << 30);
      inc[j] = KMAJOR ? BK : (int)(BK * ld);
    }
  }
  __device__ __forceinline__ void issue(int j, int, int kend, const bf16_t* lds, int wave, int) {
    const int q = wave + NW * j;
    const void* src = kk[j] < kend ? (const void*)p[j] : (const void*)g_zero;
    dma16(src, __builtin_amdgcn_readfirstlane(lds_address(lds + q * 512)));
    p[j] += KMAJOR ? BK : inc[j];
    kk[j] += BK;
  }
};

// Fragment of rows/columns r0 .. r0+15, k-step ks of an R-row tile.
template <bool KMAJOR, int R>
__device__ __forceinline__ Frag<bf16_t> frag(const bf16_t* lds, int r0, int ks, int lane) {
  Frag<bf16_t> f;
  if (KMAJOR) {
    f.v = *reinterpret_cast<const uint4*>(lds + kofs(r0 + (lane & 15), ks * 4 + (lane >> 4)));
  } else {
    const int j = lane & 15;
    const int k = ks * 32 + (lane >> 4) * 8 + (j >> 2);
    const int col = r0 + ((j & 3) << 2);
    const int c = col >> 3, half = col & 7;
    const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s_t*)(lds + mofs<R>(k, c) + half));
    const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s_t*)(lds + mofs<R>(k + 4, c) + half));
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

// Epilogue through LDS.  The accumulators of a 16x16 MFMA tile sit as four
// rows of one column per lane, so storing them straight to a row-major
// output takes one 2- or 4-byte store per element (1024 store instructions
// per 256x256 bf16 tile), which is slower than the tile's products.  Here
// the waves write their tiles to LDS in the output's row-major order (the
// stage buffers are free once the k-loop is done), then every thread copies
// whole 16-byte chunks of rows to global memory.  bf16: adjacent lanes swap
// half their values (a DPP swap) so each lane writes 4-byte pairs of
// columns.  LDS rows are BN elements; the 16-byte chunks of row R are
// XOR-permuted by (R / 4) % 4 times 32 bytes, so the four row groups one
// write instruction touches fall in different banks.  fp32 tiles go through
// LDS in two passes of BM / 2 rows.  Requires (checked by the launcher) output
// row pitches and the column split a multiple of 16 bytes and N of the
// chunk width.
template <typename OutT, int BN, int BM, bool BIAS>
__device__ __forceinline__ void store_tile_staged(const f32x4_t (&acc)[BM / 2 / 16][BN / 4 / 16],
                                                  const Out<OutT>& C, const bf16_t* bias,
                                                  bf16_t* smem, int M, int N, int m0, int n0,
                                                  int z, int wm, int wn, int wave, int lane) {
  constexpr int MI = BM / 2 / 16, NJ = BN / 4 / 16;
  constexpr int ES = sizeof(OutT);
  constexpr int ROWB = BN * ES;              // LDS bytes per tile row
  constexpr int CPR = ROWB / 16;             // 16-byte chunks per row
  constexpr int EPC = 16 / ES;               // elements per chunk
  constexpr int PASSES = ES == 2 ? 1 : 2;
  constexpr int PROWS = BM / PASSES;         // rows per pass
  unsigned char* lds = reinterpret_cast<unsigned char*>(smem);
  auto swz = [](int row, int chunk) { return chunk ^ (((row >> 2) & 3) * (32 / 16)); };
  const uint32_t odd = (lane & 1) ? 0xFFFFFFFFu : 0u;  // lane parity as a mask
  __syncthreads();  // every wave is done with the stage buffers
#pragma unroll
  for (int p = 0; p < PASSES; ++p) {
    if (PASSES == 1 || (wave >> 2) == p) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int cl = wn + j * 16 + mfma_col(lane);  // column within the tile
        const float bv = (BIAS && n0 + cl < N) ? bf16_to_f32(bias[n0 + cl]) : 0.f;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int rl = wm + i * 16 + mfma_row(lane, 0) - p * PROWS;  // first of 4 rows
          if (ES == 2) {
            // rows (0, 1) and (2, 3) of column cl, each pair rounded to bf16
            // by one hardware conversion (round to nearest; an output, not
            // a quantity compared bit for bit)
            const uint32_t p01 = pk_bf16(acc[i][j][0] + bv, acc[i][j][1] + bv);
            const uint32_t p23 = pk_bf16(acc[i][j][2] + bv, acc[i][j][3] + bv);
            // odd lanes give p01, even lanes p23 (masks, not per-lane
            // branches)
            const uint32_t give = (p01 & odd) | (p23 & ~odd);
            // quad_perm [1,0,3,2]: lane l receives lane l ^ 1
            const uint32_t got = (uint32_t)__builtin_amdgcn_mov_dpp((int)give, 0xB1, 0xF, 0xF, false);
            // even lane: rows 0, 1 of columns (cl, cl + 1); odd lane: rows 2, 3
            // of columns (cl - 1, cl).  lo / hi: the lower / upper column's pair.
            const uint32_t lo = (got & odd) | (p01 & ~odd);
            const uint32_t hi = (p23 & odd) | (got & ~odd);
            const uint32_t w0 = __builtin_amdgcn_perm(hi, lo, 0x05040100u);  // first rows
            const uint32_t w1 = __builtin_amdgcn_perm(hi, lo, 0x07060302u);  // second rows
            const int c0 = cl & ~1, r0 = rl + ((lane & 1) << 1);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int row = r0 + h;
              const int byte = c0 * 2;
              const int off = row * ROWB + swz(row, byte >> 4) * 16 + (byte & 15);
              *reinterpret_cast<uint32_t*>(lds + off) = h ? w1 : w0;
            }
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = rl + r;
              const int byte = cl * 4;
              const int off = row * ROWB + swz(row, byte >> 4) * 16 + (byte & 15);
              *reinterpret_cast<float*>(lds + off) = acc[i][j][r] + bv;
            }
          }
        }
      }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < PROWS * CPR; e += NT) {
      const int row = e / CPR, ch = e % CPR;
      const int grow = m0 + p * PROWS + row, gcol = n0 + ch * EPC;
      if (grow < M && gcol < N) {
        const uint4 v = *reinterpret_cast<const uint4*>(lds + row * ROWB + swz(row, ch) * 16);
        const bool sec = gcol >= C.split;
        OutT* cb = (sec ? C.c1 : C.c0) + (int64_t)z * C.zstride;
        const int64_t ldc = sec ? C.ld1 : C.ld0;
        const int cc = sec ? gcol - C.split : gcol;
        *reinterpret_cast<uint4*>(cb + (int64_t)grow * ldc + cc) = v;
      }
    }
    if (p + 1 < PASSES) __syncthreads();
  }
}

// LSTM cell epilogue of a gate-interleaved tile (column 4u + g is gate g of
// unit n0 / 4 + u).  Each thread takes ITEMS (row, unit) items, consecutive
// threads consecutive units of one row.  After the k-loop the items'
// operands that do not depend on the product (the input projection's four
// gates, c_{t-1}, h_{t-1}) are all loaded at once (cell_load), while the
// fp32 accumulators (the recurrent part of the gate pre-activations) go to
// LDS in row-major order; then each item runs the cell (cell_finish, with
// lstm_cell_step as lstm_cell_fwd_kernel).  The epilogue's one-time reads
// and the outputs kept for the backward are non-temporal: each XCD's tiles
// share a fixed slice of W_h's rows (2.4 MB at H = 1536, B = 512), which
// then stays in that XCD's L2 from one step to the next.  Needs BM x (BN +
// 4) x 4 bytes of LDS.
template <int BN, int BM> struct CellItems {
  static constexpr int UPR = BN / 4;                 // units per tile row
  static constexpr int ITEMS = BM * UPR / NT;
  static_assert(BM * UPR % NT == 0, "items per thread");
  uint32_t p01[ITEMS], p23[ITEMS];  // P's gates (i, f) and (g, o) as bf16 pairs
  float cp[ITEMS];
  bf16_t hp[ITEMS];
};

template <int BN, int BM>
__device__ __forceinline__ void cell_load(CellItems<BN, BM>& it, const CellArgs& c, int M,
                                          int m0, int n0) {
  using CI = CellItems<BN, BM>;
  const int H = c.hidden;
#pragma unroll
  for (int q = 0; q < CI::ITEMS; ++q) {
    const int e = threadIdx.x + q * NT;
    const int row = m0 + e / CI::UPR, j = n0 / 4 + e % CI::UPR;
    it.p01[q] = it.p23[q] = 0u;
    it.cp[q] = 0.f;
    it.hp[q] = 0;
    if (row < M && j < H) {
      // (read once: non-temporal, so that they do not evict W_h's rows)
      const bf16_t* pr = c.P + (int64_t)row * 4 * H + j;
      it.p01[q] = (uint32_t)__builtin_nontemporal_load(pr) |
                  ((uint32_t)__builtin_nontemporal_load(pr + H) << 16);
      it.p23[q] = (uint32_t)__builtin_nontemporal_load(pr + 2 * H) |
                  ((uint32_t)__builtin_nontemporal_load(pr + 3 * H) << 16);
      const int64_t o = (int64_t)row * H + j;
      if (c.cprev) it.cp[q] = __builtin_nontemporal_load(c.cprev + o);
      it.hp[q] = c.hprev[o];
    }
  }
}

template <int BN, int BM>
__device__ __forceinline__ void cell_finish(const f32x4_t (&acc)[BM / 2 / 16][BN / 4 / 16],
                                            const CellItems<BN, BM>& it, const CellArgs& c,
                                            bf16_t* smem, int M, int m0, int n0, int wm, int wn,
                                            int lane) {
  using CI = CellItems<BN, BM>;
  constexpr int MI = BM / 2 / 16, NJ = BN / 4 / 16;
  constexpr int ROWF = BN + 4;  // floats per LDS row (padded against bank conflicts)
  float* lds = reinterpret_cast<float*>(smem);
  __syncthreads();  // every wave is done with the stage buffers
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int cl = wn + j * 16 + mfma_col(lane);
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) lds[(wm + i * 16 + mfma_row(lane, r)) * ROWF + cl] = acc[i][j][r];
  }
  __syncthreads();
  const int H = c.hidden;
#pragma unroll
  for (int q = 0; q < CI::ITEMS; ++q) {
    const int e = threadIdx.x + q * NT;
    const int rl = e / CI::UPR, u = e % CI::UPR;
    const int row = m0 + rl, j = n0 / 4 + u;
    if (row >= M || j >= H) continue;
    const float4 rec = *reinterpret_cast<const float4*>(lds + rl * ROWF + 4 * u);
    const float a0 = rec.x + bf16_to_f32((bf16_t)(it.p01[q] & 0xFFFFu));
    const float a1 = rec.y + bf16_to_f32((bf16_t)(it.p01[q] >> 16));
    const float a2 = rec.z + bf16_to_f32((bf16_t)(it.p23[q] & 0xFFFFu));
    const float a3 = rec.w + bf16_to_f32((bf16_t)(it.p23[q] >> 16));
    const CellStep cs = lstm_cell_step(a0, a1, a2, a3, it.cp[q]);
    const int64_t o = (int64_t)row * H + j;
    // h_t is the next step's operand; c_t, the h_{t-1} copy and the gates
    // wait for the backward: non-temporal
    __builtin_nontemporal_store(cs.c, c.C + o);
    c.H[o] = f32_to_bf16(cs.h);
    __builtin_nontemporal_store(it.hp[q], c.Hs + o);
    const uint2 pk = pack_gates(cs.gi, cs.gf, cs.gg, cs.go);
    uint32_t* gp = reinterpret_cast<uint32_t*>(c.G + (int64_t)row * 4 * H + 4 * j);
    __builtin_nontemporal_store(pk.x, gp);
    __builtin_nontemporal_store(pk.y, gp + 1);
  }
}

// ROWSUM: A is m-major; the workgroups of the first column of tiles write
// the row sums of A over their split's k-range to rowsum[z * M + m].
// CELL: the LSTM cell epilogue (B's rows gate-interleaved; C unused).
template <bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM, int BN, int BM,
          bool CELL = false>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(
    Op A, Op B, Out<OutT> C, const bf16_t* __restrict__ bias, float* __restrict__ rowsum,
    int M, int N, int K, int kps, int tm, int tn, int S, int flags, CellArgs cell) {
  using CF = Cfg<BN, BM>;
  extern __shared__ __align__(16) bf16_t smem[];

  // XCD-contiguous tile order: workgroup b runs on XCD b % 8.
  const int G = tm * tn * S;
  const int b = blockIdx.x, x = b % NX, q = G / NX, rem = G % NX;
  const int T = x * q + min(x, rem) + b / NX;
  const int z = T / (tm * tn), t2 = T % (tm * tn);
  // tile order: n fastest (consecutive tiles share rows of A), or, with
  // few row tiles (flags & 2), m fastest (consecutive tiles share B)
  const bool mfast = (flags & 2) != 0;
  const int m0 = (mfast ? t2 % tm : t2 / tn) * BM, n0 = (mfast ? t2 / tm : t2 % tn) * BN;
  const bool staged = (flags & 1) != 0;
  const int kbeg = z * kps, kend = min(K, kbeg + kps);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = (wave >> 2) * CF::WM, wn = (wave & 3) * CF::WN;
  const bool do_sum = ROWSUM && n0 == 0 && (wave & 3) == 0;

  f32x4_t acc[CF::MI][CF::NJ];
  f32x4_t accs[ROWSUM ? CF::MI : 1];
#pragma unroll
  for (int i = 0; i < CF::MI; ++i)
#pragma unroll
    for (int j = 0; j < CF::NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < (ROWSUM ? CF::MI : 1); ++i) accs[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  Frag<bf16_t> ones;
  ones.v = make_uint4(0x3F803F80u, 0x3F803F80u, 0x3F803F80u, 0x3F803F80u);

  const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  constexpr bool PRE = !AK && !BKM;
  using LA = typename std::conditional<PRE, TileLoader<AK, BM, CF::A_IPW>,
                                       DirectLoader<AK, BM, CF::A_IPW>>::type;
  using LB = typename std::conditional<PRE, TileLoader<BKM, BN, CF::B_IPW>,
                                       DirectLoader<BKM, BN, CF::B_IPW, CELL>>::type;
  LA lda;
  LB ldb;
  lda.init(A, m0, M, kbeg, wave, lane);
  if constexpr (CELL) ldb.init(B, n0, N, kbeg, wave, lane, cell.hidden);
  else ldb.init(B, n0, N, kbeg, wave, lane);
  // direct load `idx` (< IPW) of this wave for k-tile t (each idx is issued
  // once per k-tile, in k-tile order)
  auto dma = [&](int t, int idx) {
    const bf16_t* st = smem + (t % CF::NS) * (CF::STAGE / 2);
    const int k0 = kbeg + t * BK;
    if (idx < CF::A_IPW) lda.issue(idx, k0, kend, st, wave, lane);
    else ldb.issue(idx - CF::A_IPW, k0, kend, st + CF::A_BYTES / 2, wave, lane);
  };
#pragma unroll
  for (int p = 0; p < CF::NS - 1; ++p)
    if (p < nk) {
#pragma unroll
      for (int idx = 0; idx < CF::IPW; ++idx) dma(p, idx);
    }

  // One k-tile.  DMA: the tile issues the direct loads of tile t + NS - 1
  // (a compile-time switch: the loop below runs the tiles that have such a
  // tile with it on and the last NS - 1 tiles with it off, so the loads are
  // straight-line code rather than one branch each; that alone made the
  // products 5-9 % faster).
  auto tile = [&](int t, auto with_dma) {
    constexpr bool DMA = decltype(with_dma)::value;
    // this wave's loads of tile t are done once at most the later tiles'
    // loads are outstanding; the barrier makes that true for every wave and
    // retires every read of the stage the next loads overwrite
    if (DMA || nk - 1 - t >= CF::NS - 2) wait_vm<(CF::NS - 2) * CF::IPW>();
    else wait_vm<0>();
    tile_barrier();
    const bf16_t* la = smem + (t % CF::NS) * (CF::STAGE / 2);
    const bf16_t* lb = la + CF::A_BYTES / 2;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      Frag<bf16_t> af[CF::MI], bfr[CF::NJ];
#pragma unroll
      for (int j = 0; j < CF::NJ; ++j) bfr[j] = frag<BKM, BN>(lb, wn + 16 * j, ks, lane);
#pragma unroll
      for (int i = 0; i < CF::MI; ++i) af[i] = frag<AK, BM>(la, wm + 16 * i, ks, lane);
      // The next tile's direct loads: for the weight gradients (PRE) all
      // of them right after the first k-step's fragment reads, which lets
      // the compiler move the second k-step's reads up among the first
      // one's MFMAs (the loads' asm statements order memory accesses):
      // 2.5-4 % faster there, but 7 % slower on the data gradients.
      // Elsewhere they are spread through the MFMAs (one after each row
      // tile), so that the memory pipeline works while the matrix core does,
      // instead of every wave queueing its loads at once.
      if constexpr (DMA && PRE)
        if (ks == 0) {
#pragma unroll
          for (int idx = 0; idx < CF::IPW; ++idx) dma(t + CF::NS - 1, idx);
        }
#pragma unroll
      for (int i = 0; i < CF::MI; ++i) {
#pragma unroll
        for (int j = 0; j < CF::NJ; ++j) mma_16x16x32(acc[i][j], af[i], bfr[j]);
        if (do_sum) mma_16x16x32(accs[ROWSUM ? i : 0], af[i], ones);
        const int idx = ks * CF::MI + i;
        if constexpr (DMA && !PRE)
          if (idx < CF::IPW) dma(t + CF::NS - 1, idx);
      }
    }
  };
  {
    int t = 0;
    for (; t + CF::NS - 1 < nk; ++t) tile(t, std::true_type{});
    for (; t < nk; ++t) tile(t, std::false_type{});
  }

  if (do_sum && mfma_col(lane) == 0) {
#pragma unroll
    for (int i = 0; i < CF::MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + i * 16 + mfma_row(lane, r);
        if (row < M) rowsum[(int64_t)z * M + row] = accs[ROWSUM ? i : 0][r];
      }
  }

  if constexpr (CELL) {
    // (loaded only now: the k-loop's partial vmcnt waits count its direct
    // loads alone; ordinary loads in flight there would have to be counted
    // in, relying on their order of return relative to the direct loads)
    CellItems<BN, BM> items;
    cell_load<BN, BM>(items, cell, M, m0, n0);
    cell_finish<BN, BM>(acc, items, cell, smem, M, m0, n0, wm, wn, lane);
    return;
  }
  if (staged) {
    store_tile_staged<OutT, BN, BM, BIAS>(acc, C, bias, smem, M, N, m0, n0, z, wm, wn, wave, lane);
    return;
  }
#pragma unroll
  for (int j = 0; j < CF::NJ; ++j) {
    const int col = n0 + wn + j * 16 + mfma_col(lane);
    if (col >= N) continue;
    const float bv = BIAS ? bf16_to_f32(bias[col]) : 0.f;
    const bool sec = col >= C.split;
    OutT* cb = (sec ? C.c1 : C.c0) + (int64_t)z * C.zstride;
    const int64_t ldc = sec ? C.ld1 : C.ld0;
    const int cc = sec ? col - C.split : col;
#pragma unroll
    for (int i = 0; i < CF::MI; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + i * 16 + mfma_row(lane, r);
        if (row >= M) continue;
        OutT* dst = cb + (int64_t)row * ldc + cc;
        // the fp32 results that take this path (split-K partials, weight
        // gradients in one split, a step's product for the cell kernel) are
        // each read once: non-temporal
        if constexpr (sizeof(OutT) == 4) __builtin_nontemporal_store(acc[i][j][r] + bv, dst);
        else *dst = from_f32<OutT>(acc[i][j][r] + bv);
      }
  }
}

template <bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM, int BN, int BM = BM0>
hipError_t launch(const GemmArgs& g, Out<OutT> dst, float* rowsum, int S, int kps, hipStream_t s) {
  auto kern = gemm_bf16_kernel<AK, BKM, OutT, BIAS, ROWSUM, BN, BM>;
  constexpr int lds = Cfg<BN, BM>::LDS;
  static bool attr = false;  // per instantiation
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const bf16_t* a = static_cast<const bf16_t*>(g.A);
  const bf16_t* b = static_cast<const bf16_t*>(g.B);
  const bf16_t* b2 = g.B2 ? static_cast<const bf16_t*>(g.B2) : b;
  Op A{a, g.lda, a, g.lda, 1 << 30};
  Op B{b, g.ldb, b2, g.B2 ? g.ldb2 : g.ldb, g.B2 ? g.n_split : (1 << 30)};
  const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
  // the staged epilogue writes whole 16-byte chunks
  constexpr int EPC = 16 / (int)sizeof(OutT);
  const uintptr_t al = reinterpret_cast<uintptr_t>(dst.c0) | reinterpret_cast<uintptr_t>(dst.c1);
  // (split-K fp32 partials keep the direct stores: their tiles have long
  // k-loops, 64-byte store segments, and two LDS passes cost more than
  // they save)
  const bool staged = (al & 15) == 0 && g.N % EPC == 0 && dst.ld0 % EPC == 0 &&
                      dst.ld1 % EPC == 0 && (dst.split >= g.N || dst.split % EPC == 0) &&
                      dst.zstride % EPC == 0 && (sizeof(OutT) == 2 || S == 1);
  hipLaunchKernelGGL(kern, dim3(tm * tn * S), dim3(NT), lds, s, A, B, dst,
                     static_cast<const bf16_t*>(g.bias), rowsum, g.M, g.N, g.K, kps, tm, tn, S,
                     (staged ? 1 : 0) | (tm <= 8 && tn >= 2 * tm ? 2 : 0), CellArgs{});
  return hipGetLastError();
}

// The forward step with the cell in the epilogue: A = h_{t-1} [nb][H], B =
// W_h [4H][H] read gate-interleaved, tiles of pick_small's shape.
template <int T, int TM = T>
hipError_t launch_cell(const GemmArgs& g, const CellArgs& cell, hipStream_t s) {
  auto kern = gemm_bf16_kernel<true, true, float, false, false, T, TM, true>;
  constexpr int lds = Cfg<T, TM>::LDS;
  static_assert(TM * (T + 4) * 4 <= lds, "the cell epilogue stages the fp32 tile in LDS");
  static bool attr = false;
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const bf16_t* a = static_cast<const bf16_t*>(g.A);
  const bf16_t* b = static_cast<const bf16_t*>(g.B);
  Op A{a, g.lda, a, g.lda, 1 << 30};
  Op B{b, g.ldb, b, g.ldb, 1 << 30};
  const int tm = (g.M + TM - 1) / TM, tn = (g.N + T - 1) / T;
  Out<float> none{nullptr, 0, nullptr, 0, 1 << 30, 0};
  hipLaunchKernelGGL(kern, dim3(tm * tn), dim3(NT), lds, s, A, B, none, nullptr, nullptr, g.M,
                     g.N, g.K, g.K, tm, tn, 1, (tm <= 8 && tn >= 2 * tm ? 2 : 0), cell);
  return hipGetLastError();
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

int device_cus() {
  static int cus = 0;
  if (!cus) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  return cus;
}

// Relative time of a grid of w equal workgroups of `work` units each, one
// workgroup per CU at a time.
double grid_time(int64_t w, double work) {
  const int cus = device_cus();
  return (double)((w + cus - 1) / cus) * work;
}

// Tile width: 256, or 192 when its grid keeps the CUs busier.
int pick_bn(int M, int N) {
  const int64_t tm = (M + BM0 - 1) / BM0;
  const double t256 = grid_time(tm * ((N + 255) / 256), 256.0);
  const double t192 = grid_time(tm * ((N + 191) / 192), 192.0);
  return t192 < t256 ? 192 : 256;
}

// Products with few rows (M <= 2048, e.g. one time step of the recurrence
// run as a product): tiles of 128 x 128, 64 rows x 192 columns, or 64 x 64
// where 256-row tiles would leave most CUs idle.  Relative time = rounds of
// one workgroup per CU x tile area / efficiency (smaller tiles read more LDS
// bytes per flop).  Returns the tile's columns (0: the large tiles); 192
// means 64 x 192 (e.g. B = 512 rows x 6144 columns: exactly 256 tiles,
// where 128 x 128 tiles leave 64 CUs idle).
int pick_small(int M, int N) {
  if (M > 2048) return 0;
  int best = 0;
  double tbest = 0.0;
  const struct { int tm, tn; double eff; } cand[] = {
      {256, 256, 1.0}, {128, 128, 0.8}, {64, 192, 0.8}, {64, 64, 0.55}};
  for (const auto& c : cand) {
    const int64_t tiles = (int64_t)((M + c.tm - 1) / c.tm) * ((N + c.tn - 1) / c.tn);
    const double t = grid_time(tiles, (double)c.tm * c.tn / c.eff);
    if (best == 0 || t < tbest) { best = c.tn; tbest = t; }
  }
  return best == 256 ? 0 : best;
}

template <bool AK, bool BKM, typename OutT, bool BIAS, bool ROWSUM>
hipError_t launch_bn(int bn, const GemmArgs& g, Out<OutT> dst, float* rowsum, int S, int kps,
                     hipStream_t s) {
  const int sm = pick_small(g.M, g.N);
  if (sm == 128) return launch<AK, BKM, OutT, BIAS, ROWSUM, 128, 128>(g, dst, rowsum, S, kps, s);
  if (sm == 192) return launch<AK, BKM, OutT, BIAS, ROWSUM, 192, 64>(g, dst, rowsum, S, kps, s);
  if (sm == 64) return launch<AK, BKM, OutT, BIAS, ROWSUM, 64, 64>(g, dst, rowsum, S, kps, s);
  return bn == 192 ? launch<AK, BKM, OutT, BIAS, ROWSUM, 192>(g, dst, rowsum, S, kps, s)
                   : launch<AK, BKM, OutT, BIAS, ROWSUM, 256>(g, dst, rowsum, S, kps, s);
}

// Weight gradients in S k-splits (fp32 partials and a reduction when S > 1).
template <int BN, int BM>
hipError_t weight_grads(const GemmArgs& g, int S, int ktiles, hipStream_t s) {
  if (S == 1) {
    return g.rowsum ? launch<false, false, float, false, true, BN, BM>(g, direct_out<float>(g), g.rowsum, 1, g.K, s)
                    : launch<false, false, float, false, false, BN, BM>(g, direct_out<float>(g), nullptr, 1, g.K, s);
  }
  const int kps = ((ktiles + S - 1) / S) * BK;
  float* part = g.ws;
  float* rs_part = g.ws + (int64_t)S * g.M * g.N;
  Out<float> d{part, g.N, part, g.N, 1 << 30, (int64_t)g.M * g.N};  // one slice per split
  const hipError_t e = g.rowsum ? launch<false, false, float, false, true, BN, BM>(g, d, rs_part, S, kps, s)
                                : launch<false, false, float, false, false, BN, BM>(g, d, nullptr, S, kps, s);
  if (e != hipSuccess) return e;
  return splitk_reduce_launch(part, S, g, rs_part, s);
}

}  // namespace

// C-partials [S][M][N] fp32 of a product with few rows and a long k-range
// (A k-major, B n-major), K split S ways over 128 x 128 tiles: S = the most
// splits (up to max_splits, at least 8 k-tiles each) that keep the grid
// within one workgroup per CU.  Returns S through *splits.
hipError_t gemm_bf16_splitk_rows(const GemmArgs& g, int max_splits, float* part, int* splits,
                                 hipStream_t s) {
  const int64_t tiles = (int64_t)((g.M + 127) / 128) * ((g.N + 127) / 128);
  const int ktiles = (g.K + BK - 1) / BK;
  int S = 1;
  while (S < max_splits && tiles * (S + 1) <= device_cus() && ktiles / (S + 1) >= 8) ++S;
  const int kps = ((ktiles + S - 1) / S) * BK;
  Out<float> d{part, g.N, part, g.N, 1 << 30, (int64_t)g.M * g.N};
  *splits = S;
  return launch<true, false, float, false, false, 128, 128>(g, d, nullptr, S, kps, s);
}

hipError_t gemm_bf16_lstm_fwd_step(const LstmFwdStep& a, hipStream_t s, bool* done) {
  *done = false;
  const int H = a.hidden;
  if (!a.bf16 || !a.hprev || a.nb <= 0 || H % 8 != 0) return hipSuccess;
  const int sm = pick_small(a.nb, 4 * H);
  if (sm != 128 && sm != 192 && sm != 64) return hipSuccess;
  GemmArgs g;
  g.A = a.hprev; g.lda = H;
  g.B = a.Wh; g.ldb = H;
  g.M = a.nb; g.N = 4 * H; g.K = H; g.bf16 = true;
  const CellArgs cell{static_cast<const bf16_t*>(a.P), static_cast<const bf16_t*>(a.hprev), a.cprev,
                      static_cast<bf16_t*>(a.H), static_cast<bf16_t*>(a.Hs), a.C,
                      static_cast<bf16_t*>(a.G), H};
  *done = true;
  if (sm == 192) return launch_cell<192, 64>(g, cell, s);
  return sm == 128 ? launch_cell<128>(g, cell, s) : launch_cell<64>(g, cell, s);
}

hipError_t gemm_bf16(const GemmArgs& g, hipStream_t s) {
  if (g.a_kmajor && g.b_kmajor) {  // forward projections
    const int bn = pick_bn(g.M, g.N);
    if (g.c_f32) {
      return g.bias ? launch_bn<true, true, float, true, false>(bn, g, direct_out<float>(g), nullptr, 1, g.K, s)
                    : launch_bn<true, true, float, false, false>(bn, g, direct_out<float>(g), nullptr, 1, g.K, s);
    }
    return g.bias ? launch_bn<true, true, bf16_t, true, false>(bn, g, direct_out<bf16_t>(g), nullptr, 1, g.K, s)
                  : launch_bn<true, true, bf16_t, false, false>(bn, g, direct_out<bf16_t>(g), nullptr, 1, g.K, s);
  }
  if (g.a_kmajor && !g.b_kmajor && !g.bias && !g.rowsum) {  // data gradients
    const int bn = pick_bn(g.M, g.N);
    return g.c_f32 ? launch_bn<true, false, float, false, false>(bn, g, direct_out<float>(g), nullptr, 1, g.K, s)
                   : launch_bn<true, false, bf16_t, false, false>(bn, g, direct_out<bf16_t>(g), nullptr, 1, g.K, s);
  }
  if (!g.a_kmajor && !g.b_kmajor && !g.bias && g.c_f32) {  // weight gradients
    // (the row-sum variant keeps within the register budget at BN = 192)
    constexpr int bn = 192;
    const int ktiles = (g.K + BK - 1) / BK;
    // tile height (256 or 192) and splits: least estimated time = rounds of
    // one workgroup per CU over the k-range (tiles at ~60 % of the MFMA peak
    // per CU) plus writing and re-reading the fp32 partials (~4 TB/s).  The
    // lower tiles fill the 256 CUs where 256-row tiles would leave some idle
    // (e.g. 12 x 8 tiles of 256 x 192 in 2 splits: 192 workgroups; 16 x 8 of
    // 192 x 192: 256).
    int S = 1, bm = BM0;
    if (g.ws) {
      const double t_part = (double)g.M * g.N * 8.0 / 4e12;
      double best = 1e30;
      for (int h : {BM0, 192}) {
        const int64_t tiles = (int64_t)((g.N + bn - 1) / bn) * ((g.M + h - 1) / h);
        const double t_tile = 2.0 * h * bn * (double)g.K / (2.5e15 / device_cus() * 0.6);
        for (int c = 1; c <= 8; ++c) {
          if (c > 1 && ktiles / c < 8) break;  // at least 8 k-tiles per split
          if (c > 1 && (int64_t)c * g.M * g.N + (int64_t)c * g.M > g.ws_floats) break;
          const double cost = grid_time(tiles * c, t_tile / c) + (c > 1 ? c * t_part : 0.0);
          if (cost < best - 1e-12) { best = cost; S = c; bm = h; }
        }
      }
    }
    return bm == 192 ? weight_grads<bn, 192>(g, S, ktiles, s) : weight_grads<bn, BM0>(g, S, ktiles, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace am
