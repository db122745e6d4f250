// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace am {

// C[M][N] = sum_k A(m,k) B(k,n) (+ bias[n]).
//   A(m,k) = A[m*lda + k] if a_kmajor else A[k*lda + m]
//   B(k,n) = B[n*ldb + k] if b_kmajor else B[k*ldb + n]
// Inputs are bf16 (bf16 = true) or fp32; C is fp32 (c_f32) or the input type;
// bias is per column, input type.  Requirements (checked by the caller):
// 16-byte aligned rows; a k-major K and an m/n-major M or N that is a
// multiple of 8 (bf16) / 4 (fp32).
// Optional (m/n-major B only): columns n >= n_split of B come from B2
// (row stride ldb2) and the matching columns of C go to C2 (ldc2).
// Optional (m-major A only): rowsum[m] = sum_k A(m,k) in fp32.
// Optional: ws/ws_floats, fp32 scratch that lets a TN product split K.
struct GemmArgs {
  const void* A = nullptr; int64_t lda = 0; bool a_kmajor = true;
  const void* B = nullptr; int64_t ldb = 0; bool b_kmajor = true;
  const void* B2 = nullptr; int64_t ldb2 = 0; int n_split = 0;
  void* C = nullptr; int64_t ldc = 0; bool c_f32 = false;
  void* C2 = nullptr; int64_t ldc2 = 0;
  const void* bias = nullptr;
  float* rowsum = nullptr;
  int M = 0, N = 0, K = 0;
  bool bf16 = false;
  float* ws = nullptr; int64_t ws_floats = 0;
};
hipError_t gemm(const GemmArgs& g, hipStream_t s);
// One forward LSTM step as one launch: the recurrent product h_{t-1} Wh^T
// with the cell in its epilogue (bf16, products of at most 2048 rows; W_h's
// gate rows are read interleaved, so each output tile holds all four gates
// of its units).  Same results, bit for bit, as the product into fp32
// scratch followed by lstm_cell_fwd.  *done = false: not covered (nothing
// launched; the caller runs the two-launch form).
struct LstmFwdStep;
hipError_t gemm_bf16_lstm_fwd_step(const LstmFwdStep& a, hipStream_t s, bool* done);
// The bf16 products (gemm routes bf16 arguments here).
hipError_t gemm_bf16(const GemmArgs& g, hipStream_t s);
// A k-major, B n-major, K split up to max_splits ways: fp32 partials
// part[S][M][N] (S returned in *splits), summed by the consumer in split order.
hipError_t gemm_bf16_splitk_rows(const GemmArgs& g, int max_splits, float* part, int* splits,
                                 hipStream_t s);
// Sum of S split-K partial results [S][M][N] (and partial row sums [S][M])
// into g.C / g.C2 (and g.rowsum), in split order.
hipError_t splitk_reduce_launch(const float* part, int S, const GemmArgs& g, const float* rs_part,
                                hipStream_t s);

// One forward step of one LSTM layer over the nb active rows of step t:
// gate pre-activations P (input projection + bias, rows of step t) plus
// h_{t-1} Wh^T, the cell update, and the stores BPTT needs.
struct LstmFwdStep {
  const void* P;      // [nb][4H]
  const void* Wh;     // [4H][H]
  const void* hprev;  // [nb][H] rows of h_{t-1}, or null (zero state)
  const float* cprev; // [nb][H] rows of c_{t-1}, or null
  void* H;            // [nb][H] h_t (written)
  void* Hs;           // [nb][H] copy of h_{t-1} for the Wh gradient (written)
  float* C;           // [nb][H] c_t (written)
  void* G;            // [nb][H][4] gate activations: unit j's i, f, g, o at 4j .. 4j+3 (written)
  int nb, hidden;
  bool bf16;
};
hipError_t lstm_fwd_step(const LstmFwdStep& a, hipStream_t s);

// One reverse step: dh = dHa + dA_{t+1} Wh (rows < nbn), cell backward,
// dA_t written; dc carries dc_{t+1} in and dc_t out per sequence.
struct LstmBwdStep {
  const void* dAnext; // [nbn][4H] rows of step t+1, or null
  int nbn;
  const void* WhT;    // [H][4H]
  const void* dHa;    // [nb][H] gradient from the layer above / output
  const void* G;      // [nb][4H]
  const float* C;     // [nb][H]
  const float* Cprev; // [nb][H] c_{t-1} rows, or null (zero)
  float* dc;          // [B][H]
  void* dA;           // [nb][4H] (written)
  int nb, hidden;
  bool bf16;
};
hipError_t lstm_bwd_step(const LstmBwdStep& a, hipStream_t s);
// bf16 steps as a batched product plus a cell kernel: the cell of a forward
// step from pre = h_{t-1} Wh^T ([nb][4H] fp32, or null for a zero h_{t-1});
// the cell backward from dhrec = dA_{t+1} Wh (`splits` partials
// [splits][nbn][H] fp32, summed in order).  The product's
// operands of `a` (Wh, WhT, dAnext) are not read here.
hipError_t lstm_cell_fwd(const float* pre, const LstmFwdStep& a, hipStream_t s);
hipError_t lstm_cell_bwd(const float* dhrec, int splits, const LstmBwdStep& a, hipStream_t s);

// Persistent layer kernels (all time steps in one launch of a resident grid).
// The schedule of a batch: T steps, B sequences, N frames; with varlen the
// sorted lengths (B <= 1024), else every sequence has T frames.
struct PersistSchedule {
  int T, B, N;
  int varlen;
  uint16_t lens[1024];
};
struct PersistFwd {
  const void* P;       // [N][4H] input projections (+ bias)
  const void* Wh;      // [4H][H]
  const void* h0;      // [B][H] initial h (activation type) or null (zero)
  const float* c0;     // [B][H] initial c
  void* H; void* Hs; float* C; void* G;  // [N][H], [N][H], [N][H], [N][4H] (written)
  unsigned* counters;  // one per block of 64 sequences, zero at launch
  int* err;            // set to 1 if a step barrier timed out
  int hidden;
};
struct PersistBwd {
  const void* Wh;      // [4H][H]
  const void* WhT;     // [H][4H] (the XCD-local kernel reads this layout)
  const void* dHa;     // [N][H] gradient from the layer above
  const void* G;       // [N][4H]
  const float* C;      // [N][H]
  const float* c0;     // [B][H]
  void* dA;            // [N][4H] (written)
  unsigned* counters;
  int* err;
  int hidden;
};
// XCD-local persistent layer kernels (one block of sequences per XCD, the
// exchange and the step barrier inside that XCD's L2).  Scratch: one step
// counter per block at flags[32 blk] (one cache line each), a start counter
// and the XCC id of every workgroup (xcc[grid]), all zero at launch, and the
// time-out flag (set, never cleared).
struct XcdSync {
  unsigned* flags;  // a 32-word line per block of sequences, a word per member
  int* xcc;         // the same for the members' XCD ids (check of the layout)
  int* err;
  int units;   // filled in by the launcher
  int fenced;  // nonzero: exchange with release/acquire fences even when every
               // block is found on one XCD (AM_XCD_FENCED=1, for tests)
};
bool lstm_xcd_instantiated(bool forward, int hidden, int B);
// Launch of a grid that the caller has checked fits on the device at once
// (occupancy x CUs).  With AM_COOPERATIVE=1 in the environment it goes
// through the cooperative launch (which guarantees co-residency but adds
// about 25 us of dispatch overhead around each launch); otherwise it is an
// ordinary launch, whose workgroups are all resident on an otherwise idle
// device, and every step barrier is bounded, so a grid that is not resident
// ends in the barrier time-out flag, never in a hang.
hipError_t resident_launch(const void* fn, dim3 grid, dim3 block, void** args, size_t lds,
                           hipStream_t s);
hipError_t lstm_fwd_xcd_launch(PersistFwd a, PersistSchedule ps, XcdSync y, hipStream_t s, bool* used);
hipError_t lstm_bwd_xcd_launch(PersistBwd a, PersistSchedule ps, XcdSync y, hipStream_t s, bool* used);

// Whether the persistent kernel covers this shape and its grid can be
// resident at once on the current device.
bool lstm_persistent_fits(bool forward, int hidden, int B, bool bf16, int T);
// *used is false (and nothing is launched) when the grid cannot be resident
// at once or the shape is not covered; the caller then runs single steps.
hipError_t lstm_fwd_persistent(PersistFwd a, PersistSchedule ps, bool bf16, hipStream_t s, bool* used);
hipError_t lstm_bwd_persistent(PersistBwd a, PersistSchedule ps, bool bf16, hipStream_t s, bool* used);

// Sparse soft-target cross-entropy rows (see sparse_soft_ce in the C ABI).
struct SoftCeArgs {
  int64_t N; int C; int K;
  const float* z; const int32_t* idx; const float* prob; const uint8_t* mask;
  int reduction; float* loss; void* dz; bool dz_bf16;
  float* ws_partials; int64_t n_partials; float* ws_scale;
};
int64_t soft_ce_partials(int64_t N);
hipError_t soft_ce(const SoftCeArgs& a, hipStream_t s);

// Threshold encode / decode.  The encoder's scratch: 2-bit codes (a 32-bit
// word per 16 elements, TILE elements per tile) and one count per tile, each
// region 256-byte aligned.
constexpr int64_t GTC_TILE = 4096;
constexpr int64_t gtc_tiles_c(int64_t n) { return (n + GTC_TILE - 1) / GTC_TILE; }
constexpr int64_t gtc_align256(int64_t x) { return (x + 255) & ~int64_t(255); }
constexpr int64_t gtc_codes_bytes(int64_t n) { return gtc_align256(gtc_tiles_c(n) * (GTC_TILE / 4)); }
constexpr int64_t gtc_encode_scratch_bytes(int64_t n) {
  return gtc_codes_bytes(n) + gtc_align256(gtc_tiles_c(n) * 4);
}
int64_t gtc_tiles(int64_t n);
hipError_t gtc_encode(int64_t n, const float* g, float* r, float tau, uint32_t* words,
                      int64_t* count, uint32_t* ws_mask, int32_t* ws_tile, hipStream_t s);
hipError_t gtc_decode(const uint32_t* words, const int64_t* count, int64_t capacity, float tau,
                      int64_t n, float* dense, bool accumulate, hipStream_t s);
// Decode of one stream (accumulate = 0) fused with sgd_apply: the same
// master and bf16 copy bit for bit, without the dense update.
hipError_t gtc_decode_sgd(const uint32_t* words, const int64_t* count, int64_t capacity, float tau,
                          int64_t n, float lr, float* master, uint16_t* w_bf16, hipStream_t s);
// Aggregate of `streams` workers' streams, words [streams][capacity];
// ws_start holds streams x (gtc_tiles(n) + 1) int32.
hipError_t gtc_decode_multi(int streams, const uint32_t* words, int64_t capacity,
                            const int64_t* counts, float tau, int64_t n, float* dense,
                            bool accumulate, int32_t* ws_start, hipStream_t s);

// Stacked low-frame-rate input frames (see lfr_features in the C ABI).
struct LfrArgs {
  int B, raw_dim, stack, skip, offset;
  uint16_t U[1024];    // raw frames per utterance
  const float* raw;    // [sum U][raw_dim], utterance after utterance
  const float* mean;   // [stack * raw_dim]
  const float* std;    // [stack * raw_dim]
  void* x;             // packed [N][stack * raw_dim], model dtype
};
hipError_t lfr_features(const LfrArgs& a, bool bf16, hipStream_t s);
// Targets of packed rows delayed by `delay` frames within each sequence.
struct DelayArgs {
  int T, B, K, delay;
  uint16_t len[1024];
  const int32_t* idx; const float* prob;
  int32_t* idx_out; float* prob_out; uint8_t* mask_out;
};
hipError_t delay_targets(const DelayArgs& a, hipStream_t s);

// Teacher target generation.
struct GatherRows {
  const void* src; int64_t src_ld;
  void* dst; int64_t dst_ld; int64_t dst_col;
  int width;             // elements per row (a multiple of 16 bytes)
  int64_t N;             // rows
  int T;                 // time steps of the schedule
  const int64_t* offs;   // [T + 1] packed row offsets (device)
  const int32_t* lens;   // [B] sequence lengths (device)
  int reverse;           // row (t, b) takes row (len_b - 1 - t, b)
};
hipError_t gather_rows(const GatherRows& a, bool bf16, hipStream_t s);
struct SchedTables {
  int T, B;
  uint16_t len[1024];
  int64_t* offs;  // [T + 1] out
  int32_t* lens;  // [B] out
};
hipError_t schedule_tables(const SchedTables& a, hipStream_t s);
hipError_t topk_rows(int64_t N, int C, int K, const float* z, int32_t* idx, float* val,
                     hipStream_t s);
hipError_t kbest_posteriors(int64_t N, int K, const float* val, float* prob, hipStream_t s);

// BMUF-NBM global step (count addends of stride elements, divided by workers).
hipError_t bmuf_update(int64_t n, int count, int workers, const float* models, int64_t stride,
                       float* wg, float* delta, float eta, float eta_next, float zeta,
                       float* local, uint16_t* local_bf16, hipStream_t s);

// Elementwise and data-movement helpers.
hipError_t sgd_apply_f32(int64_t n, float* master, uint16_t* w_bf16, const float* u, float lr,
                         hipStream_t s);
hipError_t cast_f32_bf16(int64_t n, const float* src, uint16_t* dst, hipStream_t s);
// dst[c][r] = src[r][c] for a rows x cols matrix of the activation type.
hipError_t transpose(const void* src, void* dst, int rows, int cols, bool bf16, hipStream_t s);
// Up to MAX bf16 matrices of one shape (rows, cols multiples of 8, 16-byte
// aligned) transposed in one launch; hipErrorInvalidValue if they are not.
struct TransposeBatch {
  static constexpr int MAX = 8;
  const void* src[MAX];
  void* dst[MAX];
};
hipError_t transpose_bf16_batch(const TransposeBatch& tb, int n, int rows, int cols, hipStream_t s);
// out[c] = sum_r in[r][c] (fp32 result, fixed summation order).
hipError_t colsum(const void* in, int64_t rows, int cols, bool bf16, float* out,
                  float* ws_partial, int n_chunks, hipStream_t s);
// dst[0..n) = +0.0 (a kernel, so the call is safe inside graph capture).
hipError_t fill_zero(float* dst, int64_t n, hipStream_t s);
hipError_t fill_zero2(float* d0, int64_t n0, float* d1, int64_t n1, hipStream_t s);
// dst[0..n) = +0.0 when *flag (device) is nonzero, else nothing.
hipError_t zero_if_set(const int* flag, float* dst, int64_t n, hipStream_t s);
// Convert fp32 [rows][cols] to the activation type (h0 for the recurrence).
hipError_t convert_rows(const float* src, void* dst, int64_t count, bool bf16, hipStream_t s);
// Final states: out[b][j] = state at row[b] (or init[b][j] / 0 if row[b] < 0).
struct GatherState {
  const void* Hrows; bool h_bf16; const float* Crows;
  const float* h0; const float* c0;
  float* hT; float* cT;
  int B, hidden;
  int rows[256];
};
hipError_t gather_state(const GatherState& a, int b0, int nb, hipStream_t s);

}  // namespace am
