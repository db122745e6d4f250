/*
 * mi355am.h -- C ABI of the MI355X (gfx950) student training step.
 *
 * The operation set is the per-worker hot path of data-parallel acoustic
 * model training in Parthasarathi et al., "Realizing Petabyte Scale Acoustic
 * Modeling": the student LSTM acoustic model (§II-B, §V-A) trained with
 * chunked BPTT (§II-B, §V-D) against sparse k-best teacher posteriors
 * (§II-C, §V-C) by mini-batch SGD (§VI, §VI-B), whose gradient is passed
 * through Gradient Threshold Compression with residual error feedback (§VI-A).
 * Two pieces of the multi-worker trainers run per GPU as well: the aggregate
 * of several workers' compressed updates (§VI-A) and the BMUF-NBM global
 * model step (§VI-B).
 *
 * Conventions for every entry point:
 *  - Pointers are device pointers unless the comment says [host].
 *  - `stream` is a hipStream_t (NULL = the default stream).  All work is
 *    enqueued on it asynchronously; nothing is synchronised unless stated.
 *  - The caller owns every buffer.  No entry point allocates device memory;
 *    scratch space is a caller-provided workspace `ws` of at least the size
 *    returned by the matching *_workspace_bytes query (256-byte aligned).
 *  - Arguments are validated on the host before anything is enqueued; on any
 *    error nothing is enqueued and no buffer is touched.  The return value is
 *    an am_status; am_last_error() gives a message for the calling thread.
 *  - Values inside device buffers (target indices, counts) are not checked,
 *    except that with AM_DEBUG=1 in the environment sparse_soft_ce
 *    synchronises its stream and checks every target index (see there).
 *
 * Model and tensor layouts:
 *  - am_model { layers L, input_dim D0, hidden H, classes C, dtype }.
 *    dtype AM_F32: parameters, inputs and activations are fp32.
 *    dtype AM_BF16: parameters (a bf16 working copy of fp32 master weights),
 *    input frames, stored activations and dlogits are bf16; every product is
 *    accumulated in fp32; cell states, logits and gradients are fp32.
 *    Requirements: H % 16 == 0; D0, H and C multiples of 8 (bf16) or 4 (f32).
 *  - Flat parameter vector (one buffer, so the whole gradient is quantised in
 *    one call): for each layer l, Wx_l [4H][D_l], Wh_l [4H][H], b_l [4H]
 *    (D_0 = D0, D_l = H), then Wo [C][H], bo [C].  Gate blocks along every
 *    4H axis are ordered input, forget, cell candidate, output.
 *  - Frames are packed time-major.  A batch is B sequences sorted by
 *    non-increasing length (`lengths`, [host] int32[B], each in [0, T]), or B
 *    sequences of T frames when `lengths` is NULL.  B_t = number of
 *    sequences longer than t; frame (t, b), b < B_t, is row off_t + b with
 *    off_t = B_0 + ... + B_{t-1}.  N = off_T rows in total; padding does not
 *    exist.  Variable-length batches allow B <= 1024.
 */
#ifndef MI355AM_H
#define MI355AM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  AM_OK = 0,
  AM_EINVAL = -1,        /* bad pointer, size, layout or ordering */
  AM_ECAPACITY = -2,     /* an output buffer is too small */
  AM_EUNSUPPORTED = -3,  /* valid but outside what the kernels handle */
  AM_EHIP = -4,          /* a HIP call failed (launch error, ...) */
  AM_EWORKSPACE = -5,    /* workspace missing or too small */
  AM_ETIMEOUT = -6       /* a step barrier timed out; the pass's results are invalid */
} am_status;

typedef enum { AM_F32 = 0, AM_BF16 = 1 } am_dtype;
typedef enum { AM_MEAN_VALID = 0, AM_SUM = 1 } am_reduction;

typedef struct {
  int32_t layers;
  int32_t input_dim;
  int32_t hidden;
  int32_t classes;
  int32_t dtype; /* am_dtype */
} am_model;

/* ---- host-only queries ------------------------------------------------- */

/* Number of parameters n of the model (24,145,848 for L=5, D0=192, H=768,
 * C=3000), or -1 if the model description is invalid. */
int64_t am_param_count(const am_model* m);

/* Writes the 3L+2 start offsets (elements) of Wx_0, Wh_0, b_0, ..., Wo, bo
 * into `offsets` [host]. */
am_status am_param_offsets(const am_model* m, int64_t* offsets);

/* Bytes of workspace lstm_am_forward/lstm_am_backward need for a batch of B
 * sequences, T steps and N packed frames; -1 if invalid. */
int64_t am_workspace_bytes(const am_model* m, int32_t T, int32_t B, int64_t N);

/* Workspace for sparse_soft_ce over N rows / for grad_threshold_encode. */
int64_t am_ce_workspace_bytes(int64_t N);
int64_t am_encode_workspace_bytes(int64_t n);

const char* am_status_string(int32_t status);
const char* am_last_error(void);

/* Which kernels run one layer's recurrence (forward = 1: the forward pass;
 * 0: BPTT) for a batch of B sequences and T steps (varlen = 1 if their
 * lengths differ), as lstm_am_forward / lstm_am_backward choose them:
 *   AM_PATH_XCD    one persistent launch per layer whose blocks of sequences
 *                  each exchange state inside one XCD's L2 (bf16, shapes the
 *                  kernels are built for; variable lengths need T <= 65535);
 *   AM_PATH_DEVICE one persistent launch per layer with a device-scope
 *                  exchange (its grid checked against the current device's
 *                  occupancy: never chosen without a device);
 *   AM_PATH_STEP   one launch per time step.
 * A persistent grid that cannot be resident at launch falls back to the
 * next path.  -1 if the model or sizes are invalid.  Host only. */
enum { AM_PATH_XCD = 1, AM_PATH_DEVICE = 2, AM_PATH_STEP = 3 };
int32_t am_recurrence_path(const am_model* m, int32_t T, int32_t B, int32_t varlen,
                           int32_t forward);

/* ---- the training step ------------------------------------------------- */

/* Forward pass of the student LSTM acoustic model (§II-B): per layer and
 * step, a = Wx x_t + Wh h_{t-1} + b; i, f, o = sigmoid, g = tanh of the gate
 * blocks; c_t = f c_{t-1} + i g; h_t = o tanh(c_t); then logits
 * z = Wo h^{L-1} + bo.
 *   params  [n] model dtype;  x [N][D0] model dtype (packed frames)
 *   lengths [host] [B] or NULL;  h0, c0 [L][B][H] fp32 or NULL (zero)
 *   logits  [N][C] fp32 (written)
 *   hT, cT  [L][B][H] fp32 or NULL: state after each sequence's last frame
 *   ws      workspace; it keeps the activations lstm_am_backward consumes and
 *           must not be modified between the two calls.                    */
am_status lstm_am_forward(const am_model* m, const void* params, const void* x,
                          const int32_t* lengths, const float* h0, const float* c0,
                          int32_t T, int32_t B, float* logits, float* hT, float* cT,
                          void* ws, int64_t ws_bytes, void* stream);

/* Cross-entropy between sparse teacher posteriors and the student softmax
 * (§II-C, §V-A; k-best targets §V-C).  Per row f with mask m_f:
 *   loss_f = -sum_j p_fj (z_{f,idx_fj} - logsumexp(z_f)),  M_f = sum_j p_fj,
 *   dlogits_f = s_f (M_f softmax(z_f) - sum_j p_fj e_{idx_fj}),
 *   loss = sum_f s_f loss_f,  s_f = m_f / sum(m) (AM_MEAN_VALID) or m_f (AM_SUM).
 * Targets are used as given (no renormalisation); idx -1 marks an empty slot;
 * repeated indices add.  An index outside [-1, C) is a caller error: release
 * builds treat it as an empty slot; with AM_DEBUG=1 in the environment the
 * call synchronises `stream` (after the work queued before it), checks every
 * index of idx and returns AM_EINVAL, with nothing enqueued, if one is out of
 * range.  Rows with m_f = 0 get zero gradient and their logits are not read.
 * Requirements: C % 4 == 0, C <= 8192, logits 16-byte aligned.
 *   logits [N][C] fp32;  idx [N][K] int32;  prob [N][K] fp32
 *   mask   [N] uint8 or NULL (all valid);  loss [1] fp32 (written)
 *   dlogits [N][C] of dlogits_dtype (AM_F32 or AM_BF16), written           */
am_status sparse_soft_ce(int64_t N, int32_t C, int32_t K, const float* logits,
                         const int32_t* idx, const float* prob, const uint8_t* mask,
                         int32_t reduction, float* loss, void* dlogits,
                         int32_t dlogits_dtype, void* ws, int64_t ws_bytes, void* stream);

/* Back-propagation through time of the forward call that filled `ws`, given
 * dL/dlogits (model dtype, [N][C]).  Writes the full gradient, fp32, in the
 * flat parameter layout, into `grads` [n] (overwritten).  The state gradient
 * is zero after each sequence's last frame (truncated BPTT within a chunk).
 * Arguments m, params, x, lengths, T, B must be those of the forward call. */
am_status lstm_am_backward(const am_model* m, const void* params, const void* x,
                           const int32_t* lengths, int32_t T, int32_t B,
                           const void* dlogits, void* ws, int64_t ws_bytes,
                           float* grads, void* stream);

/* Whether the recurrence of the last lstm_am_forward (and lstm_am_backward)
 * on `ws` completed.  The recurrence runs as one persistent launch per layer
 * whose workgroups meet at a barrier every time step; each wait is bounded,
 * and a wait that runs out (workgroups not co-resident, a stalled device)
 * sets a flag in `ws` instead of hanging.  Synchronises `stream`, then
 * returns AM_OK, or AM_ETIMEOUT when the flag is set (the outputs of that
 * pass must be discarded).  The flag is cleared by the next forward call.
 * lstm_am_backward reads the flag on the device as its last step and, when
 * it is set, overwrites `grads` with zeros, so that a caller that encodes
 * and applies the gradient before this check adds nothing to its residual
 * or weights. */
am_status am_workspace_check(const void* ws, int64_t ws_bytes, void* stream);

/* Gradient Threshold Compression encode (§VI-A), exact fp32:
 *   for i in 0..n-1:  a = residual[i] + grad[i]
 *     a >  tau: residual[i] = a - tau, emit (i << 1) | 0
 *     a < -tau: residual[i] = a + tau, emit (i << 1) | 1
 *     else:     residual[i] = a
 * Words are written to `words` in ascending i; *count (device int64) gets
 * their number.  NaN is never emitted.  n < 2^31; capacity >= n; tau > 0.
 * `residual` is updated in place and is persistent trainer state.         */
am_status grad_threshold_encode(int64_t n, const float* grad, float* residual, float tau,
                                uint32_t* words, int64_t capacity, int64_t* count,
                                void* ws, int64_t ws_bytes, void* stream);

/* For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): grad_threshold_encode with the same kernels and results, its
 * scratch held in a device array the library owns for the life of the
 * process (each GPU that runs it holds its own copy of
 * am_encode_workspace_bytes(AM_ENCODE_NOALLOC_MAX_N) = about 8.4 MB).  The
 * first call on a GPU looks up that GPU's copy (no allocation); no call
 * allocates or frees device memory.  n > AM_ENCODE_NOALLOC_MAX_N returns
 * AM_EUNSUPPORTED with nothing enqueued; other arguments and errors as
 * grad_threshold_encode.  Every call on one GPU shares that GPU's array:
 * calls that may overlap on one GPU (different streams, or threads) race and
 * must be ordered by the caller.  The array needs no clearing between calls. */
#define AM_ENCODE_NOALLOC_MAX_N (1ll << 25) /* 33,554,432 elements */
am_status grad_threshold_encode_noalloc(int64_t n, const float* grad, float* residual, float tau,
                                        uint32_t* words, int64_t capacity, int64_t* count,
                                        void* stream);

/* Decode (§VI-A): dense[i] = +tau (sign bit 0) or -tau (sign bit 1) for each
 * of the first min(*count, capacity) words (count is a device int64, so no
 * host synchronisation is needed; capacity = number of words `words` holds);
 * accumulate = 0: every other element is +0.0;  accumulate = 1: dense[i] +=
 * +-tau (one fp32 add per word) and other elements are left unchanged.
 * Words must be strictly ascending in index, as encode writes them.        */
am_status grad_threshold_decode(const uint32_t* words, const int64_t* count, int64_t capacity,
                                float tau, int64_t n, float* dense, int32_t accumulate,
                                void* stream);

/* The decode of one stream (accumulate = 0) and the SGD step on its update
 * (§VI-A decode, §VI: the update applied to the fp32 master weights) in one
 * pass: master and weights_bf16 end up exactly as after
 *   grad_threshold_decode(words, count, capacity, tau, n, update, 0, s);
 *   sgd_apply(n, master, weights_bf16, update, lr, s);
 * provided that, when lr is +0.0 or positive and finite, weights_bf16 (if
 * given) holds the round-to-nearest-even bf16 rounding of master at every
 * element no word names, and no such master is NaN.  sgd_apply and this
 * call leave the copy in that state.  With such an lr only the named
 * elements are read and written (an unnamed element's update is +0.0, and
 * w - lr * 0.0 = w), so the pass costs about 14 bytes per word rather than
 * a pass over all n; every other master and bf16 value is left as it is.
 * With any other lr (-0.0, negative, infinite, NaN) every element is
 * rewritten.  See sgd_apply for the arithmetic.  The same argument rules as
 * grad_threshold_decode: words strictly ascending in index, count [device]
 * clamped to [0, capacity], n < 2^31.                                     */
am_status grad_threshold_decode_sgd(const uint32_t* words, const int64_t* count, int64_t capacity,
                                    float tau, int64_t n, float lr, float* master,
                                    void* weights_bf16, void* stream);

/* ---- student inputs ------------------------------------------------------ */

/* Stacked frames of an utterance of raw_frames 10 ms frames: the number of
 * complete stacks of `stack` frames at a `skip` advance from frame `offset`
 * (0 <= offset < skip), i.e. max(0, (raw_frames - offset - stack) / skip + 1);
 * -1 for invalid arguments.  Host only. */
int32_t am_lfr_frames(int32_t raw_frames, int32_t stack, int32_t skip, int32_t offset);

/* The student's input frames (§II-B: 64-dim log mel energies every 10 ms,
 * stacked three at a time and sub-sampled to a 30 ms advance at one of three
 * offsets, a causal mean estimate subtracted, then global mean and variance
 * normalisation).  For utterance b with T_b = am_lfr_frames(raw_lengths[b],
 * stack, skip, offset) stacked frames, frame t (t < T_b) is
 *   y_t = [F(offset + skip t), ..., F(offset + skip t + stack - 1)]  (oldest first)
 *   z_t = y_t - (y_0 + ... + y_t) / (t + 1)
 *   out_t = (z_t - mean) / std          (per dimension)
 * evaluated in fp64 in this order without fused multiply-adds and rounded
 * once to fp32 (then to bf16 if x_dtype is AM_BF16).
 *   raw_lengths [host] [B] raw frames per utterance (<= 65535), in an order
 *               whose T_b are non-increasing; B <= 1024
 *   raw         [sum raw_lengths][raw_dim] fp32, utterance after utterance
 *   mean, std   [stack * raw_dim] fp32 (std must be non-zero)
 *   x           packed time-major model input [N][stack * raw_dim] of
 *               x_dtype: frame (t, b) is row off_t + b as in lstm_am_forward
 *               with lengths T_b; N = sum T_b.                              */
am_status lfr_features(int32_t B, const int32_t* raw_lengths, const float* raw, int32_t raw_dim,
                       int32_t stack, int32_t skip, int32_t offset, const float* mean,
                       const float* std, void* x, int32_t x_dtype, void* stream);

/* Targets for a model with a `delay`-frame look-ahead (§II-B: three frames):
 * packed row (t, b) takes the target of row (t - delay, b) of the same
 * sequence; rows with t < delay get idx -1, prob 0 and mask 0, every other
 * row mask 1.  The mask goes to sparse_soft_ce.  T, B, lengths as in
 * lstm_am_forward (B <= 1024, T <= 65535); idx, prob [N][K] in; idx_out,
 * prob_out [N][K] and mask_out [N] out (must not alias the inputs).  A caller
 * that scores the last `delay` targets of an utterance extends its input by
 * `delay` frames.                                                           */
am_status delay_targets(int32_t T, int32_t B, const int32_t* lengths, int32_t K, int32_t delay,
                        const int32_t* idx, const float* prob, int32_t* idx_out, float* prob_out,
                        uint8_t* mask_out, void* stream);

/* ---- teacher target generation ------------------------------------------ */

/* The teacher (§V-A, §VII): `layers` bidirectional LSTM layers of `hidden`
 * cells per direction over input_dim-dim frames, then a senone layer over
 * both directions' outputs.  Each direction is the student's cell; the
 * backward direction runs over each sequence from its last frame to its
 * first, from a zero state; a layer's output is [h_forward, h_backward].
 * Flat parameters: per layer, forward Wx [4H][D_l], Wh [4H][H], b [4H], then
 * the backward direction's (D_0 = input_dim, D_l = 2H); then Wo [C][2H],
 * bo [C].  The offsets query writes 6L + 2 offsets in that order. */
int64_t am_teacher_param_count(const am_model* m);
am_status am_teacher_param_offsets(const am_model* m, int64_t* offsets);
int64_t am_teacher_workspace_bytes(const am_model* m, int32_t T, int32_t B, int64_t N);

/* Teacher logits [N][C] fp32 for packed frames x (layout, lengths and dtypes
 * as lstm_am_forward; B <= 1024, T <= 65535).  Inference only: `ws` holds
 * scratch of this call alone.                                              */
am_status blstm_teacher_forward(const am_model* m, const void* params, const void* x,
                                const int32_t* lengths, int32_t T, int32_t B, float* logits,
                                void* ws, int64_t ws_bytes, void* stream);

/* The K largest logits of each row (§V-C: the teacher's targets are stored
 * as its k best logits, k = 20), in descending order, equal values by
 * ascending index, NaN after every number: idx [N][K] int32, val [N][K]
 * fp32.  K <= min(C, 64), C <= 8192.                                        */
am_status kbest_logits(int64_t N, int32_t C, int32_t K, const float* logits, int32_t* idx,
                       float* val, void* stream);

/* The posterior rebuilt from K stored logits with every missing logit at
 * -infinity (§V-C fills them with large negative values): per row, the
 * softmax over the K values, fp32 (prob [N][K]), for sparse_soft_ce.       */
am_status kbest_posteriors(int64_t N, int32_t K, const float* val, float* prob, void* stream);

/* Aggregate of the sparse updates of several workers (§VI-A: each worker
 * receives every other worker's sparse update and aggregates them).  Stream
 * s is row s of `words` [streams][capacity] (for example the result of a
 * fixed-capacity all-gather of each worker's encode output) holding
 * min(counts[s], capacity) valid words, strictly ascending in index as
 * encode writes them; counts [streams] are device int64.  With k_i = the
 * sum over all streams of +1 (sign bit 0) or -1 (sign bit 1) for the words
 * naming element i, computed exactly in integers (so the result does not
 * depend on the order of the streams), and q_i = tau * k_i rounded once to
 * fp32:
 *   accumulate = 0: dense[i] = q_i where some word names i, else +0.0;
 *   accumulate = 1: dense[i] = fl32(dense[i] + q_i) where some word names i,
 *                   other elements unchanged.
 * With one stream this equals grad_threshold_decode.  n < 2^31,
 * 0 <= streams <= 32767; workspace: am_decode_multi_workspace_bytes.        */
int64_t am_decode_multi_workspace_bytes(int32_t streams, int64_t n);
am_status grad_threshold_decode_multi(int32_t streams, const uint32_t* words, int64_t capacity,
                                      const int64_t* counts, float tau, int64_t n, float* dense,
                                      int32_t accumulate, void* ws, int64_t ws_bytes,
                                      void* stream);

/* BMUF-NBM global step that ends a block of local SGD (§VI-B, eqs. (2)-(5)),
 * per element i, in fp64 from the fp32 inputs, in this order, without fused
 * multiply-adds, each output rounded once to fp32:
 *   Wbar  = (models[0][i] + models[1][i] + ... + models[count-1][i]) / workers
 *   G     = Wbar - global_model[i]
 *   Delta = eta * delta[i] + zeta * G                     (eta = eta_t, zeta = zeta_t)
 *   W     = (global_model[i] + Delta) + eta_next * Delta  (eta_next = eta_{t+1})
 *   global_model[i] = W;  delta[i] = Delta;
 *   local_master[i] = W (or NULL);  local_bf16[i] = RNE bf16 of W (or NULL).
 * models: `count` fp32 rows `model_stride` elements apart: the N local
 * models (count = workers = N), or their all-reduced sum (count = 1,
 * workers = N).  Eq. (6) sets zeta = C N (1 - eta) for a constant C >= 1.
 * Each output may alias an input at the same index (in-place state, or the
 * restart copy written over an addend).                                    */
am_status bmuf_block_update(int64_t n, int32_t count, int32_t workers, const float* models,
                            int64_t model_stride, float* global_model, float* delta, float eta,
                            float eta_next, float zeta, float* local_master, void* local_bf16,
                            void* stream);

/* Local SGD step (§VI, §VI-B): master[i] = fl32(master[i] - lr * update[i])
 * evaluated in fp64; weights_bf16[i] (uint16 bit patterns, or NULL) =
 * round-to-nearest-even bf16 of the new master (NaN -> 0x7FC0).           */
am_status sgd_apply(int64_t n, float* master, void* weights_bf16, const float* update,
                    float lr, void* stream);

/* fp32 -> bf16 (round to nearest even, NaN -> 0x7FC0), e.g. input frames. */
am_status am_cast_f32_to_bf16(int64_t n, const float* src, void* dst_bf16, void* stream);

/* ---- kernel timing ------------------------------------------------------ */

/* Kernel classes for timing with HIP events. */
typedef enum {
  AM_K_GEMM_FWD = 0,      /* input and output projections */
  AM_K_GEMM_BWD_DATA = 1, /* gradients into activations (dlogits Wo, dA Wx) */
  AM_K_GEMM_BWD_WGT = 2,  /* weight gradients (reductions over frames) */
  AM_K_LSTM_FWD = 3,      /* recurrent product + cell (a layer's launch, or a step's) */
  AM_K_LSTM_BWD = 4,      /* recurrent product + cell backward (likewise) */
  AM_K_CE = 5,            /* soft-target cross-entropy rows */
  AM_K_ENCODE = 6,        /* threshold encode (all of its kernels) */
  AM_K_DECODE = 7,
  AM_K_SGD = 8,
  AM_K_MISC = 9,          /* casts, transposes, bias reductions, gathers */
  AM_K_BMUF = 10,         /* BMUF-NBM global step */
  AM_K_NCLASSES = 11
} am_kernel_class;

/* Starts recording: every later launch of a class whose bit is set in
 * `class_mask` is bracketed by HIP events on its stream.  Clears earlier
 * records.  Not thread-safe; one recording at a time per process. */
am_status am_profile_begin(uint32_t class_mask);
/* Records only every n-th launch of each recorded class (n >= 1; 1, the
 * default, records every launch), counted from am_profile_begin.  Each
 * bracket adds a few microseconds of queue time between kernels; sampling
 * with an n coprime to a class's launches per step still visits every
 * launch position of the step.  Returns AM_EINVAL for n < 1. */
am_status am_profile_sample_every(int32_t n);
/* Stops recording and synchronises on the recorded events. */
am_status am_profile_end(void);
/* Totals for one class since am_profile_begin: launches, summed kernel
 * milliseconds, summed algorithmic flops and algorithmic HBM bytes. */
am_status am_profile_get(int32_t kernel_class, int64_t* launches, double* ms,
                         double* flops, double* bytes);

#ifdef __cplusplus
}
#endif
#endif /* MI355AM_H */
