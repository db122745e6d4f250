// C ABI of the training step (declared in include/mi355am.h): argument
// validation, workspace planning, the launch sequence of the forward and
// backward passes, and per-class kernel timing with HIP events.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/mi355am.h"
#include "am_internal.h"

namespace {

thread_local std::string g_err;

am_status fail(am_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

am_status hip_check(hipError_t e, const char* what) {
  if (e == hipSuccess) return AM_OK;
  return fail(AM_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define AM_TRY(expr)                        \
  do {                                      \
    am_status st_ = (expr);                 \
    if (st_ != AM_OK) return st_;           \
  } while (0)

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// ---------------------------------------------------------------- timing --

struct ProfRec {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
};

struct Prof {
  bool on = false;
  uint32_t mask = 0;
  int32_t every = 1;                    // record every n-th launch of a class
  int64_t seen[AM_K_NCLASSES] = {};     // launches of the class since begin
  std::vector<hipEvent_t> pool;
  size_t next = 0;
  std::vector<ProfRec> recs;
  int64_t launches[AM_K_NCLASSES] = {};
  double ms[AM_K_NCLASSES] = {}, flops[AM_K_NCLASSES] = {}, bytes[AM_K_NCLASSES] = {};
} g_prof;

hipEvent_t prof_event() {
  if (g_prof.next == g_prof.pool.size()) {
    // timing only: no system-scope fence (cache write-back) at each record,
    // which would otherwise add a gap of several microseconds per bracket
    hipEvent_t e;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    g_prof.pool.push_back(e);
  }
  return g_prof.pool[g_prof.next++];
}

// Brackets the kernels launched during its lifetime with events when the
// class is being recorded (every n-th launch of the class when sampling).
class Timed {
 public:
  Timed(int cls, hipStream_t s, double flops, double bytes) : s_(s) {
    if (!g_prof.on || !(g_prof.mask & (1u << cls))) return;
    rec_.cls = cls;
    counted_ = true;
    if (g_prof.seen[cls]++ % g_prof.every != 0) return;
    rec_.flops = flops;
    rec_.bytes = bytes;
    rec_.a = prof_event();
    rec_.b = prof_event();
    if (rec_.a && rec_.b && hipEventRecord(rec_.a, s_) == hipSuccess) active_ = true;
  }
  ~Timed() {
    if (active_ && hipEventRecord(rec_.b, s_) == hipSuccess) g_prof.recs.push_back(rec_);
  }
  void cancel() {  // nothing was launched
    if (counted_) --g_prof.seen[rec_.cls];
    counted_ = active_ = false;
  }

 private:
  hipStream_t s_;
  ProfRec rec_{};
  bool counted_ = false;
  bool active_ = false;
};

// ------------------------------------------------------------- the model --

int vec_of(int dtype) { return dtype == AM_BF16 ? 8 : 4; }
int esz_of(int dtype) { return dtype == AM_BF16 ? 2 : 4; }

am_status check_model(const am_model* m) {
  if (!m) return fail(AM_EINVAL, "model is NULL");
  if (m->dtype != AM_F32 && m->dtype != AM_BF16) return fail(AM_EINVAL, "dtype %d unknown", m->dtype);
  if (m->layers < 1 || m->input_dim < 1 || m->hidden < 1 || m->classes < 1)
    return fail(AM_EINVAL, "model sizes must be positive");
  if (m->hidden % 16) return fail(AM_EUNSUPPORTED, "hidden %d is not a multiple of 16", m->hidden);
  const int v = vec_of(m->dtype);
  if (m->input_dim % v || m->classes % v)
    return fail(AM_EUNSUPPORTED, "input_dim and classes must be multiples of %d for this dtype", v);
  if ((int64_t)m->hidden * 4 * (int64_t)(m->hidden > m->input_dim ? m->hidden : m->input_dim) >= (1ll << 31))
    return fail(AM_EUNSUPPORTED, "layer too large");
  return AM_OK;
}

struct Offsets {
  std::vector<int64_t> wx, wh, b;
  int64_t wo, bo, n;
};

Offsets param_layout(const am_model* m) {
  Offsets o;
  const int64_t G = 4ll * m->hidden;
  int64_t pos = 0;
  for (int l = 0; l < m->layers; ++l) {
    const int64_t D = l == 0 ? m->input_dim : m->hidden;
    o.wx.push_back(pos); pos += G * D;
    o.wh.push_back(pos); pos += G * m->hidden;
    o.b.push_back(pos); pos += G;
  }
  o.wo = pos; pos += (int64_t)m->classes * m->hidden;
  o.bo = pos; pos += m->classes;
  o.n = pos;
  return o;
}

// Schedule of a batch: active counts per step and packed row offsets.
struct Schedule {
  int T = 0, B = 0;
  std::vector<int64_t> counts, offs;
  std::vector<int32_t> lens;
  int64_t N = 0;
};

am_status make_schedule(int32_t T, int32_t B, const int32_t* lengths, Schedule& s) {
  if (T < 0 || B < 1) return fail(AM_EINVAL, "need T >= 0 and B >= 1 (T=%d, B=%d)", T, B);
  s.T = T; s.B = B;
  s.lens.assign(B, T);
  if (lengths) {
    if (B > 1024) return fail(AM_EUNSUPPORTED, "variable-length batches allow B <= 1024");
    for (int b = 0; b < B; ++b) {
      if (lengths[b] < 0 || lengths[b] > T)
        return fail(AM_EINVAL, "lengths[%d] = %d outside [0, %d]", b, lengths[b], T);
      if (b > 0 && lengths[b] > lengths[b - 1])
        return fail(AM_EINVAL, "lengths must be non-increasing (lengths[%d] > lengths[%d])", b, b - 1);
      s.lens[b] = lengths[b];
    }
  }
  s.counts.assign(T, 0);
  s.offs.assign(T + 1, 0);
  int64_t nb = B;
  for (int t = 0; t < T; ++t) {
    while (nb > 0 && s.lens[nb - 1] <= t) --nb;
    s.counts[t] = nb;
    s.offs[t + 1] = s.offs[t] + nb;
  }
  s.N = s.offs[T];
  if (s.N >= (1ll << 31)) return fail(AM_EUNSUPPORTED, "too many frames");
  return AM_OK;
}

// The persistent layer kernels are used when they fit; AM_STEP_KERNELS=1 in
// the environment forces one launch per time step instead.
bool persistent_enabled() {
  const char* v = getenv("AM_STEP_KERNELS");
  if (v && v[0] && v[0] != '0') return false;
  const char* r = getenv("AM_RECURRENCE");
  return !(r && strcmp(r, "step") == 0);
}

// The bf16 per-step forward runs each step as one launch with the cell in
// the product's epilogue; AM_STEP_FUSION=0 in the environment keeps the
// product and the cell as two launches (tests compare the two bit for bit).
bool step_cell_fusion() {
  const char* v = getenv("AM_STEP_FUSION");
  return !(v && v[0] == '0' && v[1] == 0);
}

// AM_RECURRENCE=xcd|device|step picks one recurrence path (for tests);
// unset, the XCD-local kernels are tried first, then the device-scope ones.
bool xcd_enabled() {
  const char* r = getenv("AM_RECURRENCE");
  return persistent_enabled() && !(r && strcmp(r, "device") == 0);
}
bool device_persistent_enabled() {
  const char* r = getenv("AM_RECURRENCE");
  return persistent_enabled() && !(r && strcmp(r, "xcd") == 0);
}

// Scratch of the persistent kernels: the sync area at offset 0 of the
// workspace, one SYNC_BYTES slot per recurrence launch of a pass (each
// launch's step flags and XCC ids), so that one clear at the
// start of a pass serves all its launches instead of one small clear kernel
// before each.  The last word of slot 0 is the barrier time-out flag of
// every launch, zeroed once per forward pass and only ever set afterwards,
// so a time-out anywhere in a forward + backward pair stays visible to
// am_workspace_check.
constexpr int64_t SYNC_BYTES = 8192;
// k-splits of the per-step backward product dA_{t+1} W_h (five fill 240 of
// the 256 CUs with the 48 tiles of B = 512, H = 1536)
constexpr int STEP_SPLITS = 5;
constexpr int64_t SYNC_STICKY_WORD = SYNC_BYTES / 4 - 1;
void* sync_slot(void* area, int k) { return static_cast<char*>(area) + (int64_t)k * SYNC_BYTES; }
int* sync_err(void* area) { return static_cast<int*>(area) + SYNC_STICKY_WORD; }
am::XcdSync xcd_sync(void* slot, int* err) {
  unsigned* u = static_cast<unsigned*>(slot);
  am::XcdSync y;
  y.flags = u;  // flag line of block k < 16: u[32 k .. 32 k + 31], a word per member
  y.xcc = reinterpret_cast<int*>(u + 512);  // XCC line of block k: u[512 + 32 k ..], the same
  y.err = err;
  y.units = 0;
  y.fenced = 0;
  return y;
}
static_assert(512 + 512 <= SYNC_STICKY_WORD, "a slot holds the flag and XCC lines below the time-out word");

// Whether the XCD-local kernels take this layer's recurrence: bf16, the
// shape instantiated, and (variable lengths) T within the schedule's 16-bit
// lengths.
bool xcd_shape(bool forward, bool bf, int64_t H, int T, int B, bool varlen) {
  return bf && xcd_enabled() && am::lstm_xcd_instantiated(forward, (int)H, B) &&
         (!varlen || T <= 65535);
}
bool xcd_path(bool forward, bool bf, int64_t H, const Schedule& sc) {
  bool varlen = false;
  for (int b = 0; b < sc.B && !varlen; ++b) varlen = sc.lens[b] != sc.T;
  return xcd_shape(forward, bf, H, sc.T, sc.B, varlen);
}

// AM_DEBUG=1 in the environment: entry points that consume indices held in
// device buffers synchronise and check them.
bool debug_checks() {
  const char* v = getenv("AM_DEBUG");
  return v && v[0] == '1' && v[1] == 0;
}

am::PersistSchedule persist_schedule(const Schedule& sc) {
  am::PersistSchedule ps;
  ps.T = sc.T;
  ps.B = sc.B;
  ps.N = (int)sc.N;
  ps.varlen = 0;
  for (int b = 0; b < sc.B; ++b)
    if (sc.lens[b] != sc.T) ps.varlen = 1;
  memset(ps.lens, 0, sizeof ps.lens);
  if (ps.varlen)
    for (int b = 0; b < sc.B; ++b) ps.lens[b] = (uint16_t)sc.lens[b];
  return ps;
}

// Workspace carve-up (256-byte aligned regions).
struct WsLayout {
  std::vector<int64_t> h, hs, c, g;  // per layer
  int64_t p_da, dh, wht, dc, c0, h0, pre, splitk, splitk_floats, sync, total;
  static constexpr int MAX_SPLITS = 8;
};

int64_t align256(int64_t x) { return (x + 255) & ~int64_t(255); }

WsLayout ws_layout(const am_model* m, int64_t B, int64_t N) {
  WsLayout w;
  const int64_t e = esz_of(m->dtype), H = m->hidden, G = 4 * H, L = m->layers;
  int64_t pos = 0;
  auto take = [&](int64_t bytes) { int64_t at = pos; pos += align256(bytes); return at; };
  // step-barrier scratch of the persistent kernels (a slot per layer and
  // direction of the pass) and the time-out flag
  w.sync = take(2 * L * SYNC_BYTES);
  for (int l = 0; l < L; ++l) {
    w.h.push_back(take(N * H * e));
    w.hs.push_back(take(N * H * e));
    w.c.push_back(take(N * H * 4));
    w.g.push_back(take(N * G * e));
  }
  w.p_da = take(N * G * e);
  w.dh = take(N * H * e);
  w.wht = take(L * G * H * e);  // W_h^T of every layer (transposed in one launch)
  w.dc = take(B * H * 4);
  w.c0 = take(L * B * H * 4);
  w.h0 = take(L * B * H * e);
  // one step's recurrent product (per-step path): [B][4H] fp32 forward, up to
  // STEP_SPLITS k-split partials [B][H] fp32 backward
  w.pre = take(B * H * 4 * (STEP_SPLITS > 4 ? STEP_SPLITS : 4));
  // split-K partials of the weight-gradient products (plus partial row sums)
  const int64_t D0 = m->input_dim;
  const int64_t wide = (D0 > H ? D0 : H) + H;
  int64_t mn = G * wide + G;
  if ((int64_t)m->classes * H + m->classes > mn) mn = (int64_t)m->classes * H + m->classes;
  w.splitk_floats = WsLayout::MAX_SPLITS * mn;
  w.splitk = take(w.splitk_floats * 4);
  w.total = pos;
  return w;
}

template <typename P> P* at(void* base, int64_t off) {
  return reinterpret_cast<P*>(static_cast<char*>(base) + off);
}

double gemm_bytes(int64_t M, int64_t N, int64_t K, int64_t e, int64_t out) {
  return (double)(M * K + N * K) * e + (double)(M * N) * out;
}

am_status run_gemm(int cls, const am::GemmArgs& g, hipStream_t s) {
  const int64_t e = g.bf16 ? 2 : 4;
  Timed tm(cls, s, 2.0 * g.M * g.N * (double)g.K, gemm_bytes(g.M, g.N, g.K, e, g.c_f32 ? 4 : e));
  return hip_check(am::gemm(g, s), "gemm");
}

am::GemmArgs mk_gemm(const void* A, int64_t lda, bool ak, const void* B, int64_t ldb, bool bk,
                     void* C, int64_t ldc, bool cf32, const void* bias, int M, int N, int K,
                     bool bf16) {
  am::GemmArgs g;
  g.A = A; g.lda = lda; g.a_kmajor = ak;
  g.B = B; g.ldb = ldb; g.b_kmajor = bk;
  g.C = C; g.ldc = ldc; g.c_f32 = cf32;
  g.bias = bias; g.M = M; g.N = N; g.K = K; g.bf16 = bf16;
  return g;
}

// One layer's recurrence, forward in time, over the packed rows of a
// schedule: the XCD-local persistent kernel where it covers the shape, else
// the device-scope persistent kernel, else one launch per time step.
struct FwdLayer {
  const void* P;      // [N][4H] input projections + bias
  const void* Wh;     // [4H][H]
  const void* h0;     // [B][H] activation type, or null (zero)
  const float* c0;    // [B][H]
  void* H; void* Hs; float* C; void* G;  // outputs [N][H], [N][H], [N][H], [N][4H]
  void* sync;         // this launch's slot of the workspace's sync area (cleared)
  int* err;           // the time-out flag
  float* pre;         // [B][4H] fp32 scratch of the per-step path
};

am_status forward_recurrence(const FwdLayer& f, const Schedule& sc, bool bf, int64_t H,
                             hipStream_t s) {
  const int64_t e = bf ? 2 : 4, G = 4 * H;
  const int T = sc.T, B = sc.B;
  if (sc.N > 0 && persistent_enabled()) {
    am::PersistFwd pa;
    pa.P = f.P;
    pa.Wh = f.Wh;
    pa.h0 = f.h0;
    pa.c0 = f.c0;
    pa.H = f.H;
    pa.Hs = f.Hs;
    pa.C = f.C;
    pa.G = f.G;
    pa.counters = static_cast<unsigned*>(f.sync);
    pa.err = f.err;
    pa.hidden = (int)H;
    const am::PersistSchedule ps = persist_schedule(sc);
    const double flops = 2.0 * sc.N * G * H;
    const double bytes = (double)sc.N * (G * e * 2 + H * (2 * e + 4)) + (double)G * H * e;
    bool used = false;
    if (xcd_path(true, bf, H, sc)) {
      Timed tm(AM_K_LSTM_FWD, s, flops, bytes);
      AM_TRY(hip_check(am::lstm_fwd_xcd_launch(pa, ps, xcd_sync(f.sync, f.err), s, &used),
                       "lstm forward layer (xcd)"));
      if (!used) tm.cancel();
    }
    if (!used && device_persistent_enabled() && am::lstm_persistent_fits(true, (int)H, B, bf, T)) {
      Timed tm(AM_K_LSTM_FWD, s, flops, bytes);
      AM_TRY(hip_check(am::lstm_fwd_persistent(pa, ps, bf, s, &used), "lstm forward layer"));
      if (!used) tm.cancel();
    }
    if (used) return AM_OK;
  }
  const char* Hl = static_cast<const char*>(f.H);
  const float* Cl = f.C;
  const bool fuse_cell = step_cell_fusion();
  for (int t = 0; t < T; ++t) {
    const int64_t nb = sc.counts[t];
    if (nb == 0) break;
    const int64_t o = sc.offs[t];
    am::LstmFwdStep a;
    a.P = static_cast<const char*>(f.P) + o * G * e;
    a.Wh = f.Wh;
    if (t == 0) {
      a.hprev = f.h0;
      a.cprev = f.c0;
    } else {
      a.hprev = Hl + sc.offs[t - 1] * H * e;
      a.cprev = Cl + sc.offs[t - 1] * H;
    }
    a.H = static_cast<char*>(f.H) + o * H * e;
    a.Hs = static_cast<char*>(f.Hs) + o * H * e;
    a.C = f.C + o * H;
    a.G = static_cast<char*>(f.G) + o * G * e;
    a.nb = (int)nb;
    a.hidden = (int)H;
    a.bf16 = bf;
    if (bf) {
      // the step's recurrent product as a batched product (few rows: square
      // tiles that fill the CUs) with the cell in its epilogue; else the
      // product into fp32 scratch, then the cell
      float* pre = nullptr;
      if (a.hprev && fuse_cell) {
        bool done = false;
        Timed tm(AM_K_LSTM_FWD, s, 2.0 * nb * G * H,
                 gemm_bytes(nb, G, H, e, 0) + (double)nb * (G * e + H * (2 * e + 8) + G * e));
        AM_TRY(hip_check(am::gemm_bf16_lstm_fwd_step(a, s, &done), "lstm forward step (fused)"));
        if (done) continue;
        tm.cancel();
      }
      if (a.hprev) {
        AM_TRY(run_gemm(AM_K_LSTM_FWD,
                        mk_gemm(a.hprev, H, true, f.Wh, H, true, f.pre, G, true, nullptr, (int)nb,
                                (int)G, (int)H, true), s));
        pre = f.pre;
      }
      Timed tm(AM_K_LSTM_FWD, s, 0.0, (double)nb * (G * (4.0 + e) + H * (2 * e + 8) + G * e));
      AM_TRY(hip_check(am::lstm_cell_fwd(pre, a, s), "lstm forward cell"));
      continue;
    }
    const double bytes = (double)(nb * H + G * H + nb * G) * e + nb * H * 4.0 +
                         (double)nb * (H * (2 * e + 4) + G * e);
    Timed tm(AM_K_LSTM_FWD, s, 2.0 * nb * G * H, bytes);
    AM_TRY(hip_check(am::lstm_fwd_step(a, s), "lstm forward step"));
  }
  return AM_OK;
}

// Weight gradient  [C | C2] = A^T [B | B2]  (K = frames), fp32, with the
// row sums of A (the bias gradient) and split-K scratch from the workspace.
am::GemmArgs mk_wgrad(const void* A, int64_t lda, const void* B, int64_t ldb, int nB,
                      const void* B2, int64_t ldb2, int nB2, float* C, int64_t ldc, float* C2,
                      int64_t ldc2, float* rowsum, int M, int K, bool bf16, float* ws,
                      int64_t ws_floats) {
  am::GemmArgs g;
  g.A = A; g.lda = lda; g.a_kmajor = false;
  g.B = B; g.ldb = ldb; g.b_kmajor = false;
  g.C = C; g.ldc = ldc; g.c_f32 = true;
  if (B2) {
    g.B2 = B2; g.ldb2 = ldb2; g.n_split = nB;
    g.C2 = C2; g.ldc2 = ldc2;
  }
  g.rowsum = rowsum;
  g.M = M; g.N = nB + (B2 ? nB2 : 0); g.K = K; g.bf16 = bf16;
  g.ws = ws; g.ws_floats = ws_floats;
  return g;
}

// Teacher: per layer, forward Wx [4H][D_l], Wh [4H][H], b [4H], then the
// backward direction's; D_0 = input_dim, D_l = 2H; then Wo [C][2H], bo [C].
struct TeacherOffsets {
  std::vector<int64_t> wx, wh, b;  // [layer * 2 + direction]
  int64_t wo, bo, n;
};

TeacherOffsets teacher_layout(const am_model* m) {
  TeacherOffsets o;
  const int64_t H = m->hidden, G = 4 * H;
  int64_t pos = 0;
  for (int l = 0; l < m->layers; ++l) {
    const int64_t D = l == 0 ? m->input_dim : 2 * H;
    for (int d = 0; d < 2; ++d) {
      o.wx.push_back(pos); pos += G * D;
      o.wh.push_back(pos); pos += G * H;
      o.b.push_back(pos); pos += G;
    }
  }
  o.wo = pos; pos += (int64_t)m->classes * 2 * H;
  o.bo = pos; pos += m->classes;
  o.n = pos;
  return o;
}

struct TeacherWs {
  int64_t sync, offs, lens, cat0, cat1, rev, p, hdir, hs, c, g, c0, pre, total;
};

TeacherWs teacher_ws_layout(const am_model* m, int64_t T, int64_t B, int64_t N) {
  TeacherWs w;
  const int64_t e = esz_of(m->dtype), H = m->hidden, G = 4 * H;
  const int64_t Dmax = m->input_dim > 2 * H ? m->input_dim : 2 * H;
  int64_t pos = 0;
  auto take = [&](int64_t bytes) { int64_t at = pos; pos += align256(bytes); return at; };
  w.sync = take(2 * m->layers * SYNC_BYTES);  // a slot per layer and direction
  w.offs = take((T + 1) * 8);
  w.lens = take(B * 4);
  w.cat0 = take(N * 2 * H * e);
  w.cat1 = take(N * 2 * H * e);
  w.rev = take(N * Dmax * e);
  w.p = take(N * G * e);
  w.hdir = take(N * H * e);
  w.hs = take(N * H * e);
  w.c = take(N * H * 4);
  w.g = take(N * G * e);
  w.c0 = take(B * H * 4);
  w.pre = take(B * G * 4);
  w.total = pos;
  return w;
}

// ------------------------------------------------- threshold encode --

am_status check_encode_args(int64_t n, const float* grad, const float* residual, float tau,
                            const uint32_t* words, int64_t capacity, const int64_t* count) {
  if (n < 0 || n >= (1ll << 31)) return fail(AM_EINVAL, "n = %lld outside [0, 2^31)", (long long)n);
  if (!(tau > 0.f)) return fail(AM_EINVAL, "tau must be > 0");
  if (!count) return fail(AM_EINVAL, "count is NULL");
  if (n > 0 && (!grad || !residual || !words)) return fail(AM_EINVAL, "NULL pointer");
  if (capacity < n) return fail(AM_ECAPACITY, "capacity %lld < n %lld", (long long)capacity, (long long)n);
  return AM_OK;
}

// The encode launches on a scratch area of gtc_encode_scratch_bytes(n)
// (the codes, then the tile counts); every byte the kernels read there is
// written by the same call first, so the area needs no clearing.
am_status encode_with_scratch(int64_t n, const float* grad, float* residual, float tau,
                              uint32_t* words, int64_t* count, void* scratch, hipStream_t s) {
  Timed tm(AM_K_ENCODE, s, 0.0, 12.0 * n);
  uint32_t* codes = at<uint32_t>(scratch, 0);
  int32_t* tile = at<int32_t>(scratch, am::gtc_codes_bytes(n));
  return hip_check(am::gtc_encode(n, grad, residual, tau, words, count, codes, tile, s), "encode");
}

// Scratch of grad_threshold_encode_noalloc: a device array owned by the
// library for the life of the process (each GPU holds its own copy).  In
// host code its name only stands in for the symbol; the device address of
// a GPU's copy comes from hipGetSymbolAddress with that GPU current, once,
// and is kept per device.
constexpr int64_t NOALLOC_SCRATCH_BYTES = am::gtc_encode_scratch_bytes(AM_ENCODE_NOALLOC_MAX_N);
static __device__ __align__(256) unsigned char encode_scratch[NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

am_status encode_scratch_of(hipStream_t s, void** out) {
  int cur = 0, dev = 0;
  AM_TRY(hip_check(hipGetDevice(&cur), "hipGetDevice"));
  dev = cur;
  if (s) AM_TRY(hip_check(hipStreamGetDevice(s, &dev), "hipStreamGetDevice"));
  if (dev < 0 || dev >= MAX_DEVICES) return fail(AM_EUNSUPPORTED, "device %d >= %d", dev, MAX_DEVICES);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur) AM_TRY(hip_check(hipSetDevice(dev), "hipSetDevice"));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(encode_scratch));
    if (dev != cur) AM_TRY(hip_check(hipSetDevice(cur), "hipSetDevice"));
    AM_TRY(hip_check(e, "hipGetSymbolAddress(encode scratch)"));
    if (!p || !aligned(p, 256)) return fail(AM_EHIP, "encode scratch has no 256-byte aligned address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return AM_OK;
}

}  // namespace

// ================================================================= C ABI ==

extern "C" {

const char* am_status_string(int32_t st) {
  switch (st) {
    case AM_OK: return "ok";
    case AM_EINVAL: return "invalid argument";
    case AM_ECAPACITY: return "output capacity too small";
    case AM_EUNSUPPORTED: return "unsupported configuration";
    case AM_EHIP: return "HIP error";
    case AM_EWORKSPACE: return "workspace missing or too small";
    case AM_ETIMEOUT: return "step barrier timed out";
    default: return "unknown status";
  }
}

const char* am_last_error(void) { return g_err.c_str(); }

int64_t am_param_count(const am_model* m) {
  if (check_model(m) != AM_OK) return -1;
  return param_layout(m).n;
}

am_status am_param_offsets(const am_model* m, int64_t* offsets) {
  AM_TRY(check_model(m));
  if (!offsets) return fail(AM_EINVAL, "offsets is NULL");
  Offsets o = param_layout(m);
  for (int l = 0; l < m->layers; ++l) {
    offsets[3 * l] = o.wx[l];
    offsets[3 * l + 1] = o.wh[l];
    offsets[3 * l + 2] = o.b[l];
  }
  offsets[3 * m->layers] = o.wo;
  offsets[3 * m->layers + 1] = o.bo;
  return AM_OK;
}

int32_t am_recurrence_path(const am_model* m, int32_t T, int32_t B, int32_t varlen,
                           int32_t forward) {
  if (check_model(m) != AM_OK || T < 0 || B < 1) return -1;
  const bool bf = m->dtype == AM_BF16, fw = forward != 0;
  if (!persistent_enabled()) return AM_PATH_STEP;
  if (xcd_shape(fw, bf, m->hidden, T, B, varlen != 0)) return AM_PATH_XCD;
  if (device_persistent_enabled() && am::lstm_persistent_fits(fw, m->hidden, B, bf, T))
    return AM_PATH_DEVICE;
  return AM_PATH_STEP;
}

int64_t am_workspace_bytes(const am_model* m, int32_t T, int32_t B, int64_t N) {
  if (check_model(m) != AM_OK || T < 0 || B < 1 || N < 0 || N > (int64_t)T * B) return -1;
  return ws_layout(m, B, N).total;
}

int64_t am_ce_workspace_bytes(int64_t N) {
  if (N < 0) return -1;
  return align256(am::soft_ce_partials(N) * 4) + 256;
}

int64_t am_encode_workspace_bytes(int64_t n) {
  if (n < 0) return -1;
  return am::gtc_encode_scratch_bytes(n);
}

am_status am_cast_f32_to_bf16(int64_t n, const float* src, void* dst, void* stream) {
  if (n < 0) return fail(AM_EINVAL, "n < 0");
  if (n > 0 && (!src || !dst)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_MISC, s, 0.0, 6.0 * n);
  return hip_check(am::cast_f32_bf16(n, src, static_cast<uint16_t*>(dst), s), "cast");
}

am_status sgd_apply(int64_t n, float* master, void* weights_bf16, const float* update, float lr,
                    void* stream) {
  if (n < 0) return fail(AM_EINVAL, "n < 0");
  if (n > 0 && (!master || !update)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_SGD, s, 2.0 * n, (weights_bf16 ? 14.0 : 12.0) * n);
  return hip_check(am::sgd_apply_f32(n, master, static_cast<uint16_t*>(weights_bf16), update, lr, s),
                   "sgd_apply");
}

am_status grad_threshold_encode(int64_t n, const float* grad, float* residual, float tau,
                                uint32_t* words, int64_t capacity, int64_t* count, void* ws,
                                int64_t ws_bytes, void* stream) {
  AM_TRY(check_encode_args(n, grad, residual, tau, words, capacity, count));
  const int64_t need = am_encode_workspace_bytes(n);
  if (!ws || ws_bytes < need || !aligned(ws, 256))
    return fail(AM_EWORKSPACE, "encode needs %lld workspace bytes (256-aligned)", (long long)need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  return encode_with_scratch(n, grad, residual, tau, words, count, ws, s);
}

am_status grad_threshold_encode_noalloc(int64_t n, const float* grad, float* residual, float tau,
                                        uint32_t* words, int64_t capacity, int64_t* count,
                                        void* stream) {
  AM_TRY(check_encode_args(n, grad, residual, tau, words, capacity, count));
  if (n > AM_ENCODE_NOALLOC_MAX_N)
    return fail(AM_EUNSUPPORTED, "grad_threshold_encode_noalloc handles n <= %lld (n = %lld); "
                "use grad_threshold_encode with a workspace", (long long)AM_ENCODE_NOALLOC_MAX_N,
                (long long)n);
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* scratch = nullptr;
  AM_TRY(encode_scratch_of(s, &scratch));
  return encode_with_scratch(n, grad, residual, tau, words, count, scratch, s);
}

am_status grad_threshold_decode(const uint32_t* words, const int64_t* count, int64_t capacity,
                                float tau, int64_t n, float* dense, int32_t accumulate,
                                void* stream) {
  if (n < 0 || n >= (1ll << 31)) return fail(AM_EINVAL, "n outside [0, 2^31)");
  if (capacity < 0) return fail(AM_EINVAL, "capacity < 0");
  if (!count || (n > 0 && !dense) || (capacity > 0 && !words)) return fail(AM_EINVAL, "NULL pointer");
  if (accumulate != 0 && accumulate != 1) return fail(AM_EINVAL, "accumulate must be 0 or 1");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_DECODE, s, 0.0, (accumulate ? 8.0 : 4.0) * n);
  return hip_check(am::gtc_decode(words, count, capacity, tau, n, dense, accumulate != 0, s), "decode");
}

am_status grad_threshold_decode_sgd(const uint32_t* words, const int64_t* count, int64_t capacity,
                                    float tau, int64_t n, float lr, float* master,
                                    void* weights_bf16, void* stream) {
  if (n < 0 || n >= (1ll << 31)) return fail(AM_EINVAL, "n outside [0, 2^31)");
  if (capacity < 0) return fail(AM_EINVAL, "capacity < 0");
  if (!count || (n > 0 && !master) || (capacity > 0 && !words)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  // bytes: with lr +0.0 or positive and finite only the named elements are
  // touched, 14 (or 12) bytes per word, which the host cannot count without
  // reading the count: none are recorded here; otherwise the master read and
  // written and the bf16 copy written (the words not counted)
  const uint32_t lb = __builtin_bit_cast(uint32_t, lr);
  const bool named_only = lb == 0u || (lr > 0.f && lr <= 3.402823466e38f);
  Timed tm(AM_K_SGD, s, named_only ? 0.0 : 2.0 * n, named_only ? 0.0 : (weights_bf16 ? 10.0 : 8.0) * n);
  return hip_check(am::gtc_decode_sgd(words, count, capacity, tau, n, lr, master,
                                      static_cast<uint16_t*>(weights_bf16), s),
                   "decode + sgd");
}

int64_t am_decode_multi_workspace_bytes(int32_t streams, int64_t n) {
  if (streams < 0 || n < 0) return -1;
  return align256((int64_t)streams * (am::gtc_tiles(n) + 1) * 4);
}

am_status grad_threshold_decode_multi(int32_t streams, const uint32_t* words, int64_t capacity,
                                      const int64_t* counts, float tau, int64_t n, float* dense,
                                      int32_t accumulate, void* ws, int64_t ws_bytes,
                                      void* stream) {
  if (n < 0 || n >= (1ll << 31)) return fail(AM_EINVAL, "n outside [0, 2^31)");
  if (streams < 0 || streams > 32767) return fail(AM_EINVAL, "streams outside [0, 32767]");
  if (capacity < 0) return fail(AM_EINVAL, "capacity < 0");
  if ((n > 0 && !dense) || (streams > 0 && (!counts || (capacity > 0 && !words))))
    return fail(AM_EINVAL, "NULL pointer");
  if (accumulate != 0 && accumulate != 1) return fail(AM_EINVAL, "accumulate must be 0 or 1");
  const int64_t need = am_decode_multi_workspace_bytes(streams, n);
  if (need > 0 && (!ws || ws_bytes < need || !aligned(ws, 256)))
    return fail(AM_EWORKSPACE, "multi-stream decode needs %lld workspace bytes (256-aligned)",
                (long long)need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_DECODE, s, 0.0, (accumulate ? 8.0 : 4.0) * n);
  return hip_check(am::gtc_decode_multi(streams, words, capacity, counts, tau, n, dense,
                                        accumulate != 0, static_cast<int32_t*>(ws), s),
                   "multi-stream decode");
}

am_status bmuf_block_update(int64_t n, int32_t count, int32_t workers, const float* models,
                            int64_t model_stride, float* global_model, float* delta, float eta,
                            float eta_next, float zeta, float* local_master, void* local_bf16,
                            void* stream) {
  if (n < 0) return fail(AM_EINVAL, "n < 0");
  if (count < 1 || workers < 1) return fail(AM_EINVAL, "count and workers must be >= 1");
  if (count > 1 && model_stride < n) return fail(AM_EINVAL, "model_stride < n");
  if (n > 0 && (!models || !global_model || !delta)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  const double bytes = (4.0 * count + 16.0 + (local_master ? 4.0 : 0.0) + (local_bf16 ? 2.0 : 0.0)) * n;
  Timed tm(AM_K_BMUF, s, 0.0, bytes);
  return hip_check(am::bmuf_update(n, count, workers, models, model_stride, global_model, delta,
                                   eta, eta_next, zeta, local_master,
                                   static_cast<uint16_t*>(local_bf16), s),
                   "bmuf_block_update");
}

int32_t am_lfr_frames(int32_t raw_frames, int32_t stack, int32_t skip, int32_t offset) {
  if (raw_frames < 0 || stack < 1 || skip < 1 || offset < 0 || offset >= skip) return -1;
  const int32_t r = raw_frames - offset - stack;
  return r < 0 ? 0 : r / skip + 1;
}

am_status lfr_features(int32_t B, const int32_t* raw_lengths, const float* raw, int32_t raw_dim,
                       int32_t stack, int32_t skip, int32_t offset, const float* mean,
                       const float* std, void* x, int32_t x_dtype, void* stream) {
  if (B < 0 || B > 1024) return fail(AM_EUNSUPPORTED, "B must be in [0, 1024]");
  if (raw_dim < 1 || stack < 1 || skip < 1 || offset < 0 || offset >= skip)
    return fail(AM_EINVAL, "need raw_dim, stack, skip >= 1 and 0 <= offset < skip");
  if ((int64_t)stack * raw_dim > 4096) return fail(AM_EUNSUPPORTED, "stack * raw_dim > 4096");
  if (x_dtype != AM_F32 && x_dtype != AM_BF16) return fail(AM_EINVAL, "unknown x dtype");
  if (B > 0 && !raw_lengths) return fail(AM_EINVAL, "raw_lengths is NULL");
  am::LfrArgs a;
  memset(&a, 0, sizeof a);
  a.B = B; a.raw_dim = raw_dim; a.stack = stack; a.skip = skip; a.offset = offset;
  int64_t frames = 0, raws = 0;
  int32_t prev = 0;
  for (int b = 0; b < B; ++b) {
    if (raw_lengths[b] < 0 || raw_lengths[b] > 65535)
      return fail(AM_EUNSUPPORTED, "raw_lengths[%d] = %d outside [0, 65535]", b, raw_lengths[b]);
    const int32_t T = am_lfr_frames(raw_lengths[b], stack, skip, offset);
    if (b > 0 && T > prev)
      return fail(AM_EINVAL, "stacked lengths must be non-increasing (utterance %d)", b);
    prev = T;
    frames += T;
    raws += raw_lengths[b];
    a.U[b] = (uint16_t)raw_lengths[b];
  }
  if (raws > 0 && !raw) return fail(AM_EINVAL, "raw is NULL");
  if (frames > 0 && (!x || !mean || !std)) return fail(AM_EINVAL, "NULL x, mean or std");
  a.raw = raw; a.mean = mean; a.std = std; a.x = x;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const double bytes = (double)frames * stack * raw_dim * (4 + (x_dtype == AM_BF16 ? 2 : 4));
  Timed tm(AM_K_MISC, s, 0.0, bytes);
  return hip_check(am::lfr_features(a, x_dtype == AM_BF16, s), "lfr_features");
}

am_status delay_targets(int32_t T, int32_t B, const int32_t* lengths, int32_t K, int32_t delay,
                        const int32_t* idx, const float* prob, int32_t* idx_out, float* prob_out,
                        uint8_t* mask_out, void* stream) {
  if (T > 65535) return fail(AM_EUNSUPPORTED, "T > 65535");
  if (K < 0 || delay < 0) return fail(AM_EINVAL, "need K >= 0 and delay >= 0");
  Schedule sc;
  AM_TRY(make_schedule(T, B, lengths, sc));
  if (sc.N > 0 && (!mask_out || (K > 0 && (!idx || !prob || !idx_out || !prob_out))))
    return fail(AM_EINVAL, "NULL pointer");
  am::DelayArgs a;
  memset(&a, 0, sizeof a);
  if (B > 1024) return fail(AM_EUNSUPPORTED, "B > 1024");
  a.T = T; a.B = B; a.K = K; a.delay = delay;
  for (int b = 0; b < B; ++b) a.len[b] = (uint16_t)sc.lens[b];
  a.idx = idx; a.prob = prob; a.idx_out = idx_out; a.prob_out = prob_out; a.mask_out = mask_out;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_MISC, s, 0.0, (double)sc.N * (16.0 * K + 1));
  return hip_check(am::delay_targets(a, s), "delay_targets");
}

int64_t am_teacher_param_count(const am_model* m) {
  if (check_model(m) != AM_OK) return -1;
  return teacher_layout(m).n;
}

am_status am_teacher_param_offsets(const am_model* m, int64_t* offsets) {
  AM_TRY(check_model(m));
  if (!offsets) return fail(AM_EINVAL, "offsets is NULL");
  const TeacherOffsets o = teacher_layout(m);
  for (int k = 0; k < 2 * m->layers; ++k) {
    offsets[3 * k] = o.wx[k];
    offsets[3 * k + 1] = o.wh[k];
    offsets[3 * k + 2] = o.b[k];
  }
  offsets[6 * m->layers] = o.wo;
  offsets[6 * m->layers + 1] = o.bo;
  return AM_OK;
}

int64_t am_teacher_workspace_bytes(const am_model* m, int32_t T, int32_t B, int64_t N) {
  if (check_model(m) != AM_OK || T < 0 || B < 1 || N < 0 || N > (int64_t)T * B) return -1;
  return teacher_ws_layout(m, T, B, N).total;
}

am_status blstm_teacher_forward(const am_model* m, const void* params, const void* x,
                                const int32_t* lengths, int32_t T, int32_t B, float* logits,
                                void* ws, int64_t ws_bytes, void* stream) {
  AM_TRY(check_model(m));
  if (B > 1024 || T > 65535) return fail(AM_EUNSUPPORTED, "the teacher allows B <= 1024, T <= 65535");
  Schedule sc;
  AM_TRY(make_schedule(T, B, lengths, sc));
  if (!params || !ws) return fail(AM_EINVAL, "NULL params or workspace");
  if (sc.N > 0 && (!x || !logits)) return fail(AM_EINVAL, "NULL x or logits");
  if (!aligned(params, 16) || !aligned(x, 16) || !aligned(logits, 16) || !aligned(ws, 256))
    return fail(AM_EINVAL, "params, x, logits must be 16-byte and ws 256-byte aligned");
  const TeacherWs w = teacher_ws_layout(m, T, B, sc.N);
  if (ws_bytes < w.total)
    return fail(AM_EWORKSPACE, "teacher forward needs %lld workspace bytes", (long long)w.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf = m->dtype == AM_BF16;
  const int64_t e = esz_of(m->dtype), H = m->hidden, G = 4 * H, L = m->layers;
  const TeacherOffsets po = teacher_layout(m);
  const char* P8 = static_cast<const char*>(params);
  const int N = (int)sc.N;

  // schedule tables for the time reversal (built on the device from the
  // lengths passed by value); a zero initial cell state
  {
    am::SchedTables st;
    memset(&st, 0, sizeof st);
    st.T = T; st.B = B;
    for (int b = 0; b < B; ++b) st.len[b] = (uint16_t)sc.lens[b];
    st.offs = at<int64_t>(ws, w.offs);
    st.lens = at<int32_t>(ws, w.lens);
    AM_TRY(hip_check(am::schedule_tables(st, s), "schedule tables"));
  }
  AM_TRY(hip_check(am::fill_zero2(at<float>(ws, w.c0), B * H, at<float>(ws, w.sync),
                                  2 * L * SYNC_BYTES / 4, s), "c0 and sync clear"));
  auto gather = [&](const void* src, int64_t src_ld, void* dst, int64_t dst_ld, int64_t col,
                    int width, bool reverse) {
    am::GatherRows g;
    g.src = src; g.src_ld = src_ld; g.dst = dst; g.dst_ld = dst_ld; g.dst_col = col;
    g.width = width; g.N = sc.N; g.T = T;
    g.offs = at<int64_t>(ws, w.offs); g.lens = at<int32_t>(ws, w.lens);
    g.reverse = reverse ? 1 : 0;
    Timed tm(AM_K_MISC, s, 0.0, 2.0 * sc.N * width * e);
    return hip_check(am::gather_rows(g, bf, s), "gather rows");
  };

  for (int l = 0; l < L; ++l) {
    const int64_t D = l == 0 ? m->input_dim : 2 * H;
    const void* X = l == 0 ? x : at<void>(ws, (l - 1) % 2 ? w.cat1 : w.cat0);
    void* out = at<void>(ws, l % 2 ? w.cat1 : w.cat0);
    for (int d = 0; d < 2; ++d) {
      const int k = 2 * l + d;
      const void* in = X;
      if (d == 1) {  // the backward direction reads the sequences reversed
        AM_TRY(gather(X, D, at<void>(ws, w.rev), D, 0, (int)D, true));
        in = at<void>(ws, w.rev);
      }
      AM_TRY(run_gemm(AM_K_GEMM_FWD,
                      mk_gemm(in, D, true, P8 + po.wx[k] * e, D, true, at<void>(ws, w.p), G, false,
                              P8 + po.b[k] * e, N, (int)G, (int)D, bf), s));
      FwdLayer f;
      f.P = at<void>(ws, w.p);
      f.Wh = P8 + po.wh[k] * e;
      f.h0 = nullptr;
      f.c0 = at<float>(ws, w.c0);
      f.H = at<void>(ws, w.hdir);
      f.Hs = at<void>(ws, w.hs);
      f.C = at<float>(ws, w.c);
      f.G = at<void>(ws, w.g);
      f.sync = sync_slot(at<void>(ws, w.sync), k);
      f.err = sync_err(at<void>(ws, w.sync));
      f.pre = at<float>(ws, w.pre);
      AM_TRY(forward_recurrence(f, sc, bf, H, s));
      AM_TRY(gather(at<void>(ws, w.hdir), H, out, 2 * H, d * H, (int)H, d == 1));
    }
  }
  return run_gemm(AM_K_GEMM_FWD,
                  mk_gemm(at<void>(ws, (L - 1) % 2 ? w.cat1 : w.cat0), 2 * H, true, P8 + po.wo * e,
                          2 * H, true, logits, m->classes, true, P8 + po.bo * e, N, m->classes,
                          (int)(2 * H), bf), s);
}

am_status kbest_logits(int64_t N, int32_t C, int32_t K, const float* logits, int32_t* idx,
                       float* val, void* stream) {
  if (N < 0 || C < 1 || K < 0 || K > C) return fail(AM_EINVAL, "need N >= 0, C >= 1, 0 <= K <= C");
  if (K > 64) return fail(AM_EUNSUPPORTED, "K > 64");
  if (C > 8192) return fail(AM_EUNSUPPORTED, "C > 8192");
  if (N > 0 && K > 0 && (!logits || !idx || !val)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_MISC, s, 0.0, (double)N * (4.0 * C + 8.0 * K));
  return hip_check(am::topk_rows(N, C, K, logits, idx, val, s), "kbest_logits");
}

am_status kbest_posteriors(int64_t N, int32_t K, const float* val, float* prob, void* stream) {
  if (N < 0 || K < 0) return fail(AM_EINVAL, "need N >= 0 and K >= 0");
  if (N > 0 && K > 0 && (!val || !prob)) return fail(AM_EINVAL, "NULL pointer");
  hipStream_t s = static_cast<hipStream_t>(stream);
  Timed tm(AM_K_MISC, s, 0.0, (double)N * 8.0 * K);
  return hip_check(am::kbest_posteriors(N, K, val, prob, s), "kbest_posteriors");
}

am_status sparse_soft_ce(int64_t N, int32_t C, int32_t K, const float* logits, const int32_t* idx,
                         const float* prob, const uint8_t* mask, int32_t reduction, float* loss,
                         void* dlogits, int32_t dlogits_dtype, void* ws, int64_t ws_bytes,
                         void* stream) {
  if (N < 0 || C < 1 || K < 0) return fail(AM_EINVAL, "need N >= 0, C >= 1, K >= 0");
  if (C % 4) return fail(AM_EUNSUPPORTED, "C must be a multiple of 4");
  if (C > 8192) return fail(AM_EUNSUPPORTED, "C > 8192 classes");
  if (reduction != AM_MEAN_VALID && reduction != AM_SUM) return fail(AM_EINVAL, "unknown reduction");
  if (dlogits_dtype != AM_F32 && dlogits_dtype != AM_BF16) return fail(AM_EINVAL, "unknown dlogits dtype");
  if (!loss) return fail(AM_EINVAL, "loss is NULL");
  if (N > 0 && (!logits || !dlogits || (K > 0 && (!idx || !prob))))
    return fail(AM_EINVAL, "NULL pointer");
  if (!aligned(logits, 16) || !aligned(dlogits, dlogits_dtype == AM_BF16 ? 8 : 16))
    return fail(AM_EINVAL, "logits / dlogits must be 16-byte aligned");
  const int64_t need = am_ce_workspace_bytes(N);
  if (!ws || ws_bytes < need || !aligned(ws, 256))
    return fail(AM_EWORKSPACE, "soft_ce needs %lld workspace bytes (256-aligned)", (long long)need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (debug_checks() && N > 0 && K > 0) {
    // every target index in [-1, C): copied to the host after the work
    // queued before this call, then checked
    std::vector<int32_t> h((size_t)(N * K));
    AM_TRY(hip_check(hipMemcpyAsync(h.data(), idx, h.size() * 4, hipMemcpyDeviceToHost, s),
                     "AM_DEBUG index copy"));
    AM_TRY(hip_check(hipStreamSynchronize(s), "AM_DEBUG stream sync"));
    for (size_t i = 0; i < h.size(); ++i)
      if (h[i] < -1 || h[i] >= C)
        return fail(AM_EINVAL, "target index %d of row %lld, slot %lld outside [-1, %d)", h[i],
                    (long long)(i / K), (long long)(i % K), C);
  }
  am::SoftCeArgs a;
  a.N = N; a.C = C; a.K = K; a.z = logits; a.idx = idx; a.prob = prob; a.mask = mask;
  a.reduction = reduction; a.loss = loss; a.dz = dlogits; a.dz_bf16 = dlogits_dtype == AM_BF16;
  a.n_partials = am::soft_ce_partials(N);
  a.ws_partials = at<float>(ws, 0);
  a.ws_scale = at<float>(ws, align256(a.n_partials * 4));
  const double bytes = (double)N * C * (4 + (a.dz_bf16 ? 2 : 4)) + (double)N * K * 8;
  Timed tm(AM_K_CE, s, 0.0, bytes);
  return hip_check(am::soft_ce(a, s), "sparse_soft_ce");
}

am_status lstm_am_forward(const am_model* m, const void* params, const void* x,
                          const int32_t* lengths, const float* h0, const float* c0, int32_t T,
                          int32_t B, float* logits, float* hT, float* cT, void* ws,
                          int64_t ws_bytes, void* stream) {
  AM_TRY(check_model(m));
  Schedule sc;
  AM_TRY(make_schedule(T, B, lengths, sc));
  if (!params || !ws) return fail(AM_EINVAL, "NULL params or workspace");
  if (sc.N > 0 && (!x || !logits)) return fail(AM_EINVAL, "NULL x or logits");
  if (!aligned(params, 16) || !aligned(x, 16) || !aligned(logits, 16) || !aligned(ws, 256))
    return fail(AM_EINVAL, "params, x, logits must be 16-byte and ws 256-byte aligned");
  const WsLayout w = ws_layout(m, B, sc.N);
  if (ws_bytes < w.total)
    return fail(AM_EWORKSPACE, "forward needs %lld workspace bytes", (long long)w.total);

  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf = m->dtype == AM_BF16;
  const int64_t e = esz_of(m->dtype), H = m->hidden, G = 4 * H, L = m->layers;
  const Offsets po = param_layout(m);
  const char* P8 = static_cast<const char*>(params);

  // initial cell state (copied, or zero) and initial hidden state (converted)
  {
    Timed tm(AM_K_MISC, s, 0.0, 8.0 * L * B * H);
    float* c0w = at<float>(ws, w.c0);
    if (c0) AM_TRY(hip_check(am::convert_rows(c0, c0w, L * B * H, false, s), "c0 copy"));
    if (h0) AM_TRY(hip_check(am::convert_rows(h0, at<void>(ws, w.h0), L * B * H, bf, s), "h0 convert"));
    // a new forward + backward pair: every slot of the sync area and the
    // barrier time-out flag (and a zero initial cell state, in the same launch)
    AM_TRY(hip_check(am::fill_zero2(at<float>(ws, w.sync), 2 * L * SYNC_BYTES / 4, c0w,
                                    c0 ? 0 : L * B * H, s), "sync and c0 clear"));
  }

  for (int l = 0; l < L; ++l) {
    const int64_t D = l == 0 ? m->input_dim : H;
    const void* X = l == 0 ? x : at<void>(ws, w.h[l - 1]);
    void* P = at<void>(ws, w.p_da);
    AM_TRY(run_gemm(AM_K_GEMM_FWD,
                    mk_gemm(X, D, true, P8 + po.wx[l] * e, D, true, P, G, false, P8 + po.b[l] * e,
                            (int)sc.N, (int)G, (int)D, bf), s));
    FwdLayer f;
    f.P = at<void>(ws, w.p_da);
    f.Wh = P8 + po.wh[l] * e;
    f.h0 = h0 ? at<char>(ws, w.h0) + (int64_t)l * B * H * e : nullptr;
    f.c0 = at<float>(ws, w.c0) + (int64_t)l * B * H;
    f.H = at<void>(ws, w.h[l]);
    f.Hs = at<void>(ws, w.hs[l]);
    f.C = at<float>(ws, w.c[l]);
    f.G = at<void>(ws, w.g[l]);
    f.sync = sync_slot(at<void>(ws, w.sync), l);
    f.err = sync_err(at<void>(ws, w.sync));
    f.pre = at<float>(ws, w.pre);
    AM_TRY(forward_recurrence(f, sc, bf, H, s));
  }
  AM_TRY(run_gemm(AM_K_GEMM_FWD,
                  mk_gemm(at<void>(ws, w.h[L - 1]), H, true, P8 + po.wo * e, H, true, logits,
                          m->classes, true, P8 + po.bo * e, (int)sc.N, m->classes, (int)H, bf), s));

  if (hT || cT) {
    for (int l = 0; l < L; ++l) {
      for (int b0 = 0; b0 < B; b0 += 256) {
        am::GatherState g;
        g.Hrows = at<void>(ws, w.h[l]);
        g.h_bf16 = bf;
        g.Crows = at<float>(ws, w.c[l]);
        g.h0 = h0 ? h0 + (int64_t)l * B * H : nullptr;
        g.c0 = c0 ? c0 + (int64_t)l * B * H : nullptr;
        g.hT = hT ? hT + (int64_t)l * B * H : nullptr;
        g.cT = cT ? cT + (int64_t)l * B * H : nullptr;
        g.B = B;
        g.hidden = (int)H;
        const int nb = B - b0 < 256 ? B - b0 : 256;
        for (int i = 0; i < nb; ++i) {
          const int len = sc.lens[b0 + i];
          g.rows[i] = len > 0 ? (int)(sc.offs[len - 1] + b0 + i) : -1;
        }
        Timed tm(AM_K_MISC, s, 0.0, 16.0 * nb * H);
        AM_TRY(hip_check(am::gather_state(g, b0, nb, s), "final state"));
      }
    }
  }
  return AM_OK;
}

am_status lstm_am_backward(const am_model* m, const void* params, const void* x,
                           const int32_t* lengths, int32_t T, int32_t B, const void* dlogits,
                           void* ws, int64_t ws_bytes, float* grads, void* stream) {
  AM_TRY(check_model(m));
  Schedule sc;
  AM_TRY(make_schedule(T, B, lengths, sc));
  if (!params || !ws || !grads) return fail(AM_EINVAL, "NULL params, workspace or grads");
  if (sc.N > 0 && (!x || !dlogits)) return fail(AM_EINVAL, "NULL x or dlogits");
  if (!aligned(params, 16) || !aligned(x, 16) || !aligned(dlogits, 16) || !aligned(grads, 16) ||
      !aligned(ws, 256))
    return fail(AM_EINVAL, "params, x, dlogits, grads must be 16-byte and ws 256-byte aligned");
  const WsLayout w = ws_layout(m, B, sc.N);
  if (ws_bytes < w.total)
    return fail(AM_EWORKSPACE, "backward needs %lld workspace bytes", (long long)w.total);

  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf = m->dtype == AM_BF16;
  const int64_t e = esz_of(m->dtype), H = m->hidden, G = 4 * H, L = m->layers, Cc = m->classes;
  const int N = (int)sc.N;
  const Offsets po = param_layout(m);
  const char* P8 = static_cast<const char*>(params);
  float* skws = at<float>(ws, w.splitk);
  // the backward launches' slots of the sync area (not slot 0's time-out flag)
  AM_TRY(hip_check(am::fill_zero(static_cast<float*>(sync_slot(at<void>(ws, w.sync), (int)L)),
                                 L * SYNC_BYTES / 4, s), "sync clear"));

  // output layer: dWo = dZ^T H_top and dbo = column sums of dZ (one pass),
  // then dH_top = dZ Wo
  AM_TRY(run_gemm(AM_K_GEMM_BWD_WGT,
                  mk_wgrad(dlogits, Cc, at<void>(ws, w.h[L - 1]), H, (int)H, nullptr, 0, 0,
                           grads + po.wo, H, nullptr, 0, grads + po.bo, (int)Cc, N, bf, skws,
                           w.splitk_floats), s));
  void* DH = at<void>(ws, w.dh);
  AM_TRY(run_gemm(AM_K_GEMM_BWD_DATA,
                  mk_gemm(dlogits, Cc, true, P8 + po.wo * e, H, false, DH, H, false, nullptr, N,
                          (int)H, (int)Cc, bf), s));

  char* dA = at<char>(ws, w.p_da);
  auto wht = [&](int l) { return static_cast<void*>(at<char>(ws, w.wht) + (int64_t)l * G * H * e); };
  float* dc = at<float>(ws, w.dc);
  // the XCD-local recurrences read W_h^T: every layer's, transposed up front
  // in one launch (falls back to one transpose per layer below)
  bool wht_ready = false;
  if (sc.N > 0 && persistent_enabled() && xcd_path(false, bf, H, sc)) {
    Timed tm(AM_K_MISC, s, 0.0, 2.0 * L * G * H * e);
    wht_ready = true;
    for (int l0 = 0; l0 < L && wht_ready; l0 += am::TransposeBatch::MAX) {
      am::TransposeBatch tb{};
      const int n = (int)(L - l0 < am::TransposeBatch::MAX ? L - l0 : am::TransposeBatch::MAX);
      for (int i = 0; i < n; ++i) {
        tb.src[i] = P8 + po.wh[l0 + i] * e;
        tb.dst[i] = wht(l0 + i);
      }
      const hipError_t err = am::transpose_bf16_batch(tb, n, (int)G, (int)H, s);
      if (err == hipErrorInvalidValue) wht_ready = false;  // (alignment) per layer instead
      else AM_TRY(hip_check(err, "Wh transposes"));
    }
    if (!wht_ready) tm.cancel();
  }
  for (int l = L - 1; l >= 0; --l) {
    void* WhT = wht(l);
    const int64_t D = l == 0 ? m->input_dim : H;
    const char* Gl = at<char>(ws, w.g[l]);
    const float* Cl = at<float>(ws, w.c[l]);
    bool used = false;
    if (sc.N > 0 && persistent_enabled()) {
      am::PersistBwd pa;
      pa.Wh = P8 + po.wh[l] * e;
      pa.WhT = WhT;
      pa.dHa = DH;
      pa.G = Gl;
      pa.C = Cl;
      pa.c0 = at<float>(ws, w.c0) + (int64_t)l * B * H;
      pa.dA = dA;
      void* slot = sync_slot(at<void>(ws, w.sync), L + l);
      pa.counters = static_cast<unsigned*>(slot);
      pa.err = sync_err(at<void>(ws, w.sync));
      pa.hidden = (int)H;
      const am::PersistSchedule ps = persist_schedule(sc);
      const double flops = 2.0 * (sc.N - sc.counts[0]) * G * H;
      const double bytes = (double)sc.N * (G * e * 2 + H * (e + 8)) + (double)G * H * e;
      if (xcd_path(false, bf, H, sc)) {
        if (!wht_ready) {
          Timed tm(AM_K_MISC, s, 0.0, 2.0 * G * H * e);
          AM_TRY(hip_check(am::transpose(P8 + po.wh[l] * e, WhT, (int)G, (int)H, bf, s), "Wh transpose"));
        }
        Timed tm(AM_K_LSTM_BWD, s, flops, bytes);
        AM_TRY(hip_check(am::lstm_bwd_xcd_launch(pa, ps, xcd_sync(slot, pa.err), s, &used),
                         "lstm backward layer (xcd)"));
        if (!used) tm.cancel();
      }
      if (!used && device_persistent_enabled() && am::lstm_persistent_fits(false, (int)H, B, bf, T)) {
        Timed tm(AM_K_LSTM_BWD, s, flops, bytes);
        AM_TRY(hip_check(am::lstm_bwd_persistent(pa, ps, bf, s, &used), "lstm backward layer"));
        if (!used) tm.cancel();
      }
    }
    if (!used && !bf) {  // (the bf16 per-step path multiplies by Wh itself)
      Timed tm(AM_K_MISC, s, 0.0, 2.0 * G * H * e);
      AM_TRY(hip_check(am::transpose(P8 + po.wh[l] * e, WhT, (int)G, (int)H, bf, s), "Wh transpose"));
    }
    for (int t = T - 1; t >= 0 && !used; --t) {
      const int64_t nb = sc.counts[t];
      if (nb == 0) continue;
      const int64_t nbn = t + 1 < T ? sc.counts[t + 1] : 0;
      const int64_t o = sc.offs[t];
      am::LstmBwdStep a;
      a.dAnext = nbn > 0 ? dA + sc.offs[t + 1] * G * e : nullptr;
      a.nbn = (int)nbn;
      a.WhT = WhT;
      a.dHa = static_cast<char*>(DH) + o * H * e;
      a.G = Gl + o * G * e;
      a.C = Cl + o * H;
      a.Cprev = t == 0 ? at<float>(ws, w.c0) + (int64_t)l * B * H : Cl + sc.offs[t - 1] * H;
      a.dc = dc;
      a.dA = dA + o * G * e;
      a.nb = (int)nb;
      a.hidden = (int)H;
      a.bf16 = bf;
      if (bf) {
        // dA_{t+1} Wh as a batched product (few rows: square tiles), then
        // the cell backward
        // (k split up to STEP_SPLITS ways: the partials fill the fp32 scratch)
        float* dhrec = at<float>(ws, w.pre);
        int splits = 0;
        if (nbn > 0) {
          const am::GemmArgs g = mk_gemm(a.dAnext, G, true, P8 + po.wh[l] * e, H, false, dhrec, H,
                                         true, nullptr, (int)nbn, (int)H, (int)G, true);
          Timed tm(AM_K_LSTM_BWD, s, 2.0 * nbn * H * G, gemm_bytes(nbn, H, G, e, 4));
          AM_TRY(hip_check(am::gemm_bf16_splitk_rows(g, STEP_SPLITS, dhrec, &splits, s), "recurrent product"));
        }
        Timed tm(AM_K_LSTM_BWD, s, 0.0, (double)nb * (H * (4.0 * (splits > 0 ? splits : 1) + e + 16) + G * 2 * e));
        AM_TRY(hip_check(am::lstm_cell_bwd(nbn > 0 ? dhrec : nullptr, splits, a, s), "lstm backward cell"));
        continue;
      }
      const double bytes = (double)(nbn * G + G * H + nb * H + nb * G) * e +
                           nb * H * 12.0 + (double)nb * G * e;
      Timed tm(AM_K_LSTM_BWD, s, 2.0 * nbn * G * H, bytes);
      AM_TRY(hip_check(am::lstm_bwd_step(a, s), "lstm backward step"));
    }
    const void* X = l == 0 ? x : at<void>(ws, w.h[l - 1]);
    // [dWx | dWh] = dA^T [X | Hs] and db = column sums of dA, one pass
    AM_TRY(run_gemm(AM_K_GEMM_BWD_WGT,
                    mk_wgrad(dA, G, X, D, (int)D, at<void>(ws, w.hs[l]), H, (int)H,
                             grads + po.wx[l], D, grads + po.wh[l], H, grads + po.b[l], (int)G, N,
                             bf, skws, w.splitk_floats), s));
    if (l > 0)
      AM_TRY(run_gemm(AM_K_GEMM_BWD_DATA,
                      mk_gemm(dA, G, true, P8 + po.wx[l] * e, D, false, DH, H, false, nullptr, N,
                              (int)H, (int)G, bf), s));
  }
  // a step barrier of this forward + backward pair that timed out leaves the
  // gradient invalid: it is replaced by zeros on the device, so that a caller
  // that encodes and applies it before am_workspace_check adds nothing to
  // its residual or weights
  Timed tm(AM_K_MISC, s, 0.0, 4.0);
  return hip_check(am::zero_if_set(sync_err(at<void>(ws, w.sync)), grads, po.n, s), "time-out guard");
}

// ---------------------------------------------------------------- timing --

am_status am_workspace_check(const void* ws, int64_t ws_bytes, void* stream) {
  if (!ws || !aligned(ws, 256)) return fail(AM_EINVAL, "NULL or unaligned workspace");
  if (ws_bytes < SYNC_BYTES) return fail(AM_EWORKSPACE, "workspace smaller than its sync region");
  hipStream_t s = static_cast<hipStream_t>(stream);
  int flag = 0;
  AM_TRY(hip_check(hipMemcpyAsync(&flag, static_cast<const char*>(ws) + SYNC_STICKY_WORD * 4,
                                  sizeof flag, hipMemcpyDeviceToHost, s), "flag read"));
  AM_TRY(hip_check(hipStreamSynchronize(s), "stream sync"));
  if (flag) return fail(AM_ETIMEOUT, "a step barrier of a persistent recurrence kernel timed out");
  return AM_OK;
}

am_status am_profile_begin(uint32_t class_mask) {
  g_prof.on = true;
  g_prof.mask = class_mask;
  g_prof.next = 0;
  g_prof.recs.clear();
  for (int k = 0; k < AM_K_NCLASSES; ++k) {
    g_prof.seen[k] = 0;
    g_prof.launches[k] = 0;
    g_prof.ms[k] = g_prof.flops[k] = g_prof.bytes[k] = 0.0;
  }
  return AM_OK;
}

am_status am_profile_sample_every(int32_t n) {
  if (n < 1) return fail(AM_EINVAL, "sampling interval must be at least 1");
  g_prof.every = n;
  return AM_OK;
}

am_status am_profile_end(void) {
  g_prof.on = false;
  for (const ProfRec& r : g_prof.recs) {
    AM_TRY(hip_check(hipEventSynchronize(r.b), "event sync"));
    float ms = 0.f;
    AM_TRY(hip_check(hipEventElapsedTime(&ms, r.a, r.b), "event elapsed"));
    g_prof.launches[r.cls] += 1;
    g_prof.ms[r.cls] += ms;
    g_prof.flops[r.cls] += r.flops;
    g_prof.bytes[r.cls] += r.bytes;
  }
  g_prof.recs.clear();
  return AM_OK;
}

am_status am_profile_get(int32_t cls, int64_t* launches, double* ms, double* flops, double* bytes) {
  if (cls < 0 || cls >= AM_K_NCLASSES) return fail(AM_EINVAL, "unknown kernel class");
  if (launches) *launches = g_prof.launches[cls];
  if (ms) *ms = g_prof.ms[cls];
  if (flops) *flops = g_prof.flops[cls];
  if (bytes) *bytes = g_prof.bytes[cls];
  return AM_OK;
}

}  // extern "C"
