// liblede host runtime: context, KV page allocator, orchestration of the
// draft / verify passes, and the C ABI declared in include/lede.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <map>
#include <string>
#include <tuple>
#include <vector>

#include "../../include/lede.h"
#include "ctx_view.h"
#include "kernels.h"

using namespace lede;

namespace {

constexpr int PAGE = 64;
constexpr int MROWS = 16;   // rows of one verify / prefill pass
static_assert(MROWS <= KEY_PITCH && 15 + 2 <= KEY_PITCH, "a key buffer holds every row's key and every draft's");
constexpr int RECORD_INTS = 64;
constexpr int UNIF_FLOATS = 2 * SAMPLE_SLOTS + 1;  // uniforms of a sampled step

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct Layout {
  // element sizes and padded dims
  int dt, es, L, d, nq, nkv, hd, F, V, qd, kvd, Fp, H, A, max_ctx, n_pages, max_pages_seq, max_chunks, k_max;
  // weight arena offsets
  struct LayerOff { size_t attn_norm, wqkv, wo, ffn_norm, wgu, wd; };
  std::vector<LayerOff> lay;
  size_t embed, final_norm, head, qw1, qb1, qw2, qb2, ew1, eb1, ew2, eb2, wbytes;
  int He;  // exit-policy Q-network hidden width (0: none)
  // workspace offsets
  size_t h, xn, ss, q, attn_out, act, part, logits, gstats, dkeys, vkeys, qs, qhid, qv, seq_len, btab, prompt,
      record, rope, unif, dstats, trace, trace_state, trace_bak, pol_out, wsbytes;
  size_t kvbytes, kv_half;
};

const char* check_config(const lede_config* c) {
  if (!c) return "null config";
  if (c->dtype != LEDE_DTYPE_F32 && c->dtype != LEDE_DTYPE_BF16) return "dtype must be f32 or bf16";
  if (c->n_layers < 1 || c->d_model < 32 || c->n_heads < 1 || c->n_kv_heads < 1 || c->vocab < 16)
    return "bad model dims";
  if (c->head_dim != 64 && c->head_dim != 128) return "head_dim must be 64 or 128";
  if (c->n_heads % c->n_kv_heads) return "n_heads must be a multiple of n_kv_heads";
  if (c->d_model % 32 || (c->n_heads * c->head_dim) % 32) return "d_model and n_heads*head_dim must be multiples of 32";
  if (c->d_model > 8192) return "d_model above 8192 is not supported";
  if (c->ffn_dim % 8 || c->ffn_dim < 8) return "ffn_dim must be a multiple of 8";
  if (c->vocab % 16) return "vocab must be a multiple of 16";
  if (c->page_size != PAGE) return "page_size must be 64";
  if (c->max_ctx < 1 || c->n_pages < 1) return "bad KV geometry";
  if (c->k_max < 0 || c->k_max > 15) return "k_max must be in 0..15";
  if (c->qnet_hidden < 0 || c->qnet_hidden % 16) return "qnet_hidden must be a multiple of 16";
  if (c->exit_qnet_hidden < 0 || c->exit_qnet_hidden > 1024) return "exit_qnet_hidden must be in 0..1024";
  if (c->qnet_hidden > 0 || c->exit_qnet_hidden > 0) {
    if (c->n_exits < 1 || c->n_exits > 64 || c->n_lengths < 1 || c->n_lengths > 16) return "bad action grid";
    for (int i = 0; i < c->n_exits; ++i)
      if (c->exits[i] < 1 || c->exits[i] > c->n_layers || (i && c->exits[i] <= c->exits[i - 1]))
        return "exits must be ascending in 1..n_layers";
    for (int i = 0; i < c->n_lengths; ++i)
      if (c->lengths[i] < 1 || c->lengths[i] > 16) return "lengths must be in 1..16";
  }
  return nullptr;
}

Layout make_layout(const lede_config* c) {
  Layout o{};
  o.dt = c->dtype;
  o.es = c->dtype == LEDE_DTYPE_BF16 ? 2 : 4;
  o.L = c->n_layers; o.d = c->d_model; o.nq = c->n_heads; o.nkv = c->n_kv_heads; o.hd = c->head_dim;
  o.F = c->ffn_dim; o.V = c->vocab; o.qd = o.nq * o.hd; o.kvd = o.nkv * o.hd;
  const int tk = tile_k(o.dt);
  o.Fp = (o.F + tk - 1) / tk * tk;
  o.H = c->qnet_hidden; o.A = c->qnet_hidden ? c->n_exits * c->n_lengths : 0;
  o.max_ctx = c->max_ctx; o.n_pages = c->n_pages; o.k_max = c->k_max;
  o.max_pages_seq = (o.max_ctx + PAGE - 1) / PAGE;
  o.max_chunks = o.max_pages_seq;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t r = off; off += align256(bytes); return r; };
  o.lay.resize(o.L);
  for (int l = 0; l < o.L; ++l) {
    auto& x = o.lay[l];
    x.attn_norm = take((size_t)o.d * o.es);
    x.wqkv = take(tiled_bytes(o.dt, o.qd + 2 * o.kvd, o.d));
    x.wo = take(tiled_bytes(o.dt, o.d, o.qd));
    x.ffn_norm = take((size_t)o.d * o.es);
    x.wgu = take(tiled_bytes(o.dt, 2 * o.F, o.d));
    x.wd = take(tiled_bytes(o.dt, o.d, o.F));
  }
  o.embed = take((size_t)o.V * o.d * o.es);
  o.final_norm = take((size_t)o.d * o.es);
  o.head = take(tiled_bytes(o.dt, o.V, o.d));
  o.qw1 = take(o.H ? tiled_bytes(0, o.H, o.d) : 0);
  o.qb1 = take((size_t)o.H * 4);
  o.qw2 = take((size_t)o.A * o.H * 4);
  o.qb2 = take((size_t)o.A * 4);
  o.He = c->exit_qnet_hidden;
  o.ew1 = take((size_t)o.He * 3 * 4);
  o.eb1 = take((size_t)o.He * 4);
  o.ew2 = take((size_t)o.He * 2 * 4);
  o.eb2 = take(o.He ? 2 * 4 : 0);
  o.wbytes = off;

  off = 0;
  o.h = take((size_t)MROWS * o.d * 4);
  o.xn = take((size_t)MROWS * o.d * o.es);
  o.ss = take((size_t)(o.d / 16) * 16 * 4);   // split-norm partial sums [d/16][16]
  o.q = take((size_t)MROWS * o.qd * 4);
  o.attn_out = take((size_t)MROWS * o.qd * o.es);
  o.act = take((size_t)MROWS * o.Fp * o.es);
  o.part = take((size_t)MROWS * o.nq * o.max_chunks * (o.hd + 2) * 4);
  o.logits = take((size_t)2 * MROWS * o.V * 4);
  o.gstats = take((size_t)2 * MROWS * (o.V / 16) * 8);  // group statistics of sampled logits rows
  o.dkeys = take(KEY_WORDS * 8);
  o.vkeys = take(KEY_WORDS * 8);
  o.qs = take((size_t)o.d * 4);
  o.qhid = take((size_t)(o.H ? o.H : 1) * 4);
  o.qv = take((size_t)(o.A ? o.A : 1) * 4);
  o.seq_len = take(4);
  o.btab = take((size_t)o.max_pages_seq * 4);
  o.prompt = take((size_t)o.max_ctx * 4);
  o.record = take(RECORD_INTS * 4);
  o.rope = take((size_t)o.max_ctx * (o.hd / 2) * 8);
  o.unif = take(UNIF_FLOATS * 4);
  o.dstats = take(2 * SAMPLE_SLOTS * 4);
  o.trace = take(POLICY_TRACE * 4);
  o.trace_state = take(4 * 4);
  o.trace_bak = take((POLICY_TRACE + 2) * 4);
  o.pol_out = take((size_t)(c->n_exits + POLICY_MAX_DRAFT) * POLICY_LOG * 4);
  o.wsbytes = off;

  o.kv_half = align256((size_t)o.L * o.n_pages * o.nkv * PAGE * o.hd * o.es);
  o.kvbytes = 2 * o.kv_half;
  return o;
}

}  // namespace

struct lede_ctx {
  lede_config cfg;
  Layout lo;
  uint8_t *w, *kv, *ws;
  int dev;
  // host mirror of the decoding state
  int32_t seq_len = 0;
  int32_t pending = -1;
  int drafted_k = -1;  // -1: no draft outstanding
  int drafted_l = 0;
  std::deque<int32_t> free_list;
  std::vector<int32_t> table;
  int32_t* table_h = nullptr;   // pinned mirror uploaded to the device table
  int32_t* record_h = nullptr;  // pinned read-back of the step record
  float* unif_h = nullptr;      // pinned staging of a sampled step's uniforms
  float* trace_h = nullptr;     // pinned staging of the confidence trace and policy decisions
  std::vector<float> policy_log;  // decisions of the last exit-policy step, POLICY_LOG floats each
  // the last step was an exit-policy step whose decision log (device) is intact
  int policy_valid = 0, policy_l = 0, policy_a = 0;
  uint64_t* keys_h = nullptr;   // pinned read-back of argmax keys
  int use_graphs = 0, debug = 0;
  int verify_reuse = 0;  // verify from the exit layer on the draft passes' hidden states and KV
  int split_row = -1;    // the one-row residual row whose final-norm split the last pass prepared
  std::vector<int32_t> table_dev;  // the block table as the device holds it (uploads are skipped when equal)
  // pipelined steps (lede_step_submit / lede_step_collect), oldest first
  struct InFlight {
    int l, k_req, k_eff, slot;
    bool ran_q;
  };
  std::deque<InFlight> inflight;
  int32_t* rec_slots_h = nullptr;          // pinned [LEDE_MAX_IN_FLIGHT][RECORD_INTS]
  hipEvent_t rec_ev[LEDE_MAX_IN_FLIGHT] = {};
  hipEvent_t wait_ev = nullptr;            // the read-backs of a synchronous step wait on it
  // A forced step's logged Q-network runs on a second stream (default
  // priority) after its input row is normalised, beside the rest of the
  // draft pass; the record's read-back waits for it.
  hipStream_t side = nullptr;
  hipEvent_t side_in = nullptr, side_out = nullptr;
  int qnet_defer = 0, side_pending = 0;
  int next_slot = 0;
  int seq_ub = 0;                          // committed length after every step in flight, at most
  void* pipe_stream = nullptr;
  // captured draft + verify launches of a forced step, keyed by (l, k_eff, Q-net layer)
  std::map<std::tuple<int, int, int>, hipGraphExec_t> graphs;
  int last_rows = 0, last_draft_rows = 0;
  std::string err;
  // failure handling: device work issued by the current call (a failed call
  // then restores the device's copies of the state), whether it pushed to the
  // confidence trace, and the host-injected failure countdown
  // (lede_debug_inject_failure; -1: none)
  bool launched = false, trace_pushed = false;
  int fail_after = -1;

  // timing (lede_prof_*): event pairs folded into per-class totals;
  // level 1 brackets the draft and verify phases, level 2 also every launch
  struct ProfRec { int cls; hipEvent_t a, b; double bytes; };
  int prof = 0;
  std::vector<hipEvent_t> evpool;
  size_t ev_next = 0;
  std::vector<ProfRec> recs;
  double p_ms[LEDE_K_NCLASS] = {0}, p_bytes[LEDE_K_NCLASS] = {0};
  int64_t p_n[LEDE_K_NCLASS] = {0};

  // device pointers
  template <typename T> T* W(size_t off) const { return (T*)(w + off); }
  template <typename T> T* S(size_t off) const { return (T*)(ws + off); }
};

namespace {

int fail(lede_ctx* c, int code, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return code;
}

// Every device operation of a call (kernel or graph launch, copy) passes
// here first: it counts down a host-injected failure, and notes that the call
// has touched the device.
int pre_launch(lede_ctx* c) {
  if (c->fail_after >= 0 && c->fail_after-- == 0)
    return fail(c, LEDE_E_HIP, "injected failure (lede_debug_inject_failure)");
  c->launched = true;
  return LEDE_OK;
}
#define PRE()                      \
  do {                             \
    int rc_p_ = pre_launch(c);     \
    if (rc_p_) return rc_p_;       \
  } while (0)

#define HIP_CHECK(ctx, expr)                                                               \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(ctx, LEDE_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

hipStream_t S_(void* s) { return (hipStream_t)s; }

// ---- timing ------------------------------------------------------------------------

hipEvent_t next_event(lede_ctx* c) {
  if (c->ev_next == c->evpool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->evpool.push_back(e);
  }
  return c->evpool[c->ev_next++];
}

int prof_mark(lede_ctx* c, hipStream_t s, hipEvent_t* e, int level = 2) {
  *e = nullptr;
  if (c->prof < level) return LEDE_OK;
  *e = next_event(c);
  if (!*e) return fail(c, LEDE_E_HIP, "hipEventCreate failed");
  HIP_CHECK(c, hipEventRecord(*e, s));
  return LEDE_OK;
}

int prof_close(lede_ctx* c, hipStream_t s, int cls, double bytes, hipEvent_t e0) {
  if (!c->prof || !e0) return LEDE_OK;
  hipEvent_t e1 = nullptr;
  int rc = prof_mark(c, s, &e1, 1);
  if (rc) return rc;
  c->recs.push_back({cls, e0, e1, bytes});
  return LEDE_OK;
}

// Convert finished event pairs into per-class totals (synchronises).
int prof_fold(lede_ctx* c) {
  if (c->recs.empty()) { c->ev_next = 0; return LEDE_OK; }
  HIP_CHECK(c, hipEventSynchronize(c->recs.back().b));
  for (const auto& r : c->recs) {
    float ms = 0.f;
    HIP_CHECK(c, hipEventElapsedTime(&ms, r.a, r.b));
    c->p_ms[r.cls] += ms;
    c->p_bytes[r.cls] += r.bytes;
    c->p_n[r.cls] += 1;
  }
  c->recs.clear();
  c->ev_next = 0;
  return LEDE_OK;
}

// A linear launch: when timing, the dispatch records its own start / end
// events (kernel execution only).
int launch_linear_timed(lede_ctx* c, int cls, double bytes, int dt, bool mfma, const LinearArgs& a, int grid,
                        hipStream_t s) {
  PRE();
  if (c->prof < 2) {
    HIP_CHECK(c, launch_linear(dt, mfma, a, grid, s));
    return LEDE_OK;
  }
  hipEvent_t e0 = next_event(c), e1 = next_event(c);
  if (!e0 || !e1) return fail(c, LEDE_E_HIP, "hipEventCreate failed");
  HIP_CHECK(c, launch_linear(dt, mfma, a, grid, s, e0, e1));
  c->recs.push_back({cls, e0, e1, bytes});
  return LEDE_OK;
}

#define LAUNCH_LINEAR(vec, a, dt)                                                                  \
  do {                                                                                             \
    const int grid_ = linear_grid((a).n_groups, 16.0 * (a).K * ((dt) == 1 ? 2 : 4));               \
    int rc_ = launch_linear_timed(c, linear_class(dt, vec, (a).K, (a).M), linear_bytes(a, dt), dt, \
                                  !(vec), a, grid_, s);                                            \
    if (rc_) return rc_;                                                                           \
  } while (0)

// Timing class of a linear launch: one per kernel symbol.
int linear_class(int dt, bool vec, int K, int M) {
  switch (linear_x_source(dt, !vec, K, M)) {
    case XS_LDS: return LEDE_K_LINEAR_VEC;
    case XS_GLOBAL: return LEDE_K_LINEAR_VEC_GX;
    case XS_MFMA_LDS: return LEDE_K_LINEAR_MFMA_LX;
    default: return LEDE_K_LINEAR_MFMA;
  }
}

#define LAUNCH(cls, bytes, expr)                         \
  do {                                                   \
    hipEvent_t e0_ = nullptr;                            \
    PRE();                                               \
    int rc_ = prof_mark(c, s, &e0_);                     \
    if (rc_) return rc_;                                 \
    HIP_CHECK(c, (expr));                                \
    rc_ = prof_close(c, s, (cls), (bytes), e0_);         \
    if (rc_) return rc_;                                 \
  } while (0)

// Algorithmic bytes of one linear launch: weights once, input rows, outputs.
double linear_bytes(const LinearArgs& a, int dt) {
  const double es = dt == 1 ? 2.0 : 4.0;
  const double N = (double)a.n_groups * 16, K = a.K, M = a.M;
  double x = (a.x_mode == X_NORM || a.x_mode == X_EMBED_NORM || a.x_mode == X_F32) ? M * K * 4 : M * K * es;
  double y = 0;
  switch (a.epi) {
    case EPI_RESID: y = 2 * M * N * 4; break;
    case EPI_QKV: y = M * N * 4; break;
    case EPI_SWIGLU: y = M * N / 2 * es; break;
    case EPI_ARGMAX: y = M * 8 + (a.logits ? M * N * 4 : 0) + (a.gstats ? M * N / 16 * 8 : 0); break;
    default: y = M * N * 4;
  }
  if (a.ss_out) y += M * N * es + N * es + N / 16 * M * 4;  // h * gain, the gain, the partial sums
  if (a.ss_in) x += (double)a.ss_groups * M * 4;
  return N * K * es + x + y;
}

// ---- page allocator (host) ------------------------------------------------------

int ensure_pages(lede_ctx* c, int n_positions) {
  if (n_positions > c->lo.max_ctx) return fail(c, LEDE_E_CTX_OVERFLOW, "position %d exceeds max_ctx %d", n_positions, c->lo.max_ctx);
  const int need = (n_positions + PAGE - 1) / PAGE;
  if (need - (int)c->table.size() > (int)c->free_list.size())
    return fail(c, LEDE_E_KV_FULL, "KV pool exhausted (%d pages needed, %zu free)", need, c->free_list.size());
  while ((int)c->table.size() < need) {
    c->table.push_back(c->free_list.front());
    c->free_list.pop_front();
  }
  return LEDE_OK;
}

// Ints between the pinned table staging buffers (the synchronous one, then
// one per pipelined slot).
size_t table_pitch(const Layout& o) { return ((size_t)o.max_pages_seq + 63) / 64 * 64; }

void truncate_pages(lede_ctx* c, int new_len) {
  const int keep = (new_len + PAGE - 1) / PAGE;
  for (int j = (int)c->table.size() - 1; j >= keep; --j) c->free_list.push_front(c->table[j]);
  if ((int)c->table.size() > keep) c->table.resize(keep);
}

// Upload the host table if the device's differs (the acceptance kernel
// truncates the device table itself; commit_host mirrors that, and a
// pipelined step marks the entries it may clear as unknown).  `stage` is the
// pinned buffer the copy reads: a pipelined step passes its slot's, which no
// later submit overwrites before the copy has run.
int upload_table(lede_ctx* c, hipStream_t s, int32_t* stage = nullptr) {
  const int n = c->lo.max_pages_seq;
  int32_t* t = stage ? stage : c->table_h;
  bool same = (int)c->table_dev.size() == n;
  for (int j = 0; j < n; ++j) {
    t[j] = j < (int)c->table.size() ? c->table[j] : -1;
    same = same && c->table_dev[j] == t[j];
  }
  if (same) return LEDE_OK;
  PRE();
  HIP_CHECK(c, hipMemcpyAsync(c->S<int32_t>(c->lo.btab), t, n * 4, hipMemcpyHostToDevice, s));
  c->table_dev.assign(t, t + n);
  return LEDE_OK;
}

// Order the stream after a deferred Q-network (its action and maximum are in
// the record).
int join_side(lede_ctx* c, hipStream_t s) {
  if (c->side_pending) {
    HIP_CHECK(c, hipStreamWaitEvent(s, c->side_out, 0));
    c->side_pending = 0;
  }
  return LEDE_OK;
}

// Wait for the work queued on the stream so far, on an event recorded after
// it: in alternating runs of the 7B decode step this returned as soon as or
// sooner than a stream synchronize (0 to 25 us a step).
int wait_stream(lede_ctx* c, hipStream_t s) {
  HIP_CHECK(c, hipEventRecord(c->wait_ev, s));
  HIP_CHECK(c, hipEventSynchronize(c->wait_ev));
  return LEDE_OK;
}

int upload_seq_len(lede_ctx* c, int v, hipStream_t s) {
  PRE();
  c->record_h[RECORD_INTS - 1] = v;
  HIP_CHECK(c, hipMemcpyAsync(c->S<int32_t>(c->lo.seq_len), &c->record_h[RECORD_INTS - 1], 4, hipMemcpyHostToDevice, s));
  HIP_CHECK(c, hipStreamSynchronize(s));
  return LEDE_OK;
}

// ---- pass orchestration -----------------------------------------------------------

// Blocks of a linear launch (block b takes groups b, b + grid, ...), from a
// time model fitted to cold-weight measurements: the busiest CU streams its
// groups at about 19 GB/s with one resident block and 25 GB/s with two or
// more (3 blocks of 512 threads fit a CU), and each round of resident blocks
// costs about 1.6 us of ramp.  Ties go to fewer blocks.  It reproduces the
// measured best choices for the 7B shapes: gate-up 1376 groups in 459
// blocks (28.5 against 30.5 us in 1376), head 2000 groups in 500 blocks
// (41.0 against 42.1 us in 1000), QKV (768) and the 256-group projections
// at one group per block.
int linear_grid(int n_groups, double group_bytes) {
  constexpr int CUS = 256, RESIDENT = 3, GMAX = 16;
  constexpr double RATE1 = 19.0e3, RATE2 = 25.0e3;  // bytes per us per CU
  constexpr double RAMP_US = 1.6;
  int best = 1;
  double best_t = 0.0;
  for (int G = 1; G <= GMAX && G <= n_groups; ++G) {
    const int blocks = (n_groups + G - 1) / G;
    const int per_cu = (blocks + CUS - 1) / CUS;
    const int rounds = (per_cu + RESIDENT - 1) / RESIDENT;
    const double t = (double)per_cu * G * group_bytes / (per_cu >= 2 ? RATE2 : RATE1) + rounds * RAMP_US;
    if (G == 1 || t <= best_t) {
      best = G;
      best_t = t;
    }
  }
  return (n_groups + best - 1) / best;
}

// One-row passes normalise their input row in every block of the linear
// Every RMSNorm after the first of a pass is split over the kernels around
// it: the residual producer before it stores h * gain and per-group sums of
// squares, the consumer after it reads h * gain as its input and scales its
// output rows by the inverse RMS.  The first norm of a pass, whose residual
// rows come from elsewhere (the embedding, an earlier segment of the exit
// policy's pass, or the draft passes under verify reuse), normalises in the
// one-row kernel's prologue or runs the norm kernel for several rows.  A
// consumer that normalised in its own prologue would wait for the fp32
// residual row and the gain before its first tile, behind the weight stream
// of every other block; one that normalised several rows per block would
// re-read k+1 residual rows in every block.

// Arm a residual producer (EPI_RESID) to prepare the split norm with gain.
void split_norm_produce(const lede_ctx* c, LinearArgs& a, const void* gain) {
  a.ss_out = c->S<float>(c->lo.ss);
  a.xg = c->S<void>(c->lo.xn); a.ldxg = c->lo.d;
  a.xg_gain = gain;
}
// Feed a matrix-core consumer of width d from the split norm.
void split_norm_consume(const lede_ctx* c, LinearArgs& a) {
  a.x_mode = X_PLAIN; a.x = c->S<void>(c->lo.xn); a.ldx = c->lo.d;
  a.ss_in = c->S<float>(c->lo.ss); a.ss_groups = c->lo.d / 16;
}

LinearArgs base_linear(const lede_ctx* c) {
  LinearArgs a{};
  a.M = 1;
  a.eps = c->cfg.rms_eps;
  a.h = c->S<float>(c->lo.h);
  a.ldh = c->lo.d;
  return a;
}

// Run rows [0, M) at positions seq_len + pos_off + m through layers
// [l_begin, l_end).  Vector kernels for one row (draft path), matrix-core
// kernels otherwise.  qnet_after: run the Q-network after this many layers
// (0 = never).
// Layers [l_begin, l_end) for M rows.  One-row (vec) passes keep their
// residual in row vec_row of the h buffer (a draft pass i uses row i - 1, so
// that the hidden states of a step's draft inputs stay available).
int run_layers(lede_ctx* c, int M, bool vec, TokenSrc tok, int pos_off, int l_begin, int l_end, int qnet_after,
               uint64_t* zero_slot, hipStream_t s, int vec_row = 0) {
  const Layout& o = c->lo;
  const int dt = o.dt;
  c->split_row = -1;
  float* hrow = c->S<float>(o.h) + (vec ? (size_t)vec_row * o.d : 0);
  for (int j = l_begin; j < l_end; ++j) {
    const auto& lw = o.lay[j];
    const bool first = j == 0;
    // attention block: [norm] + QKV (rotary, KV append)
    LinearArgs qa = base_linear(c);
    qa.M = M;
    qa.h = hrow;
    qa.w = c->W<uint8_t>(lw.wqkv);
    qa.n_groups = (o.qd + 2 * o.kvd) / 16;
    qa.KT = k_tiles(dt, o.d);
    qa.K = o.d;
    qa.epi = EPI_QKV;
    qa.q = c->S<float>(o.q); qa.ldq = o.qd;
    qa.kcache = c->kv; qa.vcache = c->kv + o.kv_half;
    qa.layer = j; qa.n_pages = o.n_pages; qa.nq = o.nq; qa.nkv = o.nkv; qa.hd = o.hd;
    qa.block_table = c->S<int32_t>(o.btab); qa.seq_len = c->S<int32_t>(o.seq_len); qa.pos_off = pos_off;
    qa.rope = c->S<float2>(o.rope);
    if (j > l_begin) {
      split_norm_consume(c, qa);  // prepared by the previous layer's down projection
    } else if (vec) {
      qa.x_mode = first ? X_EMBED_NORM : X_NORM;
      qa.gain = c->W<void>(lw.attn_norm);
      qa.embed = c->W<void>(o.embed);
      qa.tok = tok;
      qa.vocab = o.V;
      // the pass's argmax slots are cleared by its first kernel
      if (zero_slot) { qa.zero_keys = zero_slot; qa.n_zero_keys = 1; }
    } else {
      NormArgs na{};
      na.M = M; na.d = o.d; na.ldh = o.d; na.ldx = o.d;
      na.h = c->S<float>(o.h); na.gain = c->W<void>(lw.attn_norm); na.eps = c->cfg.rms_eps;
      na.embed = first; na.embed_w = c->W<void>(o.embed); na.tok = tok; na.vocab = o.V;
      na.x = c->S<void>(o.xn);
      if (j == l_begin && zero_slot) { na.zero_keys = zero_slot; na.n_zero_keys = M; }
      LAUNCH(LEDE_K_NORM, (double)M * o.d * (4 + o.es), launch_norm(dt, na, s));
      qa.x_mode = X_PLAIN; qa.x = c->S<void>(o.xn); qa.ldx = o.d;
    }
    LAUNCH_LINEAR(vec, qa, dt);

    AttnArgs at{};
    at.q = c->S<float>(o.q); at.ldq = o.qd;
    at.kcache = c->kv; at.vcache = c->kv + o.kv_half;
    at.layer = j; at.n_pages = o.n_pages; at.nq = o.nq; at.nkv = o.nkv; at.hd = o.hd; at.M = M;
    at.block_table = c->S<int32_t>(o.btab); at.seq_len = c->S<int32_t>(o.seq_len); at.pos_off = pos_off;
    const int G = o.nq / o.nkv;
    at.rows_per_block = std::min(16, M * G);
    const int n_rs = (M * G + at.rows_per_block - 1) / at.rows_per_block;
    // about 2048 blocks, one page each where the context allows: at 4096
    // positions (13B shape, 65 pages per head) 16.05 against 16.32 ms per
    // step with 512 blocks of five pages; shorter contexts have a page per
    // block either way
    at.n_split = std::max(1, std::min(o.max_chunks, (2048 + o.nkv * n_rs - 1) / (o.nkv * n_rs)));
    at.max_chunks = o.max_chunks;
    at.part = c->S<float>(o.part);
    at.out = c->S<void>(o.attn_out); at.ldo = o.qd;
    // bf16 partials on the matrix cores for every multi-row pass (verify,
    // autoregressive, prefill: one kernel whatever the row count, so a row's
    // bits do not depend on it) and for one-row passes with grouped heads
    at.mfma = dt == 1 && (!vec || G > 1);
    const double n_pos = (double)c->seq_len + pos_off + M;
    LAUNCH(LEDE_K_ATTENTION, n_pos * o.kvd * 2.0 * o.es + 2.0 * M * o.qd * 4,
           launch_attention(dt, at, s));

    LinearArgs oa = base_linear(c);
    oa.M = M;
    oa.h = hrow;
    oa.w = c->W<uint8_t>(lw.wo);
    oa.n_groups = o.d / 16; oa.KT = k_tiles(dt, o.qd); oa.K = o.qd;
    oa.x_mode = X_PLAIN; oa.x = c->S<void>(o.attn_out); oa.ldx = o.qd;
    oa.epi = EPI_RESID;
    split_norm_produce(c, oa, c->W<void>(lw.ffn_norm));
    LAUNCH_LINEAR(vec, oa, dt);

    // feed-forward block
    LinearArgs ga = base_linear(c);
    ga.M = M;
    ga.h = hrow;
    ga.w = c->W<uint8_t>(lw.wgu);
    ga.n_groups = 2 * o.F / 16; ga.KT = k_tiles(dt, o.d); ga.K = o.d;
    ga.epi = EPI_SWIGLU; ga.act = c->S<void>(o.act); ga.ld_act = o.Fp;
    split_norm_consume(c, ga);  // prepared by the output projection
    LAUNCH_LINEAR(vec, ga, dt);

    LinearArgs da = base_linear(c);
    da.M = M;
    da.h = hrow;
    da.w = c->W<uint8_t>(lw.wd);
    da.n_groups = o.d / 16; da.KT = k_tiles(dt, o.F); da.K = o.F;
    da.x_mode = X_PLAIN; da.x = c->S<void>(o.act); da.ldx = o.Fp;
    da.epi = EPI_RESID;
    // the next norm: the next layer's attention norm, or the final norm at
    // the end of a pass that a head follows (one-row passes end at an exit)
    if (j + 1 < l_end) split_norm_produce(c, da, c->W<void>(o.lay[j + 1].attn_norm));
    else if (vec || l_end == o.L) split_norm_produce(c, da, c->W<void>(o.final_norm));
    LAUNCH_LINEAR(vec, da, dt);

    if (qnet_after == j + 1 && o.H > 0) {
      NormArgs na{};
      na.M = 1; na.d = o.d; na.ldh = o.d; na.ldx = o.d;
      na.h = hrow; na.gain = c->W<void>(o.final_norm); na.eps = c->cfg.rms_eps;
      na.x = c->S<void>(o.qs); na.f32_out = 1;
      LAUNCH(LEDE_K_QNET, (double)o.d * 8, launch_norm(dt, na, s));
      // the hidden and output layers read only the normalised row: on the
      // second stream when the step's caller does not wait for the action
      const bool defer = c->qnet_defer && c->side && !c->prof;
      hipStream_t qstream = s;
      if (defer) {
        HIP_CHECK(c, hipEventRecord(c->side_in, s));
        HIP_CHECK(c, hipStreamWaitEvent(c->side, c->side_in, 0));
        qstream = c->side;
      }
      LinearArgs la = base_linear(c);
      la.w = c->W<uint8_t>(o.qw1);
      la.n_groups = o.H / 16; la.KT = k_tiles(0, o.d); la.K = o.d;
      la.x_mode = X_F32; la.x = c->S<void>(o.qs);
      la.epi = EPI_BIAS_RELU; la.out = c->S<float>(o.qhid); la.bias = c->W<float>(o.qb1);
      QnetOutArgs qo{};
      qo.hid = c->S<float>(o.qhid); qo.H = o.H;
      qo.w2 = c->W<float>(o.qw2); qo.b2 = c->W<float>(o.qb2); qo.A = o.A;
      qo.qv = c->S<float>(o.qv); qo.action = c->S<int32_t>(o.record) + 48;
      if (defer) {
        PRE();
        HIP_CHECK(c, launch_linear(0, false, la, la.n_groups, qstream));
        PRE();
        HIP_CHECK(c, launch_qnet_out(qo, qstream));
        HIP_CHECK(c, hipEventRecord(c->side_out, qstream));
        c->side_pending = 1;
      } else {
        LAUNCH(LEDE_K_QNET, linear_bytes(la, 0), launch_linear(0, false, la, la.n_groups, s));
        LAUNCH(LEDE_K_QNET, (double)o.A * (o.H + 2) * 4, launch_qnet_out(qo, s));
      }
    }
  }
  // a one-row pass's last down projection prepared the final norm's split
  // for its row (a multi-row pass's head reads it through its `split` flag)
  if (vec && l_end > l_begin) c->split_row = vec_row;
  return LEDE_OK;
}

// Shared final RMSNorm + LM head + argmax for rows [0, M) into keys[0..M).
// split: a multi-row pass through the last layer prepared the final norm
// (one-row heads use the split when the last one-row pass ended on their row).
// gstats (with logits): also the rows' 16-token group statistics at inv_t.
int run_head(lede_ctx* c, int M, bool vec, uint64_t* keys, float* logits, hipStream_t s, int vec_row = 0,
             bool split = false, float2* gstats = nullptr, float inv_t = 0.f) {
  if (vec) split = c->split_row == vec_row;
  else c->split_row = -1;
  const Layout& o = c->lo;
  LinearArgs ha = base_linear(c);
  ha.M = M;
  if (vec) ha.h += (size_t)vec_row * o.d;
  ha.w = c->W<uint8_t>(o.head);
  ha.n_groups = o.V / 16; ha.KT = k_tiles(o.dt, o.d); ha.K = o.d;
  ha.epi = EPI_ARGMAX; ha.keys = keys; ha.vocab = o.V;
  ha.logits = logits; ha.ld_logits = o.V;
  if (logits && gstats) { ha.gstats = gstats; ha.ld_gstats = o.V / 16; ha.inv_t = inv_t; }
  if (split) {
    split_norm_consume(c, ha);
  } else if (vec) {
    ha.x_mode = X_NORM; ha.gain = c->W<void>(o.final_norm);
  } else {
    NormArgs na{};
    na.M = M; na.d = o.d; na.ldh = o.d; na.ldx = o.d;
    na.h = c->S<float>(o.h); na.gain = c->W<void>(o.final_norm); na.eps = c->cfg.rms_eps;
    na.x = c->S<void>(o.xn);
    LAUNCH(LEDE_K_NORM, (double)M * o.d * (4 + o.es), launch_norm(o.dt, na, s));
    ha.x_mode = X_PLAIN; ha.x = c->S<void>(o.xn); ha.ldx = o.d;
  }
  LAUNCH_LINEAR(vec, ha, o.dt);
  return LEDE_OK;
}

// Logits rows in the workspace: verify / prefill rows first, draft rows after
// them.  Greedy steps write them only in debug mode; sampled steps always.
float* draft_logits(lede_ctx* c, int i, bool always = false) {
  return (c->debug || always) ? c->S<float>(c->lo.logits) + (size_t)(MROWS + i) * c->lo.V : nullptr;
}
float* verify_logits(lede_ctx* c, bool always = false) {
  return (c->debug || always) ? c->S<float>(c->lo.logits) : nullptr;
}
// Group statistics of logits row r (same row order as the logits).
float2* logits_gstats(lede_ctx* c, int r) { return c->S<float2>(c->lo.gstats) + (size_t)r * (c->lo.V / 16); }

// Draft passes i = i0..k (1-based): token i-1 -> layers [0, l) -> head -> key i.
// qnet_after applies to pass 1 only.  inv_t > 0: draft i is drawn from
// softmax(z / T) with the step's uniform i-1 instead of taken as the argmax.
int launch_drafts(lede_ctx* c, int l, int i0, int k, int qnet_after, int pass1_begin, hipStream_t s,
                  float inv_t = 0.f) {
  uint64_t* dk = c->S<uint64_t>(c->lo.dkeys);
  const bool sampled = inv_t > 0.f;
  for (int i = i0; i <= k; ++i) {
    TokenSrc tok{nullptr, dk + (i - 1)};
    const int begin = i == 1 ? pass1_begin : 0;
    int rc = run_layers(c, 1, true, tok, i - 1, begin, l, i == 1 ? qnet_after : 0, dk + i, s, i - 1);
    if (rc) return rc;
    rc = run_head(c, 1, true, dk + i, draft_logits(c, i - 1, sampled), s, i - 1, false,
                  sampled ? logits_gstats(c, MROWS + i - 1) : nullptr, inv_t);
    if (rc) return rc;
    if (sampled) {
      SampleArgs sa{};
      sa.logits = draft_logits(c, i - 1, true); sa.vocab = c->lo.V; sa.inv_t = inv_t;
      sa.u = c->S<float>(c->lo.unif); sa.u_index = i - 1;
      sa.key_out = dk + i; sa.stats_out = c->S<float>(c->lo.dstats) + 2 * (i - 1);
      sa.gstats = logits_gstats(c, MROWS + i - 1); sa.n_groups = c->lo.V / 16;
      LAUNCH(LEDE_K_ACCEPT, (double)c->lo.V / 16 * 8 + 64, launch_sample(sa, s));
    }
  }
  c->last_draft_rows = k;
  return LEDE_OK;
}

// Confidence trace of the exit policy: push -log max p of `rows` logits rows
// (or of record[0] + 1 rows when record is set).
int push_trace(lede_ctx* c, const float* logits, int rows, const int32_t* record, hipStream_t s) {
  TracePushArgs ta{};
  ta.logits = logits; ta.vocab = c->lo.V; ta.ld = c->lo.V;
  ta.record = record; ta.n_rows = rows;
  ta.trace = c->S<float>(c->lo.trace); ta.trace_state = c->S<int32_t>(c->lo.trace_state);
  ta.backup = c->S<float>(c->lo.trace_bak);
  LAUNCH(LEDE_K_ACCEPT, (double)(rows ? rows : 2) * c->lo.V * 4, launch_trace_push(ta, s));
  c->trace_pushed = true;
  return LEDE_OK;
}

// The pass of draft input k (the last draft) through layers [0, l) without a
// head: with it, rows 0..k of the h buffer hold every verify row's hidden
// state at layer l and the KV of positions c..c+k is written below l.
int extend_drafts(lede_ctx* c, int l, int k, hipStream_t s) {
  uint64_t* dk = c->S<uint64_t>(c->lo.dkeys);
  return run_layers(c, 1, true, TokenSrc{nullptr, dk + k}, k, 0, l, 0, nullptr, s, k);
}

// The verify pass of rows [pending, d_1..d_k]: all layers from the embedding
// (from_layer = 0), or layers [from_layer, L) on the hidden states the draft
// passes left in rows 0..k (verify reuse), then the head and acceptance.
int launch_verify(lede_ctx* c, int k, hipStream_t s, float inv_t = 0.f, int from_layer = 0) {
  uint64_t* dk = c->S<uint64_t>(c->lo.dkeys);
  uint64_t* vk = c->S<uint64_t>(c->lo.vkeys);
  const bool sampled = inv_t > 0.f;
  const bool trace = c->lo.He > 0;
  TokenSrc tok{nullptr, dk};
  int rc;
  if (from_layer >= c->lo.L) {
    // no layer left: the head's argmax slots are cleared here
    PRE();
    HIP_CHECK(c, launch_fill_u64(vk, 0, KEY_WORDS, s));
  } else if ((rc = run_layers(c, k + 1, false, tok, 0, from_layer, c->lo.L, 0, vk, s))) {
    return rc;
  }
  rc = run_head(c, k + 1, false, vk, verify_logits(c, sampled || trace), s, 0, from_layer < c->lo.L,
                sampled ? logits_gstats(c, 0) : nullptr, inv_t);
  if (rc) return rc;
  AcceptArgs aa{};
  aa.dkeys = dk; aa.vkeys = vk; aa.k = k;
  aa.seq_len = c->S<int32_t>(c->lo.seq_len);
  aa.block_table = c->S<int32_t>(c->lo.btab);
  aa.pending_out = dk;
  aa.record = c->S<int32_t>(c->lo.record);
  if (sampled) {
    SampledAcceptArgs sa{};
    sa.acc = aa;
    sa.dlogits = draft_logits(c, 0, true); sa.dstats = c->S<float>(c->lo.dstats);
    sa.vlogits = verify_logits(c, true);
    sa.vocab = c->lo.V; sa.inv_t = inv_t;
    sa.u = c->S<float>(c->lo.unif);
    sa.vgstats = logits_gstats(c, 0); sa.n_groups = c->lo.V / 16;
    LAUNCH(LEDE_K_ACCEPT, (double)(2 * k + 1) * c->lo.V * 4, launch_accept_sampled(sa, s));
  } else {
    LAUNCH(LEDE_K_ACCEPT, 256.0, launch_accept(aa, s));
  }
  if (trace && (rc = push_trace(c, verify_logits(c, true), 0, aa.record, s))) return rc;
  c->last_rows = k + 1;
  return LEDE_OK;
}

// Draft passes (k > 0) and the verify pass of a forced step, captured once per
// (l, k, Q-net layer) into a HIP graph and replayed on the stream.
int step_graph(lede_ctx* c, int l, int k, int qa, hipStream_t s) {
  const auto key = std::make_tuple(l, k, qa);
  auto it = c->graphs.find(key);
  if (it == c->graphs.end()) {
    HIP_CHECK(c, hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal));
    int rc = k > 0 ? launch_drafts(c, l, 1, k, qa, 0, s) : LEDE_OK;
    if (!rc) rc = launch_verify(c, k, s);
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(s, &g);
    if (rc) {
      if (g) (void)hipGraphDestroy(g);
      return rc;
    }
    if (e != hipSuccess) return fail(c, LEDE_E_HIP, "hipStreamEndCapture: %s", hipGetErrorString(e));
    hipGraphExec_t ex = nullptr;
    const hipError_t ei = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (ei != hipSuccess) return fail(c, LEDE_E_HIP, "hipGraphInstantiate: %s", hipGetErrorString(ei));
    it = c->graphs.emplace(key, ex).first;
  }
  PRE();
  HIP_CHECK(c, hipGraphLaunch(it->second, s));
  if (k > 0) c->last_draft_rows = k;  // as the eager launches leave them
  c->last_rows = k + 1;
  return LEDE_OK;
}

// The acceptance record, and the Q-network's action and value (slots 48..49,
// written there by the Q-network's output kernel), in one read-back.
int read_record(lede_ctx* c, hipStream_t s) {
  if (int rc = join_side(c, s)) return rc;
  PRE();
  HIP_CHECK(c, hipMemcpyAsync(c->record_h, c->S<int32_t>(c->lo.record), 50 * 4, hipMemcpyDeviceToHost, s));
  return wait_stream(c, s);
}

// Restore the decoding state a failed call started from: committed length
// c0, pending token pending0, the page table of c0 positions (pages freed by
// truncate_pages go back to the front of the free list in logical order, so
// re-taking them rebuilds the same table), no outstanding draft.  When the
// call had issued device work, the device's copies (length, pending token,
// table, confidence trace) are rewritten after the stream drains.  Keeps the
// error text of the original failure; best effort when the device itself
// has failed.
void rollback(lede_ctx* c, hipStream_t s, int c0, int pending0) {
  const std::string keep = c->err;
  c->fail_after = -1;
  truncate_pages(c, c0);
  (void)ensure_pages(c, c0);
  c->seq_len = c0;
  c->pending = pending0;
  c->drafted_k = -1;
  c->policy_valid = 0;
  c->split_row = -1;
  if (c->launched) {
    (void)hipStreamSynchronize(s);
    (void)hipStreamSynchronize(c->side);
    c->side_pending = 0;
    c->table_dev.assign(c->lo.max_pages_seq, -3);  // not a value the host ever uploads
    (void)upload_table(c, s);
    (void)upload_seq_len(c, c0, s);
    if (pending0 >= 0) (void)launch_set_token(c->S<uint64_t>(c->lo.dkeys), 0, pending0, s);
    if (c->trace_pushed) {
      (void)hipMemcpyAsync(c->S<float>(c->lo.trace), c->S<float>(c->lo.trace_bak), POLICY_TRACE * 4,
                           hipMemcpyDeviceToDevice, s);
      (void)hipMemcpyAsync(c->S<int32_t>(c->lo.trace_state), c->S<float>(c->lo.trace_bak) + POLICY_TRACE, 2 * 4,
                           hipMemcpyDeviceToDevice, s);
    }
    (void)hipStreamSynchronize(s);
  }
  c->launched = c->trace_pushed = false;
  c->err = keep;
}

// A call that changes the decoding state: when it fails after it has
// allocated pages or issued device work (or always, with force), the state
// it started from is restored (rollback).  A failed argument or state check
// changes nothing.
struct Txn {
  lede_ctx* c;
  hipStream_t s;
  int c0, pending0;
  size_t n_table0;
  bool force;
  Txn(lede_ctx* c_, hipStream_t s_, bool force_ = false)
      : c(c_), s(s_), c0(c_->seq_len), pending0(c_->pending), n_table0(c_->table.size()), force(force_) {
    c->launched = c->trace_pushed = false;
  }
  int done(int rc) {
    if (rc != LEDE_OK && (force || c->launched || c->table.size() != n_table0)) rollback(c, s, c0, pending0);
    return rc;
  }
};

// Apply a finished verify (record read back) to the host mirror.
void commit_host(lede_ctx* c) {
  c->policy_valid = 0;
  c->seq_len = c->record_h[2];
  c->pending = c->record_h[3];
  truncate_pages(c, c->seq_len);
  // the acceptance kernel cleared the device entries past the kept pages
  for (size_t j = c->table.size(); j < c->table_dev.size(); ++j) c->table_dev[j] = -1;
  c->drafted_k = -1;
}

}  // namespace

// ---- C ABI -------------------------------------------------------------------------

extern "C" {

int lede_region_bytes(const lede_config* cfg, size_t* wb, size_t* kvb, size_t* wsb) {
  if (const char* why = check_config(cfg)) { (void)why; return cfg ? LEDE_E_UNSUPPORTED : LEDE_E_ARG; }
  Layout o = make_layout(cfg);
  if (wb) *wb = o.wbytes;
  if (kvb) *kvb = o.kvbytes;
  if (wsb) *wsb = o.wsbytes;
  return LEDE_OK;
}

const char* lede_last_error(const lede_ctx* c) { return c ? c->err.c_str() : "null context"; }

int lede_create(const lede_config* cfg, void* warena, size_t wbytes, void* kv, size_t kvbytes, void* ws,
                size_t wsbytes, lede_ctx** out) {
  if (!out) return LEDE_E_ARG;
  *out = nullptr;
  if (!cfg || !warena || !kv || !ws) return LEDE_E_ARG;
  if (check_config(cfg)) return LEDE_E_UNSUPPORTED;
  Layout o = make_layout(cfg);
  if (wbytes < o.wbytes || kvbytes < o.kvbytes || wsbytes < o.wsbytes) return LEDE_E_ARG;
  if (((uintptr_t)warena | (uintptr_t)kv | (uintptr_t)ws) & 255) return LEDE_E_ARG;
  lede_ctx* c = new lede_ctx();
  c->cfg = *cfg;
  c->lo = o;
  c->w = (uint8_t*)warena;
  c->kv = (uint8_t*)kv;
  c->ws = (uint8_t*)ws;
  (void)hipGetDevice(&c->dev);
  for (int i = 0; i < o.n_pages; ++i) c->free_list.push_back(i);
  if (hipHostMalloc((void**)&c->table_h, (size_t)(1 + LEDE_MAX_IN_FLIGHT) * table_pitch(o) * 4, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->record_h, RECORD_INTS * 4, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->unif_h, UNIF_FLOATS * 4, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->trace_h, 64 * 4, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->keys_h, 2 * KEY_WORDS * 8, 0) != hipSuccess ||
      hipHostMalloc((void**)&c->rec_slots_h, LEDE_MAX_IN_FLIGHT * RECORD_INTS * 4, 0) != hipSuccess) {
    lede_destroy(c);
    return LEDE_E_HIP;
  }
  // zero the workspace (padding columns of activations must be finite)
  if (hipMemset(ws, 0, o.wsbytes) != hipSuccess) { lede_destroy(c); return LEDE_E_HIP; }
  // rotary table: angle pos * base^(-2i/hd) in fp64, stored as fp32 (cos, sin)
  std::vector<float> rope((size_t)o.max_ctx * o.hd);
  for (int p = 0; p < o.max_ctx; ++p)
    for (int i = 0; i < o.hd / 2; ++i) {
      const double ang = (double)p * std::pow((double)cfg->rope_base, -2.0 * i / o.hd);
      rope[((size_t)p * (o.hd / 2) + i) * 2] = (float)std::cos(ang);
      rope[((size_t)p * (o.hd / 2) + i) * 2 + 1] = (float)std::sin(ang);
    }
  if (hipMemcpy(c->S<void>(o.rope), rope.data(), rope.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    lede_destroy(c);
    return LEDE_E_HIP;
  }
  std::vector<int32_t> bt(o.max_pages_seq, -1);
  if (hipMemcpy(c->S<void>(o.btab), bt.data(), bt.size() * 4, hipMemcpyHostToDevice) != hipSuccess) {
    lede_destroy(c);
    return LEDE_E_HIP;
  }
  c->table_dev = bt;
  for (hipEvent_t& e : c->rec_ev)
    if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) {
      lede_destroy(c);
      return LEDE_E_HIP;
    }
  if (hipEventCreateWithFlags(&c->wait_ev, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->side_in, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&c->side_out, hipEventDisableTiming) != hipSuccess ||
      hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess) {
    lede_destroy(c);
    return LEDE_E_HIP;
  }
  *out = c;
  return LEDE_OK;
}

void lede_destroy(lede_ctx* c) {
  if (!c) return;
  // pipelined steps still copy their records into the host slots
  for (const auto& f : c->inflight) (void)hipEventSynchronize(c->rec_ev[f.slot]);
  for (hipEvent_t e : c->rec_ev)
    if (e) (void)hipEventDestroy(e);
  if (c->wait_ev) (void)hipEventDestroy(c->wait_ev);
  if (c->side) {
    (void)hipStreamSynchronize(c->side);
    (void)hipStreamDestroy(c->side);
  }
  if (c->side_in) (void)hipEventDestroy(c->side_in);
  if (c->side_out) (void)hipEventDestroy(c->side_out);
  if (c->rec_slots_h) (void)hipHostFree(c->rec_slots_h);
  for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.second);
  for (hipEvent_t e : c->evpool) (void)hipEventDestroy(e);
  if (c->table_h) (void)hipHostFree(c->table_h);
  if (c->record_h) (void)hipHostFree(c->record_h);
  if (c->unif_h) (void)hipHostFree(c->unif_h);
  if (c->trace_h) (void)hipHostFree(c->trace_h);
  if (c->keys_h) (void)hipHostFree(c->keys_h);
  delete c;
}

int lede_load_tensor(lede_ctx* c, int32_t kind, int32_t layer, const void* src, void* stream) {
  if (!c || !src) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  const Layout& o = c->lo;
  hipStream_t s = S_(stream);
  const bool per_layer = kind >= LEDE_T_ATTN_NORM && kind <= LEDE_T_WD;
  if (per_layer && (layer < 0 || layer >= o.L)) return fail(c, LEDE_E_ARG, "layer %d out of range", layer);
  auto copy = [&](size_t off, size_t bytes) -> int {
    HIP_CHECK(c, hipMemcpyAsync(c->w + off, src, bytes, hipMemcpyDeviceToDevice, s));
    return LEDE_OK;
  };
  auto repack = [&](size_t off, int N, int K, int group0, int n_groups, int order, int dt) -> int {
    RepackArgs ra{};
    ra.src = src; ra.N = N; ra.K = K; ra.dst = c->w + off; ra.KT = k_tiles(dt, K);
    ra.group0 = group0; ra.n_groups = n_groups; ra.order = order; ra.hd = o.hd;
    HIP_CHECK(c, launch_repack(dt, ra, s));
    return LEDE_OK;
  };
  const auto* lw = per_layer ? &o.lay[layer] : nullptr;
  const size_t ed = (size_t)o.d * o.es;
  switch (kind) {
    case LEDE_T_EMBED: return copy(o.embed, (size_t)o.V * ed);
    case LEDE_T_FINAL_NORM: return copy(o.final_norm, ed);
    case LEDE_T_HEAD: return repack(o.head, o.V, o.d, 0, o.V / 16, ROWS_PLAIN, o.dt);
    case LEDE_T_ATTN_NORM: return copy(lw->attn_norm, ed);
    case LEDE_T_FFN_NORM: return copy(lw->ffn_norm, ed);
    case LEDE_T_WQ: return repack(lw->wqkv, o.qd, o.d, 0, o.qd / 16, ROWS_ROPE, o.dt);
    case LEDE_T_WK: return repack(lw->wqkv, o.kvd, o.d, o.qd / 16, o.kvd / 16, ROWS_ROPE, o.dt);
    case LEDE_T_WV: return repack(lw->wqkv, o.kvd, o.d, (o.qd + o.kvd) / 16, o.kvd / 16, ROWS_PLAIN, o.dt);
    case LEDE_T_WO: return repack(lw->wo, o.d, o.qd, 0, o.d / 16, ROWS_PLAIN, o.dt);
    case LEDE_T_WG: return repack(lw->wgu, o.F, o.d, 0, o.F / 8, ROWS_GATE, o.dt);
    case LEDE_T_WU: return repack(lw->wgu, o.F, o.d, 0, o.F / 8, ROWS_UP, o.dt);
    case LEDE_T_WD: return repack(lw->wd, o.d, o.F, 0, o.d / 16, ROWS_PLAIN, o.dt);
    case LEDE_T_QNET_W1:
      if (!o.H) return fail(c, LEDE_E_STATE, "config has no Q-network");
      return repack(o.qw1, o.H, o.d, 0, o.H / 16, ROWS_PLAIN, 0);
    case LEDE_T_QNET_B1: if (!o.H) return fail(c, LEDE_E_STATE, "config has no Q-network"); return copy(o.qb1, (size_t)o.H * 4);
    case LEDE_T_QNET_W2: if (!o.H) return fail(c, LEDE_E_STATE, "config has no Q-network"); return copy(o.qw2, (size_t)o.A * o.H * 4);
    case LEDE_T_QNET_B2: if (!o.H) return fail(c, LEDE_E_STATE, "config has no Q-network"); return copy(o.qb2, (size_t)o.A * 4);
    case LEDE_T_EXIT_W1: if (!o.He) return fail(c, LEDE_E_STATE, "config has no exit policy"); return copy(o.ew1, (size_t)o.He * 3 * 4);
    case LEDE_T_EXIT_B1: if (!o.He) return fail(c, LEDE_E_STATE, "config has no exit policy"); return copy(o.eb1, (size_t)o.He * 4);
    case LEDE_T_EXIT_W2: if (!o.He) return fail(c, LEDE_E_STATE, "config has no exit policy"); return copy(o.ew2, (size_t)o.He * 2 * 4);
    case LEDE_T_EXIT_B2: if (!o.He) return fail(c, LEDE_E_STATE, "config has no exit policy"); return copy(o.eb2, 2 * 4);
  }
  return fail(c, LEDE_E_ARG, "unknown tensor kind %d", kind);
}

int lede_set_free_list(lede_ctx* c, const int32_t* order, int32_t n) {
  if (!c || !order) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (!c->table.empty()) return fail(c, LEDE_E_STATE, "pages are allocated");
  if (n != c->lo.n_pages) return fail(c, LEDE_E_ARG, "order must list all %d pages", c->lo.n_pages);
  std::vector<char> seen(n, 0);
  for (int i = 0; i < n; ++i) {
    if (order[i] < 0 || order[i] >= n || seen[order[i]]) return fail(c, LEDE_E_ARG, "order is not a permutation");
    seen[order[i]] = 1;
  }
  c->free_list.assign(order, order + n);
  return LEDE_OK;
}

int lede_set_options(lede_ctx* c, int32_t use_graphs, int32_t debug) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  // a captured step keeps the logits pointers of the debug mode it was
  // captured in: a change of either option drops the captures
  if ((debug != 0) != (c->debug != 0) || (use_graphs != 0) != (c->use_graphs != 0)) {
    for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.second);
    c->graphs.clear();
  }
  c->use_graphs = use_graphs;
  c->debug = debug;
  return LEDE_OK;
}

int lede_debug_inject_failure(lede_ctx* c, int32_t n_ops) {
  if (!c) return LEDE_E_ARG;
  c->fail_after = n_ops < 0 ? -1 : n_ops;
  return LEDE_OK;
}

int lede_load_weights(lede_ctx* c, const lede_weights* w, void* stream) {
  if (!c || !w) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  const Layout& o = c->lo;
  if (w->n_layers < 0 || w->first_layer < 0 || w->first_layer + w->n_layers > o.L)
    return fail(c, LEDE_E_ARG, "layers [%d, %d) outside the model's %d", w->first_layer,
                w->first_layer + w->n_layers, o.L);
  if (w->n_layers > 0 && !w->layer) return fail(c, LEDE_E_ARG, "null layer table");
  if (!o.H && (w->qnet_w1 || w->qnet_b1 || w->qnet_w2 || w->qnet_b2))
    return fail(c, LEDE_E_STATE, "config has no Q-network");
  if (!o.He && (w->exit_w1 || w->exit_b1 || w->exit_w2 || w->exit_b2))
    return fail(c, LEDE_E_STATE, "config has no exit policy");
  // every tensor named is repacked or copied in order; a null entry is left as it is
  struct Item { int kind, layer; const void* src; };
  std::vector<Item> items = {{LEDE_T_EMBED, 0, w->embed}, {LEDE_T_FINAL_NORM, 0, w->final_norm},
                             {LEDE_T_HEAD, 0, w->head}};
  for (int j = 0; j < w->n_layers; ++j)
    for (int t = 0; t < LEDE_LAYER_TENSORS; ++t)
      items.push_back({LEDE_T_ATTN_NORM + t, w->first_layer + j, w->layer[(size_t)j * LEDE_LAYER_TENSORS + t]});
  const void* rest[8] = {w->qnet_w1, w->qnet_b1, w->qnet_w2, w->qnet_b2, w->exit_w1, w->exit_b1, w->exit_w2, w->exit_b2};
  for (int t = 0; t < 8; ++t) items.push_back({LEDE_T_QNET_W1 + t, 0, rest[t]});
  for (const Item& it : items) {
    if (!it.src) continue;
    const int rc = lede_load_tensor(c, it.kind, it.layer, it.src, stream);
    if (rc) return rc;
  }
  return LEDE_OK;
}

int lede_debug_logits(lede_ctx* c, int32_t which, float* host, size_t cap_floats, int32_t* rows, void* stream) {
  if (!c) return LEDE_E_ARG;
  if (which != LEDE_LOGITS_VERIFY && which != LEDE_LOGITS_DRAFT)
    return fail(c, LEDE_E_ARG, "which must be LEDE_LOGITS_VERIFY or LEDE_LOGITS_DRAFT");
  return lede_debug_read(c, which == LEDE_LOGITS_VERIFY ? 0 : 3, host, cap_floats, rows, stream);
}

int lede_set_verify_reuse(lede_ctx* c, int32_t enable) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  c->verify_reuse = enable != 0;
  return LEDE_OK;
}

static int prefill_impl(lede_ctx* c, const int32_t* tokens, int32_t n, hipStream_t s, int32_t* next_token) {
  c->policy_valid = 0;
  const int c0 = c->seq_len;
  int rc = ensure_pages(c, c0 + n);
  if (rc) return rc;
  if ((rc = upload_table(c, s)) || (rc = upload_seq_len(c, c0, s))) return rc;
  int32_t* pd = c->S<int32_t>(c->lo.prompt);
  PRE();
  HIP_CHECK(c, hipMemcpyAsync(pd, tokens, (size_t)n * 4, hipMemcpyHostToDevice, s));
  uint64_t* vk = c->S<uint64_t>(c->lo.vkeys);
  int last_m = 0;
  for (int off = 0; off < n; off += MROWS) {
    const int M = std::min(MROWS, n - off);
    TokenSrc tok{pd + off, nullptr};
    if ((rc = run_layers(c, M, false, tok, off, 0, c->lo.L, 0, vk, s))) return rc;
    if (off + M == n) {
      const bool trace = c->lo.He > 0;
      if ((rc = run_head(c, M, false, vk, verify_logits(c, trace), s, 0, true))) return rc;
      if (trace && (rc = push_trace(c, verify_logits(c, true) + (size_t)(M - 1) * c->lo.V, 1, nullptr, s)))
        return rc;
    }
    last_m = M;
  }
  c->last_rows = last_m;
  PRE();
  HIP_CHECK(c, hipMemcpyAsync(c->keys_h, vk, KEY_WORDS * 8, hipMemcpyDeviceToHost, s));
  HIP_CHECK(c, hipStreamSynchronize(s));
  const int next = key_token(key_value(c->keys_h, last_m - 1));
  PRE();
  HIP_CHECK(c, launch_set_token(c->S<uint64_t>(c->lo.dkeys), 0, next, s));
  if ((rc = upload_seq_len(c, c0 + n, s))) return rc;
  c->seq_len = c0 + n;
  c->pending = next;
  if (next_token) *next_token = next;
  return LEDE_OK;
}

int lede_prefill(lede_ctx* c, const int32_t* tokens, int32_t n, void* stream, int32_t* next_token) {
  if (!c || !tokens || n < 1) return fail(c, LEDE_E_ARG, "bad prefill arguments");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  for (int i = 0; i < n; ++i)
    if (tokens[i] < 0 || tokens[i] >= c->lo.V) return fail(c, LEDE_E_ARG, "token %d out of range", tokens[i]);
  hipStream_t s = S_(stream);
  Txn t(c, s);
  return t.done(prefill_impl(c, tokens, n, s, next_token));
}

int lede_set_pending(lede_ctx* c, int32_t token, void* stream) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (token < 0 || token >= c->lo.V) return fail(c, LEDE_E_ARG, "token out of range");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  hipStream_t s = S_(stream);
  Txn t(c, s);
  c->policy_valid = 0;
  int rc = pre_launch(c);
  if (!rc && launch_set_token(c->S<uint64_t>(c->lo.dkeys), 0, token, s) != hipSuccess)
    rc = fail(c, LEDE_E_HIP, "launch_set_token failed");
  if (!rc && hipStreamSynchronize(s) != hipSuccess) rc = fail(c, LEDE_E_HIP, "hipStreamSynchronize failed");
  if (!rc) c->pending = token;
  return t.done(rc);
}

int lede_truncate(lede_ctx* c, int32_t new_len, void* stream) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (new_len < 0 || new_len > c->seq_len) return fail(c, LEDE_E_ARG, "new_len %d not in [0, %d]", new_len, c->seq_len);
  hipStream_t s = S_(stream);
  // a failed truncation leaves the state as it was, outstanding draft aside
  Txn t(c, s);
  c->policy_valid = 0;
  truncate_pages(c, new_len);
  c->drafted_k = -1;
  int rc = upload_table(c, s);
  if (!rc) rc = upload_seq_len(c, new_len, s);
  if (!rc) c->seq_len = new_len;
  return t.done(rc);
}

static int draft_impl(lede_ctx* c, int l, int k, hipStream_t s) {
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is already outstanding");
  if (c->pending < 0) return fail(c, LEDE_E_STATE, "no pending token (prefill first)");
  if (l < 1 || l > c->lo.L) return fail(c, LEDE_E_ARG, "exit layer %d not in 1..%d", l, c->lo.L);
  if (k < 1 || k > c->lo.k_max) return fail(c, LEDE_E_ARG, "draft length %d not in 1..%d", k, c->lo.k_max);
  int rc = ensure_pages(c, c->seq_len + k + 1);
  if (rc) return rc;
  if ((rc = upload_table(c, s))) return rc;
  rc = launch_drafts(c, l, 1, k, 0, 0, s);
  if (rc) return rc;
  c->drafted_k = k;
  c->drafted_l = l;
  return LEDE_OK;
}

int lede_draft(lede_ctx* c, int32_t l, int32_t k, void* stream, int32_t* drafts) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  hipStream_t s = S_(stream);
  Txn t(c, s);
  int rc = draft_impl(c, l, k, s);
  if (rc) return t.done(rc);
  c->policy_valid = 0;
  if (drafts) {
    rc = pre_launch(c);
    if (!rc && (hipMemcpyAsync(c->keys_h, c->S<uint64_t>(c->lo.dkeys), KEY_WORDS * 8, hipMemcpyDeviceToHost, s) !=
                    hipSuccess ||
                hipStreamSynchronize(s) != hipSuccess))
      rc = fail(c, LEDE_E_HIP, "draft read-back failed");
    if (rc) return t.done(rc);
    for (int i = 0; i < k; ++i) drafts[i] = key_token(key_value(c->keys_h, i + 1));
  }
  return LEDE_OK;
}

static int verify_impl(lede_ctx* c, hipStream_t s, int32_t* accepted, int32_t* tokens, int32_t* n_emitted,
                       int32_t* verify) {
  const int k = c->drafted_k < 0 ? 0 : c->drafted_k;
  int rc;
  if (c->drafted_k < 0) {
    if ((rc = ensure_pages(c, c->seq_len + 1))) return rc;
    if ((rc = upload_table(c, s))) return rc;
  }
  const int from = (c->verify_reuse && k > 0) ? c->drafted_l : 0;
  rc = from ? extend_drafts(c, from, k, s) : LEDE_OK;
  if (!rc) rc = launch_verify(c, k, s, 0.f, from);
  if (rc) return rc;
  if (verify) {
    PRE();
    HIP_CHECK(c, hipMemcpyAsync(c->keys_h + KEY_WORDS, c->S<uint64_t>(c->lo.vkeys), KEY_WORDS * 8,
                                hipMemcpyDeviceToHost, s));
  }
  if ((rc = read_record(c, s))) return rc;
  commit_host(c);
  const int a = c->record_h[0];
  if (accepted) *accepted = a;
  if (n_emitted) *n_emitted = a + 1;
  if (tokens) for (int i = 0; i <= a; ++i) tokens[i] = c->record_h[4 + i];
  if (verify) for (int i = 0; i <= k; ++i) verify[i] = key_token(key_value(c->keys_h + KEY_WORDS, i));
  return LEDE_OK;
}

int lede_verify(lede_ctx* c, void* stream, int32_t* accepted, int32_t* tokens, int32_t* n_emitted, int32_t* verify) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (c->pending < 0) return fail(c, LEDE_E_STATE, "no pending token (prefill first)");
  hipStream_t s = S_(stream);
  // a failed verify also discards the outstanding draft: the transition
  // (draft, verify, commit) rolls back to the committed state it started from
  Txn t(c, s, true);
  return t.done(verify_impl(c, s, accepted, tokens, n_emitted, verify));
}

}  // extern "C"

namespace {

// One step (greedy when temperature == 0, speculative sampling otherwise).
// A step's host record from its device record r (acceptance record, and the
// Q-network's action and value in slots 48..49).
void fill_record(const lede_ctx* c, const int32_t* r, int l, int k, int k_eff, bool ran_q, lede_step_record* rec) {
  const int a = r[0];
  rec->l = l;
  rec->k_req = k;
  rec->k_eff = k_eff;
  rec->accepted = a;
  rec->n_emitted = a + 1;
  for (int i = 0; i <= a; ++i) rec->tokens[i] = r[4 + i];
  for (int i = 0; i < k_eff; ++i) rec->drafts[i] = r[24 + i];
  rec->seq_len = r[2];
  rec->pending = r[3];
  if (ran_q) {
    rec->q_action = r[48];
    int32_t bits = r[49];
    memcpy(&rec->q_max, &bits, 4);
  } else {
    rec->q_action = -1;
    rec->q_max = NAN;
  }
  // Section 3.1.3 reward, summed over the drafts up to the first rejection
  rec->reward = 0.f;
  if (k_eff > 0) {
    const double lam = (double)(c->lo.L - l) / c->lo.L;
    rec->reward = (float)(a * (1.0 + lam) + (a < k_eff ? (-2.0 + lam) : 0.0));
  }
}

int step_body(lede_ctx* c, const lede_action* forced, int32_t log_qnet, int32_t n_remaining, float temperature,
              const float* uniforms, void* stream, lede_step_record* rec) {
  if (!c || !rec) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (n_remaining < 1) return fail(c, LEDE_E_ARG, "n_remaining must be >= 1");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  if (c->pending < 0) return fail(c, LEDE_E_STATE, "no pending token (prefill first)");
  const Layout& o = c->lo;
  if (!forced && !o.H) return fail(c, LEDE_E_STATE, "no Q-network configured");
  const bool sampled = temperature != 0.f;
  if (sampled) {
    if (!(temperature > 0.f) || !std::isfinite(temperature))
      return fail(c, LEDE_E_ARG, "temperature must be finite and > 0");
    if (!uniforms) return fail(c, LEDE_E_ARG, "null uniforms");
    for (int i = 0; i < UNIF_FLOATS; ++i)
      if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return fail(c, LEDE_E_ARG, "uniform %d not in [0, 1)", i);
  }
  const float inv_t = sampled ? 1.f / temperature : 0.f;
  hipStream_t s = S_(stream);
  int rc0 = 0;
  memset(rec, 0, sizeof *rec);
  rec->q_action = -1;
  const int c0 = c->seq_len;
  int l = forced ? forced->l : 0, k = forced ? forced->k : 0;
  if (forced) {
    if (l < 1 || l > o.L) return fail(c, LEDE_E_ARG, "exit layer %d not in 1..%d", l, o.L);
    if (k < 0 || k > o.k_max) return fail(c, LEDE_E_ARG, "draft length %d not in 0..%d", k, o.k_max);
  }
  if (sampled) {
    memcpy(c->unif_h, uniforms, UNIF_FLOATS * 4);
    PRE();
    HIP_CHECK(c, hipMemcpyAsync(c->S<float>(o.unif), c->unif_h, UNIF_FLOATS * 4, hipMemcpyHostToDevice, s));
  }
  const int l_min = o.H ? c->cfg.exits[0] : 0;
  const bool want_q = o.H && (!forced || log_qnet);
  hipEvent_t ph0 = nullptr;
  if ((rc0 = prof_mark(c, s, &ph0, 1))) return rc0;
  int k_eff = forced ? std::min(k, n_remaining - 1) : std::min(o.k_max, n_remaining - 1);
  bool ran_q = false;
  int rc;
  (void)rc0;
  if (k_eff > 0) {
    if (!forced) {
      // the agent decides at the first candidate layer of the first draft's
      // forward pass; the step continues once its action is known
      if ((rc = ensure_pages(c, c0 + 1)) || (rc = upload_table(c, s))) return rc;
      uint64_t* dk = c->S<uint64_t>(o.dkeys);
      rc = run_layers(c, 1, true, TokenSrc{nullptr, dk}, 0, 0, l_min, l_min, dk + 1, s);
      if (rc) return rc;
      PRE();
      HIP_CHECK(c, hipMemcpyAsync(c->record_h + 48, c->S<int32_t>(o.record) + 48, 2 * 4, hipMemcpyDeviceToHost, s));
      if ((rc = wait_stream(c, s))) return rc;
      const int a = c->record_h[48];
      if (a < 0 || a >= o.A) return fail(c, LEDE_E_HIP, "Q-network action %d out of range", a);
      l = c->cfg.exits[a / c->cfg.n_lengths];
      k = c->cfg.lengths[a % c->cfg.n_lengths];
      k_eff = std::min(std::min(k, o.k_max), n_remaining - 1);
      ran_q = true;
      if ((rc = ensure_pages(c, c0 + k_eff + 1)) || (rc = upload_table(c, s))) return rc;
      rc = launch_drafts(c, l, 1, k_eff, 0, l_min, s, inv_t);
      if (rc) return rc;
    } else {
      if ((rc = ensure_pages(c, c0 + k_eff + 1)) || (rc = upload_table(c, s))) return rc;
      const int qa = (want_q && l_min <= l) ? l_min : 0;
      ran_q = qa > 0;
      if (c->use_graphs && !c->prof && s && !sampled && !c->verify_reuse) {
        // the whole step as one graph: every launch reads positions, tokens
        // and pages from device memory, so a capture serves every step of
        // the same shape
        if ((rc = step_graph(c, l, k_eff, qa, s))) return rc;
        goto verified;
      }
      c->qnet_defer = 1;
      rc = launch_drafts(c, l, 1, k_eff, qa, 0, s, inv_t);
      c->qnet_defer = 0;
      if (rc) return rc;
    }
  } else {
    k_eff = 0;
    if ((rc = ensure_pages(c, c0 + 1)) || (rc = upload_table(c, s))) return rc;
    if (forced && c->use_graphs && !c->prof && s && !sampled) {
      if ((rc = step_graph(c, l, 0, 0, s))) return rc;
      goto verified;
    }
  }
  {
    const int from = (c->verify_reuse && k_eff > 0) ? l : 0;
    if (from && (rc = extend_drafts(c, l, k_eff, s))) return rc;
    if (k_eff > 0 && (rc = prof_close(c, s, LEDE_K_DRAFT_PHASE, 0.0, ph0))) return rc;
    hipEvent_t ph1 = nullptr;
    if ((rc = prof_mark(c, s, &ph1, 1))) return rc;
    rc = launch_verify(c, k_eff, s, inv_t, from);
    if (rc) return rc;
    if ((rc = prof_close(c, s, LEDE_K_VERIFY_PHASE, 0.0, ph1))) return rc;
  }
verified:
  rc = read_record(c, s);
  if (rc) return rc;
  commit_host(c);
  if ((rc = prof_fold(c))) return rc;
  fill_record(c, c->record_h, l, k, k_eff, ran_q, rec);
  return LEDE_OK;
}

int step_impl(lede_ctx* c, const lede_action* forced, int32_t log_qnet, int32_t n_remaining, float temperature,
              const float* uniforms, void* stream, lede_step_record* rec) {
  if (!c) return LEDE_E_ARG;
  Txn t(c, S_(stream));
  return t.done(step_body(c, forced, log_qnet, n_remaining, temperature, uniforms, stream, rec));
}

}  // namespace

extern "C" {

int lede_step(lede_ctx* c, const lede_action* forced, int32_t log_qnet, int32_t n_remaining, void* stream,
              lede_step_record* rec) {
  return step_impl(c, forced, log_qnet, n_remaining, 0.f, nullptr, stream, rec);
}

static int submit_body(lede_ctx* c, const lede_action* action, int32_t log_qnet, int32_t n_remaining,
                       void* stream);

// A failed submit: the steps in flight before it stay queued; the pages and
// the device's copies of the state return to what those steps leave (their
// records have arrived once the stream has drained).
static void submit_rollback(lede_ctx* c, hipStream_t s, int ub_prev) {
  const std::string keep = c->err;
  c->fail_after = -1;
  truncate_pages(c, ub_prev);
  (void)ensure_pages(c, ub_prev);
  c->policy_valid = 0;
  c->split_row = -1;
  if (c->launched) {
    (void)hipStreamSynchronize(s);
    (void)hipStreamSynchronize(c->side);
    c->side_pending = 0;
    int len = c->seq_len, pend = c->pending;
    if (!c->inflight.empty()) {
      const int32_t* r = c->rec_slots_h + (size_t)c->inflight.back().slot * RECORD_INTS;
      len = r[2];
      pend = r[3];
    }
    c->table_dev.assign(c->lo.max_pages_seq, -3);
    (void)upload_table(c, s);
    (void)upload_seq_len(c, len, s);
    (void)launch_set_token(c->S<uint64_t>(c->lo.dkeys), 0, pend, s);
    (void)hipStreamSynchronize(s);
  }
  c->launched = c->trace_pushed = false;
  c->err = keep;
}

int lede_step_submit(lede_ctx* c, const lede_action* action, int32_t log_qnet, int32_t n_remaining, void* stream) {
  if (!c) return LEDE_E_ARG;
  const int ub_prev = c->inflight.empty() ? c->seq_len : c->seq_ub;
  const size_t n_table0 = c->table.size();
  c->launched = c->trace_pushed = false;
  const int rc = submit_body(c, action, log_qnet, n_remaining, stream);
  if (rc != LEDE_OK && (c->launched || c->table.size() != n_table0)) submit_rollback(c, S_(stream), ub_prev);
  return rc;
}

static int submit_body(lede_ctx* c, const lede_action* action, int32_t log_qnet, int32_t n_remaining,
                       void* stream) {
  if (!c || !action) return fail(c, LEDE_E_ARG, "null argument");
  if (n_remaining < 1) return fail(c, LEDE_E_ARG, "n_remaining must be >= 1");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  if (c->pending < 0) return fail(c, LEDE_E_STATE, "no pending token (prefill first)");
  if ((int)c->inflight.size() >= LEDE_MAX_IN_FLIGHT)
    return fail(c, LEDE_E_STATE, "%d steps are already outstanding", LEDE_MAX_IN_FLIGHT);
  if (!c->inflight.empty() && stream != c->pipe_stream) return fail(c, LEDE_E_STATE, "submit on the collecting stream");
  if (c->use_graphs || c->prof || c->verify_reuse)
    return fail(c, LEDE_E_STATE, "graph replay, profiling and verify reuse are not pipelined");
  const Layout& o = c->lo;
  const int l = action->l, k = action->k;
  if (l < 1 || l > o.L) return fail(c, LEDE_E_ARG, "exit layer %d not in 1..%d", l, o.L);
  if (k < 0 || k > o.k_max) return fail(c, LEDE_E_ARG, "draft length %d not in 0..%d", k, o.k_max);
  hipStream_t s = S_(stream);
  const int k_eff = std::min(k, n_remaining - 1);
  // the step starts at the committed length after the steps in flight, which
  // the device knows; pages cover their longest acceptances
  const int ub = c->inflight.empty() ? c->seq_len : c->seq_ub;
  int rc = ensure_pages(c, ub + k_eff + 1);
  if (rc) return rc;
  const int slot = c->next_slot;
  if ((rc = upload_table(c, s, c->table_h + (1 + slot) * table_pitch(o)))) return rc;
  // the acceptance clears the entries from the first page wholly past the
  // committed length to the last page the step wrote; the step starts at a
  // length in [lo, ub] (every step in flight commits at least one token), so
  // the host no longer knows the device's entries in that range
  const int lo = c->seq_len + (int)c->inflight.size();
  for (int j = (lo + 1 + PAGE - 1) / PAGE; j < (ub + k_eff + 1 + PAGE - 1) / PAGE && j < (int)c->table_dev.size(); ++j)
    c->table_dev[j] = -2;
  const int l_min = o.H ? c->cfg.exits[0] : 0;
  const int qa = (o.H && log_qnet && l_min <= l && k_eff > 0) ? l_min : 0;
  c->policy_valid = 0;
  c->qnet_defer = 1;
  rc = k_eff > 0 ? launch_drafts(c, l, 1, k_eff, qa, 0, s) : LEDE_OK;
  c->qnet_defer = 0;
  if (rc) return rc;
  if ((rc = launch_verify(c, k_eff, s))) return rc;
  if ((rc = join_side(c, s))) return rc;
  PRE();
  HIP_CHECK(c, hipMemcpyAsync(c->rec_slots_h + (size_t)slot * RECORD_INTS, c->S<int32_t>(o.record), 50 * 4,
                              hipMemcpyDeviceToHost, s));
  HIP_CHECK(c, hipEventRecord(c->rec_ev[slot], s));
  c->next_slot = (slot + 1) % LEDE_MAX_IN_FLIGHT;
  c->inflight.push_back(lede_ctx::InFlight{l, k, k_eff, slot, qa > 0});
  c->seq_ub = ub + k_eff + 1;
  c->pipe_stream = stream;
  return LEDE_OK;
}

int lede_step_collect(lede_ctx* c, void* stream, lede_step_record* rec) {
  if (!c || !rec) return fail(c, LEDE_E_ARG, "null argument");
  if (c->inflight.empty()) return fail(c, LEDE_E_STATE, "no step submitted");
  if (stream != c->pipe_stream) return fail(c, LEDE_E_STATE, "collect on the submitting stream");
  const lede_ctx::InFlight f = c->inflight.front();
  HIP_CHECK(c, hipEventSynchronize(c->rec_ev[f.slot]));
  c->inflight.pop_front();
  const int32_t* r = c->rec_slots_h + (size_t)f.slot * RECORD_INTS;
  c->seq_len = r[2];
  c->pending = r[3];
  int ub = c->seq_len;
  for (const auto& g : c->inflight) ub += g.k_eff + 1;
  c->seq_ub = ub;
  truncate_pages(c, ub);  // keeps the pages the remaining steps may still write
  memset(rec, 0, sizeof *rec);
  fill_record(c, r, f.l, f.k_req, f.k_eff, f.ran_q, rec);
  return LEDE_OK;
}

int lede_step_sampled(lede_ctx* c, const lede_action* forced, int32_t log_qnet, int32_t n_remaining,
                      float temperature, const float* uniforms, void* stream, lede_step_record* rec) {
  if (c && !(temperature > 0.f)) return fail(c, LEDE_E_ARG, "temperature must be > 0");
  return step_impl(c, forced, log_qnet, n_remaining, temperature, uniforms, stream, rec);
}

static int policy_body(lede_ctx* c, int32_t n_remaining, hipStream_t s, lede_step_record* rec) {
  const Layout& o = c->lo;
  memset(rec, 0, sizeof *rec);
  rec->q_action = -1;
  rec->q_max = NAN;
  c->policy_log.clear();
  c->policy_valid = 0;
  const int c0 = c->seq_len;
  const int k_lim = std::max(0, std::min(std::min(POLICY_MAX_DRAFT, o.k_max), n_remaining - 1));
  int rc;
  if ((rc = ensure_pages(c, c0 + k_lim + 1)) || (rc = upload_table(c, s))) return rc;
  hipEvent_t ph0 = nullptr;
  if ((rc = prof_mark(c, s, &ph0, 1))) return rc;
  uint64_t* dk = c->S<uint64_t>(o.dkeys);
  ExitPolicyArgs pa{};
  pa.vocab = o.V; pa.hidden = o.He;
  pa.w1 = c->W<float>(o.ew1); pa.b1 = c->W<float>(o.eb1); pa.w2 = c->W<float>(o.ew2); pa.b2 = c->W<float>(o.eb2);
  pa.trace = c->S<float>(o.trace); pa.trace_state = c->S<int32_t>(o.trace_state);
  float* log_dev = c->S<float>(o.pol_out);
  // one decision: the state of the head's logits, scored on the device (kept in
  // the device decision log), read back
  auto decide = [&](const float* logits, int kind, int index, int* action) -> int {
    pa.out = log_dev + c->policy_log.size();
    pa.logits = logits; pa.kind = (float)kind; pa.index = (float)index;
    PRE();
    HIP_CHECK(c, launch_exit_policy(pa, s));
    PRE();
    HIP_CHECK(c, hipMemcpyAsync(c->trace_h, pa.out, POLICY_LOG * 4, hipMemcpyDeviceToHost, s));
    if (int rc = wait_stream(c, s)) return rc;
    c->policy_log.insert(c->policy_log.end(), c->trace_h, c->trace_h + POLICY_LOG);
    *action = c->trace_h[7] > 0.5f ? 1 : 0;
    return LEDE_OK;
  };
  int l_star = c->cfg.exits[c->cfg.n_exits - 1], k = 0;
  bool ran_last = false;  // the pass of draft input k (the last draft) has run
  if (k_lim > 0) {
    // exit layer: up the candidate layers with the pending token (draft pass 1)
    int begin = 0;
    for (int e = 0; e < c->cfg.n_exits; ++e) {
      const int l = c->cfg.exits[e];
      rc = run_layers(c, 1, true, TokenSrc{nullptr, dk}, 0, begin, l, 0, dk + 1, s);
      if (!rc) rc = run_head(c, 1, true, dk + 1, draft_logits(c, 0, true), s);
      int act = 0;
      if (!rc) rc = decide(draft_logits(c, 0, true), 0, l, &act);
      if (rc) return rc;
      begin = l;
      if (act == 1 || e == c->cfg.n_exits - 1) {
        l_star = l;
        break;
      }
    }
    k = 1;
    // draft length: each further pass at l* continues on 'exit'
    while (k < k_lim) {
      rc = run_layers(c, 1, true, TokenSrc{nullptr, dk + k}, k, 0, l_star, 0, dk + k + 1, s, k);
      if (!rc) rc = run_head(c, 1, true, dk + k + 1, draft_logits(c, k, true), s, k);
      int act = 0;
      if (!rc) rc = decide(draft_logits(c, k, true), 1, k + 1, &act);
      if (rc) return rc;
      ran_last = act != 1;  // 'continue': this pass was the last draft's input pass
      if (act != 1) break;
      ++k;
    }
    c->last_draft_rows = k;
  }
  const int from = (c->verify_reuse && k > 0) ? l_star : 0;
  if (from && !ran_last && (rc = extend_drafts(c, l_star, k, s))) return rc;
  // the draft phase includes the decisions' read-backs (the stream idles
  // while the host waits for each)
  if (k > 0 && (rc = prof_close(c, s, LEDE_K_DRAFT_PHASE, 0.0, ph0))) return rc;
  hipEvent_t ph1 = nullptr;
  if ((rc = prof_mark(c, s, &ph1, 1))) return rc;
  if ((rc = launch_verify(c, k, s, 0.f, from))) return rc;
  if ((rc = prof_close(c, s, LEDE_K_VERIFY_PHASE, 0.0, ph1))) return rc;
  if ((rc = read_record(c, s))) return rc;
  commit_host(c);
  if ((rc = prof_fold(c))) return rc;
  const int a = c->record_h[0];
  c->policy_valid = 1;
  c->policy_l = l_star;
  c->policy_a = a;
  rec->l = l_star;
  rec->k_req = POLICY_MAX_DRAFT;
  rec->k_eff = k;
  rec->accepted = a;
  rec->n_emitted = a + 1;
  for (int i = 0; i <= a; ++i) rec->tokens[i] = c->record_h[4 + i];
  for (int i = 0; i < k; ++i) rec->drafts[i] = c->record_h[24 + i];
  rec->seq_len = c->record_h[2];
  rec->pending = c->record_h[3];
  if (k > 0) {
    const double lam = (double)(o.L - l_star) / o.L;
    rec->reward = (float)(a * (1.0 + lam) + (a < k ? (-2.0 + lam) : 0.0));
  }
  return LEDE_OK;
}

int lede_step_policy(lede_ctx* c, int32_t n_remaining, void* stream, lede_step_record* rec) {
  if (!c || !rec) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (n_remaining < 1) return fail(c, LEDE_E_ARG, "n_remaining must be >= 1");
  if (c->drafted_k >= 0) return fail(c, LEDE_E_STATE, "a draft is outstanding");
  if (c->pending < 0) return fail(c, LEDE_E_STATE, "no pending token (prefill first)");
  if (!c->lo.He) return fail(c, LEDE_E_STATE, "no exit policy configured");
  hipStream_t s = S_(stream);
  Txn t(c, s);
  const int rc = t.done(policy_body(c, n_remaining, s, rec));
  if (rc) c->policy_log.clear();
  return rc;
}

int lede_set_trace(lede_ctx* c, const float* values, int32_t n, void* stream) {
  if (!c || (n > 0 && !values)) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (!c->lo.He) return fail(c, LEDE_E_STATE, "no exit policy configured");
  if (n < 0 || n > POLICY_TRACE) return fail(c, LEDE_E_ARG, "trace length %d not in 0..%d", n, POLICY_TRACE);
  hipStream_t s = S_(stream);
  for (int i = 0; i < POLICY_TRACE; ++i) c->trace_h[i] = i < n ? values[i] : 0.f;
  int32_t* st = (int32_t*)(c->trace_h + 32);
  st[0] = n;
  st[1] = n % POLICY_TRACE;
  HIP_CHECK(c, hipMemcpyAsync(c->S<float>(c->lo.trace), c->trace_h, POLICY_TRACE * 4, hipMemcpyHostToDevice, s));
  HIP_CHECK(c, hipMemcpyAsync(c->S<int32_t>(c->lo.trace_state), st, 2 * 4, hipMemcpyHostToDevice, s));
  HIP_CHECK(c, hipStreamSynchronize(s));
  return LEDE_OK;
}

int lede_get_trace(lede_ctx* c, float* values, int32_t* n, void* stream) {
  if (!c || !values || !n) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (!c->lo.He) return fail(c, LEDE_E_STATE, "no exit policy configured");
  hipStream_t s = S_(stream);
  HIP_CHECK(c, hipMemcpyAsync(c->trace_h, c->S<float>(c->lo.trace), POLICY_TRACE * 4, hipMemcpyDeviceToHost, s));
  HIP_CHECK(c, hipMemcpyAsync(c->trace_h + 32, c->S<int32_t>(c->lo.trace_state), 2 * 4, hipMemcpyDeviceToHost, s));
  HIP_CHECK(c, hipStreamSynchronize(s));
  const int32_t* st = (const int32_t*)(c->trace_h + 32);
  const int cnt = st[0], next = st[1];
  // oldest first: the ring holds the last cnt values ending just before `next`
  for (int i = 0; i < cnt; ++i) values[i] = c->trace_h[(next - cnt + i + 2 * POLICY_TRACE) % POLICY_TRACE];
  *n = cnt;
  return LEDE_OK;
}

int lede_op_sample(const float* logits, int32_t V, float temperature, float u, int32_t* token, void* stream) {
  if (!logits || !token || V < 1) return LEDE_E_ARG;
  if (!(temperature > 0.f) || !std::isfinite(temperature) || !(u >= 0.f && u < 1.f)) return LEDE_E_ARG;
  hipStream_t s = S_(stream);
  uint64_t* key = nullptr;
  if (hipMalloc((void**)&key, KEY_WORDS * 8) != hipSuccess) return LEDE_E_HIP;
  SampleArgs sa{};
  sa.logits = logits; sa.vocab = V; sa.inv_t = 1.f / temperature;
  sa.u = nullptr; sa.u_imm = u; sa.key_out = key; sa.stats_out = nullptr;
  uint64_t h = 0;
  int rc = LEDE_OK;
  if (launch_sample(sa, s) != hipSuccess || hipMemcpyAsync(&h, key, 8, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    rc = LEDE_E_HIP;
  (void)hipFree(key);
  if (rc == LEDE_OK) *token = key_token(h);  // a single writer: word 0 holds the key
  return rc;
}

int lede_get_kv_state(lede_ctx* c, int32_t* seq_len, int32_t* pending, int32_t* bt, int32_t cap, int32_t* n_table) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (seq_len) *seq_len = c->seq_len;
  if (pending) *pending = c->pending;
  if (n_table) *n_table = (int32_t)c->table.size();
  if (bt) {
    if (cap < (int)c->table.size()) return fail(c, LEDE_E_ARG, "block table capacity %d < %zu", cap, c->table.size());
    for (size_t i = 0; i < c->table.size(); ++i) bt[i] = c->table[i];
  }
  return LEDE_OK;
}

int lede_debug_read(lede_ctx* c, int32_t which, float* host, size_t cap, int32_t* rows, void* stream) {
  if (!c || !host) return fail(c, LEDE_E_ARG, "null argument");
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  if (!c->debug && which != 4) return fail(c, LEDE_E_STATE, "debug mode is off");
  hipStream_t s = S_(stream);
  const Layout& o = c->lo;
  const float* src;
  size_t n;
  int r;
  switch (which) {
    case 0: r = c->last_rows; src = c->S<float>(o.logits); n = (size_t)r * o.V; break;
    case 1: r = 1; src = c->S<float>(o.qv); n = (size_t)o.A; break;
    case 2: r = 1; src = c->S<float>(o.qs); n = (size_t)o.d; break;
    case 3: r = c->last_draft_rows; src = c->S<float>(o.logits) + (size_t)MROWS * o.V; n = (size_t)r * o.V; break;
    case 4: {
      const size_t m = c->policy_log.size();
      if (cap < m) return fail(c, LEDE_E_ARG, "capacity %zu < %zu", cap, m);
      std::copy(c->policy_log.begin(), c->policy_log.end(), host);
      if (rows) *rows = (int)(m / POLICY_LOG);
      return LEDE_OK;
    }
    default: return fail(c, LEDE_E_ARG, "unknown debug buffer %d", which);
  }
  if (cap < n) return fail(c, LEDE_E_ARG, "capacity %zu < %zu", cap, n);
  HIP_CHECK(c, hipMemcpyAsync(host, src, n * 4, hipMemcpyDeviceToHost, s));
  HIP_CHECK(c, hipStreamSynchronize(s));
  if (rows) *rows = r;
  return LEDE_OK;
}

int lede_prof_enable(lede_ctx* c, int32_t on) {
  if (!c) return LEDE_E_ARG;
  if (!c->inflight.empty()) return fail(c, LEDE_E_STATE, "pipelined steps are outstanding");
  int rc = prof_fold(c);
  if (rc) return rc;
  if (on < 0 || on > 2) return fail(c, LEDE_E_ARG, "timing level %d not in 0..2", on);
  c->prof = on;
  return LEDE_OK;
}

int lede_prof_read(lede_ctx* c, lede_prof_entry* out, int32_t reset) {
  if (!c || !out) return fail(c, LEDE_E_ARG, "null argument");
  int rc = prof_fold(c);
  if (rc) return rc;
  for (int i = 0; i < LEDE_K_NCLASS; ++i) {
    out[i].ms = c->p_ms[i];
    out[i].bytes = c->p_bytes[i];
    out[i].launches = c->p_n[i];
    if (reset) c->p_ms[i] = c->p_bytes[i] = 0, c->p_n[i] = 0;
  }
  return LEDE_OK;
}

size_t lede_op_tiled_bytes(int32_t dtype, int32_t N, int32_t K) {
  if ((dtype != 0 && dtype != 1) || N < 1 || K < 1) return 0;
  return tiled_bytes(dtype, N, K);
}

int lede_op_repack(int32_t dtype, const void* src, int32_t N, int32_t K, void* tiled, void* stream) {
  if ((dtype != 0 && dtype != 1) || !src || !tiled || N < 1 || K < 1) return LEDE_E_ARG;
  if (N % 16) return LEDE_E_UNSUPPORTED;
  RepackArgs ra{};
  ra.src = src; ra.N = N; ra.K = K; ra.dst = tiled; ra.KT = k_tiles(dtype, K);
  ra.group0 = 0; ra.n_groups = N / 16; ra.order = ROWS_PLAIN; ra.hd = 0;
  return launch_repack(dtype, ra, S_(stream)) == hipSuccess ? LEDE_OK : LEDE_E_HIP;
}

int lede_op_linear(int32_t dtype, const void* tiled, int32_t N, int32_t K, const void* x, int32_t ldx, int32_t M,
                   float* y, int32_t use_mfma, void* stream) {
  if ((dtype != 0 && dtype != 1) || !tiled || !x || !y || N < 1 || K < 1) return LEDE_E_ARG;
  if (N % 16) return LEDE_E_UNSUPPORTED;
  if (M < 1 || M > 16 || (!use_mfma && M != 1)) return LEDE_E_ARG;
  // the kernels read whole tiles of every row: rows padded to the tile width
  if (ldx < k_tiles(dtype, K) * tile_k(dtype)) return LEDE_E_ARG;
  LinearArgs a{};
  a.w = (const uint8_t*)tiled;
  a.n_groups = N / 16; a.KT = k_tiles(dtype, K); a.K = K; a.M = M;
  a.x_mode = X_PLAIN; a.x = x; a.ldx = ldx;
  a.epi = EPI_STORE; a.out = y; a.ldo = N;
  return launch_linear(dtype, use_mfma != 0, a, std::min(a.n_groups, 4096), S_(stream)) == hipSuccess ? LEDE_OK
                                                                                                  : LEDE_E_HIP;
}

int lede_op_read_probe(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream, float* kernel_ms) {
  if (!src || !sink || bytes == 0) return LEDE_E_ARG;
  if (bytes % 16 || grid < 1 || grid > 65535) return LEDE_E_ARG;
  if (!kernel_ms)
    return launch_read_probe(src, bytes, sink, grid, S_(stream)) == hipSuccess ? LEDE_OK : LEDE_E_HIP;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess) return LEDE_E_HIP;
  if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return LEDE_E_HIP; }
  int rc = LEDE_OK;
  if (launch_read_probe(src, bytes, sink, grid, S_(stream), e0, e1) != hipSuccess ||
      hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(kernel_ms, e0, e1) != hipSuccess)
    rc = LEDE_E_HIP;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return rc;
}

int lede_op_read_groups(const void* src, int32_t n_groups, int32_t tiles, uint32_t* sink, void* stream,
                        float* kernel_ms) {
  if (!src || !sink || n_groups < 1 || n_groups > 65535 || tiles < 1) return LEDE_E_ARG;
  if (!kernel_ms)
    return launch_read_groups(src, n_groups, tiles, sink, S_(stream)) == hipSuccess ? LEDE_OK : LEDE_E_HIP;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess) return LEDE_E_HIP;
  if (hipEventCreate(&e1) != hipSuccess) { (void)hipEventDestroy(e0); return LEDE_E_HIP; }
  int rc = LEDE_OK;
  if (launch_read_groups(src, n_groups, tiles, sink, S_(stream), e0, e1) != hipSuccess ||
      hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(kernel_ms, e0, e1) != hipSuccess)
    rc = LEDE_E_HIP;
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  return rc;
}

}  // extern "C"

// ---- views for the policy trainer (dqn.cpp) ----------------------------------------

namespace lede {

int policy_step_take(lede_ctx* c, PolicyStepView* v) {
  if (!c->policy_valid) return LEDE_E_STATE;
  c->policy_valid = 0;
  v->log = c->S<float>(c->lo.pol_out);
  v->n_dec = (int)(c->policy_log.size() / POLICY_LOG);
  v->l_star = c->policy_l;
  v->accepted = c->policy_a;
  v->n_layers = c->lo.L;
  return LEDE_OK;
}

int exit_weights_view(lede_ctx* c, ExitWeightsView* v) {
  const Layout& o = c->lo;
  if (!o.He) return LEDE_E_STATE;
  v->w1 = c->W<float>(o.ew1);
  v->b1 = c->W<float>(o.eb1);
  v->w2 = c->W<float>(o.ew2);
  v->b2 = c->W<float>(o.eb2);
  v->hidden = o.He;
  return LEDE_OK;
}

}  // namespace lede
