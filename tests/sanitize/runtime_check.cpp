// Host sanitizer run of the runtime's host code (liblede built with
// AddressSanitizer and UndefinedBehaviorSanitizer on its host side only).
// Without a GPU it drives what the host does on its own: region sizing over
// the supported shapes and the rejected ones, argument checks of every entry
// point, and context creation failing cleanly when the device calls do.
// With a GPU it also decodes on a tiny fp32 model whose KV pool holds four
// pages, so that the host's pager, rollback and pipelining paths run: prefill,
// forced, Q-network, sampled and exit-policy steps, truncation and resume, a
// permuted free list, injected failures (the state must come back
// unchanged), two steps in flight, and the pool and context running out.
// Exit status 0 when everything ran clean and returned the documented codes.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstring>
#include <vector>

#include "../../include/lede.h"

static int failures = 0;
#define EXPECT(cond)                                                   \
  do {                                                                 \
    if (!(cond)) {                                                     \
      std::fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                      \
    }                                                                  \
  } while (0)

static lede_config config(int L, int d, int nq, int nkv, int hd, int F, int V, int dtype) {
  lede_config c;
  std::memset(&c, 0, sizeof c);
  c.n_layers = L; c.d_model = d; c.n_heads = nq; c.n_kv_heads = nkv; c.head_dim = hd;
  c.ffn_dim = F; c.vocab = V; c.rms_eps = 1e-5f; c.rope_base = 10000.f; c.dtype = dtype;
  c.max_ctx = 832; c.page_size = 64; c.n_pages = 16;
  c.qnet_hidden = 64; c.n_exits = 4; c.n_lengths = 8;
  for (int i = 0; i < 4; ++i) c.exits[i] = i + 1;
  for (int i = 0; i < 8; ++i) c.lengths[i] = i + 1;
  c.k_max = 8;
  c.exit_qnet_hidden = 16;
  return c;
}


// ---- with a GPU: a tiny fp32 model through the decoding state machine ---------

struct KvState {
  int32_t seq_len = 0, pending = 0, n_table = 0;
  std::vector<int32_t> table = std::vector<int32_t>(64, -7);
  bool operator==(const KvState& o) const {
    return seq_len == o.seq_len && pending == o.pending && n_table == o.n_table &&
           std::vector<int32_t>(table.begin(), table.begin() + n_table) ==
               std::vector<int32_t>(o.table.begin(), o.table.begin() + o.n_table);
  }
};
static KvState kv_state(lede_ctx* ctx) {
  KvState k;
  EXPECT(lede_get_kv_state(ctx, &k.seq_len, &k.pending, k.table.data(), 64, &k.n_table) == LEDE_OK);
  return k;
}

static uint32_t rng = 88172645u;
static float frand() {
  rng ^= rng << 13;
  rng ^= rng >> 17;
  rng ^= rng << 5;
  return (float)((rng >> 8) / 8388608.0 - 1.0);
}

static void decode_on_gpu(lede_ctx* ctx, const lede_config& c) {
  // weights: one device buffer per tensor, random values
  const int d = c.d_model, qd = c.n_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim, F = c.ffn_dim, V = c.vocab;
  const int A = c.n_exits * c.n_lengths, H = c.qnet_hidden, He = c.exit_qnet_hidden;
  std::vector<void*> bufs;
  auto load = [&](int kind, int layer, size_t n, float scale, float offset) {
    std::vector<float> h(n);
    for (float& x : h) x = offset + scale * frand();
    void* dv = nullptr;
    EXPECT(hipMalloc(&dv, n * 4) == hipSuccess);
    EXPECT(hipMemcpy(dv, h.data(), n * 4, hipMemcpyHostToDevice) == hipSuccess);
    bufs.push_back(dv);
    EXPECT(lede_load_tensor(ctx, kind, layer, dv, nullptr) == LEDE_OK);
  };
  load(LEDE_T_EMBED, 0, (size_t)V * d, 1.f, 0.f);
  load(LEDE_T_FINAL_NORM, 0, d, 0.1f, 1.f);
  load(LEDE_T_HEAD, 0, (size_t)V * d, 0.05f, 0.f);
  for (int l = 0; l < c.n_layers; ++l) {
    load(LEDE_T_ATTN_NORM, l, d, 0.1f, 1.f);
    load(LEDE_T_WQ, l, (size_t)qd * d, 0.05f, 0.f);
    load(LEDE_T_WK, l, (size_t)kvd * d, 0.05f, 0.f);
    load(LEDE_T_WV, l, (size_t)kvd * d, 0.05f, 0.f);
    load(LEDE_T_WO, l, (size_t)d * qd, 0.05f, 0.f);
    load(LEDE_T_FFN_NORM, l, d, 0.1f, 1.f);
    load(LEDE_T_WG, l, (size_t)F * d, 0.05f, 0.f);
    load(LEDE_T_WU, l, (size_t)F * d, 0.05f, 0.f);
    load(LEDE_T_WD, l, (size_t)d * F, 0.05f, 0.f);
  }
  load(LEDE_T_QNET_W1, 0, (size_t)H * d, 0.05f, 0.f);
  load(LEDE_T_QNET_B1, 0, H, 0.f, 0.f);
  load(LEDE_T_QNET_W2, 0, (size_t)A * H, 0.05f, 0.f);
  load(LEDE_T_QNET_B2, 0, A, 0.f, 0.f);
  load(LEDE_T_EXIT_W1, 0, (size_t)He * 3, 0.5f, 0.f);
  load(LEDE_T_EXIT_B1, 0, He, 0.5f, 0.f);
  load(LEDE_T_EXIT_W2, 0, (size_t)2 * He, 0.5f, 0.f);
  load(LEDE_T_EXIT_B2, 0, 2, 0.f, 0.f);
  EXPECT(hipDeviceSynchronize() == hipSuccess);

  // a permuted free list, then a prompt over two pages
  const int32_t order[4] = {2, 0, 3, 1};
  EXPECT(lede_set_free_list(ctx, order, 4) == LEDE_OK);
  std::vector<int32_t> prompt(70);
  for (size_t i = 0; i < prompt.size(); ++i) prompt[i] = (int32_t)((i * 37 + 11) % V);
  int32_t next = -1;
  EXPECT(lede_prefill(ctx, prompt.data(), (int32_t)prompt.size(), nullptr, &next) == LEDE_OK);
  EXPECT(next >= 0 && next < V);
  KvState k0 = kv_state(ctx);
  EXPECT(k0.seq_len == 70 && k0.n_table == 2 && k0.table[0] == 2 && k0.table[1] == 0);
  EXPECT(lede_set_free_list(ctx, order, 4) == LEDE_E_STATE);  // pages are allocated

  lede_step_record rec;
  float unif[LEDE_SAMPLE_STRIDE];
  for (float& u : unif) u = 0.5f * (frand() + 1.f) * 0.999f;
  for (int i = 0; i < 6; ++i) {
    lede_action act = {1 + i % c.n_layers, 1 + i % 5};
    EXPECT(lede_step(ctx, &act, i & 1, 40, nullptr, &rec) == LEDE_OK);
    EXPECT(rec.n_emitted == rec.accepted + 1 && rec.seq_len == kv_state(ctx).seq_len);
  }
  EXPECT(lede_step(ctx, nullptr, 0, 40, nullptr, &rec) == LEDE_OK);           // the Q-network's action
  EXPECT(lede_step_sampled(ctx, nullptr, 0, 40, 0.6f, unif, nullptr, &rec) == LEDE_OK);
  EXPECT(lede_step_policy(ctx, 40, nullptr, &rec) == LEDE_OK);                // the paper's exit policy
  float trace[20];
  int32_t n_trace = 0;
  EXPECT(lede_get_trace(ctx, trace, &n_trace, nullptr) == LEDE_OK && n_trace > 0);

  // injected failures: every operation index of a forced step, state unchanged
  for (int n_ops = 1; n_ops <= 12; ++n_ops) {
    const KvState before = kv_state(ctx);
    EXPECT(lede_debug_inject_failure(ctx, n_ops) == LEDE_OK);
    lede_action act = {2, 4};
    const int rc = lede_step(ctx, &act, 1, 40, nullptr, &rec);
    EXPECT(rc == LEDE_OK || rc == LEDE_E_HIP);
    if (rc != LEDE_OK) EXPECT(kv_state(ctx) == before);
    EXPECT(lede_debug_inject_failure(ctx, -1) == LEDE_OK);
  }

  // two steps in flight
  {
    lede_action act = {1, 3};
    EXPECT(lede_step_submit(ctx, &act, 0, 40, nullptr) == LEDE_OK);
    EXPECT(lede_step_submit(ctx, &act, 0, 40, nullptr) == LEDE_OK);
    EXPECT(lede_step_submit(ctx, &act, 0, 40, nullptr) == LEDE_E_STATE);
    EXPECT(lede_step(ctx, &act, 0, 40, nullptr, &rec) == LEDE_E_STATE);
    EXPECT(lede_step_collect(ctx, nullptr, &rec) == LEDE_OK);
    EXPECT(lede_step_collect(ctx, nullptr, &rec) == LEDE_OK);
    EXPECT(lede_step_collect(ctx, nullptr, &rec) == LEDE_E_STATE);
  }

  // draft, truncate (discards it) and resume by re-prefill
  {
    int32_t drafts[4];
    const KvState before = kv_state(ctx);
    EXPECT(lede_draft(ctx, 2, 4, nullptr, drafts) == LEDE_OK);
    EXPECT(lede_draft(ctx, 2, 4, nullptr, drafts) == LEDE_E_STATE);
    EXPECT(lede_truncate(ctx, before.seq_len - 5, nullptr) == LEDE_OK);
    EXPECT(lede_truncate(ctx, before.seq_len, nullptr) == LEDE_E_ARG);
    EXPECT(lede_prefill(ctx, prompt.data(), 5, nullptr, &next) == LEDE_OK);
    EXPECT(kv_state(ctx).seq_len == before.seq_len);
  }

  // the pool (4 pages = 256 positions) and the context (max_ctx) run out
  {
    int rc = LEDE_OK;
    for (int i = 0; i < 400 && rc == LEDE_OK; ++i) {
      const KvState before = kv_state(ctx);
      lede_action act = {2, 8};
      rc = lede_step(ctx, &act, 0, 100, nullptr, &rec);
      if (rc != LEDE_OK) EXPECT(kv_state(ctx) == before);
    }
    EXPECT(rc == LEDE_E_KV_FULL || rc == LEDE_E_CTX_OVERFLOW);
    EXPECT(lede_truncate(ctx, 0, nullptr) == LEDE_OK && kv_state(ctx).n_table == 0);
    std::vector<int32_t> big(300, 5);
    EXPECT(lede_prefill(ctx, big.data(), (int32_t)big.size(), nullptr, &next) == LEDE_E_KV_FULL ||
           lede_prefill(ctx, big.data(), (int32_t)big.size(), nullptr, &next) == LEDE_E_CTX_OVERFLOW);
    EXPECT(kv_state(ctx).seq_len == 0);
  }
  for (void* b : bufs) (void)hipFree(b);
}

int main() {
  // region sizes of the supported shapes
  const lede_config shapes[] = {config(4, 256, 4, 4, 64, 688, 1024, LEDE_DTYPE_F32),
                                config(32, 4096, 32, 32, 128, 11008, 32000, LEDE_DTYPE_BF16),
                                config(32, 4096, 32, 8, 128, 14336, 128256, LEDE_DTYPE_BF16),
                                config(40, 5120, 40, 40, 128, 13824, 32000, LEDE_DTYPE_BF16)};
  for (const lede_config& c : shapes) {
    size_t wb = 0, kvb = 0, wsb = 0;
    EXPECT(lede_region_bytes(&c, &wb, &kvb, &wsb) == LEDE_OK);
    EXPECT(wb > 0 && kvb > 0 && wsb > 0);
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_OK);
  }
  // rejected shapes
  {
    lede_config c = shapes[0];
    c.head_dim = 96;
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_E_UNSUPPORTED);
    c = shapes[0]; c.page_size = 32;
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_E_UNSUPPORTED);
    c = shapes[0]; c.k_max = 16;
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_E_UNSUPPORTED);
    c = shapes[0]; c.exits[1] = 1;  // not ascending
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_E_UNSUPPORTED);
    c = shapes[0]; c.n_heads = 6;   // not a multiple of n_kv_heads
    EXPECT(lede_region_bytes(&c, nullptr, nullptr, nullptr) == LEDE_E_UNSUPPORTED);
    EXPECT(lede_region_bytes(nullptr, nullptr, nullptr, nullptr) == LEDE_E_ARG);
  }
  // context creation: bad arguments, then a valid request
  {
    const lede_config& c = shapes[0];
    size_t wb = 0, kvb = 0, wsb = 0;
    lede_region_bytes(&c, &wb, &kvb, &wsb);
    std::vector<unsigned char> w(wb + 256), kv(kvb + 256), ws(wsb + 256);
    auto al = [](std::vector<unsigned char>& v) {
      return (void*)(((uintptr_t)v.data() + 255) & ~(uintptr_t)255);
    };
    lede_ctx* ctx = (lede_ctx*)1;
    EXPECT(lede_create(&c, al(w), wb, al(kv), kvb, al(ws), wsb, nullptr) == LEDE_E_ARG);
    EXPECT(lede_create(nullptr, al(w), wb, al(kv), kvb, al(ws), wsb, &ctx) == LEDE_E_ARG && ctx == nullptr);
    EXPECT(lede_create(&c, al(w), wb - 1, al(kv), kvb, al(ws), wsb, &ctx) == LEDE_E_ARG);
    EXPECT(lede_create(&c, (unsigned char*)al(w) + 16, wb, al(kv), kvb, al(ws), wsb, &ctx) == LEDE_E_ARG);
    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev == 0) {
      // no GPU: the first device call of a valid request fails and the partly
      // built context is torn down (with a GPU, host buffers are never passed)
      const int rc = lede_create(&c, al(w), wb, al(kv), kvb, al(ws), wsb, &ctx);
      EXPECT(rc == LEDE_E_HIP && ctx == nullptr);
    } else {
      // a GPU: the same shape over device regions, with a four-page KV pool
      lede_config g = c;
      g.n_pages = 4;
      g.max_ctx = 300;
      EXPECT(lede_region_bytes(&g, &wb, &kvb, &wsb) == LEDE_OK);
      void *dw = nullptr, *dkv = nullptr, *dws = nullptr;
      EXPECT(hipMalloc(&dw, wb) == hipSuccess && hipMalloc(&dkv, kvb) == hipSuccess &&
             hipMalloc(&dws, wsb) == hipSuccess);
      lede_ctx* gctx = nullptr;
      EXPECT(lede_create(&g, dw, wb, dkv, kvb, dws, wsb, &gctx) == LEDE_OK);
      if (gctx) {
        decode_on_gpu(gctx, g);
        lede_destroy(gctx);
        std::printf("decoded on the GPU\n");
      }
      (void)hipFree(dw);
      (void)hipFree(dkv);
      (void)hipFree(dws);
    }
  }
  // every context entry point rejects a null context
  {
    int32_t i32[64] = {0};
    float f32[64] = {0};
    lede_action act = {1, 1};
    lede_step_record rec;
    lede_prof_entry prof[LEDE_K_NCLASS];
    lede_weights lw;
    std::memset(&lw, 0, sizeof lw);
    EXPECT(lede_load_tensor(nullptr, LEDE_T_EMBED, 0, f32, nullptr) == LEDE_E_ARG);
    EXPECT(lede_load_weights(nullptr, &lw, nullptr) == LEDE_E_ARG);
    EXPECT(lede_set_free_list(nullptr, i32, 1) == LEDE_E_ARG);
    EXPECT(lede_set_options(nullptr, 0, 0) == LEDE_E_ARG);
    EXPECT(lede_set_verify_reuse(nullptr, 0) == LEDE_E_ARG);
    EXPECT(lede_prefill(nullptr, i32, 4, nullptr, i32) == LEDE_E_ARG);
    EXPECT(lede_set_pending(nullptr, 1, nullptr) == LEDE_E_ARG);
    EXPECT(lede_truncate(nullptr, 0, nullptr) == LEDE_E_ARG);
    EXPECT(lede_draft(nullptr, 1, 1, nullptr, i32) == LEDE_E_ARG);
    EXPECT(lede_verify(nullptr, nullptr, i32, i32, i32, i32) == LEDE_E_ARG);
    EXPECT(lede_step(nullptr, &act, 0, 8, nullptr, &rec) == LEDE_E_ARG);
    EXPECT(lede_step_submit(nullptr, &act, 0, 8, nullptr) == LEDE_E_ARG);
    EXPECT(lede_step_collect(nullptr, nullptr, &rec) == LEDE_E_ARG);
    EXPECT(lede_step_sampled(nullptr, &act, 0, 8, 0.6f, f32, nullptr, &rec) == LEDE_E_ARG);
    EXPECT(lede_step_policy(nullptr, 8, nullptr, &rec) == LEDE_E_ARG);
    EXPECT(lede_set_trace(nullptr, f32, 1, nullptr) == LEDE_E_ARG);
    EXPECT(lede_get_trace(nullptr, f32, i32, nullptr) == LEDE_E_ARG);
    EXPECT(lede_get_kv_state(nullptr, i32, i32, i32, 64, i32) == LEDE_E_ARG);
    EXPECT(lede_debug_read(nullptr, 0, f32, 64, i32, nullptr) == LEDE_E_ARG);
    EXPECT(lede_debug_logits(nullptr, 0, f32, 64, i32, nullptr) == LEDE_E_ARG);
    EXPECT(lede_debug_inject_failure(nullptr, 1) == LEDE_E_ARG);
    EXPECT(lede_prof_enable(nullptr, 1) == LEDE_E_ARG);
    EXPECT(lede_prof_read(nullptr, prof, 1) == LEDE_E_ARG);
    EXPECT(std::strlen(lede_last_error(nullptr)) > 0);
    lede_destroy(nullptr);
  }
  // the trainer's handle: sizes, rejected configurations, creation
  {
    lede_dqn_config q;
    std::memset(&q, 0, sizeof q);
    q.hidden = 16; q.capacity = 64; q.batch = 8; q.n_step = 3; q.gamma = 0.99f; q.lr = 6.25e-5f;
    q.beta1 = 0.9f; q.beta2 = 0.999f; q.adam_eps = 1.5e-4f; q.sigma0 = 0.1f;
    const size_t bytes = lede_dqn_region_bytes(&q);
    EXPECT(bytes > 0);
    lede_dqn_config bad = q;
    bad.batch = 0;
    EXPECT(lede_dqn_region_bytes(&bad) == 0);
    EXPECT(lede_dqn_region_bytes(nullptr) == 0);
    float f32[16] = {0};
    std::vector<unsigned char> region(bytes + 256);
    void* r = (void*)(((uintptr_t)region.data() + 255) & ~(uintptr_t)255);
    lede_dqn* h = nullptr;
    EXPECT(lede_dqn_create(&q, r, bytes - 1, &h) == LEDE_E_ARG);
    EXPECT(lede_dqn_create(&q, (unsigned char*)r + 4, bytes, &h) == LEDE_E_ARG);
    EXPECT(lede_dqn_create(&bad, r, bytes, &h) != LEDE_OK);
    // the handle stages read-backs in pinned host memory: without a GPU its
    // creation fails cleanly
    const int rc = lede_dqn_create(&q, r, bytes, &h);
    if (rc == LEDE_OK) {
      EXPECT(h != nullptr);
      EXPECT(lede_dqn_push(h, f32, -1, nullptr) == LEDE_E_ARG);
      EXPECT(std::strlen(lede_dqn_last_error(h)) > 0);
      EXPECT(lede_dqn_record(h, nullptr, 0, nullptr) == LEDE_E_ARG);
      EXPECT(lede_dqn_act(h, nullptr, nullptr, nullptr) == LEDE_E_ARG);
      lede_dqn_destroy(h);
    } else {
      EXPECT(rc == LEDE_E_HIP);
    }
    EXPECT(lede_dqn_push(nullptr, f32, 1, nullptr) == LEDE_E_ARG);
    EXPECT(lede_dqn_update(nullptr, f32, f32, nullptr, f32) == LEDE_E_ARG);
    lede_dqn_destroy(nullptr);
    EXPECT(std::strlen(lede_dqn_last_error(nullptr)) > 0);
  }
  // the stateless operations' argument checks
  {
    int32_t tok = 0;
    float f32[16] = {0};
    EXPECT(lede_op_tiled_bytes(LEDE_DTYPE_BF16, 48, 1000) > 0);
    EXPECT(lede_op_sample(nullptr, 16, 1.f, 0.5f, &tok, nullptr) == LEDE_E_ARG);
    EXPECT(lede_op_sample(f32, 16, 1.f, 0.5f, nullptr, nullptr) == LEDE_E_ARG);
  }
  std::printf(failures ? "runtime sanitizer run: %d FAILED\n" : "runtime sanitizer run: clean\n", failures);
  return failures ? 1 : 0;
}
