// Host sanitizer run of the runtime's host code (liblede built with
// AddressSanitizer and UndefinedBehaviorSanitizer on its host side only).
// Without a GPU it drives what the host does on its own: region sizing over
// the supported shapes and the rejected ones, argument checks of every entry
// point, and context creation failing cleanly when the device calls do.
// Exit status 0 when everything ran clean and returned the documented codes.
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
  // context creation: bad arguments, then a valid request whose device
  // calls fail without a GPU (the partly built context is torn down)
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
    const int rc = lede_create(&c, al(w), wb, al(kv), kvb, al(ws), wsb, &ctx);
    if (rc == LEDE_OK) {
      lede_destroy(ctx);  // a GPU is present after all
    } else {
      EXPECT(rc == LEDE_E_HIP && ctx == nullptr);
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
