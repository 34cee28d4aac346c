// liblede policy trainer: the C ABI of the offline optimisation of the exit
// policy's Q-network declared in include/lede.h, over the kernels of dqn.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/lede.h"
#include "ctx_view.h"
#include "kernels.h"

using namespace lede;

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct DqnLayout {
  size_t theta, target, m, v, ring, loss, bytes;
};

// "" when cfg is usable, else the reason; *code the status to return
const char* check(const lede_dqn_config& c, int* code) {
  *code = LEDE_E_UNSUPPORTED;
  if (c.hidden < 1 || c.hidden > DQN_MAX_HIDDEN) return "hidden not in 1..128";
  if (c.capacity < 2 || c.capacity > (1 << 24)) return "capacity not in 2..2^24";
  if (c.batch < 1 || c.batch > DQN_MAX_BATCH) return "batch not in 1..256";
  if ((int64_t)c.batch * c.hidden > DQN_MAX_BH) return "batch * hidden above 4096";
  if (c.n_step < 1 || c.n_step > DQN_MAX_N) return "n_step not in 1..16";
  *code = LEDE_E_ARG;
  if (!(c.gamma >= 0.f && c.gamma <= 1.f)) return "gamma not in [0, 1]";
  if (!(c.lr > 0.f) || !std::isfinite(c.lr)) return "lr not finite and > 0";
  if (!(c.beta1 >= 0.f && c.beta1 < 1.f) || !(c.beta2 >= 0.f && c.beta2 < 1.f)) return "betas not in [0, 1)";
  if (!(c.adam_eps > 0.f) || !std::isfinite(c.adam_eps)) return "adam_eps not finite and > 0";
  if (!(c.sigma0 >= 0.f) || !std::isfinite(c.sigma0)) return "sigma0 not finite and >= 0";
  *code = LEDE_OK;
  return "";
}

DqnLayout layout(const lede_dqn_config& c) {
  DqnLayout o{};
  const size_t set2 = 2 * (size_t)dqn_params(c.hidden) * 4;
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t r = off; off += align256(bytes); return r; };
  o.theta = take(set2);
  o.target = take(set2);
  o.m = take(set2);
  o.v = take(set2);
  o.ring = take((size_t)c.capacity * DQN_SLOT * 4);
  o.loss = take(4);
  o.bytes = off;
  return o;
}

}  // namespace

struct lede_dqn {
  lede_dqn_config cfg;
  DqnLayout lo;
  uint8_t* r;
  int P;
  int head = 0, count = 0;  // next ring slot written, transitions stored
  int64_t t = 0;            // Adam steps taken
  float* stage = nullptr;   // pinned host staging of the loss
  std::string err;
  float* F(size_t off) const { return (float*)(r + off); }
};

namespace {

int fail(lede_dqn* q, int code, const char* fmt, ...) {
  if (q) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    q->err = buf;
  }
  return code;
}

#define DQN_HIP(q, expr)                                                                    \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return fail(q, LEDE_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

hipStream_t S_(void* s) { return (hipStream_t)s; }

void advance(lede_dqn* q, int64_t n) {
  q->head = (int)(((int64_t)q->head + n) % q->cfg.capacity);
  q->count = (int)std::min<int64_t>((int64_t)q->count + n, q->cfg.capacity);
}

}  // namespace

extern "C" {

size_t lede_dqn_region_bytes(const lede_dqn_config* cfg) {
  int code;
  if (!cfg || *check(*cfg, &code)) return 0;
  return layout(*cfg).bytes;
}

int lede_dqn_create(const lede_dqn_config* cfg, void* region, size_t bytes, lede_dqn** out) {
  if (!cfg || !region || !out) return LEDE_E_ARG;
  int code;
  if (*check(*cfg, &code)) return code;
  const DqnLayout lo = layout(*cfg);
  if (bytes < lo.bytes || ((uintptr_t)region & 255)) return LEDE_E_ARG;
  lede_dqn* q = new lede_dqn();
  q->cfg = *cfg;
  q->lo = lo;
  q->r = (uint8_t*)region;
  q->P = dqn_params(cfg->hidden);
  if (hipHostMalloc((void**)&q->stage, 64, hipHostMallocDefault) != hipSuccess) {
    delete q;
    return LEDE_E_HIP;
  }
  *out = q;
  return LEDE_OK;
}

void lede_dqn_destroy(lede_dqn* q) {
  if (!q) return;
  if (q->stage) (void)hipHostFree(q->stage);
  delete q;
}

const char* lede_dqn_last_error(const lede_dqn* q) { return q ? q->err.c_str() : "null handle"; }

int lede_dqn_init(lede_dqn* q, const float* u, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (!u) return fail(q, LEDE_E_ARG, "null uniforms");
  DqnInitArgs a{};
  a.u = u;
  a.H = q->cfg.hidden;
  a.sigma0 = q->cfg.sigma0;
  a.theta = q->F(q->lo.theta);
  a.target = q->F(q->lo.target);
  a.m = q->F(q->lo.m);
  a.v = q->F(q->lo.v);
  DQN_HIP(q, launch_dqn_init(a, S_(stream)));
  q->head = q->count = 0;
  q->t = 0;
  return LEDE_OK;
}

int lede_dqn_push(lede_dqn* q, const float* transitions, int32_t n, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (n < 0 || (n > 0 && !transitions)) return fail(q, LEDE_E_ARG, "bad transitions (n = %d)", n);
  if (n == 0) return LEDE_OK;
  DqnPushArgs a{};
  a.src = transitions;
  a.n = n;
  a.ring = q->F(q->lo.ring);
  a.capacity = q->cfg.capacity;
  a.head = q->head;
  DQN_HIP(q, launch_dqn_push(a, S_(stream)));
  advance(q, n);
  return LEDE_OK;
}

int lede_dqn_record(lede_dqn* q, lede_ctx* ctx, int32_t episode_end, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (!ctx) return fail(q, LEDE_E_ARG, "null context");
  PolicyStepView v{};
  if (policy_step_take(ctx, &v) != LEDE_OK)
    return fail(q, LEDE_E_STATE, "the context's last step is not an exit-policy step (or was recorded)");
  const double lam = (double)(v.n_layers - v.l_star) / v.n_layers;
  DqnRecordArgs a{};
  a.log = v.log;
  a.n_dec = v.n_dec;
  a.l_star = v.l_star;
  a.accepted = v.accepted;
  a.r_accept = (float)(1.0 + lam);
  a.r_reject = (float)(-2.0 + lam);
  a.r_continue = -0.01f;
  a.ring = q->F(q->lo.ring);
  a.capacity = q->cfg.capacity;
  a.head = q->head;
  a.end_episode = episode_end != 0;
  a.prev_newest = q->count ? (q->head - 1 + q->cfg.capacity) % q->cfg.capacity : -1;
  DQN_HIP(q, launch_dqn_record(a, S_(stream)));
  advance(q, v.n_dec);
  return LEDE_OK;
}

int lede_dqn_end_episode(lede_dqn* q, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (!q->count) return LEDE_OK;
  DqnRecordArgs a{};
  a.n_dec = 0;
  a.ring = q->F(q->lo.ring);
  a.capacity = q->cfg.capacity;
  a.head = q->head;
  a.end_episode = 1;
  a.prev_newest = (q->head - 1 + q->cfg.capacity) % q->cfg.capacity;
  DQN_HIP(q, launch_dqn_record(a, S_(stream)));
  return LEDE_OK;
}

int lede_dqn_update(lede_dqn* q, const float* u, const float* noise, void* stream, float* loss) {
  if (!q) return LEDE_E_ARG;
  if (!u || !noise) return fail(q, LEDE_E_ARG, "null uniforms or noise");
  const lede_dqn_config& c = q->cfg;
  const int n_valid = q->count - c.n_step;
  if (n_valid < 1)
    return fail(q, LEDE_E_STATE, "%d transitions stored; an update needs more than n_step = %d", q->count, c.n_step);
  const int64_t t = q->t + 1;
  DqnUpdateArgs a{};
  a.theta = q->F(q->lo.theta);
  a.target = q->F(q->lo.target);
  a.m = q->F(q->lo.m);
  a.v = q->F(q->lo.v);
  a.ring = q->F(q->lo.ring);
  a.capacity = c.capacity;
  a.oldest = (q->head - q->count + c.capacity) % c.capacity;
  a.n_valid = n_valid;
  a.u = u;
  a.noise = noise;
  a.H = c.hidden;
  a.B = c.batch;
  a.n = c.n_step;
  a.gamma = c.gamma;
  a.gamma_n = (float)std::pow((double)c.gamma, (double)c.n_step);
  a.lr = c.lr;
  a.beta1 = c.beta1;
  a.beta2 = c.beta2;
  a.eps = c.adam_eps;
  a.bc1 = (float)(1.0 - std::pow((double)c.beta1, (double)t));
  a.bc2 = (float)(1.0 - std::pow((double)c.beta2, (double)t));
  a.loss_out = q->F(q->lo.loss);
  hipStream_t s = S_(stream);
  DQN_HIP(q, launch_dqn_update(a, s));
  q->t = t;
  if (loss) {
    DQN_HIP(q, hipMemcpyAsync(q->stage, a.loss_out, 4, hipMemcpyDeviceToHost, s));
    DQN_HIP(q, hipStreamSynchronize(s));
    *loss = q->stage[0];
  }
  return LEDE_OK;
}

int lede_dqn_sync_target(lede_dqn* q, void* stream) {
  if (!q) return LEDE_E_ARG;
  DQN_HIP(q, launch_dqn_copy(q->F(q->lo.theta), q->F(q->lo.target), 2 * q->P, S_(stream)));
  return LEDE_OK;
}

int lede_dqn_act(lede_dqn* q, lede_ctx* ctx, const float* noise, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (!ctx) return fail(q, LEDE_E_ARG, "null context");
  ExitWeightsView w{};
  if (exit_weights_view(ctx, &w) != LEDE_OK || w.hidden != q->cfg.hidden)
    return fail(q, LEDE_E_STATE, "the context has no exit policy of hidden width %d", q->cfg.hidden);
  DqnActArgs a{};
  a.theta = q->F(q->lo.theta);
  a.noise = noise;
  a.H = q->cfg.hidden;
  a.w1 = w.w1;
  a.b1 = w.b1;
  a.w2 = w.w2;
  a.b2 = w.b2;
  DQN_HIP(q, launch_dqn_act(a, S_(stream)));
  return LEDE_OK;
}

int lede_dqn_read(lede_dqn* q, int32_t which, float* host, size_t cap_floats, int32_t* count, void* stream) {
  if (!q) return LEDE_E_ARG;
  if (!host || !count) return fail(q, LEDE_E_ARG, "null argument");
  hipStream_t s = S_(stream);
  if (which >= 0 && which <= 3) {
    const size_t off[4] = {q->lo.theta, q->lo.target, q->lo.m, q->lo.v};
    const size_t n = 2 * (size_t)q->P;
    if (cap_floats < n) return fail(q, LEDE_E_ARG, "%zu floats needed", n);
    DQN_HIP(q, hipMemcpyAsync(host, q->F(off[which]), n * 4, hipMemcpyDeviceToHost, s));
    DQN_HIP(q, hipStreamSynchronize(s));
    *count = (int32_t)n;
    return LEDE_OK;
  }
  if (which == 4) {
    const int cap = q->cfg.capacity;
    if (cap_floats < (size_t)q->count * 6) return fail(q, LEDE_E_ARG, "%zu floats needed", (size_t)q->count * 6);
    std::vector<float> ring((size_t)cap * DQN_SLOT);
    DQN_HIP(q, hipMemcpyAsync(ring.data(), q->F(q->lo.ring), ring.size() * 4, hipMemcpyDeviceToHost, s));
    DQN_HIP(q, hipStreamSynchronize(s));
    for (int j = 0; j < q->count; ++j) {
      const size_t slot = (size_t)((q->head - q->count + j + cap) % cap);
      std::copy(ring.begin() + slot * DQN_SLOT, ring.begin() + slot * DQN_SLOT + 6, host + (size_t)j * 6);
    }
    *count = q->count;
    return LEDE_OK;
  }
  return fail(q, LEDE_E_ARG, "which = %d not in 0..4", which);
}

}  // extern "C"
