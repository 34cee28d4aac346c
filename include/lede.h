/*
 * liblede -- batch-1 self-speculative decoding with learned (exit layer,
 * draft length) control, for AMD Instinct MI355X (gfx950).
 *
 * The method (Zhu et al., "Experience-Driven Dynamic Exits for LLMs with
 * Reinforcement Learning"): the model's own first l* layers draft k tokens,
 * each read out through the shared final RMSNorm and LM head (Section 2.2;
 * Section 3.1.1 -- the next-token distribution at layer l is computed from
 * the layer-l hidden state); the full L-layer model then verifies the k
 * drafts in one parallel pass (Section 1); a small MLP Q-network chooses
 * (l*, k) inside the loop (Sections 3.2, 3.3).  Decoding is greedy
 * (Section 4.1): the longest prefix of drafts equal to the full model's
 * argmax is accepted, followed by the full model's own next token.
 *
 * Conventions for every entry point:
 *  - Return value: LEDE_OK (0) or a negative lede_status.  On error the
 *    decoding state (KV length, pending token, page table, the exit policy's
 *    confidence trace) is the one the call started from -- a call that fails
 *    after it has allocated pages or issued device work drains the stream
 *    and rewrites the device's copies of that state -- and lede_last_error()
 *    describes the failure.  A failed draft, verify or step also leaves no
 *    draft outstanding: the transition of Section 3.1 (draft, verify,
 *    commit) rolls back to the committed state.  KV entries past the
 *    committed length may have been overwritten; they are never read.  No
 *    exception crosses the ABI.
 *  - Device pointers are HIP device addresses on the current device; host
 *    pointers are ordinary process memory.  The caller owns every buffer it
 *    passes (weights staging, weight arena, KV pool, workspace) and the
 *    stream; the library owns only its host-side context.  No hot call
 *    allocates device memory.
 *  - `stream` is a hipStream_t passed as void*.  All device work is ordered
 *    on it.  Calls that return host values synchronise the stream.
 *  - A context is used by one host thread at a time.
 *
 * Model: Llama-style decoder -- RMSNorm, rotary position embedding
 * (rotate-half pairs (i, i + hd/2), angle pos * base^(-2i/hd)), grouped-query
 * attention (query head h reads KV head h / (n_heads / n_kv_heads)), SwiGLU
 * feed-forward, untied LM head.  Weights are bf16 or fp32; for bf16 models
 * the inputs of every linear layer and the cached K/V are rounded to bf16
 * (nearest-even) and everything else is accumulated in fp32.
 */
#ifndef LEDE_H
#define LEDE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lede_ctx lede_ctx;

typedef enum {
  LEDE_OK = 0,
  LEDE_E_ARG = -1,           /* bad argument: null pointer, size, range */
  LEDE_E_STATE = -2,         /* call not valid in the current decoding state */
  LEDE_E_KV_FULL = -3,       /* no free KV page left in the pool */
  LEDE_E_CTX_OVERFLOW = -4,  /* position would exceed max_ctx */
  LEDE_E_HIP = -5,           /* a HIP runtime call failed */
  LEDE_E_UNSUPPORTED = -6    /* shape outside what the kernels handle */
} lede_status;

enum { LEDE_DTYPE_F32 = 0, LEDE_DTYPE_BF16 = 1 };

/* Model shape, KV pool geometry and the Q-network's action grid. */
typedef struct {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps;     /* RMSNorm epsilon */
  float rope_base;   /* rotary base (10000, 500000, ...) */
  int32_t dtype;     /* LEDE_DTYPE_F32 or LEDE_DTYPE_BF16 */
  int32_t max_ctx;   /* largest KV length (positions) a sequence may reach */
  int32_t page_size; /* tokens per KV page; must be 64 */
  int32_t n_pages;   /* pages in the KV pool */
  int32_t qnet_hidden;         /* Q-network hidden width H (0: no Q-network) */
  int32_t n_exits, n_lengths;  /* action grid E x K, row-major (exit major) */
  int32_t exits[64];           /* candidate exit layers, ascending, 1..n_layers */
  int32_t lengths[16];         /* candidate draft lengths, 1..16 */
  int32_t k_max;               /* largest draft length any call may use (<= 15) */
  int32_t exit_qnet_hidden;    /* hidden width of the exit policy's 2-action Q-network
                                  (0: no exit policy; <= 1024); its candidate layers
                                  are exits[0 .. n_exits) */
} lede_config;

/* Tensor kinds for lede_load_tensor.  Logical layouts (row-major [out][in]):
 * EMBED, HEAD [vocab][d]; FINAL_NORM, ATTN_NORM, FFN_NORM [d];
 * WQ [n_heads*hd][d]; WK, WV [n_kv*hd][d]; WO [d][n_heads*hd];
 * WG, WU [ffn][d]; WD [d][ffn]; all in the model dtype.
 * QNET_W1 [H][d], QNET_B1 [H], QNET_W2 [E*K][H], QNET_B2 [E*K]: fp32.
 * EXIT_W1 [He][3], EXIT_B1 [He], EXIT_W2 [2][He], EXIT_B2 [2]: fp32, the
 * exit policy's Q-network (state: top-5 confidence, entropy, confidence
 * trace; outputs: continue, exit). */
typedef enum {
  LEDE_T_EMBED = 0, LEDE_T_FINAL_NORM, LEDE_T_HEAD,
  LEDE_T_ATTN_NORM, LEDE_T_WQ, LEDE_T_WK, LEDE_T_WV, LEDE_T_WO,
  LEDE_T_FFN_NORM, LEDE_T_WG, LEDE_T_WU, LEDE_T_WD,
  LEDE_T_QNET_W1, LEDE_T_QNET_B1, LEDE_T_QNET_W2, LEDE_T_QNET_B2,
  LEDE_T_EXIT_W1, LEDE_T_EXIT_B1, LEDE_T_EXIT_W2, LEDE_T_EXIT_B2
} lede_tensor;

/* Every tensor of the model at once, for lede_load_weights: device pointers
 * (non-owning; read on the stream of the call) in the logical layouts of
 * lede_load_tensor.  A null pointer leaves that tensor as it is, so a
 * caller short of device memory may load a model in several calls (for
 * example a range of layers at a time).  `layer` is a host array of
 * n_layers * LEDE_LAYER_TENSORS pointers for layers first_layer ..
 * first_layer + n_layers - 1, in the order attn_norm, wq, wk, wv, wo,
 * ffn_norm, wg, wu, wd. */
#define LEDE_LAYER_TENSORS 9
typedef struct {
  const void *embed, *final_norm, *head;
  int32_t first_layer, n_layers;
  const void* const* layer;
  const float *qnet_w1, *qnet_b1, *qnet_w2, *qnet_b2;  /* the (exit, length) Q-network */
  const float *exit_w1, *exit_b1, *exit_w2, *exit_b2;  /* the exit policy's 2-action Q-network */
} lede_weights;

/* An action of the agent: exit layer l* (1..L) and draft length k. */
typedef struct {
  int32_t l, k;
} lede_action;

/* One logged transition (Section 3.2 stores (s, a, r, s') tuples): the
 * action, what verification accepted, the tokens committed and the
 * Section 3.1.3 reward summed over the step's scored drafts. */
typedef struct {
  int32_t l;           /* exit layer used */
  int32_t k_req;       /* requested draft length */
  int32_t k_eff;       /* draft length after clamping to the tokens left */
  int32_t accepted;    /* accepted drafts a (0..k_eff) */
  int32_t n_emitted;   /* a + 1 */
  int32_t tokens[17];  /* committed tokens d_1..d_a, then the verify token */
  int32_t drafts[16];  /* the k_eff draft tokens */
  int32_t q_action;    /* argmax index of the Q-network (-1 if not run) */
  float q_max;         /* its Q-value */
  float reward;        /* Section 3.1.3 reward of this step */
  int32_t seq_len;     /* committed KV length after the step */
  int32_t pending;     /* next pending token (not yet in the cache) */
} lede_step_record;

/* Bytes of the three device regions the caller allocates for `cfg`:
 * the weight arena (repacked weights), the KV pool and the workspace.
 * Returns LEDE_E_UNSUPPORTED for shapes the kernels do not handle
 * (head_dim not 64/128, d_model or q_dim not a multiple of 32, d_model above
 * 8192, ffn_dim not a multiple of 8, page_size != 64, k_max > 15, ...). */
int lede_region_bytes(const lede_config* cfg, size_t* weight_bytes, size_t* kv_bytes,
                      size_t* workspace_bytes);

/* Create a context on the current device over caller-owned regions of at
 * least the sizes above (256-byte aligned).  Uploads the RoPE table to the
 * workspace (synchronous).  The page free list starts as 0..n_pages-1. */
int lede_create(const lede_config* cfg, void* weight_arena, size_t weight_bytes, void* kv_pool,
                size_t kv_bytes, void* workspace, size_t workspace_bytes, lede_ctx** out);

void lede_destroy(lede_ctx* ctx);

/* Text of the last error on this context (never NULL). */
const char* lede_last_error(const lede_ctx* ctx);

/* Repack one tensor from the caller's device buffer `src` (logical layout
 * above) into the weight arena (tiled for the kernels).  `layer` is ignored
 * for non-layer tensors.  `src` may be reused once the stream has passed
 * this call. */
int lede_load_tensor(lede_ctx* ctx, int32_t kind, int32_t layer, const void* src, void* stream);

/* Load the weights of the decoder the MDP runs on (Section 3.1: the states
 * are its hidden states, the actions its exit layers; Section 2.2: the draft
 * model is its own first layers with the shared final norm and LM head) and
 * of its Q-networks (Section 3.2), repacking every non-null tensor of *w as
 * lede_load_tensor does, in the order embed, final_norm, head, layers, Q-network,
 * exit policy.  LEDE_E_ARG on a null ctx or w, a layer range outside the
 * model or a null layer table with n_layers > 0; LEDE_E_STATE when a
 * Q-network tensor is given to a config without that network; LEDE_E_HIP on
 * a failed repack (tensors before it are loaded).  Stream-ordered; the
 * sources may be reused once the stream has passed the call. */
int lede_load_weights(lede_ctx* ctx, const lede_weights* w, void* stream);

/* Seed the KV page free list with a permutation of 0..n_pages-1 (allocation
 * pops the front).  Only valid while no page is allocated. */
int lede_set_free_list(lede_ctx* ctx, const int32_t* order, int32_t n);

/* Options: use_graphs -- replay each step shape as a captured HIP graph;
 * debug -- keep the fp32 logits of the last draft / verify / prefill head
 * and the Q-values for lede_debug_read.  Changing either drops the captured
 * graphs (a capture holds the debug mode it was made in). */
int lede_set_options(lede_ctx* ctx, int32_t use_graphs, int32_t debug);

/* Verify reuse (the self-speculative decoding the paper builds on, Section
 * 4.1 and Section 2.2: the draft layers are the model's own first layers).
 * With enable != 0, the verify of a step with k > 0 drafts at exit layer l*
 * runs only layers l*+1..L, on the layer-l* hidden states of rows [pending,
 * d_1 .. d_k]: the draft passes leave those of the pending token and d_1 ..
 * d_{k-1}, and one more one-row pass takes d_k through layers 1..l* (the
 * exit policy's last pass already does when it ended drafting); the KV the
 * draft passes wrote below l* is kept.  At batch 1 this reads the same weight
 * bytes as a full verify and saves FLOPs and launches.  The verify rows'
 * layers up to l* then come from the one-row kernels, so committed tokens
 * equal greedy decoding up to rounding, not bit for bit.  Steps with reuse
 * run eagerly (no graphs).  Applies to lede_step, lede_step_sampled,
 * lede_step_policy and lede_verify.  LEDE_E_STATE while a draft is
 * outstanding. */
int lede_set_verify_reuse(lede_ctx* ctx, int32_t enable);

/* Prefill (the paper does not describe it; decoding in Section 4.1 starts
 * from a prompt at batch 1): append n prompt tokens (host int32, each in
 * [0, vocab)) at positions seq_len .. seq_len+n-1 through all L layers in
 * 16-row passes of the verify kernels, writing their K/V; the full model's
 * argmax at the last row becomes the pending token and is returned in
 * *next_token (host), and its -log max p enters the confidence trace.
 * Valid when no draft is outstanding (LEDE_E_STATE); LEDE_E_ARG on a null
 * pointer, n < 1 or a token out of range; LEDE_E_CTX_OVERFLOW /
 * LEDE_E_KV_FULL when the positions do not fit.  Synchronises. */
int lede_prefill(lede_ctx* ctx, const int32_t* tokens, int32_t n, void* stream, int32_t* next_token);

/* Replace the pending token (teacher forcing / resume).  Synchronous. */
int lede_set_pending(lede_ctx* ctx, int32_t token, void* stream);

/* KV rollback (the paper leaves it implicit: a transition of Section 3.1
 * commits only the accepted drafts and the verify token, so the positions
 * of rejected drafts are dropped; this call exposes the same truncation for
 * resume and teacher forcing): roll the sequence back to new_len <= seq_len
 * positions, free the pages wholly past it (pushed to the front of the free
 * list in descending logical order) and discard any outstanding draft.  The
 * pending token is unchanged (lede_set_pending or lede_prefill sets the next
 * one).  LEDE_E_ARG when new_len is outside [0, seq_len]. */
int lede_truncate(lede_ctx* ctx, int32_t new_len, void* stream);

/* Draft k >= 1 tokens from the pending token by running layers 1..l (Section
 * 2.2) and the shared final RMSNorm + LM head + argmax, writing each draft's
 * K/V at layers 1..l.  drafts (host, nullable, [k]) receives the tokens
 * (then the call synchronises).  Leaves a draft outstanding for
 * lede_verify.  LEDE_E_STATE if a draft is already outstanding. */
int lede_draft(lede_ctx* ctx, int32_t l, int32_t k, void* stream, int32_t* drafts);

/* Verify (Section 1: the full model checks the k drafts in one parallel
 * pass; Section 4.1: greedy decoding, so a draft is kept while it equals the
 * full model's argmax) the outstanding drafts, or, with none, take one
 * autoregressive step: rows [pending, d_1..d_k] at positions
 * seq_len..seq_len+k through all L layers in one pass, greedy acceptance,
 * commit of d_1..d_a and the verify token y_a, KV truncation to seq_len+a+1.
 * Outputs (host): accepted a, tokens [k+1] (d_1..d_a, y_a), n_emitted = a+1,
 * verify (nullable, [k+1]) the full model's argmax of every row.  On failure
 * the outstanding draft is discarded with the rest of the transition.
 * LEDE_E_STATE without a pending token.  Synchronises. */
int lede_verify(lede_ctx* ctx, void* stream, int32_t* accepted, int32_t* tokens,
                int32_t* n_emitted, int32_t* verify);

/* One decoding step of the MDP (Section 3.1): the Q-network observes the
 * final-normed hidden state of the pending token at the smallest candidate
 * exit layer and scores the (exit, length) grid; the action is `forced` if
 * non-NULL (the Q-network still runs and is logged when log_qnet != 0), else
 * its argmax.  k is clamped to n_remaining - 1 (n_remaining = tokens still
 * to produce, >= 1); with k_eff = 0 the step is one autoregressive step.
 * Then draft, verify, accept, truncate; *rec is filled.  Synchronises once
 * at the end (twice when the Q-network chooses the action). */
int lede_step(lede_ctx* ctx, const lede_action* forced, int32_t log_qnet, int32_t n_remaining,
              void* stream, lede_step_record* rec);

/* Pipelined steps (the same step as lede_step with a forced action: drafts
 * and verify of Section 2.2, greedy acceptance and rollback of Section 3.3,
 * the Section 3.1.3 reward in the record): lede_step_submit enqueues the whole step on `stream` (drafts,
 * verify, acceptance, and the record's read-back into a host slot) and
 * returns without waiting; lede_step_collect waits for the oldest submitted
 * step and fills *rec exactly as lede_step would have.  The device holds the
 * committed length, the pending token and the page table, so step n+1 needs
 * nothing from step n's record and can be queued behind it: the host's work
 * between steps overlaps the GPU's.  Pages are allocated for the longest
 * acceptance of every step in flight and returned at collection, so a
 * submit can fail with LEDE_E_CTX_OVERFLOW or LEDE_E_KV_FULL where a
 * synchronous step would not (collect and retry, or step synchronously).
 * k is clamped to n_remaining - 1 with the n_remaining given at submission.
 * Errors: LEDE_E_ARG for a null ctx or action, n_remaining < 1, or l or k
 * out of range; LEDE_E_HIP when a launch or copy fails.  At
 * most LEDE_MAX_IN_FLIGHT steps may be outstanding (LEDE_E_STATE beyond, or
 * when collecting with none); while any is, every other decoding call
 * returns LEDE_E_STATE.  Submit and collect must use the same stream.
 * Graph replay, profiling, verify reuse and sampling are not pipelined
 * (LEDE_E_STATE when enabled). */
#define LEDE_MAX_IN_FLIGHT 2
int lede_step_submit(lede_ctx* ctx, const lede_action* action, int32_t log_qnet, int32_t n_remaining,
                     void* stream);
int lede_step_collect(lede_ctx* ctx, void* stream, lede_step_record* rec);

/* ---- speculative sampling (Section 4.1: sampling at temperature T, e.g.
 * 0.6, with speculative-sampling acceptance) -------------------------------
 * A step as lede_step, except that
 *  - draft i is drawn from softmax(z_draft / T) by inverse CDF in index
 *    order with uniforms[i-1];
 *  - draft i is kept while uniforms[16 + i - 1] * q(d) < p(d), q the draft
 *    distribution and p the full model's at that position;
 *  - the token after the kept drafts is drawn (uniforms[32]) from the
 *    normalised residual max(0, p - q) at the first rejection, else from p
 *    after the last draft.
 * uniforms: host pointer to LEDE_SAMPLE_STRIDE floats, each in [0, 1); the
 * caller owns the random numbers, so a step is a pure function of its
 * inputs.  temperature must be finite and > 0 (LEDE_E_ARG otherwise, state
 * unchanged).  rec->drafts holds the drawn drafts.  Not captured in graphs.
 * Synchronises as lede_step. */
#define LEDE_SAMPLE_SLOTS 16
#define LEDE_SAMPLE_STRIDE 33
int lede_step_sampled(lede_ctx* ctx, const lede_action* forced, int32_t log_qnet, int32_t n_remaining,
                      float temperature, const float* uniforms, void* stream, lede_step_record* rec);

/* ---- the paper's exit policy (Sections 3.1.1, 3.1.2, 3.3) -----------------
 * Needs exit_qnet_hidden > 0.  One greedy step: the pending token goes up
 * the candidate exit layers exits[0..n_exits) in order; at each, the state
 * (C_5 = mean -log p of the 5 most likely tokens, H = entropy in nats, both
 * of softmax(z) of that layer's shared final norm + LM head, and C_trace)
 * is scored by the exit Q-network, and the first 'exit' (forced at the last
 * candidate) fixes l*; draft 1 is that head's argmax.  Each further draft
 * pass at l* is scored the same way: 'exit' keeps its argmax as the next
 * draft, 'continue' ends drafting (its token is not kept); at most
 * min(12, k_max, n_remaining - 1) drafts.  Then verify, greedy acceptance,
 * truncation.  The host reads each decision back (one synchronisation per
 * decision).  rec->k_req = 12, rec->l = l*.  The decisions are read with
 * lede_debug_read(which = 4).
 *
 * C_trace is the mean of -log max p of the full model at the last 20
 * committed positions (0 while none): every prefill (its last row) and every
 * verify (the accepted rows and the bonus row) of a context with an exit
 * policy push to the window, whichever call made them.  lede_truncate does
 * not rewind it; lede_set_trace replaces it (host values, oldest first,
 * n <= 20), lede_get_trace reads it (n receives the count). */
int lede_step_policy(lede_ctx* ctx, int32_t n_remaining, void* stream, lede_step_record* rec);
int lede_set_trace(lede_ctx* ctx, const float* values, int32_t n, void* stream);
int lede_get_trace(lede_ctx* ctx, float* values /* [20] */, int32_t* n, void* stream);

/* ---- offline optimisation of the exit policy's Q-network ------------------
 * Section 3.2 (experience replay, n-step TD error to a target network,
 * greedy target action) with the training setup of Section 4.1 (Adam,
 * factorised Gaussian noisy layers, mini-batches, periodic target copies).
 * The network is the exit policy's 3 -> H -> 2 MLP; every weight w of it is
 * mu + sigma * f(eps_out) f(eps_in), f(x) = sgn(x) sqrt(|x|) (NoisyNet,
 * factorised), with standard normals supplied by the caller.
 *
 * Device memory, caller-owned, lede_dqn_region_bytes bytes (256-aligned):
 * online parameters [mu, sigma] (2P floats, P = 6H + 2, each set laid out W1
 * [H][3], b1 [H], W2 [2][H], b2 [2]), target parameters, Adam moments m and
 * v, and the replay ring (capacity slots of 8 floats: state C_5, H, C_trace,
 * action, reward, terminal, 2 unused).  The handle keeps host-side counters
 * (ring head and count, Adam step t); calls are stream-ordered and a handle
 * is not thread-safe.  Every entry returns a lede_status; errors leave the
 * handle unchanged and set lede_dqn_last_error. */
typedef struct lede_dqn lede_dqn;
typedef struct {
  int32_t hidden;    /* H, 1..128 (the exit policy's exit_qnet_hidden) */
  int32_t capacity;  /* replay slots, 2..2^24 */
  int32_t batch;     /* mini-batch, 1..256, batch * hidden <= 4096 */
  int32_t n_step;    /* n of the n-step target, 1..16 */
  float gamma;       /* discount, [0, 1] */
  float lr;          /* Adam step size, > 0 */
  float beta1, beta2;  /* Adam moment decays, [0, 1) */
  float adam_eps;    /* Adam epsilon, > 0 */
  float sigma0;      /* noisy-layer initial scale, >= 0 */
} lede_dqn_config;

/* Bytes of the device region for cfg; 0 for an invalid cfg. */
size_t lede_dqn_region_bytes(const lede_dqn_config* cfg);
/* Handle over a caller region of at least lede_dqn_region_bytes (device,
 * 256-byte aligned).  Allocates host memory only.  LEDE_E_ARG on a null
 * pointer, a small or misaligned region; LEDE_E_UNSUPPORTED on sizes outside
 * the ranges above. */
int lede_dqn_create(const lede_dqn_config* cfg, void* region, size_t bytes, lede_dqn** out);
void lede_dqn_destroy(lede_dqn* q);
const char* lede_dqn_last_error(const lede_dqn* q);

/* Initialisation (NoisyNet, factorised): mu = (2u - 1) / sqrt(p) from the
 * device uniforms u [P] in [0, 1), sigma = sigma0 / sqrt(p), p the layer's
 * fan-in (3, then H); target = online; Adam moments zero, t = 0; the ring is
 * emptied. */
int lede_dqn_init(lede_dqn* q, const float* u, void* stream);

/* Appends n >= 0 caller transitions (device [n][6] floats: state (3),
 * action 0 / 1, reward, terminal 0 / 1) in order; when n exceeds the
 * capacity only the last capacity land.  The newest overwrite the oldest. */
int lede_dqn_push(lede_dqn* q, const float* transitions, int32_t n, void* stream);

/* Appends the decisions of ctx's last lede_step_policy as transitions, in
 * decision order (Section 3.3): the state of the decision, the executed
 * action (the last candidate layer's forced exit is stored as exit), and the
 * Section 3.1.3 reward with lambda = (L - l*) / L: 'continue' -0.01; an exit
 * at a candidate layer scores draft 1, an exit after a further draft pass
 * scores the draft it keeps, +1 + lambda when that draft is among the
 * accepted ones, -2 + lambda otherwise.  The next transition's state is the
 * successor state.  episode_end != 0 marks the newest stored transition
 * terminal (the generation ended).  Must follow the policy step before any
 * other step, prefill, truncation or set_pending on ctx (LEDE_E_STATE
 * otherwise).  ctx and q share the device and stream order. */
int lede_dqn_record(lede_dqn* q, lede_ctx* ctx, int32_t episode_end, void* stream);

/* Marks the newest stored transition terminal (no-op on an empty ring). */
int lede_dqn_end_episode(lede_dqn* q, void* stream);

/* One learning update.  u: device [batch] uniforms, each m / 2^24 with an
 * integer m; sample b is the transition at position floor(m_b * n_valid /
 * 2^24) of the stored ones, oldest first, n_valid = count - n_step (a
 * transition is sampled once its n successors are stored; LEDE_E_STATE when
 * n_valid < 1).  noise: device [2][2H + 5] standard normals, eps_in (3) and
 * eps_out (H) of layer 1 then eps_in (H) and eps_out (2) of layer 2, for the
 * online network and then the target network.  Target y = sum_{k<n} gamma^k
 * r_{t+k} (stopping after a terminal transition) + gamma^n max_a'
 * Qbar(s_{t+n}, a') (only without a terminal); loss = mean (Q(s_t, a_t) -
 * y)^2; Adam (t += 1) on every mu and sigma.  loss (nullable host pointer)
 * receives the loss, which synchronises the stream. */
int lede_dqn_update(lede_dqn* q, const float* u, const float* noise, void* stream, float* loss);

/* Copies the online parameters into the target network. */
int lede_dqn_sync_target(lede_dqn* q, void* stream);

/* Writes the acting network into ctx's exit-policy Q-network: mu + sigma *
 * noise for noise = device [2H + 5] standard normals (exploration), or the
 * means for noise = NULL.  LEDE_E_STATE when ctx has no exit policy of width
 * H. */
int lede_dqn_act(lede_dqn* q, lede_ctx* ctx, const float* noise, void* stream);

/* Host read-back (synchronises): which = 0 online [mu, sigma], 1 target,
 * 2 Adam m, 3 Adam v (2P floats each); 4 the stored transitions, oldest
 * first, 6 floats each.  *count receives the number of floats (or
 * transitions for 4); LEDE_E_ARG when cap_floats is too small. */
int lede_dqn_read(lede_dqn* q, int32_t which, float* host, size_t cap_floats, int32_t* count, void* stream);

/* The agent's view of the KV state between transitions (Section 3.1: the
 * state is read at the committed length; the paper does not describe the
 * cache's layout): committed KV length, pending token and the page table,
 * logical page i -> pool page block_table[i] (host copies).  LEDE_E_ARG when
 * cap < the table's length (n_table receives it). */
int lede_get_kv_state(lede_ctx* ctx, int32_t* seq_len, int32_t* pending, int32_t* block_table,
                      int32_t cap, int32_t* n_table);

/* Debug read-back (needs set_options(debug=1)); which = 0: logits of the
 * last verify / prefill head launch [rows][vocab] fp32; 1: Q-values of the
 * last Q-network run [E*K]; 2: the Q-network's input state [d] fp32; 3:
 * logits of the last step's draft heads [rows][vocab]; 4 (debug mode not
 * needed): the exit-policy decisions of the last lede_step_policy, 8 floats
 * each (kind 0 = candidate layer / 1 = draft pass, layer or draft index,
 * C_5, H, C_trace, Q(continue), Q(exit), action).  *rows receives the row
 * count.  Synchronises. */
int lede_debug_read(lede_ctx* ctx, int32_t which, float* host, size_t cap_floats, int32_t* rows,
                    void* stream);

/* The next-token logits behind the last transition's decisions (Section
 * 3.1.1: the distribution at layer l comes from the shared head over that
 * layer's hidden state): which = LEDE_LOGITS_VERIFY, the full model's rows
 * of the last verify or prefill head [rows][vocab] fp32; LEDE_LOGITS_DRAFT,
 * the exit head's rows of the last step's drafts.  Needs
 * set_options(debug = 1) (LEDE_E_STATE); LEDE_E_ARG on a bad `which` or
 * cap_floats below rows * vocab.  Synchronises. */
enum { LEDE_LOGITS_VERIFY = 0, LEDE_LOGITS_DRAFT = 1 };
int lede_debug_logits(lede_ctx* ctx, int32_t which, float* host, size_t cap_floats, int32_t* rows, void* stream);

/* For callers that test failure handling: the (n_ops + 1)-th device
 * operation (kernel or graph launch, or copy) that a call on ctx issues from
 * now on fails with LEDE_E_HIP before it is issued; one-shot; n_ops < 0
 * disables it.  Nothing faults on the device. */
int lede_debug_inject_failure(lede_ctx* ctx, int32_t n_ops);

/* ---- timing for roofline reports ------------------------------------------
 * Level 1 brackets the draft phase and the verify phase of each lede_step
 * with HIP events on its stream.  Level 2 also has every kernel launch record
 * its own start / end events and attributes it to a kernel class (the extra
 * events slow the phases down, so phase rates are read at level 1).  Reading
 * synchronises, converts the event pairs to milliseconds and (reset != 0)
 * clears the totals.  bytes is the algorithmic HBM traffic of the launches:
 * weights and KV read once, plus activations in and out. */
enum {
  LEDE_K_LINEAR_VEC = 0,  /* one-row linear kernel, input row staged in LDS (draft path) */
  LEDE_K_LINEAR_MFMA,     /* matrix-core linear kernel, input rows read from global memory (verify / prefill path) */
  LEDE_K_ATTENTION,       /* paged attention partial + combine */
  LEDE_K_NORM,            /* RMSNorm rows */
  LEDE_K_QNET,            /* Q-network layers */
  LEDE_K_ACCEPT,          /* acceptance scan + KV truncation */
  LEDE_K_DRAFT_PHASE,     /* all draft passes of a step */
  LEDE_K_VERIFY_PHASE,    /* the verify pass + acceptance of a step */
  LEDE_K_LINEAR_VEC_GX,   /* one-row linear kernel, input row read from global memory (rows > 32 KiB) */
  LEDE_K_LINEAR_MFMA_LX,  /* matrix-core linear kernel, input rows staged in LDS (all rows <= 48 KiB) */
  LEDE_K_NCLASS
};
typedef struct {
  double ms;
  double bytes;
  int64_t launches;
} lede_prof_entry;

int lede_prof_enable(lede_ctx* ctx, int32_t level /* 0 off, 1 phases, 2 phases + launches; else LEDE_E_ARG */);
int lede_prof_read(lede_ctx* ctx, lede_prof_entry* out /* [LEDE_K_NCLASS] */, int32_t reset);

/* ---- single-operation entry points (kernel-level tests and tooling) ----- */

/* Bytes of a tiled weight matrix of N x K (dtype LEDE_DTYPE_*). */
size_t lede_op_tiled_bytes(int32_t dtype, int32_t N, int32_t K);

/* Repack a logical row-major N x K device matrix into the tiled layout the
 * linear kernels stream (16-row x 1 KiB tiles, K zero-padded). */
int lede_op_repack(int32_t dtype, const void* src, int32_t N, int32_t K, void* tiled, void* stream);

/* y[m][n] = sum_k W[n][k] x[m][k] (fp32 accumulate) for m < M <= 16 with a
 * tiled W (N multiple of 16, any K) and x [M][ldx] in the model dtype
 * (device).  The kernels read whole tiles: ldx must be at least K rounded up
 * to the tile width (32 bf16 / 16 fp32 columns; LEDE_E_ARG otherwise) and
 * the columns K..ldx-1 must hold finite values (they meet the tiles' zero
 * padding).  use_mfma = 0 requires M = 1 (the draft path's vector kernel); 1
 * uses the matrix-core kernel of the verify path. */
int lede_op_linear(int32_t dtype, const void* tiled, int32_t N, int32_t K, const void* x, int32_t ldx,
                   int32_t M, float* y, int32_t use_mfma, void* stream);

/* One draw from softmax(logits / temperature) by inverse CDF in index order
 * with the uniform u in [0, 1), as the sampled step draws its drafts: logits
 * is a device fp32 row of V, *token (host) receives the index.  Allocates a
 * 16-byte device buffer and synchronises (a test and tooling entry point).
 * LEDE_E_ARG on a null pointer, V < 1, temperature not finite and > 0, or u
 * outside [0, 1). */
int lede_op_sample(const float* logits, int32_t V, float temperature, float u, int32_t* token, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops and harnesses that forbid hipMalloc): the draws of
 * lede_op_sample for n_rows rows at once, with no allocation.  Row r is the
 * device fp32 row logits + r * ld (V used entries, ld >= V), drawn with the
 * host uniform u[r] in [0, 1); tokens (host, [n_rows]) receives the draws.
 * The draws' keys live in a library-owned static device array of 32 keys
 * (2 KiB per device, held until the process ends): n_rows above 32 is
 * LEDE_E_ARG, as are null pointers, V < 1, ld < V, a temperature that is not
 * finite and > 0 and a uniform outside [0, 1).  Every call on a device
 * shares that device's array: calls that overlap on one GPU (other threads,
 * other streams) race.  Synchronises the stream. */
int lede_op_sample_noalloc(const float* logits, int32_t n_rows, int32_t ld, int32_t V, float temperature,
                           const float* u, int32_t* tokens, void* stream);

/* Achievable HBM read bandwidth: reads `bytes` (a multiple of 16, > 0) of the
 * device buffer src once, with the same non-temporal 16-byte loads the
 * linear kernels use for weights, on `grid` (1..65535) blocks of 256 threads;
 * one uint32 per block goes to the device buffer sink [grid] so that no load
 * is dropped.  kernel_ms (nullable host pointer): when given, the dispatch
 * records its own start / end events, the call waits for them and stores the
 * kernel's duration.  LEDE_E_ARG on bad arguments, LEDE_E_HIP on a HIP error. */
int lede_op_read_probe(const void* src, size_t bytes, uint32_t* sink, int32_t grid, void* stream,
                       float* kernel_ms);

/* The one-row linear kernel's memory access alone: reads n_groups (1..65535)
 * groups of `tiles` (>= 1) contiguous 1 KiB weight tiles from the device
 * buffer src (n_groups * tiles KiB) with that kernel's load structure, one
 * group per block of 8 wavefronts, 4 non-temporal 16-byte loads per lane in
 * flight; one uint32 per block goes to the device buffer sink [n_groups].
 * The per-launch read rate of a matrix shape without any arithmetic, to set
 * the kernel's times against.  kernel_ms as for lede_op_read_probe.
 * LEDE_E_ARG on bad arguments, LEDE_E_HIP on a HIP error. */
int lede_op_read_groups(const void* src, int32_t n_groups, int32_t tiles, uint32_t* sink, void* stream,
                        float* kernel_ms);

#ifdef __cplusplus
}
#endif

#endif /* LEDE_H */
