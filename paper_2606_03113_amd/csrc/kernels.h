// Internal interface between the runtime (runtime.cpp) and the gfx950
// kernels (linear.hip, norm.hip, attention.hip, accept.hip, policy.hip,
// dqn.hip, misc.hip).  Not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "linear.h"

namespace lede {

struct NormArgs {
  int M, d, ldh, ldx;
  float* h;                // fp32 residual rows
  const void* gain; float eps;
  int embed; const void* embed_w; TokenSrc tok;  // h[m] = embed[tok(m)] first
  int vocab;
  void* x;                 // output rows
  int f32_out;             // 1: fp32 output, not rounded
  uint64_t* zero_keys; int n_zero_keys;
};

struct AttnArgs {
  const float* q; int ldq;        // [M][nq*hd] (rotated)
  const void* kcache; const void* vcache;
  int layer, n_pages, nq, nkv, hd, M;
  const int32_t* block_table; const int32_t* seq_len; int pos_off;
  int n_split;                     // blocks per (kv head, row slice); chunks strided
  int rows_per_block;              // <= 16 query rows (m, head-in-group) per block
  int max_chunks;
  float* part;                     // [M][nq][max_chunks][hd + 2]
  void* out; int ldo;              // combine output [M][nq*hd], model dtype
  int mfma;                        // bf16: partials on the matrix cores (rows of verify, prefill, AR)
};

struct QnetOutArgs {
  const float* hid; int H;
  const float* w2; const float* b2; int A;
  float* qv; int32_t* action;     // action[0] = argmax, action[1] = bits of max
};

struct AcceptArgs {
  const uint64_t* dkeys;   // [0] pending, [1..k] drafts
  const uint64_t* vkeys;   // [0..k] verify argmax
  int k;
  int32_t* seq_len;
  int32_t* block_table;
  uint64_t* pending_out;   // dkeys[0]
  int32_t* record;         // [0] a, [1] n_emitted, [2] seq_len, [3] pending, [4..] tokens, [24..] drafts
};

// Speculative sampling at temperature T (inv_t = 1 / T).  Draft and verify
// logits are fp32 rows of `vocab`; stats rows hold (max logit, sum of
// exp((z - max) * inv_t)).  Uniforms per step: drafts [0, 16), acceptance
// tests [16, 32), residual / bonus draw [32].
constexpr int SAMPLE_SLOTS = 16;
struct SampleArgs {
  const float* logits; int vocab; float inv_t;
  const float* u; int u_index;   // the draw uses u[u_index] (u_imm when u is null)
  float u_imm;
  uint64_t* key_out;             // argmax-style key of the drawn token
  float* stats_out;              // (max, sum) of the row
  const float2* gstats;          // optional: the row's 16-token group statistics (vocab = 16 n_groups)
  int n_groups;
};
struct SampledAcceptArgs {
  AcceptArgs acc;                // keys, k, commit targets
  const float* dlogits;          // [k][vocab] draft rows (row i drew draft i+1)
  const float* dstats;           // [k][2]
  const float* vlogits;          // [k+1][vocab]
  int vocab; float inv_t;
  const float* u;                // the step's uniforms
  const float2* vgstats;         // optional: [k+1][n_groups] group statistics of the verify rows
  int n_groups;
};

// The paper's exit policy: state features of a next-token distribution and
// the 2-action Q-network (rows of w2: continue, exit), and the window of
// committed confidences the state's trace feature averages.
constexpr int POLICY_TOPK = 5, POLICY_TRACE = 20, POLICY_MAX_DRAFT = 12, POLICY_LOG = 8;
struct ExitPolicyArgs {
  const float* logits; int vocab;
  const float* w1; const float* b1; const float* w2; const float* b2; int hidden;  // fp32, W1 [H][3], W2 [2][H]
  const float* trace; const int32_t* trace_state;  // ring [POLICY_TRACE]; state[0] = count
  float* out;                                      // [POLICY_LOG]: kind, index, C_k, H, C_trace, Q0, Q1, action
  float kind, index;
};
struct TracePushArgs {
  const float* logits; int vocab; int ld;          // rows of logits, row stride
  const int32_t* record;                           // rows = record[0] + 1 when set, else n_rows
  int n_rows;
  float* trace; int32_t* trace_state;              // state[0] = count, state[1] = next slot
  float* backup;                                   // [POLICY_TRACE + 2]: the ring and state before the push
};

// Offline optimisation of the exit policy's Q-network (3 -> H -> 2 MLP with
// factorised noisy layers).  A parameter set is one flat fp32 vector: W1
// [H][3], b1 [H], W2 [2][H], b2 [2] (P = 6H + 2 entries); theta = [mu, sigma]
// (2P).  One network's noise is 3 + 2H + 2 standard normals: eps_in and
// eps_out of layer 1, then of layer 2.  A replay slot is 8 floats: state (3),
// action, reward, terminal, 2 unused.
constexpr int DQN_SLOT = 8, DQN_MAX_HIDDEN = 128, DQN_MAX_BATCH = 256, DQN_MAX_BH = 4096, DQN_MAX_N = 16;
constexpr int DQN_THREADS = 256;
__host__ __device__ inline int dqn_params(int H) { return 6 * H + 2; }
__host__ __device__ inline int dqn_noise(int H) { return 2 * H + 5; }
struct DqnInitArgs {
  const float* u; int H; float sigma0;
  float* theta; float* target; float* m; float* v;
};
struct DqnUpdateArgs {
  float* theta; const float* target; float* m; float* v;
  const float* ring; int capacity, oldest, n_valid;
  const float* u;                  // [B] uniforms m / 2^24
  const float* noise;              // [2][3 + 2H + 2]: online, then target
  int H, B, n;
  float gamma, gamma_n, lr, beta1, beta2, eps, bc1, bc2;  // bc = 1 - beta^t
  float* loss_out;                 // [1]
};
struct DqnRecordArgs {
  const float* log; int n_dec;     // POLICY_LOG floats per decision
  int l_star, accepted;
  float r_accept, r_reject, r_continue;
  float* ring; int capacity, head;
  int end_episode, prev_newest;    // prev_newest: slot marked terminal when n_dec = 0 (-1: none)
};
struct DqnPushArgs {
  const float* src; int n;         // [n][6]: state (3), action, reward, terminal
  float* ring; int capacity, head;
};
struct DqnActArgs {
  const float* theta; const float* noise;  // noise may be null: the means
  int H;
  float *w1, *b1, *w2, *b2;
};

// Launchers (one per kernel family, next to its kernels).  All return
// hipError_t of the launch.
hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t s);
hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s);
hipError_t launch_qnet_out(const QnetOutArgs& a, hipStream_t s);
hipError_t launch_accept(const AcceptArgs& a, hipStream_t s);
hipError_t launch_sample(const SampleArgs& a, hipStream_t s);
hipError_t launch_exit_policy(const ExitPolicyArgs& a, hipStream_t s);
hipError_t launch_trace_push(const TracePushArgs& a, hipStream_t s);
hipError_t launch_accept_sampled(const SampledAcceptArgs& a, hipStream_t s);
hipError_t launch_fill_u64(uint64_t* p, uint64_t v, int n, hipStream_t s);
// Reads bytes (a multiple of 16) of src once; e0 / e1 (may be null) bracket
// the kernel's execution.
hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, int grid, hipStream_t s,
                             hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// Reads n_groups groups of `tiles` weight tiles (contiguous) with the one-row
// linear kernel's load structure, one group per block.
hipError_t launch_read_groups(const void* src, int n_groups, int tiles, uint32_t* sink, hipStream_t s,
                              hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t launch_set_token(uint64_t* keys, int idx, int token, hipStream_t s);
hipError_t launch_dqn_init(const DqnInitArgs& a, hipStream_t s);
hipError_t launch_dqn_update(const DqnUpdateArgs& a, hipStream_t s);
hipError_t launch_dqn_record(const DqnRecordArgs& a, hipStream_t s);
hipError_t launch_dqn_push(const DqnPushArgs& a, hipStream_t s);
hipError_t launch_dqn_copy(const float* src, float* dst, int n, hipStream_t s);
hipError_t launch_dqn_act(const DqnActArgs& a, hipStream_t s);


}  // namespace lede
