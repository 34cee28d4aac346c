// The paper's exit policy on the device (gfx950): the state of a candidate
// exit layer (Section 3.1.1) from that layer's next-token logits, the
// 2-action Q-network (Section 3.2), and the window of committed confidences.
#include "rowops.h"

namespace lede {

// Keep the POLICY_TOPK largest values seen, in descending order: x bubbles
// down the list (static indices, no branches).
__device__ __forceinline__ void top_insert(float (&t)[POLICY_TOPK], float x) {
#pragma unroll
  for (int j = 0; j < POLICY_TOPK; ++j) {
    const float hi = fmaxf(t[j], x), lo = fminf(t[j], x);
    t[j] = hi;
    x = lo;
  }
}

// One block: features (top-k confidence, entropy, trace) of softmax(logits)
// at temperature 1, Q-values and the greedy action (ties: continue).
//   C_k = log S - mean_{top k} (z - m),  H = log S - sum e (z - m) / S,
// with m the max logit, e = exp(z - m), S = sum e.
__global__ __launch_bounds__(SB) void k_exit_policy(ExitPolicyArgs a) {
  __shared__ float red[SW];
  __shared__ float tops[SW][POLICY_TOPK];
  __shared__ float hid[SB];
  const float* z = a.logits;
  const int V = a.vocab;
  const int C = chunk_len(V), v0 = threadIdx.x * C, v1 = min(V, v0 + C);
  // pass 1 over this thread's chunk (batched loads): the max and the top k
  float m = -INFINITY;
  float t[POLICY_TOPK];
#pragma unroll
  for (int j = 0; j < POLICY_TOPK; ++j) t[j] = -INFINITY;
  for (int b = v0; b < v1; b += CB) {
    float r[CB];
    load_batch(z, v1, b, r);
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const float x = b + j < v1 ? r[j] : -INFINITY;
      m = fmaxf(m, x);
      top_insert(t, x);
    }
  }
  m = block_max_f(m, red);
  // the top-k lists of a wavefront merged pairwise through shuffles, then
  // the waves' lists by one thread below
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    float u[POLICY_TOPK];
#pragma unroll
    for (int j = 0; j < POLICY_TOPK; ++j) u[j] = __shfl_xor(t[j], o);
#pragma unroll
    for (int j = 0; j < POLICY_TOPK; ++j) top_insert(t, u[j]);
  }
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int j = 0; j < POLICY_TOPK; ++j) tops[threadIdx.x >> 6][j] = t[j];
  // pass 2: S = sum e and W = sum e (z - m), each in index order
  float s_e = 0.f, s_w = 0.f;
  for (int b = v0; b < v1; b += CB) {
    float r[CB];
    load_batch(z, v1, b, r);
#pragma unroll
    for (int j = 0; j < CB; ++j)
      if (b + j < v1) {
        const float d = r[j] - m, e = expf(d);
        s_e += e;
        s_w += e * d;
      }
  }
  float S, wtot;
  (void)block_excl_scan(s_e, red, S);
  __syncthreads();
  (void)block_excl_scan(s_w, red, wtot);
  __syncthreads();
  __shared__ float state[3];
  if (threadIdx.x == 0) {
    float t[POLICY_TOPK];
#pragma unroll
    for (int j = 0; j < POLICY_TOPK; ++j) t[j] = -INFINITY;
    for (int i = 0; i < SW; ++i)
#pragma unroll
      for (int j = 0; j < POLICY_TOPK; ++j) top_insert(t, tops[i][j]);
    const int kk = min(POLICY_TOPK, V);
    float ts = 0.f;
    for (int j = 0; j < kk; ++j) ts += t[j] - m;
    const float logS = logf(S);
    const int n = min(a.trace_state[0], POLICY_TRACE);
    float tr = 0.f;
    for (int i = 0; i < n; ++i) tr += a.trace[i];
    state[0] = logS - ts / (float)kk;
    state[1] = logS - wtot / S;
    state[2] = n ? tr / (float)n : 0.f;
  }
  __syncthreads();
  for (int h = threadIdx.x; h < a.hidden; h += SB) {
    float x = a.b1[h];
    for (int i = 0; i < 3; ++i) x = fmaf(a.w1[h * 3 + i], state[i], x);
    hid[h] = fmaxf(x, 0.f);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float q[2];
    for (int o = 0; o < 2; ++o) {
      float x = a.b2[o];
      for (int h = 0; h < a.hidden; ++h) x = fmaf(a.w2[o * a.hidden + h], hid[h], x);
      q[o] = x;
    }
    a.out[0] = a.kind;
    a.out[1] = a.index;
    a.out[2] = state[0];
    a.out[3] = state[1];
    a.out[4] = state[2];
    a.out[5] = q[0];
    a.out[6] = q[1];
    a.out[7] = q[1] > q[0] ? 1.f : 0.f;
  }
}

// Push -log max p (= log S at temperature 1) of each committed row into the
// window, oldest first.
__global__ __launch_bounds__(SB) void k_trace_push(TracePushArgs a) {
  __shared__ float red[SW];
  const int n = a.record ? a.record[0] + 1 : a.n_rows;
  // the window as it was, kept so that a failed call can be rolled back
  static_assert(SB >= POLICY_TRACE, "one thread per slot");
  if (threadIdx.x < POLICY_TRACE) a.backup[threadIdx.x] = a.trace[threadIdx.x];
  if (threadIdx.x < 2) ((int32_t*)(a.backup + POLICY_TRACE))[threadIdx.x] = a.trace_state[threadIdx.x];
  __syncthreads();
  for (int j = 0; j < n; ++j) {
    const float2 st = row_stats(a.logits + (size_t)j * a.ld, a.vocab, 1.f, red);
    if (threadIdx.x == 0) {
      const int slot = a.trace_state[1];
      a.trace[slot] = logf(st.y);
      a.trace_state[1] = (slot + 1) % POLICY_TRACE;
      a.trace_state[0] = min(a.trace_state[0] + 1, POLICY_TRACE);
    }
    __syncthreads();
  }
}

hipError_t launch_exit_policy(const ExitPolicyArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_exit_policy, dim3(1), dim3(SB), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_trace_push(const TracePushArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_trace_push, dim3(1), dim3(SB), 0, s, a);
  return hipGetLastError();
}

}  // namespace lede
