// Acceptance and commit of a step: greedy prefix match, and speculative
// sampling at temperature T (gfx950).
#include "rowops.h"

namespace lede {

// ---- greedy acceptance scan + commit + KV truncation --------------------------

// Commit of a verified step: the record, the new length, the pending token
// and the device block table (pages wholly past the committed length go back
// to the pool).  One thread.  drafts: the decoded drafts (index 1..k) if
// the caller has them, else they are decoded from the keys here.
__device__ void commit_step(const AcceptArgs& a, int acc, int y, const int* drafts = nullptr) {
  TokenSrc dk = {nullptr, a.dkeys};
  const int k = a.k;
  const int c = *a.seq_len;
  const int c_new = c + acc + 1;
  for (int i = 0; i < acc; ++i) a.record[4 + i] = drafts ? drafts[i + 1] : dk.get(i + 1);
  a.record[4 + acc] = y;
  for (int i = 0; i < k; ++i) a.record[24 + i] = drafts ? drafts[i + 1] : dk.get(i + 1);
  a.record[0] = acc;
  a.record[1] = acc + 1;
  a.record[2] = c_new;
  a.record[3] = y;
  *a.seq_len = c_new;
  key_store_token(a.pending_out, 0, y);
  const int keep = (c_new + 63) / 64, used = (c + k + 1 + 63) / 64;
  for (int j = keep; j < used; ++j) a.block_table[j] = -1;
}

// Lanes 0..k decode verify row i's argmax and draft i at once (each the
// largest of a key's slot words); lane 0 then scans for the first mismatch
// and commits.  k is at most 15 (the configuration's limit on k_max).
__global__ void k_accept(AcceptArgs a) {
  constexpr int KM = 15;
  __shared__ int dtok[KM + 1], vtok[KM + 1];
  const int i = threadIdx.x, k = min(a.k, KM);
  if (blockIdx.x != 0) return;
  if (i <= k) {
    vtok[i] = TokenSrc{nullptr, a.vkeys}.get(i);
    dtok[i] = i ? TokenSrc{nullptr, a.dkeys}.get(i) : 0;
  }
  __syncthreads();
  if (i != 0) return;
  int acc = 0;
  while (acc < k && dtok[acc + 1] == vtok[acc]) ++acc;
  commit_step(a, acc, vtok[acc], dtok);
}

// ---- speculative sampling -------------------------------------------------------

__global__ __launch_bounds__(SB) void k_sample(SampleArgs a) {
  __shared__ float red[SW];
  __shared__ int ired[SW];
  const float u = a.u ? a.u[a.u_index] : a.u_imm;
  const float it = a.inv_t;
  float2 st;
  int tok;
  if (a.gstats) {  // from the head's group statistics: no pass over the row
    st = group_row_stats(a.gstats, a.n_groups, it, red);
    tok = group_draw(a.gstats, a.logits, a.n_groups, st.x, it, u, red, ired);
  } else {
    st = row_stats(a.logits, a.vocab, it, red);
    const float m = st.x;
    tok = block_draw([&](float x, float) { return expf((x - m) * it); }, a.logits, nullptr, a.vocab, u, red, ired);
  }
  if (threadIdx.x == 0) {
    key_store_token(a.key_out, 0, tok);
    if (a.stats_out) {
      a.stats_out[0] = st.x;
      a.stats_out[1] = st.y;
    }
  }
}

// Speculative-sampling acceptance of the k drafts, the draw of the token
// after them, and the commit.
__global__ __launch_bounds__(SB) void k_accept_sampled(SampledAcceptArgs a) {
  __shared__ float red[SW];
  __shared__ int ired[SW];
  __shared__ float vst[2 * (SAMPLE_SLOTS + 1)];
  __shared__ int acc_s;
  const int k = a.acc.k, V = a.vocab;
  const float it = a.inv_t;
  for (int j = 0; j <= k; ++j) {
    const float2 st = a.vgstats ? group_row_stats(a.vgstats + (size_t)j * a.n_groups, a.n_groups, it, red)
                                : row_stats(a.vlogits + (size_t)j * V, V, it, red);
    if (threadIdx.x == 0) {
      vst[2 * j] = st.x;
      vst[2 * j + 1] = st.y;
    }
  }
  if (threadIdx.x == 0) {
    TokenSrc dk = {nullptr, a.acc.dkeys};
    int acc = 0;
    while (acc < k) {
      const int d = (int)min((unsigned)dk.get(acc + 1), (unsigned)(V - 1));  // non-finite logits aside, in range
      const float p = expf((a.vlogits[(size_t)acc * V + d] - vst[2 * acc]) * it) / vst[2 * acc + 1];
      const float q = expf((a.dlogits[(size_t)acc * V + d] - a.dstats[2 * acc]) * it) / a.dstats[2 * acc + 1];
      if (!(a.u[SAMPLE_SLOTS + acc] * q < p)) break;
      ++acc;
    }
    acc_s = acc;
  }
  __syncthreads();
  const int acc = acc_s;
  const float* zp = a.vlogits + (size_t)acc * V;
  const float mp = vst[2 * acc], sp = vst[2 * acc + 1];
  const float ur = a.u[2 * SAMPLE_SLOTS];
  int y;
  if (acc < k) {
    const float* zq = a.dlogits + (size_t)acc * V;
    const float mq = a.dstats[2 * acc], sq = a.dstats[2 * acc + 1];
    y = block_draw([&](float xp, float xq) { return fmaxf(expf((xp - mp) * it) / sp - expf((xq - mq) * it) / sq, 0.f); },
                   zp, zq, V, ur, red, ired);
    // rounding can leave no positive residual weight; the target row is
    // then the residual's only possible limit
    if (y < 0) y = block_draw([&](float x, float) { return expf((x - mp) * it); }, zp, nullptr, V, ur, red, ired);
  } else if (a.vgstats) {
    y = group_draw(a.vgstats + (size_t)acc * a.n_groups, zp, a.n_groups, mp, it, ur, red, ired);
  } else {
    y = block_draw([&](float x, float) { return expf((x - mp) * it); }, zp, nullptr, V, ur, red, ired);
  }
  if (threadIdx.x == 0) commit_step(a.acc, acc, y < 0 ? 0 : y);  // y < 0 only for non-finite logits
}

// ---- launchers ----------------------------------------------------------------

hipError_t launch_accept(const AcceptArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_accept, dim3(1), dim3(64), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_sample(const SampleArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_sample, dim3(1), dim3(SB), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_accept_sampled(const SampledAcceptArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_accept_sampled, dim3(1), dim3(SB), 0, s, a);
  return hipGetLastError();
}

}  // namespace lede
