// Acceptance and commit of a step: greedy prefix match, and speculative
// sampling at temperature T (gfx950).
#include "device.h"

namespace lede {

// ---- greedy acceptance scan + commit + KV truncation --------------------------

// Commit of a verified step: the record, the new length, the pending token
// and the device block table (pages wholly past the committed length go back
// to the pool).  One thread.
__device__ void commit_step(const AcceptArgs& a, int acc, int y) {
  TokenSrc dk = {nullptr, a.dkeys};
  const int k = a.k;
  const int c = *a.seq_len;
  const int c_new = c + acc + 1;
  for (int i = 0; i < acc; ++i) a.record[4 + i] = dk.get(i + 1);
  a.record[4 + acc] = y;
  for (int i = 0; i < k; ++i) a.record[24 + i] = dk.get(i + 1);
  a.record[0] = acc;
  a.record[1] = acc + 1;
  a.record[2] = c_new;
  a.record[3] = y;
  *a.seq_len = c_new;
  a.pending_out[0] = (uint64_t)(0xFFFFFFFFu - (uint32_t)y);
  const int keep = (c_new + 63) / 64, used = (c + k + 1 + 63) / 64;
  for (int j = keep; j < used; ++j) a.block_table[j] = -1;
}

__global__ void k_accept(AcceptArgs a) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  TokenSrc dk = {nullptr, a.dkeys}, vk = {nullptr, a.vkeys};
  const int k = a.k;
  int acc = 0;
  while (acc < k && dk.get(acc + 1) == vk.get(acc)) ++acc;
  commit_step(a, acc, vk.get(acc));
}

// ---- speculative sampling -------------------------------------------------------
// One block of SB threads per row.  Thread t owns the contiguous chunk
// [t C, (t+1) C) of the vocabulary (C = ceil(V / SB) rounded up to 4) and
// requests it in batches of CB elements (vector loads when the row is 16-byte
// aligned).  A thread sums its chunk in index order; the chunk sums are
// combined by one block scan in thread order.  Every sum therefore runs in
// one fixed order, and a row's statistics and draw depend on nothing but its
// inputs.

constexpr int SB = 1024, SW = SB / 64, CB = 16;

__device__ __forceinline__ int chunk_len(int V) { return ((V + SB - 1) / SB + 3) / 4 * 4; }

// Elements [b, b + CB) of row z (zero from `end` on) into r; b is a multiple
// of 4, so a 16-byte aligned row takes vector loads.
__device__ __forceinline__ void load_batch(const float* z, int end, int b, float (&r)[CB]) {
  if (((uintptr_t)z & 15) == 0 && b + CB <= end) {
#pragma unroll
    for (int j = 0; j < CB; j += 4) *(float4*)&r[j] = *(const float4*)(z + b + j);
  } else {
#pragma unroll
    for (int j = 0; j < CB; ++j) r[j] = b + j < end ? z[b + j] : 0.f;
  }
}

__device__ __forceinline__ float block_max_f(float v, float* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float m = red[0];
  for (int w = 1; w < SW; ++w) m = fmaxf(m, red[w]);
  return m;
}

__device__ __forceinline__ int block_max_i(int v, int* red) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int m = red[0];
  for (int w = 1; w < SW; ++w) m = max(m, red[w]);
  return m;
}

// Exclusive prefix of v over the threads in index order, and the total.
__device__ __forceinline__ float block_excl_scan(float v, float* red, float& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float x = v;
  for (int o = 1; o < 64; o <<= 1) {
    const float y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  float ex = __shfl_up(x, 1);
  if (lane == 0) ex = 0.f;
  __syncthreads();
  if (lane == 63) red[wave] = x;
  __syncthreads();
  float base = 0.f;
  for (int w = 0; w < wave; ++w) base += red[w];
  total = base;
  for (int w = wave; w < SW; ++w) total += red[w];
  return base + ex;
}

// Sum of f(v, z1[v], z2[v]) over this thread's chunk, in index order.
template <typename F>
__device__ float chunk_sum(F f, const float* z1, const float* z2, int V) {
  const int C = chunk_len(V), v0 = threadIdx.x * C, v1 = min(V, v0 + C);
  float s = 0.f;
  for (int b = v0; b < v1; b += CB) {
    float r1[CB], r2[CB];
    load_batch(z1, v1, b, r1);
    if (z2) load_batch(z2, v1, b, r2);
#pragma unroll
    for (int j = 0; j < CB; ++j)
      if (b + j < v1) s += f(r1[j], z2 ? r2[j] : 0.f);
  }
  return s;
}

// Inverse-CDF draw from the non-negative weights f(z1[v], z2[v]): the first
// index whose running sum exceeds u * total, else (rounding) the last index
// of positive weight in the owning chunk.  Returns -1 when every weight is 0.
template <typename F>
__device__ int block_draw(F f, const float* z1, const float* z2, int V, float u, float* red, int* ired) {
  const float s = chunk_sum(f, z1, z2, V);
  float total;
  const float pre = block_excl_scan(s, red, total);
  const float thr = u * total;
  const int owner = block_max_i((s > 0.f && pre <= thr) ? (int)threadIdx.x : -1, ired);
  __shared__ int tok;
  if ((int)threadIdx.x == owner) {
    const int C = chunk_len(V), v0 = owner * C, v1 = min(V, v0 + C);
    float acc = pre;
    int hit = -1, last = -1;
    for (int b = v0; b < v1 && hit < 0; b += CB) {
      float r1[CB], r2[CB];
      load_batch(z1, v1, b, r1);
      if (z2) load_batch(z2, v1, b, r2);
      for (int j = 0; j < CB && b + j < v1; ++j) {
        const float w = f(r1[j], z2 ? r2[j] : 0.f);
        if (w > 0.f) last = b + j;
        acc += w;
        if (acc > thr) {
          hit = b + j;
          break;
        }
      }
    }
    tok = hit >= 0 ? hit : last;
  }
  if (threadIdx.x == 0 && owner < 0) tok = -1;
  __syncthreads();
  return tok;
}

// (max, sum of exp((z - max) * inv_t)) of one row.
__device__ float2 row_stats(const float* z, int V, float inv_t, float* red) {
  float m = -INFINITY;
  {
    const int C = chunk_len(V), v0 = threadIdx.x * C, v1 = min(V, v0 + C);
    for (int b = v0; b < v1; b += CB) {
      float r[CB];
      load_batch(z, v1, b, r);
#pragma unroll
      for (int j = 0; j < CB; ++j)
        if (b + j < v1) m = fmaxf(m, r[j]);
    }
  }
  m = block_max_f(m, red);
  const float s = chunk_sum([&](float x, float) { return expf((x - m) * inv_t); }, z, nullptr, V);
  float total;
  (void)block_excl_scan(s, red, total);
  __syncthreads();
  return make_float2(m, total);
}

__global__ __launch_bounds__(SB) void k_sample(SampleArgs a) {
  __shared__ float red[SW];
  __shared__ int ired[SW];
  const float2 st = row_stats(a.logits, a.vocab, a.inv_t, red);
  const float m = st.x, it = a.inv_t;
  const float u = a.u ? a.u[a.u_index] : a.u_imm;
  const int tok = block_draw([&](float x, float) { return expf((x - m) * it); }, a.logits, nullptr, a.vocab, u,
                             red, ired);
  if (threadIdx.x == 0) {
    *a.key_out = (uint64_t)(0xFFFFFFFFu - (uint32_t)tok);
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
    const float2 st = row_stats(a.vlogits + (size_t)j * V, V, it, red);
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
