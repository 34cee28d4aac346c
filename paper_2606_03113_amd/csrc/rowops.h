// Block-level row reductions over a vocabulary-sized fp32 row (gfx950):
// statistics, fixed-order sums and inverse-CDF draws, used by the sampling
// and exit-policy kernels.
#pragma once

#include "device.h"

namespace lede {

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
__device__ inline float2 row_stats(const float* z, int V, float inv_t, float* red) {
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

// ---- the same from per-group statistics --------------------------------------
// A row of V = 16 G tokens summarised by its groups' (max m_g, sum of
// exp((z - m_g) * inv_t)): thread t owns the contiguous groups
// [t D, (t+1) D) (D = ceil(G / SB)), and every sum runs in group order within
// a thread and in thread order across the block.

__device__ __forceinline__ int group_chunk(int G) { return (G + SB - 1) / SB; }

// Weight of group g relative to the row maximum mx: sum over its tokens of
// exp((z - mx) * inv_t).
__device__ __forceinline__ float group_weight(float2 st, float mx, float inv_t) {
  return st.x > -INFINITY ? st.y * expf((st.x - mx) * inv_t) : 0.f;
}

// (max, sum of exp((z - max) * inv_t)) of the row from its group statistics.
__device__ inline float2 group_row_stats(const float2* gs, int G, float inv_t, float* red) {
  const int D = group_chunk(G), g0 = threadIdx.x * D, g1 = min(G, g0 + D);
  float m = -INFINITY;
  for (int g = g0; g < g1; ++g) m = fmaxf(m, gs[g].x);
  m = block_max_f(m, red);
  float s = 0.f;
  for (int g = g0; g < g1; ++g) s += group_weight(gs[g], m, inv_t);
  float total;
  (void)block_excl_scan(s, red, total);
  __syncthreads();
  return make_float2(m, total);
}

// Inverse-CDF draw at temperature 1 / inv_t from the row z with group
// statistics gs and row maximum mx: the group whose running weight crosses
// u * total, then the token within it whose running weight does (else, by
// rounding, the group's last token of positive weight).  -1 when the total
// weight is 0.
__device__ int group_draw(const float2* gs, const float* z, int G, float mx, float inv_t, float u, float* red,
                          int* ired) {
  const int D = group_chunk(G), g0 = threadIdx.x * D, g1 = min(G, g0 + D);
  float s = 0.f;
  for (int g = g0; g < g1; ++g) s += group_weight(gs[g], mx, inv_t);
  float total;
  const float pre = block_excl_scan(s, red, total);
  const float thr = u * total;
  const int owner = block_max_i((s > 0.f && pre <= thr) ? (int)threadIdx.x : -1, ired);
  __shared__ int tok;
  if ((int)threadIdx.x == owner) {
    float acc = pre;  // running weight before group g
    int gsel = -1, glast = -1;
    for (int g = g0; g < g1; ++g) {
      const float w = group_weight(gs[g], mx, inv_t);
      if (w > 0.f) glast = g;
      if (w > 0.f && acc + w > thr) {
        gsel = g;
        break;
      }
      acc += w;
    }
    const int gg = gsel >= 0 ? gsel : glast;  // glast: rounding left the crossing past the chunk
    int hit = -1, last = -1;
    for (int j = 0; j < 16; ++j) {
      const float w = expf((z[gg * 16 + j] - mx) * inv_t);
      if (w > 0.f) last = gg * 16 + j;
      acc += w;
      if (gsel >= 0 && hit < 0 && acc > thr) hit = gg * 16 + j;
    }
    tok = hit >= 0 ? hit : last;
  }
  if (threadIdx.x == 0 && owner < 0) tok = -1;
  __syncthreads();
  return tok;
}

}  // namespace lede
