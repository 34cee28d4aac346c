// Split-KV attention over the paged KV cache (gfx950).
#include "device.h"

namespace lede {

// ---- attention over the paged KV cache --------------------------------------

// Eight consecutive cache elements as fp32.
template <int DT>
__device__ __forceinline__ void load8(const void* base, size_t idx, float* o) {
  if (DT == 1) {
    const uint4 u = ld16((const uint16_t*)base + idx);
    o[0] = bf16lo(u.x); o[1] = bf16hi(u.x); o[2] = bf16lo(u.y); o[3] = bf16hi(u.y);
    o[4] = bf16lo(u.z); o[5] = bf16hi(u.z); o[6] = bf16lo(u.w); o[7] = bf16hi(u.w);
  } else {
    const float4 a = *(const float4*)((const float*)base + idx);
    const float4 b = *(const float4*)((const float*)base + idx + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
}

// Partial attention of up to 16 query rows (row = (m, query head of the
// group)) against whole 64-token pages; pages are strided over the blocks of
// a split.  For every (row, page): running max, sum of exp and the
// exp-weighted value sum, stored for the combine kernel.  A row's partials
// do not depend on which other rows share the block.
template <int DT, int HD>
__global__ __launch_bounds__(256) void k_attn_partial(AttnArgs a) {
  constexpr int NPC = HD / 32;  // 8-element pieces per thread in the score phase
  constexpr int PV_DG = HD / 8, PV_TG = 256 / PV_DG, TPT = 64 / PV_TG;
  __shared__ float qs[16][HD];
  __shared__ float ss[16][64];
  __shared__ float st_m[16], st_l[16];
  __shared__ float red[4][16][HD];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int G = a.nq / a.nkv;
  const int R = a.M * G;
  const int n_rs = (R + a.rows_per_block - 1) / a.rows_per_block;
  const int kvh = blockIdx.x / n_rs, rs = blockIdx.x % n_rs;
  const int r0 = rs * a.rows_per_block;
  const int nr = min(a.rows_per_block, R - r0);
  const int pos0 = *a.seq_len + a.pos_off;
  const int pmax = pos0 + a.M - 1;
  const int n_chunks = pmax / 64 + 1;
  if ((int)blockIdx.y >= n_chunks) return;
  const float scale = rsqrtf((float)HD);
  // thread roles: scores (token t, part p covering dims p*8 + 32c + e);
  // values (dims dg*8.., tokens tg + PV_TG u)
  const int dg = tid % PV_DG, tg = tid / PV_DG;
  float vf[TPT][8], kf[NPC * 8];
  auto load_page = [&](int jj) {
    const int page = a.block_table[jj];
    const size_t base = (((size_t)a.layer * a.n_pages + page) * a.nkv + kvh) * 64 * HD;
    const int nvalid = min(64, pmax - jj * 64 + 1);
#pragma unroll
    for (int u = 0; u < TPT; ++u) {
      const int t = tg + PV_TG * u;
      if (t < nvalid) load8<DT>(a.vcache, base + (size_t)t * HD + dg * 8, vf[u]);
      else
#pragma unroll
        for (int e = 0; e < 8; ++e) vf[u][e] = 0.f;
    }
    const int t = tid >> 2, p = tid & 3;
    if (t < nvalid) {
#pragma unroll
      for (int c = 0; c < NPC; ++c) load8<DT>(a.kcache, base + (size_t)t * HD + p * 8 + 32 * c, kf + 8 * c);
    } else {
#pragma unroll
      for (int e = 0; e < NPC * 8; ++e) kf[e] = 0.f;
    }
  };
  load_page(blockIdx.y);  // the first page's keys and values are in flight with the query loads

  for (int idx = tid; idx < nr * (HD / 4); idx += 256) {
    const int r = idx / (HD / 4), i = 4 * (idx % (HD / 4));
    const int rr = r0 + r, m = rr / G, head = kvh * G + rr % G;
    const float4 v = *(const float4*)(a.q + (size_t)m * a.ldq + head * HD + i);
    qs[r][i] = v.x * scale;
    qs[r][i + 1] = v.y * scale;
    qs[r][i + 2] = v.z * scale;
    qs[r][i + 3] = v.w * scale;
  }
  __syncthreads();

  for (int j = blockIdx.y; j < n_chunks; j += a.n_split) {
    const int tok0 = j * 64;
    {
      const int t = tid >> 2, p = tid & 3;
      for (int r = 0; r < nr; ++r) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < NPC; ++c)
#pragma unroll
          for (int e = 0; e < 8; ++e) s = fmaf(qs[r][p * 8 + 32 * c + e], kf[8 * c + e], s);
        s += __shfl_xor(s, 1);
        s += __shfl_xor(s, 2);
        const int m = (r0 + r) / G;
        if (p == 0) ss[r][t] = (tok0 + t <= pos0 + m) ? s : -INFINITY;
      }
    }
    __syncthreads();
    for (int r = wave; r < nr; r += 4) {  // softmax statistics, one lane per token
      const float v = ss[r][lane];
      const float mx = wave_max(v);
      const float e = (v == -INFINITY) ? 0.f : __expf(v - mx);
      const float l = wave_sum(e);
      ss[r][lane] = e;
      if (lane == 0) {
        st_m[r] = mx;
        st_l[r] = l;
      }
    }
    __syncthreads();
    {  // exp-weighted values: thread (dim group dg, token group tg)
      for (int r = 0; r < nr; ++r) {
        float o[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = 0.f;
#pragma unroll
        for (int u = 0; u < TPT; ++u) {
          const float w = ss[r][tg + PV_TG * u];
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = fmaf(w, vf[u][e], o[e]);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e)
          for (int off = PV_DG; off < 64; off <<= 1) o[e] += __shfl_xor(o[e], off);
        if (lane < PV_DG) {
#pragma unroll
          for (int e = 0; e < 8; ++e) red[wave][r][dg * 8 + e] = o[e];
        }
      }
    }
    __syncthreads();
    if (j + a.n_split < n_chunks) load_page(j + a.n_split);  // the next page of this block
    for (int idx = tid; idx < nr * HD; idx += 256) {
      const int r = idx / HD, i = idx % HD;
      const int rr = r0 + r, m = rr / G, head = kvh * G + rr % G;
      float* p = a.part + (((size_t)m * a.nq + head) * a.max_chunks + j) * (HD + 2);
      p[2 + i] = ((red[0][r][i] + red[1][r][i]) + red[2][r][i]) + red[3][r][i];
      if (i == 0) {
        p[0] = st_m[r];
        p[1] = st_l[r];
      }
    }
    __syncthreads();
  }
}

// Combine the per-page partials of every (row, head) in page order.
template <int DT, int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(AttnArgs a) {
  const int m = blockIdx.x / a.nq, head = blockIdx.x % a.nq, i = threadIdx.x;
  const int pos = *a.seq_len + a.pos_off + m;
  const int nc = pos / 64 + 1;
  const float* p = a.part + ((size_t)m * a.nq + head) * a.max_chunks * (HD + 2);
  float mx = -INFINITY, l = 0.f, acc = 0.f;
  for (int j0 = 0; j0 < nc; j0 += 8) {
    float pm[8], pl[8], pa[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float* q = p + (size_t)(j0 + u) * (HD + 2);
      const bool ok = j0 + u < nc;
      pm[u] = ok ? q[0] : -INFINITY;
      pl[u] = ok ? q[1] : 0.f;
      pa[u] = ok ? q[2 + i] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (j0 + u >= nc) break;
      const float nm = fmaxf(mx, pm[u]);
      const float so = (mx == -INFINITY) ? 0.f : __expf(mx - nm);
      const float sn = __expf(pm[u] - nm);
      l = l * so + pl[u] * sn;
      acc = acc * so + pa[u] * sn;
      mx = nm;
    }
  }
  Elem<DT>::store(a.out, (size_t)m * a.ldo + head * HD + i, acc / l);
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  const int G = a.nq / a.nkv;
  const int n_rs = (a.M * G + a.rows_per_block - 1) / a.rows_per_block;
  dim3 grid(a.nkv * n_rs, a.n_split);
  const int combine_grid = a.M * a.nq;
  if (dtype == 1) {
    if (a.hd == 128) {
      hipLaunchKernelGGL((k_attn_partial<1, 128>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<1, 128>), dim3(combine_grid), dim3(128), 0, s, a);
    } else {
      hipLaunchKernelGGL((k_attn_partial<1, 64>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<1, 64>), dim3(combine_grid), dim3(64), 0, s, a);
    }
  } else {
    if (a.hd == 128) {
      hipLaunchKernelGGL((k_attn_partial<0, 128>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<0, 128>), dim3(combine_grid), dim3(128), 0, s, a);
    } else {
      hipLaunchKernelGGL((k_attn_partial<0, 64>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<0, 64>), dim3(combine_grid), dim3(64), 0, s, a);
    }
  }
  return hipGetLastError();
}

}  // namespace lede
