// Split-KV attention over the paged KV cache (gfx950).
#include "device.h"

namespace lede {

// ---- attention over the paged KV cache --------------------------------------

// At most this many thread groups in the combine kernel (16 pages each per
// round of loads); a launch uses ceil(max_chunks / 16) of them.
constexpr int COMBINE_GROUPS = 8;

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
  // Every token slot of an allocated page is readable, so the loads are
  // unconditional and tokens past the length are zeroed afterwards: guarded
  // loads compile to one branch and one wait per load.
  auto load_page = [&](int jj) {
    const int page = a.block_table[jj];
    const size_t base = (((size_t)a.layer * a.n_pages + page) * a.nkv + kvh) * 64 * HD;
    const int nvalid = min(64, pmax - jj * 64 + 1);
#pragma unroll
    for (int u = 0; u < TPT; ++u) load8<DT>(a.vcache, base + (size_t)(tg + PV_TG * u) * HD + dg * 8, vf[u]);
    const int t = tid >> 2, p = tid & 3;
#pragma unroll
    for (int c = 0; c < NPC; ++c) load8<DT>(a.kcache, base + (size_t)t * HD + p * 8 + 32 * c, kf + 8 * c);
#pragma unroll
    for (int u = 0; u < TPT; ++u)
#pragma unroll
      for (int e = 0; e < 8; ++e) vf[u][e] = tg + PV_TG * u < nvalid ? vf[u][e] : 0.f;
#pragma unroll
    for (int e = 0; e < NPC * 8; ++e) kf[e] = t < nvalid ? kf[e] : 0.f;
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

// One step of the page-ordered combine: fold a page's (max, sum, weighted
// value) into the running (mx, l, acc).
__device__ __forceinline__ void fold_step(float& mx, float& l, float& acc, float pm, float pl, float pa) {
  const float nm = fmaxf(mx, pm);
  const float so = (mx == -INFINITY) ? 0.f : __expf(mx - nm);
  const float sn = __expf(pm - nm);
  l = l * so + pl * sn;
  acc = acc * so + pa * sn;
  mx = nm;
}

// Combine the per-page partials of every (row, head): S = blockDim / HD
// groups of HD threads, group s folding pages 16 s .. 16 s + 15 (then
// 16 s + 16 S, ...) in page order, one thread per dim; the groups' running
// states are then folded in group order.  Up to 16 pages only group 0 has
// pages and the result is the plain page-ordered fold.  The loads are
// unconditional (a page index past the buffer is clamped to its last page,
// and pages past the row's position are loaded but not folded), so each
// group's 16 issue together, and before the sequence length arrives.
template <int DT, int HD>
__global__ __launch_bounds__(HD * COMBINE_GROUPS) void k_attn_combine(AttnArgs a) {
  constexpr int B = 16;
  __shared__ float st[COMBINE_GROUPS][3][HD];
  const int S = blockDim.x / HD;
  const int m = blockIdx.x / a.nq, head = blockIdx.x % a.nq;
  const int i = threadIdx.x % HD, sg = threadIdx.x / HD;
  const float* p = a.part + ((size_t)m * a.nq + head) * a.max_chunks * (HD + 2);
  float pm[B], pl[B], pa[B];
  auto load = [&](int j0) {
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const float* q = p + (size_t)min(j0 + u, a.max_chunks - 1) * (HD + 2);
      pm[u] = q[0];
      pl[u] = q[1];
      pa[u] = q[2 + i];
    }
  };
  load(sg * B);
  const int pos = *a.seq_len + a.pos_off + m;
  const int nc = pos / 64 + 1;
  float mx = -INFINITY, l = 0.f, acc = 0.f;
  for (int j0 = sg * B; j0 < nc; j0 += S * B) {
    if (j0 > sg * B) load(j0);
#pragma unroll
    for (int u = 0; u < B; ++u)
      if (j0 + u < nc) fold_step(mx, l, acc, pm[u], pl[u], pa[u]);
  }
  st[sg][0][i] = mx;
  st[sg][1][i] = l;
  st[sg][2][i] = acc;
  __syncthreads();
  if (sg == 0) {
    for (int q = 1; q < S && q * B < nc; ++q) fold_step(mx, l, acc, st[q][0][i], st[q][1][i], st[q][2][i]);
    Elem<DT>::store(a.out, (size_t)m * a.ldo + head * HD + i, acc / l);
  }
}

// Eight fp32 values as bf16 high parts and the bf16 rounding of what is left,
// packed as two matrix-core fragments: x ~= hi + lo to about 16 bits.
__device__ __forceinline__ void split8(const float* x, uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint16_t h0 = f32_to_bf16(x[2 * i]), h1 = f32_to_bf16(x[2 * i + 1]);
    const uint16_t l0 = f32_to_bf16(x[2 * i] - bf16_to_f32(h0)), l1 = f32_to_bf16(x[2 * i + 1] - bf16_to_f32(h1));
    h[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
    l[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// Partial attention on the matrix cores (bf16 cache), the same partials as
// k_attn_partial for up to 16 query rows per block: per page, wavefront w
// scores the page's tokens 16w..16w+15 against all rows (S^T = K Q^T as
// 16x16x32 tiles, q split into bf16 high and low parts), the page's per-row
// max and sum combine the four wavefronts in order through LDS, and
// wavefront w forms its HD/4 output dims as V^T P^T (the weights split the
// same way; the wavefront's value columns are staged in LDS and read back
// transposed).  Every output element is a fixed-order function of its own
// row, so a row's partials do not depend on the rows sharing its block.
// Five waves per SIMD (at most 96 VGPRs, no spills) keeps five blocks per
// CU instead of four.
template <int HD>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5))) void k_attn_mfma(AttnArgs a) {
  constexpr int KS = HD / 32;          // k-steps of the scores
  constexpr int DW = HD / 4;           // output dims per wavefront
  constexpr int DT = DW / 16;          // 16-dim output tiles per wavefront
  constexpr int VS = DW + 4;           // LDS row stride (elements) of the staged values
  __shared__ float smax[4][16], ssum[4][16];
  __shared__ float ps[16][64 + 4];
  __shared__ uint16_t vs[4][64 * VS];
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, lr = l & 15, lg = l >> 4;
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
  // this lane's query row as a matrix-core operand (rows past nr are zero)
  const bool row_ok = lr < nr;
  const int rr = r0 + lr, m_row = row_ok ? rr / G : 0, head = kvh * G + (row_ok ? rr % G : 0);
  const int row_pos = pos0 + m_row;
  uint4 qh[KS], ql[KS];
  {
    const float scale = rsqrtf((float)HD);
    const float* qp = a.q + (size_t)m_row * a.ldq + head * HD + lg * 8;
    // unconditional loads (a row past nr reads row 0's query, then zeroes it)
    float4 qu[KS], qv[KS];
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      qu[s2] = *(const float4*)(qp + 32 * s2);
      qv[s2] = *(const float4*)(qp + 32 * s2 + 4);
    }
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      const float4 u = qu[s2], v = qv[s2];
      float x[8];
      x[0] = row_ok ? u.x * scale : 0.f; x[1] = row_ok ? u.y * scale : 0.f;
      x[2] = row_ok ? u.z * scale : 0.f; x[3] = row_ok ? u.w * scale : 0.f;
      x[4] = row_ok ? v.x * scale : 0.f; x[5] = row_ok ? v.y * scale : 0.f;
      x[6] = row_ok ? v.z * scale : 0.f; x[7] = row_ok ? v.w * scale : 0.f;
      split8(x, qh[s2], ql[s2]);
    }
  }
  const uint16_t* kc = (const uint16_t*)a.kcache;
  const uint16_t* vc = (const uint16_t*)a.vcache;
  for (int j = blockIdx.y; j < n_chunks; j += a.n_split) {
    const int page = a.block_table[j];
    const size_t base = (((size_t)a.layer * a.n_pages + page) * a.nkv + kvh) * 64 * HD;
    const int nvalid = min(64, pmax - j * 64 + 1);
    // keys of tokens 16w + lr, dims 32 s + 8 lg; values of this wavefront's dims
    // (unconditional loads within the page, tokens past the length zeroed after)
    uint4 kf[KS];
    const int tk = 16 * w + lr;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) kf[s2] = ld16(kc + base + (size_t)tk * HD + 32 * s2 + 8 * lg);
    constexpr int VC = 64 * DW / 8 / 64;   // 16-byte value chunks per lane
    uint4 vf[VC];
#pragma unroll
    for (int c = 0; c < VC; ++c) {
      const int idx = l + 64 * c, t = idx / (DW / 8), d8 = idx % (DW / 8);
      vf[c] = ld16(vc + base + (size_t)t * HD + w * DW + 8 * d8);
    }
    // (masks, not selects of whole vectors: those select addresses and
    // put the arrays in scratch)
    const uint32_t km = tk < nvalid ? ~0u : 0u;
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      kf[s2].x &= km; kf[s2].y &= km; kf[s2].z &= km; kf[s2].w &= km;
    }
#pragma unroll
    for (int c = 0; c < VC; ++c) {
      const uint32_t vm = (l + 64 * c) / (DW / 8) < nvalid ? ~0u : 0u;
      vf[c].x &= vm; vf[c].y &= vm; vf[c].z &= vm; vf[c].w &= vm;
    }
    // S^T tile: lane holds tokens 16w + 4 lg + i of row lr
    f32x4 sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < KS; ++s2) {
      sc = mfma_tile<1>(kf[s2], qh[s2], sc);
      sc = mfma_tile<1>(kf[s2], ql[s2], sc);
    }
    float sv[4], mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int t = j * 64 + 16 * w + 4 * lg + i;
      sv[i] = (row_ok && t <= row_pos) ? sc[i] : -INFINITY;
      mx = fmaxf(mx, sv[i]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (lg == 0) smax[w][lr] = mx;
#pragma unroll
    for (int c = 0; c < VC; ++c) {
      const int idx = l + 64 * c, t = idx / (DW / 8), d8 = idx % (DW / 8);
      uint16_t* dst = &vs[w][t * VS + 8 * d8];
      *(uint2*)dst = make_uint2(vf[c].x, vf[c].y);
      *(uint2*)(dst + 4) = make_uint2(vf[c].z, vf[c].w);
    }
    __syncthreads();
    const float pm = fmaxf(fmaxf(fmaxf(smax[0][lr], smax[1][lr]), smax[2][lr]), smax[3][lr]);
    float pv[4], sum = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      pv[i] = sv[i] == -INFINITY ? 0.f : __expf(sv[i] - pm);
      sum += pv[i];
    }
    sum += __shfl_xor(sum, 16);
    sum += __shfl_xor(sum, 32);
    if (lg == 0) ssum[w][lr] = sum;
    *(float4*)&ps[lr][16 * w + 4 * lg] = make_float4(pv[0], pv[1], pv[2], pv[3]);
    __syncthreads();
    // this wavefront's dims: D^T = V^T P^T over the page's 64 tokens
    f32x4 oc[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      float px[8];
      const float4 u = *(const float4*)&ps[lr][32 * ks + 8 * lg], v = *(const float4*)&ps[lr][32 * ks + 8 * lg + 4];
      px[0] = u.x; px[1] = u.y; px[2] = u.z; px[3] = u.w; px[4] = v.x; px[5] = v.y; px[6] = v.z; px[7] = v.w;
      uint4 ph, pl;
      split8(px, ph, pl);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d = 16 * dt + lr;
        uint32_t e[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int t = 32 * ks + 8 * lg + 2 * i;
          e[i] = (uint32_t)vs[w][t * VS + d] | ((uint32_t)vs[w][(t + 1) * VS + d] << 16);
        }
        const uint4 vt = make_uint4(e[0], e[1], e[2], e[3]);
        oc[dt] = mfma_tile<1>(vt, ph, oc[dt]);
        oc[dt] = mfma_tile<1>(vt, pl, oc[dt]);
      }
    }
    // partials of row lr: dims w * DW + 16 dt + 4 lg + i
    if (row_ok) {
      float* p = a.part + (((size_t)m_row * a.nq + head) * a.max_chunks + j) * (HD + 2);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const int d0 = w * DW + 16 * dt + 4 * lg;
#pragma unroll
        for (int i = 0; i < 4; ++i) p[2 + d0 + i] = oc[dt][i];
      }
      if (w == 0 && lg == 0) {
        p[0] = pm;
        p[1] = ((ssum[0][lr] + ssum[1][lr]) + ssum[2][lr]) + ssum[3][lr];
      }
    }
    __syncthreads();  // the next page rewrites the staging
  }
}

hipError_t launch_attention(int dtype, const AttnArgs& a, hipStream_t s) {
  const int G = a.nq / a.nkv;
  const int n_rs = (a.M * G + a.rows_per_block - 1) / a.rows_per_block;
  dim3 grid(a.nkv * n_rs, a.n_split);
  const int combine_grid = a.M * a.nq;
  const int groups = (a.max_chunks + 15) / 16 < COMBINE_GROUPS ? (a.max_chunks + 15) / 16 : COMBINE_GROUPS;
  if (dtype == 1) {
    if (a.hd == 128) {
      if (a.mfma) hipLaunchKernelGGL((k_attn_mfma<128>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_partial<1, 128>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<1, 128>), dim3(combine_grid), dim3(128 * groups), 0, s, a);
    } else {
      if (a.mfma) hipLaunchKernelGGL((k_attn_mfma<64>), grid, dim3(256), 0, s, a);
      else hipLaunchKernelGGL((k_attn_partial<1, 64>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<1, 64>), dim3(combine_grid), dim3(64 * groups), 0, s, a);
    }
  } else {
    if (a.hd == 128) {
      hipLaunchKernelGGL((k_attn_partial<0, 128>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<0, 128>), dim3(combine_grid), dim3(128 * groups), 0, s, a);
    } else {
      hipLaunchKernelGGL((k_attn_partial<0, 64>), grid, dim3(256), 0, s, a);
      hipLaunchKernelGGL((k_attn_combine<0, 64>), dim3(combine_grid), dim3(64 * groups), 0, s, a);
    }
  }
  return hipGetLastError();
}

}  // namespace lede
