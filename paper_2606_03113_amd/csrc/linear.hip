// Weight-streaming linear kernels of the decode step (gfx950).
//
// Memory-bound batch-1 decoding: every weight byte is streamed from HBM once
// per pass.  Weights live in the tiled layout of kernels.h (one coalesced
// 1 KiB wave load per 16-row x TK tile).  The draft path (one row) uses the
// vector dot2 instructions; the verify path (k+1 <= 16 rows) uses the
// 16x16x32 bf16 (or 16x16x4 fp32) matrix-core instructions with the weight
// tile as the A operand, so one weight read serves every verify row.
//
// Determinism: every reduction runs in a fixed order, and the matrix-core
// result for a row does not depend on the other rows of the call, so a row
// gives the same bits in a prefill chunk, a verify pass or a one-row
// autoregressive step.
#include "device.h"

namespace lede {

// ---- repack: logical row-major -> tiled -------------------------------------

template <int DT>
__global__ __launch_bounds__(256) void k_repack(RepackArgs a) {
  typedef Tile<DT> TL;
  typedef typename Elem<DT>::T ET;
  const size_t total = (size_t)a.n_groups * a.KT * 64;
  for (size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (size_t)gridDim.x * 256) {
    const int lane = (int)(idx & 63);
    const size_t rest = idx >> 6;
    const int t = (int)(rest % a.KT);
    const int gl = (int)(rest / a.KT);  // group within this call
    const int r = lane & 15;
    int row;
    bool valid = true;
    switch (a.order) {
      case ROWS_ROPE: {
        const int gph = a.hd / 16;
        const int head = gl / gph, tt = gl % gph;
        row = head * a.hd + (r < 8 ? 8 * tt + r : a.hd / 2 + 8 * tt + (r - 8));
        break;
      }
      case ROWS_GATE: row = 8 * gl + r; valid = r < 8; break;
      case ROWS_UP: row = 8 * gl + (r - 8); valid = r >= 8; break;
      default: row = 16 * gl + r;
    }
    if (!valid) continue;  // the other source fills these rows
    ET vals[TL::EPL];
    const int k0 = t * TL::TK + (lane >> 4) * TL::EPL;
#pragma unroll
    for (int e = 0; e < TL::EPL; ++e) {
      const int k = k0 + e;
      vals[e] = (row < a.N && k < a.K) ? ((const ET*)a.src)[(size_t)row * a.K + k] : (ET)0;
    }
    uint8_t* dst = (uint8_t*)a.dst + ((size_t)(a.group0 + gl) * a.KT + t) * TILE_BYTES + lane * 16;
    *(uint4*)dst = *(const uint4*)vals;
  }
}

// ---- linear: y = W x with fused prologue / epilogue --------------------------

// What the QKV epilogue of thread tid needs from the sequence length c
// alone: the rotary pair of its (row, dim) in q / k groups and the cache page
// of its row.  Fetched before the weights stream for the block's first group.
struct QkvPre {
  float2 cs;
  int page;
};
__device__ __forceinline__ QkvPre qkv_fetch(const LinearArgs& a, int g, int c) {
  const int tid = threadIdx.x, m = tid & 15;
  const int gph = a.hd / 16, qg = a.nq * gph, kg = a.nkv * gph;
  QkvPre p = {make_float2(1.f, 0.f), 0};
  if (tid >= 256 || m >= a.M) return p;
  const int pos = c + m;
  if (g >= qg) p.page = a.block_table[pos >> 6];
  if (g < qg + kg && tid < 128) {
    const int gl = g < qg ? g : g - qg;
    p.cs = a.rope[(size_t)pos * (a.hd / 2) + 8 * (gl % gph) + (tid >> 4)];
  }
  return p;
}

template <int DT, bool GS>
__device__ __forceinline__ void epilogue(const LinearArgs& a, int g, float (*ct)[17], uint64_t& best, int qkv_c,
                                         const QkvPre& pre) {
  const int tid = threadIdx.x;
  const int M = a.M;
  switch (a.epi) {
    case EPI_STORE: {
      const int n = tid >> 4, m = tid & 15;
      if (m < M) a.out[(size_t)m * a.ldo + g * 16 + n] = ct[n][m];
      break;
    }
    case EPI_BIAS_RELU: {
      if (tid < 16) {
        const int row = g * 16 + tid;
        a.out[row] = fmaxf(ct[tid][0] + a.bias[row], 0.f);
      }
      break;
    }
    case EPI_RESID: {
      const int n = tid >> 4, m = tid & 15;
      if (m < M) {
        const int col = g * 16 + n;
        float* hp = a.h + (size_t)m * a.ldh + col;
        // the gain is read before the residual is stored, so that the two
        // loads share one round trip (after the store they could alias)
        const float gn = a.ss_out ? Elem<DT>::load(a.xg_gain, col) : 0.f;
        const float hn = *hp + ct[n][m];
        *hp = hn;
        if (a.ss_out) {
          Elem<DT>::store(a.xg, (size_t)m * a.ldxg + col, hn * gn);
          ct[n][m] = hn;  // squared and summed per row once the block has synchronised
        }
      }
      break;
    }
    case EPI_SWIGLU: {
      if (tid < 128) {
        const int r = tid >> 4, m = tid & 15;
        if (m < M) {
          const float gt = ct[r][m], up = ct[r + 8][m];
          const float s = gt / (1.f + __expf(-gt));
          Elem<DT>::store(a.act, (size_t)m * a.ld_act + 8 * g + r, s * up);
        }
      }
      break;
    }
    case EPI_QKV: {
      const int hd = a.hd, gph = hd / 16;
      const int qg = a.nq * gph, kg = a.nkv * gph;
      const int c = qkv_c;
      const QkvPre p = g == (int)blockIdx.x ? pre : qkv_fetch(a, g, c);
      if (g < qg + kg) {
        if (tid < 128) {
          const int r = tid >> 4, m = tid & 15;
          if (m < M) {
            const bool isq = g < qg;
            const int gl = isq ? g : g - qg;
            const int head = gl / gph, i = 8 * (gl % gph) + r;
            const int pos = c + m;
            const float2 cs = p.cs;
            const float x0 = ct[r][m], x1 = ct[r + 8][m];
            const float y0 = x0 * cs.x - x1 * cs.y;
            const float y1 = x1 * cs.x + x0 * cs.y;
            if (isq) {
              float* q = a.q + (size_t)m * a.ldq + head * hd;
              q[i] = y0;
              q[i + hd / 2] = y1;
            } else {
              const size_t base = ((((size_t)a.layer * a.n_pages + p.page) * a.nkv + head) * 64 + (pos & 63)) * hd;
              Elem<DT>::store(a.kcache, base + i, y0);
              Elem<DT>::store(a.kcache, base + i + hd / 2, y1);
            }
          }
        }
      } else {
        const int n = tid >> 4, m = tid & 15;
        if (m < M) {
          const int dim = (g - qg - kg) * 16 + n;
          const int head = dim / hd, i = dim % hd;
          const int pos = c + m;
          const size_t base = ((((size_t)a.layer * a.n_pages + p.page) * a.nkv + head) * 64 + (pos & 63)) * hd;
          Elem<DT>::store(a.vcache, base + i, ct[n][m]);
        }
      }
      break;
    }
    case EPI_ARGMAX: {
      const int n = tid >> 4, m = tid & 15;
      const int row = g * 16 + n;
      if (m < M && a.logits) a.logits[(size_t)m * a.ld_logits + row] = ct[n][m];
      if (tid < 16 && tid < M) {
        for (int nn = 0; nn < 16; ++nn) {
          const int rr = g * 16 + nn;
          if (rr < a.vocab) {
            const uint64_t key = argmax_key(ct[nn][tid], rr);
            best = key > best ? key : best;
          }
        }
        if (GS) {  // the group's sampling statistics, in token order
          float gm = -INFINITY, gs = 0.f;
          for (int nn = 0; nn < 16; ++nn)
            if (g * 16 + nn < a.vocab) gm = fmaxf(gm, ct[nn][tid]);
          for (int nn = 0; nn < 16; ++nn)
            if (g * 16 + nn < a.vocab && gm > -INFINITY) gs += expf((ct[nn][tid] - gm) * a.inv_t);
          a.gstats[(size_t)tid * a.ld_gstats + g] = make_float2(gm, gs);
        }
      }
      break;
    }
  }
}


// 16 bytes from LDS through an LDS-typed pointer: a select between such a
// load and a register constant cannot become a load through a selected
// pointer (which would put the constant in scratch memory).
__device__ __forceinline__ uint4 lds_ld16(const uint8_t* p) {
  const u32x4 v = *(const __attribute__((address_space(3))) u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Deterministic sum over the NW wavefronts of a block (every thread takes
// part in the barriers).
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* scratch) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  __syncthreads();
  if (lane == 0) scratch[wave] = v;
  __syncthreads();
  float s = scratch[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) s += scratch[w];
  return s;
}

// Normalise the single input row of the vector kernel into LDS with every
// thread of the block: thread t holds elements 4t + 4 NT j of the row and of
// the gain in registers (both requested together), sums the squares in j
// order, and the block sums the threads' partials in wave order.  The row is
// zero-padded to the batch size the main loop reads.  The loads
// (norm_row_load) are issued together with the block's other prologue loads
// and consumed (norm_row_stage) before the weights are requested.
template <int NW>
struct NormRow {
  static constexpr int NT = NW * 64, J = (8192 + 4 * NT - 1) / (4 * NT);  // rows of up to 8192 elements
  float4 v[J], g[J];
};

template <int DT, int NW>
__device__ __forceinline__ void norm_row_load(const LinearArgs& a, NormRow<NW>& nr) {
  constexpr int NT = NormRow<NW>::NT, J = NormRow<NW>::J;
  const int tid = threadIdx.x;
  const float* h = a.h;
  const void* row = nullptr;
  if (a.x_mode == X_EMBED_NORM) {
    const int tok = (int)min((unsigned)a.tok.get(0), (unsigned)(a.vocab - 1));
    row = (const uint8_t*)a.embed + (size_t)tok * a.K * Elem<DT>::ES_;
    h = nullptr;
  }
  // unconditional loads (a lane past the row re-reads its first elements),
  // zeroed afterwards: guarded loads compile to a branch and a wait each
  // (the gain first, then the row from a source chosen once, outside the
  // loops, so that no branch separates the loads)
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int i = 4 * tid + 4 * NT * j;
    nr.g[j] = row_load4<DT>(nullptr, a.gain, i < a.K ? i : 0);
  }
  if (h) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int i = 4 * tid + 4 * NT * j;
      nr.v[j] = row_load4<DT>(h, nullptr, i < a.K ? i : 0);
    }
  } else {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int i = 4 * tid + 4 * NT * j;
      nr.v[j] = row_load4<DT>(nullptr, row, i < a.K ? i : 0);
    }
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool in = 4 * tid + 4 * NT * j < a.K;
    nr.v[j].x = in ? nr.v[j].x : 0.f; nr.v[j].y = in ? nr.v[j].y : 0.f;
    nr.v[j].z = in ? nr.v[j].z : 0.f; nr.v[j].w = in ? nr.v[j].w : 0.f;
    nr.g[j].x = in ? nr.g[j].x : 0.f; nr.g[j].y = in ? nr.g[j].y : 0.f;
    nr.g[j].z = in ? nr.g[j].z : 0.f; nr.g[j].w = in ? nr.g[j].w : 0.f;
  }
}

template <int DT, int NW>
__device__ void norm_row_stage(const LinearArgs& a, const NormRow<NW>& nr, uint8_t* lds, float* scratch) {
  constexpr int NT = NormRow<NW>::NT, J = NormRow<NW>::J;
  const int tid = threadIdx.x;
  const int row_bytes = a.K * Elem<DT>::ES_, pad_bytes = lin_x_tiles(a.KT) * Tile<DT>::TK * Elem<DT>::ES_;
  for (int i = row_bytes + tid * 4; i < pad_bytes; i += NT * 4) *(uint32_t*)(lds + i) = 0u;
  float* h_out = (a.x_mode == X_EMBED_NORM && blockIdx.x == 0) ? a.h : nullptr;
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    ss = fmaf(nr.v[j].x, nr.v[j].x, ss);
    ss = fmaf(nr.v[j].y, nr.v[j].y, ss);
    ss = fmaf(nr.v[j].z, nr.v[j].z, ss);
    ss = fmaf(nr.v[j].w, nr.v[j].w, ss);
  }
  ss = block_sum<NW>(ss, scratch);
  const float inv = rsqrtf(ss / (float)a.K + a.eps);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int i = 4 * tid + 4 * NT * j;
    if (i < a.K) {
      float4 y;
      y.x = (nr.v[j].x * inv) * nr.g[j].x;
      y.y = (nr.v[j].y * inv) * nr.g[j].y;
      y.z = (nr.v[j].z * inv) * nr.g[j].z;
      y.w = (nr.v[j].w * inv) * nr.g[j].w;
      if (h_out) *(float4*)(h_out + i) = nr.v[j];
      store4<DT>(lds, i, y);
    }
  }
  __syncthreads();
}

// Copy the vector kernel's input row (KT tiles of the model dtype) into LDS
// and zero the padding up to pad bytes, loaded (copy_row_load) and stored
// (copy_row_stage) like the normalised row.
template <int NW>
struct CopyRow {
  static constexpr int C = LIN_LDS_X_MAX / (NW * 64 * 16);  // 16-byte chunks per thread
  uint4 c[C];
};

template <int NW>
__device__ __forceinline__ void copy_row_load(const void* x, int bytes, CopyRow<NW>& cr) {
#pragma unroll
  for (int u = 0; u < CopyRow<NW>::C; ++u) {
    const int i = (threadIdx.x + NW * 64 * u) * 16;
    cr.c[u] = i < bytes ? ld16((const uint8_t*)x + i) : make_uint4(0u, 0u, 0u, 0u);
  }
}

template <int NW>
__device__ void copy_row_stage(const CopyRow<NW>& cr, int pad, uint8_t* lds) {
#pragma unroll
  for (int u = 0; u < CopyRow<NW>::C; ++u) {
    const int i = (threadIdx.x + NW * 64 * u) * 16;
    if (i < pad) *(uint4*)(lds + i) = cr.c[u];
  }
  __syncthreads();
}

// y = W x over 16-row groups, one group per block pass.  Eight wavefronts
// split K (wave w takes tiles w, w + 8, ...), four tiles per wave in flight,
// and the partials are summed in wave order.
//   XS = XS_LDS:    one input row, staged in LDS in the prologue (normalised
//                   for X_NORM / X_EMBED_NORM, copied otherwise); dot2 math.
//   XS = XS_GLOBAL: one input row read from global memory per tile (rows too
//                   long for LDS); dot2 math.
//   XS = XS_MFMA:   up to 16 rows read from global memory per tile, 16x16
//                   matrix-core tiles.
//   XS = XS_MFMA_LDS: the same, with the rows staged in LDS in the prologue:
//                   each wavefront copies the tiles it will use (direct
//                   global-to-LDS loads issued before its weights) into a
//                   region of its own, [row m][tile j][64 bytes], so that it
//                   waits for its own loads only.
// GS: the argmax epilogue also writes the sampling group statistics (a
// separate kernel, so that the others carry none of its registers).
template <int DT, int XS, bool GS>
__device__ __forceinline__ void linear_main(const LinearArgs& a) {
  typedef Tile<DT> TL;
  constexpr int NW = LIN_WAVES, U = 4;  // tiles per wave per batch
  constexpr bool MFMA = XS == XS_MFMA || XS == XS_MFMA_LDS;
  constexpr bool XL = XS == XS_MFMA_LDS;
  static_assert(TL::TK * TL::ES == 64, "64 bytes of a row per tile");
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float red[NW][16][16];
  __shared__ float ct[16][17];
  __shared__ float scratch[NW];
  __shared__ float inv_s[16];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KT = a.KT, NG = a.n_groups;
  const uint4 zero = {0u, 0u, 0u, 0u};

  if (blockIdx.x == 0 && a.zero_keys && tid < KEY_WORDS && (tid % KEY_PITCH) < a.n_zero_keys) a.zero_keys[tid] = 0;

  // staged matrix-core rows: 16 (row, tile) units of 64 bytes per load
  // instruction, lane L carrying bytes 16 (L & 3) of unit L >> 2; a region
  // holds xj tiles per row (a wavefront with fewer leaves the rest unused)
  const int xj = (KT + NW - 1) / NW;                                    // tiles per row of a region
  uint8_t* xw = smem + (size_t)wave * xj * a.M * (TL::TK * TL::ES);     // this wavefront's region
  if (XL) {
    const int jw = (KT - wave + NW - 1) / NW, units = xj * a.M;
    for (int i = 0; i * 16 < units; ++i) {
      const int u = i * 16 + (lane >> 2);
      const int m = u / xj, j = u - m * xj;
      const uint8_t* src = (const uint8_t*)a.x + ((size_t)m * a.ldx * TL::ES + (size_t)(wave + NW * j) * 64 + (lane & 3) * 16);
      if (u < units && j < jw)
        __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(xw + i * 1024), 16,
                                         0, 0);
    }
  }

  // split norm: the producer's partial sums, requested with the rows (vector
  // loads complete in issue order: a wait for a load issued after the first
  // weight batch would wait for the weights too)
  static_assert(NW * 64 == 512 && SS_MAX_GROUPS <= 512, "32 threads per row of partial sums; one per thread");
  constexpr int SSJ = SS_MAX_GROUPS / 32;
  const bool split_norm = (MFMA || XS == XS_LDS) && a.ss_in;
  float ssv[SSJ];
  if (split_norm) {
    if (MFMA) {
      const int m = tid & 15, j0 = tid >> 4;
      const float* row = a.ss_in + (m < a.M ? m : 0) * a.ss_groups;
      const int nj = m < a.M ? a.ss_groups : 0;
#pragma unroll
      for (int i = 0; i < SSJ; ++i) ssv[i] = j0 + 32 * i < nj ? row[j0 + 32 * i] : 0.f;
    } else {  // one row: thread t holds group t's partial
      ssv[0] = tid < a.ss_groups ? a.ss_in[tid] : 0.f;
    }
  }

  // QKV: the sequence length is requested first (a scalar load, waited for
  // only after the weights are issued)
  const int qkv_c = a.epi == EPI_QKV ? *a.seq_len + a.pos_off : 0;
  const bool norm_row = XS == XS_LDS && (a.x_mode == X_NORM || a.x_mode == X_EMBED_NORM);
  NormRow<NW> nrow;
  CopyRow<NW> crow;
  if (norm_row) norm_row_load<DT, NW>(a, nrow);
  else if (XS == XS_LDS) copy_row_load<NW>(a.x, KT * TL::TK * TL::ES, crow);

  int g = blockIdx.x;
  // The input rows are staged before the first weight batch is requested.
  // Every block starts within about 0.6 us, and a row requested alongside
  // the weights waits behind every block's first batch: its first read
  // misses the L2 (the previous kernel wrote it).  Waiting for the rows
  // first and then streaming measured 5.756 against 5.774 ms per step.
  if (XS == XS_LDS) {
    if (norm_row) norm_row_stage<DT, NW>(a, nrow, smem, scratch);
    else copy_row_stage<NW>(crow, lin_x_tiles(KT) * TL::TK * TL::ES, smem);
  }
  if (XL) __builtin_amdgcn_s_waitcnt(0);  // this wavefront's staged tiles (and partial sums)
  uint4 w[U];
  {
    const uint8_t* wg = a.w + (size_t)(g < NG ? g : 0) * KT * TILE_BYTES + lane * 16;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = wave + NW * u;
      w[u] = (g < NG && t < KT) ? ld16_stream(wg + (size_t)t * TILE_BYTES) : zero;
    }
  }
  if (split_norm && !MFMA) {
    const float t = block_sum<NW>(ssv[0], scratch);  // wave order
    if (tid == 0) inv_s[0] = rsqrtf(t / (float)a.K + a.eps);
    __syncthreads();
  } else if (split_norm) {
    // row m's sum: thread partials in i order, then the 32 threads in order
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < SSJ; ++i) s += ssv[i];
    float* ssr = &red[0][0][0];  // [32][16], free until the main loop's partials
    ssr[tid] = s;                // = ssr[j0 * 16 + m]
    __syncthreads();
    if (tid < 16) {
      float t = 0.f;
      for (int j = 0; j < 32; ++j) t += ssr[j * 16 + tid];
      inv_s[tid] = rsqrtf(t / (float)a.K + a.eps);
    }
    __syncthreads();
  }

  QkvPre qpre = {make_float2(1.f, 0.f), 0};
  if (a.epi == EPI_QKV) qpre = qkv_fetch(a, blockIdx.x, qkv_c);
  // the staged rows: the compiler does not track the direct-to-LDS loads
  // (waited for above, before the weights were requested)

  uint64_t best = 0;
  bool first = true;
  for (; g < NG; g += gridDim.x, first = false) {
    const uint8_t* wg = a.w + (size_t)g * KT * TILE_BYTES + lane * 16;
    float acc0 = 0.f, acc1 = 0.f;
    f32x4 c0 = {0.f, 0.f, 0.f, 0.f}, c1 = {0.f, 0.f, 0.f, 0.f};
    const int m = MFMA ? (lane & 15) : 0;
    const bool has = !MFMA || m < a.M;
    const uint8_t* xg = (const uint8_t*)a.x + ((size_t)m * a.ldx + (lane >> 4) * TL::EPL) * TL::ES;
    const uint8_t* xs = smem + (lane >> 4) * 16;
    // staged rows: tile j of this lane's row at LDS byte xl + 64 j
    const uint32_t xl = (uint32_t)(xw - smem) + m * xj * 64 + (lane >> 4) * 16;
    int xrow0 = 0;
    for (int t = wave; t < KT; t += NW * U, xrow0 += U) {
      if (!(first && t == wave)) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int tt = t + NW * u;
          w[u] = tt < KT ? ld16_stream(wg + (size_t)tt * TILE_BYTES) : zero;
        }
      }
      if (XS == XS_LDS) {
#pragma unroll
        for (int u = 0; u < U; u += 2) {
          const int t0 = t + NW * u, t1 = t0 + NW;  // the staged row is zero-padded past KT
          const uint4 x0 = *(const uint4*)(xs + (size_t)t0 * TL::TK * TL::ES);
          const uint4 x1 = *(const uint4*)(xs + (size_t)t1 * TL::TK * TL::ES);
          acc0 = dot16<DT>(w[u], x0, acc0);
          acc1 = dot16<DT>(w[u + 1], x1, acc1);
        }
      } else {
        uint4 x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int tt = t + NW * u;
          if (XL) {
            x[u] = (has && tt < KT) ? lds_ld16(smem + xl + (uint32_t)(xrow0 + u) * 64) : zero;
          } else {
            x[u] = (has && tt < KT) ? ld16(xg + (size_t)tt * TL::TK * TL::ES) : zero;
          }
        }
#pragma unroll
        for (int u = 0; u < U; u += 2) {
          if (MFMA) {
            c0 = mfma_tile<DT>(w[u], x[u], c0);
            c1 = mfma_tile<DT>(w[u + 1], x[u + 1], c1);
          } else {
            acc0 = dot16<DT>(w[u], x[u], acc0);
            acc1 = dot16<DT>(w[u + 1], x[u + 1], acc1);
          }
        }
      }
    }
    if (MFMA) {
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave][4 * (lane >> 4) + i][lane & 15] = c0[i] + c1[i];
    } else {
      float acc = acc0 + acc1;
      acc += __shfl_xor(acc, 16);
      acc += __shfl_xor(acc, 32);
      if (lane < 16) red[wave][lane][0] = acc;
    }
    __syncthreads();
    if (tid < 256) {
      const int n = tid >> 4, mm = tid & 15;
      if (MFMA || mm == 0) {
        float s = red[0][n][mm];
#pragma unroll
        for (int q = 1; q < NW; ++q) s += red[q][n][mm];
        ct[n][mm] = split_norm ? s * inv_s[mm] : s;
      }
    }
    __syncthreads();
    if (tid < 256) epilogue<DT, GS>(a, g, ct, best, qkv_c, qpre);
    __syncthreads();
    if (a.epi == EPI_RESID && a.ss_out && tid < 16) {
      float s = 0.f;
      if (tid < a.M)
        for (int n = 0; n < 16; ++n) s = fmaf(ct[n][tid], ct[n][tid], s);
      a.ss_out[tid * NG + g] = s;
    }
  }
  if (a.epi == EPI_ARGMAX && tid < 16 && tid < a.M && best)
    atomicMax((unsigned long long*)&a.keys[(blockIdx.x % KEY_SLOTS) * KEY_PITCH + tid], (unsigned long long)best);
}

// Six waves per SIMD (at most 80 VGPRs) keeps three blocks per CU.
template <int DT, int XS>
__global__ __launch_bounds__(LIN_WAVES * 64) __attribute__((amdgpu_waves_per_eu(6))) void k_linear(LinearArgs a) {
  linear_main<DT, XS, false>(a);
}
// The heads of sampled passes (2 blocks per CU): no occupancy target.
template <int DT, int XS>
__global__ __launch_bounds__(LIN_WAVES * 64) void k_linear_gs(LinearArgs a) {
  linear_main<DT, XS, true>(a);
}

// ---- launchers ----------------------------------------------------------------

hipError_t launch_repack(int dtype, const RepackArgs& a, hipStream_t s) {
  const size_t total = (size_t)a.n_groups * a.KT * 64;
  const int grid = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
  if (dtype == 1) hipLaunchKernelGGL(k_repack<1>, dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_repack<0>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

// LDS bytes of matrix-core rows staged per wavefront region.
static size_t mfma_lds_bytes(int dtype, int K, int M) {
  const int tk = dtype == 1 ? 32 : 16;
  const int KT = (K + tk - 1) / tk;
  return (size_t)LIN_WAVES * ((KT + LIN_WAVES - 1) / LIN_WAVES) * M * 64;
}

int linear_x_source(int dtype, bool mfma, int K, int M) {
  if (mfma) return mfma_lds_bytes(dtype, K, M) <= LIN_MFMA_LDS_X_MAX ? XS_MFMA_LDS : XS_MFMA;
  const int tk = dtype == 1 ? 32 : 16, es = dtype == 1 ? 2 : 4;
  return (size_t)lin_x_tiles((K + tk - 1) / tk) * tk * es <= LIN_LDS_X_MAX ? XS_LDS : XS_GLOBAL;
}

size_t linear_lds_bytes(int dtype, bool mfma, int x_mode, int K, int M) {
  (void)x_mode;
  const int xs = linear_x_source(dtype, mfma, K, M);
  if (xs == XS_MFMA_LDS) return mfma_lds_bytes(dtype, K, M);
  if (xs != XS_LDS) return 0;
  const int tk = dtype == 1 ? 32 : 16, es = dtype == 1 ? 2 : 4;
  return (size_t)lin_x_tiles((K + tk - 1) / tk) * tk * es;
}

// With events, the start / stop timestamps are taken by the dispatch itself
// (the kernel's own execution, as a kernel trace measures it).
template <int DT, int XS>
static void launch_linear_t(const LinearArgs& a, int grid, size_t lds, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  if (a.gstats) {
    if (e0)
      hipExtLaunchKernelGGL((k_linear_gs<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), (uint32_t)lds, s, e0, e1, 0, a);
    else
      hipLaunchKernelGGL((k_linear_gs<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), lds, s, a);
  } else if (e0) {
    hipExtLaunchKernelGGL((k_linear<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), (uint32_t)lds, s, e0, e1, 0, a);
  } else {
    hipLaunchKernelGGL((k_linear<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), lds, s, a);
  }
}

hipError_t launch_linear(int dtype, bool mfma, const LinearArgs& a, int grid, hipStream_t s, hipEvent_t e0,
                         hipEvent_t e1) {
  const size_t lds = linear_lds_bytes(dtype, mfma, a.x_mode, a.K, a.M);
  const int xs = linear_x_source(dtype, mfma, a.K, a.M);
  if (dtype == 1) {
    if (xs == XS_MFMA_LDS) launch_linear_t<1, XS_MFMA_LDS>(a, grid, lds, s, e0, e1);
    else if (xs == XS_MFMA) launch_linear_t<1, XS_MFMA>(a, grid, lds, s, e0, e1);
    else if (xs == XS_LDS) launch_linear_t<1, XS_LDS>(a, grid, lds, s, e0, e1);
    else launch_linear_t<1, XS_GLOBAL>(a, grid, lds, s, e0, e1);
  } else {
    if (xs == XS_MFMA_LDS) launch_linear_t<0, XS_MFMA_LDS>(a, grid, lds, s, e0, e1);
    else if (xs == XS_MFMA) launch_linear_t<0, XS_MFMA>(a, grid, lds, s, e0, e1);
    else if (xs == XS_LDS) launch_linear_t<0, XS_LDS>(a, grid, lds, s, e0, e1);
    else launch_linear_t<0, XS_GLOBAL>(a, grid, lds, s, e0, e1);
  }
  return hipGetLastError();
}

}  // namespace lede
