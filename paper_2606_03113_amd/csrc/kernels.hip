// gfx950 kernels of the self-speculative decode step.
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
#include "kernels.h"

#include <hip/hip_ext.h>
#include <math.h>

namespace lede {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// ---- scalar helpers -------------------------------------------------------

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round fp32 to bf16, nearest-even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <int DT> struct Elem;
template <> struct Elem<0> {
  typedef float T;
  static constexpr int ES_ = 4;
  static __device__ __forceinline__ float load(const void* p, size_t i) { return ((const float*)p)[i]; }
  static __device__ __forceinline__ void store(void* p, size_t i, float v) { ((float*)p)[i] = v; }
  static __device__ __forceinline__ float round(float v) { return v; }
};
template <> struct Elem<1> {
  typedef uint16_t T;
  static constexpr int ES_ = 2;
  static __device__ __forceinline__ float load(const void* p, size_t i) { return bf16_to_f32(((const uint16_t*)p)[i]); }
  static __device__ __forceinline__ void store(void* p, size_t i, float v) { ((uint16_t*)p)[i] = f32_to_bf16(v); }
  static __device__ __forceinline__ float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
};

// Orderable 64-bit argmax key: larger value first, then lower index.
__device__ __forceinline__ uint64_t argmax_key(float v, int idx) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// 16-byte loads.
__device__ __forceinline__ uint4 ld16(const void* p) { return *(const uint4*)p; }

// Dot product of one 16-byte weight fragment with one 16-byte x fragment.
template <int DT> __device__ __forceinline__ float dot16(uint4 w, uint4 x, float acc);
template <> __device__ __forceinline__ float dot16<1>(uint4 w, uint4 x, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.x), __builtin_bit_cast(bf16x2, x.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.y), __builtin_bit_cast(bf16x2, x.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.z), __builtin_bit_cast(bf16x2, x.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w.w), __builtin_bit_cast(bf16x2, x.w), acc, false);
  return acc;
}
template <> __device__ __forceinline__ float dot16<0>(uint4 w, uint4 x, float acc) {
  acc = fmaf(__uint_as_float(w.x), __uint_as_float(x.x), acc);
  acc = fmaf(__uint_as_float(w.y), __uint_as_float(x.y), acc);
  acc = fmaf(__uint_as_float(w.z), __uint_as_float(x.z), acc);
  acc = fmaf(__uint_as_float(w.w), __uint_as_float(x.w), acc);
  return acc;
}

// One matrix-core step over a 16 x TK tile: c[n][m] += W[n][k] X[m][k].
template <int DT> __device__ __forceinline__ f32x4 mfma_tile(uint4 w, uint4 x, f32x4 c);
template <> __device__ __forceinline__ f32x4 mfma_tile<1>(uint4 w, uint4 x, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, w), __builtin_bit_cast(bf16x8, x), c, 0, 0, 0);
}
template <> __device__ __forceinline__ f32x4 mfma_tile<0>(uint4 w, uint4 x, f32x4 c) {
  // four K=4 steps; slot j of every lane covers column (l >> 4) * 4 + j
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.x), __uint_as_float(x.x), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.y), __uint_as_float(x.y), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.z), __uint_as_float(x.z), c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(w.w), __uint_as_float(x.w), c, 0, 0, 0);
  return c;
}

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

// ---- RMSNorm ------------------------------------------------------------------

__device__ __forceinline__ float bf16lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

// Four consecutive elements of a row: fp32 residual h, or a model-dtype row.
template <int DT>
__device__ __forceinline__ float4 row_load4(const float* h, const void* row, int i) {
  if (h) return *(const float4*)(h + i);
  if (DT == 1) {
    const uint2 u = *(const uint2*)((const uint16_t*)row + i);
    return make_float4(bf16lo(u.x), bf16hi(u.x), bf16lo(u.y), bf16hi(u.y));
  }
  return *(const float4*)((const float*)row + i);
}

template <int DT>
__device__ __forceinline__ void store4(uint8_t* base, int i, float4 y) {
  if (DT == 1) {
    const uint32_t lo = (uint32_t)f32_to_bf16(y.x) | ((uint32_t)f32_to_bf16(y.y) << 16);
    const uint32_t hi = (uint32_t)f32_to_bf16(y.z) | ((uint32_t)f32_to_bf16(y.w) << 16);
    *(uint2*)(base + (size_t)i * 2) = make_uint2(lo, hi);
  } else {
    *(float4*)(base + (size_t)i * 4) = y;
  }
}

// RMSNorm rows for the verify / prefill path and the Q-network's state: one
// block of 256 threads per row, every load issued before the first use
// (thread t holds elements 4t + 1024 j in registers).
template <int DT>
__global__ __launch_bounds__(256) void k_norm(NormArgs a) {
  __shared__ float scratch[4];
  const int m = blockIdx.x, tid = threadIdx.x;
  if (m == 0 && a.zero_keys && tid < a.n_zero_keys) a.zero_keys[tid] = 0;
  float* h = a.h + (size_t)m * a.ldh;
  const float* src = h;
  const void* row = nullptr;
  if (a.embed) {
    // a token outside the vocabulary can only come from a fault upstream;
    // clamping keeps the read inside the table
    const int tok = (int)min((unsigned)a.tok.get(m), (unsigned)(a.vocab - 1));
    row = (const uint8_t*)a.embed_w + (size_t)tok * a.d * Elem<DT>::ES_;
    src = nullptr;
  }
  float4 v[8], g[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int i = 4 * tid + 1024 * j;
    v[j] = i < a.d ? row_load4<DT>(src, row, i) : make_float4(0.f, 0.f, 0.f, 0.f);
    g[j] = i < a.d ? row_load4<DT>(nullptr, a.gain, i) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    ss = fmaf(v[j].x, v[j].x, ss);
    ss = fmaf(v[j].y, v[j].y, ss);
    ss = fmaf(v[j].z, v[j].z, ss);
    ss = fmaf(v[j].w, v[j].w, ss);
  }
  ss = wave_sum(ss);
  if ((tid & 63) == 0) scratch[tid >> 6] = ss;
  __syncthreads();
  ss = ((scratch[0] + scratch[1]) + scratch[2]) + scratch[3];
  const float inv = rsqrtf(ss / (float)a.d + a.eps);
  uint8_t* out = (uint8_t*)a.x + (size_t)m * a.ldx * (a.f32_out ? 4 : Elem<DT>::ES_);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int i = 4 * tid + 1024 * j;
    if (i < a.d) {
      float4 y;
      y.x = (v[j].x * inv) * g[j].x;
      y.y = (v[j].y * inv) * g[j].y;
      y.z = (v[j].z * inv) * g[j].z;
      y.w = (v[j].w * inv) * g[j].w;
      if (a.embed) *(float4*)(h + i) = v[j];
      if (a.f32_out) store4<0>(out, i, y);
      else store4<DT>(out, i, y);
    }
  }
}

// ---- linear: y = W x with fused prologue / epilogue --------------------------

template <int DT>
__device__ __forceinline__ void epilogue(const LinearArgs& a, int g, float (*ct)[17], uint64_t& best) {
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
      if (m < M) a.h[(size_t)m * a.ldh + g * 16 + n] += ct[n][m];
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
      const int c = *a.seq_len + a.pos_off;
      if (g < qg + kg) {
        if (tid < 128) {
          const int r = tid >> 4, m = tid & 15;
          if (m < M) {
            const bool isq = g < qg;
            const int gl = isq ? g : g - qg;
            const int head = gl / gph, i = 8 * (gl % gph) + r;
            const int pos = c + m;
            const float2 cs = a.rope[(size_t)pos * (hd / 2) + i];
            const float x0 = ct[r][m], x1 = ct[r + 8][m];
            const float y0 = x0 * cs.x - x1 * cs.y;
            const float y1 = x1 * cs.x + x0 * cs.y;
            if (isq) {
              float* q = a.q + (size_t)m * a.ldq + head * hd;
              q[i] = y0;
              q[i + hd / 2] = y1;
            } else {
              const int page = a.block_table[pos >> 6];
              const size_t base = ((((size_t)a.layer * a.n_pages + page) * a.nkv + head) * 64 + (pos & 63)) * hd;
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
          const int page = a.block_table[pos >> 6];
          const size_t base = ((((size_t)a.layer * a.n_pages + page) * a.nkv + head) * 64 + (pos & 63)) * hd;
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
      }
      break;
    }
  }
}

// Weights are streamed once per pass: non-temporal loads keep them from
// displacing the activations and KV pages in the caches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const void* p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load((const u32x4*)p));
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
// zero-padded to the batch size the main loop reads.
template <int DT, int NW>
__device__ void stage_norm_row(const LinearArgs& a, uint8_t* lds, float* scratch) {
  constexpr int NT = NW * 64, J = (8192 + 4 * NT - 1) / (4 * NT);  // rows of up to 8192 elements
  const int tid = threadIdx.x;
  const int row_bytes = a.K * Elem<DT>::ES_, pad_bytes = lin_x_tiles(a.KT) * Tile<DT>::TK * Elem<DT>::ES_;
  for (int i = row_bytes + tid * 4; i < pad_bytes; i += NT * 4) *(uint32_t*)(lds + i) = 0u;
  const float* h = a.h;
  const void* row = nullptr;
  float* h_out = nullptr;
  if (a.x_mode == X_EMBED_NORM) {
    const int tok = (int)min((unsigned)a.tok.get(0), (unsigned)(a.vocab - 1));
    row = (const uint8_t*)a.embed + (size_t)tok * a.K * Elem<DT>::ES_;
    if (blockIdx.x == 0) h_out = a.h;
    h = nullptr;
  }
  float4 v[J], g[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int i = 4 * tid + 4 * NT * j;
    const bool in = i < a.K;
    v[j] = in ? row_load4<DT>(h, row, i) : make_float4(0.f, 0.f, 0.f, 0.f);
    g[j] = in ? row_load4<DT>(nullptr, a.gain, i) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    ss = fmaf(v[j].x, v[j].x, ss);
    ss = fmaf(v[j].y, v[j].y, ss);
    ss = fmaf(v[j].z, v[j].z, ss);
    ss = fmaf(v[j].w, v[j].w, ss);
  }
  ss = block_sum<NW>(ss, scratch);
  const float inv = rsqrtf(ss / (float)a.K + a.eps);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int i = 4 * tid + 4 * NT * j;
    if (i < a.K) {
      float4 y;
      y.x = (v[j].x * inv) * g[j].x;
      y.y = (v[j].y * inv) * g[j].y;
      y.z = (v[j].z * inv) * g[j].z;
      y.w = (v[j].w * inv) * g[j].w;
      if (h_out) *(float4*)(h_out + i) = v[j];
      store4<DT>(lds, i, y);
    }
  }
  __syncthreads();
}

// Copy the vector kernel's input row (KT tiles of the model dtype) into LDS
// and zero the padding up to pad bytes.
template <int NW>
__device__ void stage_copy_row(const void* x, int bytes, int pad, uint8_t* lds) {
  for (int i = threadIdx.x * 16; i < pad; i += NW * 64 * 16)
    *(uint4*)(lds + i) = i < bytes ? ld16((const uint8_t*)x + i) : make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
}

// y = W x over 16-row groups, one group per block pass.  Eight wavefronts
// split K (wave w takes tiles w, w + 8, ...), four tiles per wave in flight,
// and the partials are summed in wave order.
//   XS = XS_LDS:    one input row, staged in LDS in the prologue (normalised
//                   for X_NORM / X_EMBED_NORM, copied otherwise); dot2 math.
//   XS = XS_GLOBAL: one input row read from global memory per tile (rows too
//                   long for LDS); dot2 math.
//   XS = XS_MFMA:   up to 16 rows read from global memory (normalised by the
//                   norm kernel), 16x16 matrix-core tiles.
template <int DT, int XS>
__global__ __launch_bounds__(LIN_WAVES * 64) void k_linear(LinearArgs a) {
  typedef Tile<DT> TL;
  constexpr int NW = LIN_WAVES, U = 4;  // tiles per wave per batch
  constexpr bool MFMA = XS == XS_MFMA;
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ float red[NW][16][16];
  __shared__ float ct[16][17];
  __shared__ float scratch[NW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int KT = a.KT, NG = a.n_groups;
  const uint4 zero = {0u, 0u, 0u, 0u};

  if (blockIdx.x == 0 && a.zero_keys && tid < a.n_zero_keys) a.zero_keys[tid] = 0;

  int g = blockIdx.x;
  // the weights do not depend on the input: the first batch is in flight
  // while the prologue stages the input row
  uint4 w[U];
  {
    const uint8_t* wg = a.w + (size_t)(g < NG ? g : 0) * KT * TILE_BYTES + lane * 16;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = wave + NW * u;
      w[u] = (g < NG && t < KT) ? ld16_stream(wg + (size_t)t * TILE_BYTES) : zero;
    }
  }
  if (XS == XS_LDS) {
    if (a.x_mode == X_NORM || a.x_mode == X_EMBED_NORM) stage_norm_row<DT, NW>(a, smem, scratch);
    else stage_copy_row<NW>(a.x, KT * TL::TK * TL::ES, lin_x_tiles(KT) * TL::TK * TL::ES, smem);
  }

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
    for (int t = wave; t < KT; t += NW * U) {
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
          x[u] = (has && tt < KT) ? ld16(xg + (size_t)tt * TL::TK * TL::ES) : zero;
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
        ct[n][mm] = s;
      }
    }
    __syncthreads();
    if (tid < 256) epilogue<DT>(a, g, ct, best);
    __syncthreads();
  }
  if (a.epi == EPI_ARGMAX && tid < 16 && tid < a.M && best)
    atomicMax((unsigned long long*)&a.keys[tid], (unsigned long long)best);
}

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

// ---- Q-network output layer + argmax ----------------------------------------

// One wavefront per action: q[j] = sum_i W2[j][i] hid[i] + b2[j]; argmax with
// the lowest index on ties.
__global__ __launch_bounds__(256) void k_qnet_out(QnetOutArgs a) {
  __shared__ unsigned long long best[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  uint64_t b = 0;
  for (int j = wave; j < a.A; j += 4) {
    float s = 0.f;
    for (int i = lane; i < a.H; i += 64) s = fmaf(a.w2[(size_t)j * a.H + i], a.hid[i], s);
    s = wave_sum(s) + a.b2[j];
    if (lane == 0) a.qv[j] = s;
    const uint64_t key = argmax_key(s, j);
    b = key > b ? key : b;
  }
  if (lane == 0) best[wave] = b;
  __syncthreads();
  if (tid == 0) {
    uint64_t m = best[0];
    for (int w = 1; w < 4; ++w) m = best[w] > m ? best[w] : m;
    const int idx = (int)(0xFFFFFFFFu - (uint32_t)(m & 0xFFFFFFFFull));
    a.action[0] = idx;
    uint32_t u = (uint32_t)(m >> 32);
    u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;  // undo the key's ordering transform
    a.action[1] = (int)u;
  }
}

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

__global__ void k_fill_u64(uint64_t* p, uint64_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_set_token(uint64_t* keys, int idx, int token) {
  if (threadIdx.x == 0) keys[idx] = (uint64_t)(0xFFFFFFFFu - (uint32_t)token);
}

// Achievable-bandwidth probe: every 16-byte chunk of src is read once with
// the same non-temporal loads the linear kernels stream weights with, eight
// loads in flight per lane; the XOR of the data goes to sink[block] so that no
// load can be dropped.
__global__ __launch_bounds__(256) void k_read_probe(const uint8_t* src, size_t n16, uint32_t* sink) {
  const size_t stride = (size_t)gridDim.x * 256;
  size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    uint4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = ld16_stream(src + (i + u * stride) * 16);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const uint4 v = ld16_stream(src + i * 16);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  __shared__ uint32_t red[4];
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

// ---- launchers ----------------------------------------------------------------

hipError_t launch_repack(int dtype, const RepackArgs& a, hipStream_t s) {
  const size_t total = (size_t)a.n_groups * a.KT * 64;
  const int grid = (int)((total + 255) / 256 < 65536 ? (total + 255) / 256 : 65536);
  if (dtype == 1) hipLaunchKernelGGL(k_repack<1>, dim3(grid), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_repack<0>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t s) {
  if (dtype == 1) hipLaunchKernelGGL(k_norm<1>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_norm<0>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

int linear_x_source(int dtype, bool mfma, int K) {
  if (mfma) return XS_MFMA;
  const int tk = dtype == 1 ? 32 : 16, es = dtype == 1 ? 2 : 4;
  return (size_t)lin_x_tiles((K + tk - 1) / tk) * tk * es <= LIN_LDS_X_MAX ? XS_LDS : XS_GLOBAL;
}

size_t linear_lds_bytes(int dtype, bool mfma, int x_mode, int K, int M) {
  (void)M;
  if (linear_x_source(dtype, mfma, K) != XS_LDS) return 0;
  const int tk = dtype == 1 ? 32 : 16, es = dtype == 1 ? 2 : 4;
  const size_t row = (size_t)lin_x_tiles((K + tk - 1) / tk) * tk * es;
  (void)x_mode;
  return row;
}

// With events, the start / stop timestamps are taken by the dispatch itself
// (the kernel's own execution, as a kernel trace measures it).
template <int DT, int XS>
static void launch_linear_t(const LinearArgs& a, int grid, size_t lds, hipStream_t s, hipEvent_t e0,
                            hipEvent_t e1) {
  if (e0)
    hipExtLaunchKernelGGL((k_linear<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), (uint32_t)lds, s, e0, e1, 0, a);
  else
    hipLaunchKernelGGL((k_linear<DT, XS>), dim3(grid), dim3(LIN_WAVES * 64), lds, s, a);
}

hipError_t launch_linear(int dtype, bool mfma, const LinearArgs& a, int grid, hipStream_t s, hipEvent_t e0,
                         hipEvent_t e1) {
  const size_t lds = linear_lds_bytes(dtype, mfma, a.x_mode, a.K, a.M);
  const int xs = linear_x_source(dtype, mfma, a.K);
  if (dtype == 1) {
    if (xs == XS_MFMA) launch_linear_t<1, XS_MFMA>(a, grid, lds, s, e0, e1);
    else if (xs == XS_LDS) launch_linear_t<1, XS_LDS>(a, grid, lds, s, e0, e1);
    else launch_linear_t<1, XS_GLOBAL>(a, grid, lds, s, e0, e1);
  } else {
    if (xs == XS_MFMA) launch_linear_t<0, XS_MFMA>(a, grid, lds, s, e0, e1);
    else if (xs == XS_LDS) launch_linear_t<0, XS_LDS>(a, grid, lds, s, e0, e1);
    else launch_linear_t<0, XS_GLOBAL>(a, grid, lds, s, e0, e1);
  }
  return hipGetLastError();
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

hipError_t launch_qnet_out(const QnetOutArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_qnet_out, dim3(1), dim3(256), 0, s, a);
  return hipGetLastError();
}

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

hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* sink, int grid, hipStream_t s,
                             hipEvent_t e0, hipEvent_t e1) {
  if (e0)
    hipExtLaunchKernelGGL(k_read_probe, dim3(grid), dim3(256), 0, s, e0, e1, 0, (const uint8_t*)src, bytes / 16,
                          sink);
  else
    hipLaunchKernelGGL(k_read_probe, dim3(grid), dim3(256), 0, s, (const uint8_t*)src, bytes / 16, sink);
  return hipGetLastError();
}

hipError_t launch_fill_u64(uint64_t* p, uint64_t v, int n, hipStream_t s) {
  hipLaunchKernelGGL(k_fill_u64, dim3((n + 255) / 256), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

hipError_t launch_set_token(uint64_t* keys, int idx, int token, hipStream_t s) {
  hipLaunchKernelGGL(k_set_token, dim3(1), dim3(64), 0, s, keys, idx, token);
  return hipGetLastError();
}

}  // namespace lede
