// Device-side helpers shared by the gfx950 kernels of the decode step:
// bf16 conversions, element access by model dtype, argmax keys, wavefront
// reductions, and the tile dot products of the weight-streaming kernels.
#pragma once

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

// Weights are streamed once per pass: non-temporal loads keep them from
// displacing the activations and KV pages in the caches.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld16_stream(const void* p) {
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load((const u32x4*)p));
}

// ---- row access --------------------------------------------------------------

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

}  // namespace lede
