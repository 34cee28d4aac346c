// RMSNorm rows of the verify / prefill path and the Q-network state (gfx950).
#include "device.h"

namespace lede {

// RMSNorm rows for the verify / prefill path and the Q-network's state: one
// block of 256 threads per row, every load issued before the first use
// (thread t holds elements 4t + 1024 j in registers).
template <int DT>
__global__ __launch_bounds__(256) void k_norm(NormArgs a) {
  __shared__ float scratch[4];
  const int m = blockIdx.x, tid = threadIdx.x;
  if (m == 0 && a.zero_keys && tid < KEY_WORDS && (tid % KEY_PITCH) < a.n_zero_keys) a.zero_keys[tid] = 0;
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
  // unconditional loads (a thread past the row re-reads its first elements),
  // zeroed afterwards, and the row's source chosen outside the loops: a
  // guarded load compiles to a branch and a wait
  float4 v[8], g[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int i = 4 * tid + 1024 * j;
    g[j] = row_load4<DT>(nullptr, a.gain, i < a.d ? i : 0);
  }
  if (src) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = 4 * tid + 1024 * j;
      v[j] = row_load4<DT>(src, nullptr, i < a.d ? i : 0);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int i = 4 * tid + 1024 * j;
      v[j] = row_load4<DT>(nullptr, row, i < a.d ? i : 0);
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const bool in = 4 * tid + 1024 * j < a.d;
    v[j].x = in ? v[j].x : 0.f; v[j].y = in ? v[j].y : 0.f; v[j].z = in ? v[j].z : 0.f; v[j].w = in ? v[j].w : 0.f;
    g[j].x = in ? g[j].x : 0.f; g[j].y = in ? g[j].y : 0.f; g[j].z = in ? g[j].z : 0.f; g[j].w = in ? g[j].w : 0.f;
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

hipError_t launch_norm(int dtype, const NormArgs& a, hipStream_t s) {
  if (dtype == 1) hipLaunchKernelGGL(k_norm<1>, dim3(a.M), dim3(256), 0, s, a);
  else hipLaunchKernelGGL(k_norm<0>, dim3(a.M), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace lede
