// Small kernels of the decode step: the Q-network output layer, key fills,
// and the achievable-bandwidth probe (gfx950).
#include "device.h"

namespace lede {

// ---- Q-network output layer + argmax ----------------------------------------

// q[j] = sum_i W2[j][i] hid[i] + b2[j] for every action j, with 16
// wavefronts taking actions j = w, w + 16, ...; argmax with the lowest index
// on ties.  Lane l sums i = l, l + 64, ... in order.  Up to QNA actions per
// wavefront and QNC 64-wide chunks of the hidden layer, every load is issued
// before the first sum (one memory round trip); larger networks loop.
constexpr int QNW = 16, QNA = 4, QNC = 4;
__global__ __launch_bounds__(QNW * 64) void k_qnet_out(QnetOutArgs a) {
  __shared__ unsigned long long best[QNW];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  uint64_t b = 0;
  if (a.A <= QNW * QNA && a.H <= 64 * QNC) {
    float hv[QNC], wv[QNA][QNC], bv[QNA];
#pragma unroll
    for (int c = 0; c < QNC; ++c) hv[c] = lane + 64 * c < a.H ? a.hid[lane + 64 * c] : 0.f;
#pragma unroll
    for (int q = 0; q < QNA; ++q) {
      const int j = wave + QNW * q;
      bv[q] = j < a.A ? a.b2[j] : 0.f;
#pragma unroll
      for (int c = 0; c < QNC; ++c)
        wv[q][c] = (j < a.A && lane + 64 * c < a.H) ? a.w2[(size_t)j * a.H + lane + 64 * c] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < QNA; ++q) {
      const int j = wave + QNW * q;
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < QNC; ++c) s = fmaf(wv[q][c], hv[c], s);
      s = wave_sum(s) + bv[q];
      if (j < a.A) {
        if (lane == 0) a.qv[j] = s;
        const uint64_t key = argmax_key(s, j);
        b = key > b ? key : b;
      }
    }
  } else {
    for (int j = wave; j < a.A; j += QNW) {
      float s = 0.f;
      for (int i = lane; i < a.H; i += 64) s = fmaf(a.w2[(size_t)j * a.H + i], a.hid[i], s);
      s = wave_sum(s) + a.b2[j];
      if (lane == 0) a.qv[j] = s;
      const uint64_t key = argmax_key(s, j);
      b = key > b ? key : b;
    }
  }
  if (lane == 0) best[wave] = b;
  __syncthreads();
  if (tid == 0) {
    uint64_t m = best[0];
    for (int w = 1; w < QNW; ++w) m = best[w] > m ? best[w] : m;
    const int idx = (int)(0xFFFFFFFFu - (uint32_t)(m & 0xFFFFFFFFull));
    a.action[0] = idx;
    uint32_t u = (uint32_t)(m >> 32);
    u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;  // undo the key's ordering transform
    a.action[1] = (int)u;
  }
}

__global__ void k_fill_u64(uint64_t* p, uint64_t v, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_set_token(uint64_t* keys, int idx, int token) {
  if (threadIdx.x == 0) key_store_token(keys, idx, token);
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

// Reads n_groups x tiles tiles of TILE_BYTES with the one-row linear kernel's
// load structure and nothing else: one group per block, LIN_WAVES wavefronts
// splitting the group's tiles, LIN_TILES_PER_WAVE non-temporal 16-byte loads
// per lane in flight per batch.  The XOR of the data goes to sink[block].
__global__ __launch_bounds__(LIN_WAVES * 64) void k_read_groups(const uint8_t* src, int tiles, uint32_t* sink) {
  constexpr int NW = LIN_WAVES, U = LIN_TILES_PER_WAVE;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint8_t* base = src + (size_t)blockIdx.x * tiles * TILE_BYTES + lane * 16;
  uint32_t acc = 0;
  for (int t0 = wave; t0 < tiles; t0 += NW * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + NW * u;
      v[u] = t < tiles ? ld16_stream(base + (size_t)t * TILE_BYTES) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  __shared__ uint32_t red[NW];
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  if (lane == 0) red[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = 0;
    for (int w = 0; w < NW; ++w) x ^= red[w];
    sink[blockIdx.x] = x;
  }
}

// ---- launchers ----------------------------------------------------------------

hipError_t launch_qnet_out(const QnetOutArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_qnet_out, dim3(1), dim3(QNW * 64), 0, s, a);
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

hipError_t launch_read_groups(const void* src, int n_groups, int tiles, uint32_t* sink, hipStream_t s,
                              hipEvent_t e0, hipEvent_t e1) {
  if (e0)
    hipExtLaunchKernelGGL(k_read_groups, dim3(n_groups), dim3(LIN_WAVES * 64), 0, s, e0, e1, 0, (const uint8_t*)src,
                          tiles, sink);
  else
    hipLaunchKernelGGL(k_read_groups, dim3(n_groups), dim3(LIN_WAVES * 64), 0, s, (const uint8_t*)src, tiles, sink);
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
