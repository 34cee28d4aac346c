// Inverse-CDF draws for callers that cannot allocate device memory (code
// under HIP graph capture, serving loops and harnesses that forbid
// hipMalloc).  lede_op_sample allocates a key buffer per call; this variant
// keeps the keys of up to NOALLOC_MAX_ROWS draws in a file-scope device
// array instead, so that a call allocates nothing.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/lede.h"
#include "kernels.h"

namespace {

using lede::KEY_PITCH;
using lede::KEY_WORDS;

// One key per row in the key-buffer layout of the argmax heads (row r's
// slot s at word s * KEY_PITCH + r): KEY_PITCH = 32 rows, 2 KiB.  Each device
// the library runs on holds its own copy until the process ends.  Every word
// a call reads is written by that call (the sampling kernel stores its key's
// slot 0 and clears the other slots), so nothing is cleared beforehand.
constexpr int NOALLOC_MAX_ROWS = KEY_PITCH;
static __device__ __align__(256) uint64_t scratch[KEY_WORDS];

constexpr int MAX_DEVICES = 64;
uint64_t* g_scratch[MAX_DEVICES] = {};  // device address of each device's copy (null: not looked up yet)
std::mutex g_mu;

// The device address of the current device's copy of the array, looked up
// once per device with that device current.  In host code the array's name
// is only a host-side stand-in, never a device address.
int scratch_address(uint64_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return LEDE_E_HIP;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LEDE_E_HIP;
    g_scratch[dev] = (uint64_t*)p;
  }
  *out = g_scratch[dev];
  return LEDE_OK;
}

}  // namespace

extern "C" int lede_op_sample_noalloc(const float* logits, int32_t n_rows, int32_t ld, int32_t V,
                                      float temperature, const float* u, int32_t* tokens, void* stream) {
  if (!logits || !u || !tokens || V < 1 || n_rows < 1 || ld < V) return LEDE_E_ARG;
  if (n_rows > NOALLOC_MAX_ROWS) return LEDE_E_ARG;  // more rows than the static key array holds
  if (!(temperature > 0.f) || !(temperature <= 3.402823466e38f)) return LEDE_E_ARG;
  for (int r = 0; r < n_rows; ++r)
    if (!(u[r] >= 0.f && u[r] < 1.f)) return LEDE_E_ARG;
  uint64_t* keys = nullptr;
  if (int rc = scratch_address(&keys)) return rc;
  hipStream_t s = (hipStream_t)stream;
  for (int r = 0; r < n_rows; ++r) {
    lede::SampleArgs sa{};
    sa.logits = logits + (size_t)r * ld;
    sa.vocab = V;
    sa.inv_t = 1.f / temperature;
    sa.u = nullptr;
    sa.u_imm = u[r];
    sa.key_out = keys + r;
    sa.stats_out = nullptr;
    if (lede::launch_sample(sa, s) != hipSuccess) return LEDE_E_HIP;
  }
  uint64_t h[KEY_WORDS];
  if (hipMemcpyAsync(h, keys, sizeof h, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return LEDE_E_HIP;
  for (int r = 0; r < n_rows; ++r) tokens[r] = lede::key_token(lede::key_value(h, r));
  return LEDE_OK;
}
