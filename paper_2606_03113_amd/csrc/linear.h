// Interface of the weight-streaming linear kernels (linear.hip): the tiled
// weight layout, the argument block, the kernel shape and the launchers.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lede {

// Tiled weight layout streamed by the linear kernels.  A tile is 16 rows x
// TK columns stored as 64 lanes x 16 bytes: lane l holds row (l & 15) and
// the EPL consecutive columns starting at (l >> 4) * EPL.  This is the A
// operand layout of the 16x16 matrix-core instructions, so a tile is one
// coalesced 1 KiB wave load for both the vector and the matrix kernels.
// The tiles of a 16-row group are contiguous along K.
constexpr int TILE_BYTES = 1024;
template <int DT> struct Tile;
template <> struct Tile<0> { static constexpr int TK = 16, EPL = 4, ES = 4; };  // fp32
template <> struct Tile<1> { static constexpr int TK = 32, EPL = 8, ES = 2; };  // bf16

inline int tile_k(int dtype) { return dtype == 1 ? 32 : 16; }
inline int k_tiles(int dtype, int K) { int tk = tile_k(dtype); return (K + tk - 1) / tk; }
inline size_t tiled_bytes(int dtype, int N, int K) {
  return (size_t)((N + 15) / 16) * k_tiles(dtype, K) * TILE_BYTES;
}

// Row orders of a tiled matrix (row r of tile-group g holds logical row ...).
enum RowOrder : int {
  ROWS_PLAIN = 0,   // 16g + r
  ROWS_ROPE = 1,    // rotary pairs: within each head of `hd` rows, group t holds dims
                    // 8t..8t+7 (r < 8) and hd/2 + 8t .. (r >= 8)
  ROWS_GATE = 2,    // gate/up interleave, source A: rows 0..7 of group t = A[8t..8t+7]
  ROWS_UP = 3,      // source B: rows 8..15 of group t = B[8t..8t+7]
};

struct RepackArgs {
  const void* src;  // logical [N][K] row-major, model dtype
  int N, K;         // logical rows / columns of src
  void* dst;        // tiled matrix
  int KT;           // tiles along K in dst
  int group0;       // first tile-group of dst written
  int n_groups;     // tile-groups written
  int order;        // RowOrder
  int hd;           // head dim for ROWS_ROPE
};

// Where a linear kernel's input rows come from.
enum XMode : int {
  X_PLAIN = 0,     // x [M][ldx] in model dtype, used as is
  X_NORM = 1,      // RMSNorm(h[m]) * gain, rounded to model dtype (h fp32 [M][ldh])
  X_EMBED_NORM = 2,// as X_NORM, but h[m] = embed[token m] (also stored to h by block 0)
  X_F32 = 3,       // x fp32 [M][ldx] (the Q-network's fp32 layers)
};

// Argmax keys.  Logical key i of a key buffer is spread over KEY_SLOTS words,
// keys[s * KEY_PITCH + i] for s < KEY_SLOTS, 256 bytes apart: block b of a
// head raises word b mod KEY_SLOTS with its atomic maximum, so that the
// blocks of one launch contend on eight addresses instead of one, and the
// key is the largest of its words.  A single writer stores word 0 and clears
// the others.  A key buffer holds KEY_PITCH logical keys.
constexpr int KEY_SLOTS = 8;
constexpr int KEY_PITCH = 32;
constexpr int KEY_WORDS = KEY_SLOTS * KEY_PITCH;

__host__ __device__ inline uint64_t key_value(const uint64_t* keys, int i) {
  uint64_t m = keys[i];
  for (int s = 1; s < KEY_SLOTS; ++s) {
    const uint64_t v = keys[s * KEY_PITCH + i];
    m = v > m ? v : m;
  }
  return m;
}
__host__ __device__ inline int key_token(uint64_t key) { return (int)(0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFull)); }
__host__ __device__ inline void key_store_token(uint64_t* keys, int i, int token) {
  keys[i] = (uint64_t)(0xFFFFFFFFu - (uint32_t)token);
  for (int s = 1; s < KEY_SLOTS; ++s) keys[s * KEY_PITCH + i] = 0;
}

// Token sources: int32 array, or argmax keys.
struct TokenSrc {
  const int32_t* ids;   // if non-null
  const uint64_t* keys; // else decode logical key i
  __host__ __device__ int get(int i) const { return ids ? ids[i] : key_token(key_value(keys, i)); }
};

// Epilogues.
enum Epi : int {
  EPI_STORE = 0,   // out[m][n] = acc
  EPI_RESID = 1,   // h[m][n] += acc
  EPI_QKV = 2,     // rotary on q/k, q -> qbuf, k/v rounded into the paged cache
  EPI_SWIGLU = 3,  // act[m][f] = round(silu(gate) * up)
  EPI_ARGMAX = 4,  // logits (debug) + per-row argmax key (atomic max)
  EPI_BIAS_RELU = 5// out[n] = max(acc + bias[n], 0)  (fp32, M = 1)
};

struct LinearArgs {
  const uint8_t* w;  // tiled weights
  int n_groups;      // 16-row groups
  int KT;            // tiles along K
  int K;             // logical K (columns of x used)
  int M;             // rows of x (1..16)
  int groups_per_block;
  // input
  int x_mode;
  const void* x; int ldx;          // X_PLAIN / X_F32
  float* h; int ldh;               // X_NORM / X_EMBED_NORM (and EPI_RESID target)
  const void* gain; float eps;
  const void* embed; TokenSrc tok;
  uint64_t* zero_keys; int n_zero_keys;  // logical keys cleared by block 0 (every slot; of a later head)
  // epilogue
  int epi;
  float* out; int ldo;             // EPI_STORE / EPI_BIAS_RELU
  const float* bias;
  // EPI_QKV
  float* q; int ldq;               // [M][nq*hd]
  void* kcache; void* vcache;      // [L][n_pages][nkv][64][hd]
  int layer, n_pages, nq, nkv, hd;
  const int32_t* block_table; const int32_t* seq_len; int pos_off;
  const float2* rope;              // [max_ctx][hd/2] (cos, sin)
  // EPI_SWIGLU
  void* act; int ld_act;
  // EPI_ARGMAX
  uint64_t* keys; float* logits; int ld_logits; int vocab;
  // optional, with logits: per 16-token group g of row m, (max z, sum of
  // exp((z - max) * inv_t)) at gstats[m * ld_gstats + g]
  float2* gstats; int ld_gstats; float inv_t;
  // RMSNorm split over two kernels.  A residual producer (EPI_RESID) with
  // ss_out also stores xg[m][n] = h[m][n] * xg_gain[n] in the model dtype and,
  // per 16-column group g of its n_groups, the sum of squares of its columns
  // of each new residual row, ss_out[m * n_groups + g] (rows 0..15).  A
  // consumer with ss_in (the matrix-core kernel, or the one-row kernel with
  // x_mode X_PLAIN) reads x = xg and scales output row m by
  // 1 / sqrt(sum over the ss_groups partials of row m / K + eps).
  float* ss_out; const void* xg_gain; void* xg; int ldxg;
  const float* ss_in; int ss_groups;
};
constexpr int SS_MAX_GROUPS = 512;  // rows of up to 8192 elements

// Linear kernel shape: wavefronts per block, and where the input row comes
// from (see k_linear).  Rows longer than LIN_LDS_X_MAX bytes are read from
// global memory instead of being staged in LDS.
constexpr int LIN_WAVES = 8;
constexpr int LIN_LDS_X_MAX = 32768;
constexpr int LIN_TILES_PER_WAVE = 4;  // tiles each wavefront has in flight per batch
enum XSource { XS_LDS = 0, XS_GLOBAL = 1, XS_MFMA = 2, XS_MFMA_LDS = 3 };
// Matrix-core input rows are staged in LDS when they take at most this many
// bytes (three blocks of 512 threads still fit a CU's 160 KiB).
constexpr int LIN_MFMA_LDS_X_MAX = 48 * 1024;
// K tiles the staged row is zero-padded to, so that every batch reads it
// without bounds checks.
__host__ __device__ inline int lin_x_tiles(int KT) {
  const int b = LIN_WAVES * LIN_TILES_PER_WAVE;
  return (KT + b - 1) / b * b;
}
int linear_x_source(int dtype, bool mfma, int K, int M);

// Bytes of dynamic LDS the linear kernels use for the staged input row.
size_t linear_lds_bytes(int dtype, bool mfma, int x_mode, int K, int M);

hipError_t launch_repack(int dtype, const RepackArgs& a, hipStream_t s);
// e0 / e1 (optional): events recorded by the dispatch at kernel start / end.
hipError_t launch_linear(int dtype, bool mfma, const LinearArgs& a, int grid, hipStream_t s,
                         hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);

}  // namespace lede
