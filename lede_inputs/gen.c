/*
 * Seeded synthetic-input generator shared by the CPU oracle and the GPU path.
 *
 * It holds none of the decoding method's arithmetic: it only turns
 * (seed, stream, element index) into numbers.  Every element is a pure
 * function of that triple, so any slice of any tensor can be regenerated
 * independently and the output does not depend on the thread count.
 *
 * Bit source: Philox4x32-10, the counter-based generator published by
 * Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as
 * 1, 2, 3" (SC'11).  Key = (seed, stream); counter = (i_lo, i_hi, 0, 0).
 *
 * Normal deviates: the Box-Muller transform (Box and Muller, 1958) of two
 * 53-bit uniforms taken from one Philox block, evaluated in double.  Element
 * e uses block e/2; even elements take the cosine branch, odd the sine.
 * A weight is (float)(std * z) (round-to-nearest-even), and a bf16 weight
 * is that float rounded to nearest-even at 8 significant bits.
 *
 * Integers: lo + (u64 mod (hi - lo + 1)) with u64 from block e.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox4x32_10(uint32_t ctr[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * ctr[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * ctr[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ ctr[1] ^ k0;
    uint32_t n2 = hi0 ^ ctr[3] ^ k1;
    ctr[0] = n0;
    ctr[1] = lo1;
    ctr[2] = n2;
    ctr[3] = lo0;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
}

static inline void block(uint32_t seed, uint32_t stream, uint64_t i, uint32_t out[4]) {
  out[0] = (uint32_t)i;
  out[1] = (uint32_t)(i >> 32);
  out[2] = 0;
  out[3] = 0;
  philox4x32_10(out, seed, stream);
}

/* Standard normal deviate for element e of (seed, stream). */
static inline double normal_at(uint32_t seed, uint32_t stream, uint64_t e) {
  uint32_t x[4];
  block(seed, stream, e >> 1, x);
  uint64_t a = (((uint64_t)x[1] << 32) | x[0]) >> 11; /* 53 bits */
  uint64_t b = (((uint64_t)x[3] << 32) | x[2]) >> 11;
  double u1 = ((double)a + 1.0) * 0x1.0p-53; /* (0, 1] */
  double u2 = (double)b * 0x1.0p-53;         /* [0, 1) */
  double r = sqrt(-2.0 * log(u1));
  double t = 6.283185307179586476925286766559 * u2;
  return (e & 1) ? r * sin(t) : r * cos(t);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

void lede_gen_normal_f32(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, double std,
                         float* out) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < (int64_t)n; ++j) out[j] = (float)(std * normal_at(seed, stream, offset + (uint64_t)j));
}

void lede_gen_normal_bf16(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, double std,
                          uint16_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t j = 0; j < (int64_t)n; ++j)
    out[j] = f32_to_bf16_rne((float)(std * normal_at(seed, stream, offset + (uint64_t)j)));
}

void lede_gen_uniform_int(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, int32_t lo,
                          int32_t hi, int32_t* out) {
  uint64_t span = (uint64_t)((int64_t)hi - (int64_t)lo + 1);
  for (uint64_t j = 0; j < n; ++j) {
    uint32_t x[4];
    block(seed, stream, offset + j, x);
    uint64_t u = ((uint64_t)x[1] << 32) | x[0];
    out[j] = (int32_t)((int64_t)lo + (int64_t)(u % span));
  }
}

/* Uniform floats in [0, 1): element j takes the first word of Philox block
 * (offset + j) and keeps its top 24 bits, so every value is an exact float. */
void lede_gen_uniform01(uint32_t seed, uint32_t stream, uint64_t offset, uint64_t n, float* out) {
  for (uint64_t j = 0; j < n; ++j) {
    uint32_t x[4];
    block(seed, stream, offset + j, x);
    out[j] = (float)(x[0] >> 8) * (1.0f / 16777216.0f);
  }
}

/* Raw Philox block, exported so tests can check the generator against the
 * known-answer vectors published with the Random123 library. */
void lede_gen_philox_block(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0, uint32_t k1,
                           uint32_t out[4]) {
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
  philox4x32_10(out, k0, k1);
}
