/*
 * Host sanitizer run of the CPU oracle (test infrastructure): the oracle's C
 * source is compiled into this driver with AddressSanitizer and
 * UndefinedBehaviorSanitizer, and every exported routine runs on a tiny
 * grouped-query model in both precisions.  Besides memory and UB errors it
 * checks one invariant the oracle states: a row's result does not depend on
 * the other rows of the call (a batch of T tokens equals T one-token calls).
 * Exit status 0 when everything ran clean.
 */
#include "../../oracle/lede_oracle.c"

#include <stdio.h>

static uint32_t rng = 2463534242u;
static double urand(void) {  /* xorshift32, uniform in [-1, 1) */
  rng ^= rng << 13;
  rng ^= rng >> 17;
  rng ^= rng << 5;
  return (rng >> 8) / 8388608.0 - 1.0;
}

/* n weights with scale s: bf16 bit patterns or float32 */
static void* weights(int is_bf16, size_t n, double s) {
  if (is_bf16) {
    uint16_t* w = malloc(n * 2);
    for (size_t i = 0; i < n; ++i) {
      float f = (float)(urand() * s);
      uint32_t u;
      memcpy(&u, &f, 4);
      w[i] = (uint16_t)(u >> 16);
    }
    return w;
  }
  float* w = malloc(n * 4);
  for (size_t i = 0; i < n; ++i) w[i] = (float)(urand() * s);
  return w;
}

static int run(int is_bf16) {
  OracleModel M;
  memset(&M, 0, sizeof M);
  M.n_layers = 2; M.d = 64; M.nq = 4; M.nkv = 2; M.hd = 16; M.ffn = 96; M.vocab = 50;
  M.is_bf16 = is_bf16; M.max_ctx = 24; M.eps = 1e-5; M.rope_base = 10000.0;
  const int d = M.d, qd = M.nq * M.hd, kvd = M.nkv * M.hd, F = M.ffn, L = M.n_layers;
  M.embed = weights(is_bf16, (size_t)M.vocab * d, 1.0);
  M.final_norm = weights(is_bf16, d, 1.0);
  M.head = weights(is_bf16, (size_t)M.vocab * d, 0.2);
  const void** tab[9];
  for (int i = 0; i < 9; ++i) tab[i] = malloc(sizeof(void*) * L);
  for (int l = 0; l < L; ++l) {
    tab[0][l] = weights(is_bf16, d, 1.0);
    tab[1][l] = weights(is_bf16, (size_t)qd * d, 0.2);
    tab[2][l] = weights(is_bf16, (size_t)kvd * d, 0.2);
    tab[3][l] = weights(is_bf16, (size_t)kvd * d, 0.2);
    tab[4][l] = weights(is_bf16, (size_t)d * qd, 0.2);
    tab[5][l] = weights(is_bf16, d, 1.0);
    tab[6][l] = weights(is_bf16, (size_t)F * d, 0.2);
    tab[7][l] = weights(is_bf16, (size_t)F * d, 0.2);
    tab[8][l] = weights(is_bf16, (size_t)d * F, 0.2);
  }
  M.attn_norm = tab[0]; M.wq = tab[1]; M.wk = tab[2]; M.wv = tab[3]; M.wo = tab[4];
  M.ffn_norm = tab[5]; M.wg = tab[6]; M.wu = tab[7]; M.wd = tab[8];
  const size_t cache = (size_t)L * M.max_ctx * kvd;
  M.kcache = calloc(cache, sizeof(double));
  M.vcache = calloc(cache, sizeof(double));

  enum { T = 9 };
  int32_t tok[T];
  for (int t = 0; t < T; ++t) tok[t] = (int32_t)((urand() + 1.0) * 0.5 * M.vocab) % M.vocab;
  double* hb = malloc(sizeof(double) * T * d);
  double* h1 = malloc(sizeof(double) * T * d);
  int bad = 0;
  /* a batch of T rows, then the same rows one at a time over the same cache */
  bad |= oracle_forward(&M, tok, T, 0, L, hb) != 0;
  for (int t = 0; t < T; ++t) bad |= oracle_forward(&M, tok + t, 1, t, L, h1 + (size_t)t * d) != 0;
  for (size_t i = 0; i < (size_t)T * d; ++i)
    if (hb[i] != h1[i]) {
      fprintf(stderr, "row %zu differs between batch and one-row calls\n", i / d);
      bad = 1;
      break;
    }
  /* an early exit and the head on every row */
  double* he = malloc(sizeof(double) * T * d);
  bad |= oracle_forward(&M, tok, T, 0, 1, he) != 0;
  double* logits = malloc(sizeof(double) * T * M.vocab);
  double* normed = malloc(sizeof(double) * T * d);
  bad |= oracle_head(&M, hb, T, logits, normed) != 0;
  bad |= oracle_head(&M, he, T, logits, NULL) != 0;
  /* rejected arguments */
  bad |= oracle_forward(&M, tok, T, M.max_ctx - 2, L, hb) != -1;
  int32_t wrong = M.vocab;
  bad |= oracle_forward(&M, &wrong, 1, 0, L, hb) != -1;
  bad |= oracle_forward(&M, tok, 1, 0, L + 1, hb) != -1;
  /* the exported pieces */
  double q[16], K[5 * 16], V[5 * 16], out[16], pr[5], g[16], y[16];
  for (int i = 0; i < 16; ++i) { q[i] = urand(); g[i] = 1.0 + 0.1 * urand(); }
  for (int i = 0; i < 5 * 16; ++i) { K[i] = urand(); V[i] = urand(); }
  oracle_attend(q, K, V, 5, 16, out, pr);
  double psum = 0.0;
  for (int j = 0; j < 5; ++j) psum += pr[j];
  bad |= fabs(psum - 1.0) > 1e-12;
  oracle_rope(q, 16, 7, 10000.0);
  oracle_rmsnorm_f64(q, g, 16, 1e-5, y);
  float wf[3 * 16], bf[3];
  for (int i = 0; i < 3 * 16; ++i) wf[i] = (float)urand();
  for (int i = 0; i < 3; ++i) bf[i] = (float)urand();
  oracle_linear_f32(wf, bf, 3, 16, y, out);
  oracle_matvec(M.head, is_bf16, M.vocab, d, hb, 2, logits);
  bad |= oracle_round_bf16(1.0 + 1.0 / 512.0) != 1.0;  /* ties to even */

  free(hb); free(h1); free(he); free(logits); free(normed);
  free(M.kcache); free(M.vcache);
  free((void*)M.embed); free((void*)M.final_norm); free((void*)M.head);
  for (int i = 0; i < 9; ++i) {
    for (int l = 0; l < L; ++l) free((void*)tab[i][l]);
    free(tab[i]);
  }
  return bad;
}

int main(void) {
  int bad = run(0) | run(1);
  printf(bad ? "oracle sanitizer run: FAILED\n" : "oracle sanitizer run: clean\n");
  return bad;
}
