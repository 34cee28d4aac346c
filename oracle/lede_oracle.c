/*
 * CPU ORACLE -- test infrastructure only.  Only tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this file's library.  It shares no
 * code with the GPU path.
 *
 * A plain, slow, fp64 implementation of the Llama-style decoder that the
 * self-speculative decoding method runs (paper: Section 1 -- every token
 * passes the full layer stack; Section 2.2 -- the model's own early layers
 * draft; Section 3.1.1 -- the next-token distribution at layer l is computed
 * from the hidden state at layer l).  The early-exit head at layer l applies
 * the shared final RMSNorm and LM head to the layer-l hidden state; l = L is
 * the full model.
 *
 * Per token at position p, per layer (standard Llama definition):
 *   u = RMSNorm(x; g_attn);  q,k,v = Wq u, Wk u, Wv u;  RoPE(q, p), RoPE(k, p)
 *   head h attends with KV head floor(h / (nq/nkv)) over positions <= p,
 *   scores q.k / sqrt(hd), softmax;  x += Wo o
 *   n = RMSNorm(x; g_ffn);  x += Wd (SiLU(Wg n) * (Wu n))
 * RMSNorm(x; g) = x / sqrt(mean(x^2) + eps) * g.  SiLU(z) = z / (1 + e^-z).
 * RoPE (rotate-half pairing): for i < hd/2, theta_i = base^(-2i/hd) and the
 * pair (x_i, x_{i+hd/2}) is rotated by the angle p * theta_i.
 *
 * Precision.  All arithmetic is fp64; every dot product is summed in index
 * order.  For bf16 models the values that the GPU stores in bf16 are rounded
 * to bf16 (nearest-even at 8 significant bits) at the same points: the input
 * of every linear layer (both RMSNorm outputs, the attention output, the
 * SiLU-gated product, the final-norm output) and K, V when written to the
 * cache.  For fp32 models nothing is rounded.
 *
 * Rows.  A call processes T rows at consecutive positions pos0..pos0+T-1.
 * Each row's arithmetic does not depend on T or on the other rows (row t
 * only reads cache positions <= pos0+t), so a row gives the same bits
 * whether it is run alone or in a batch.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int n_layers, d, nq, nkv, hd, ffn, vocab, is_bf16, max_ctx;
  double eps, rope_base;
  /* weights: bf16 bit patterns (uint16) if is_bf16, else float32; row-major [out][in] */
  const void* embed;      /* [vocab][d] */
  const void* final_norm; /* [d] */
  const void* head;       /* [vocab][d] */
  const void** attn_norm; /* per layer [d] */
  const void** wq;        /* [nq*hd][d] */
  const void** wk;        /* [nkv*hd][d] */
  const void** wv;        /* [nkv*hd][d] */
  const void** wo;        /* [d][nq*hd] */
  const void** ffn_norm;  /* [d] */
  const void** wg;        /* [ffn][d] */
  const void** wu;        /* [ffn][d] */
  const void** wd;        /* [d][ffn] */
  /* KV cache owned by the caller: [n_layers][max_ctx][nkv][hd] doubles */
  double* kcache;
  double* vcache;
} OracleModel;

/* ---- scalar helpers ---------------------------------------------------- */

static inline double bf16_bits_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* Round to the nearest value with 8 significant bits (bf16), ties to even. */
double oracle_round_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);        /* x = m * 2^e, 0.5 <= |m| < 1 */
  double r = nearbyint(m * 256.0); /* 8 significant bits, current mode = nearest-even */
  return ldexp(r, e - 8);
}

static inline double wget(const OracleModel* M, const void* w, size_t i) {
  if (M->is_bf16) return bf16_bits_to_double(((const uint16_t*)w)[i]);
  return (double)((const float*)w)[i];
}

static inline double act_round(const OracleModel* M, double x) { return M->is_bf16 ? oracle_round_bf16(x) : x; }

/*
 * y[t][n] = sum_k W[n][k] * x[t][k] for t < T.  Every sum runs over k in
 * increasing order with separately rounded multiply and add (the library is
 * built with -ffp-contract=off), so y[t][n] does not depend on T.  Rows are
 * visited RB at a time with x transposed only so that one pass over W serves
 * RB rows; that changes no arithmetic.
 */
#define RB 16
static void matvec_rows(const OracleModel* M, const void* W, int N, int K, const double* x, int T,
                        double* y) {
  double* xt = malloc(sizeof(double) * (size_t)K * RB);
  for (int t0 = 0; t0 < T; t0 += RB) {
    int tb = T - t0 < RB ? T - t0 : RB;
    for (int k = 0; k < K; ++k)
      for (int r = 0; r < RB; ++r) xt[(size_t)k * RB + r] = r < tb ? x[(size_t)(t0 + r) * K + k] : 0.0;
#pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
      double acc[RB];
      for (int r = 0; r < RB; ++r) acc[r] = 0.0;
      for (int k = 0; k < K; ++k) {
        double w = wget(M, W, (size_t)n * K + k);
        const double* xk = xt + (size_t)k * RB;
        for (int r = 0; r < RB; ++r) acc[r] += w * xk[r];
      }
      for (int r = 0; r < tb; ++r) y[(size_t)(t0 + r) * N + n] = acc[r];
    }
  }
  free(xt);
}

static void rmsnorm(const OracleModel* M, const double* x, const void* g, int d, double eps, double* out) {
  double ss = 0.0;
  for (int i = 0; i < d; ++i) ss += x[i] * x[i];
  double inv = 1.0 / sqrt(ss / d + eps);
  for (int i = 0; i < d; ++i) out[i] = x[i] * inv * wget(M, g, i);
}

static void rope(double* v, int hd, int pos, double base) {
  int half = hd / 2;
  for (int i = 0; i < half; ++i) {
    double theta = pow(base, -2.0 * i / hd);
    double a = pos * theta;
    double c = cos(a), s = sin(a);
    double x0 = v[i], x1 = v[i + half];
    v[i] = x0 * c - x1 * s;
    v[i + half] = x1 * c + x0 * s;
  }
}

/* ---- public entry points ------------------------------------------------- */

/* RoPE of one head vector, exported so the tests can pin it on its own. */
void oracle_rope(double* v, int hd, int pos, double base) { rope(v, hd, pos, base); }

/* RMSNorm of one vector with a gain given as double. */
void oracle_rmsnorm_f64(const double* x, const double* g, int d, double eps, double* out) {
  double ss = 0.0;
  for (int i = 0; i < d; ++i) ss += x[i] * x[i];
  double inv = 1.0 / sqrt(ss / d + eps);
  for (int i = 0; i < d; ++i) out[i] = x[i] * inv * g[i];
}

/* Softmax attention of one query row (head dim hd) over n keys/values given
 * row-major [n][hd]; exported so the tests can pin attention on its own. */
void oracle_attend(const double* q, const double* K, const double* V, int n, int hd, double* out,
                   double* probs) {
  double scale = 1.0 / sqrt((double)hd);
  double mx = -INFINITY;
  for (int j = 0; j < n; ++j) {
    double s = 0.0;
    for (int i = 0; i < hd; ++i) s += q[i] * K[(size_t)j * hd + i];
    probs[j] = s * scale;
    if (probs[j] > mx) mx = probs[j];
  }
  double sum = 0.0;
  for (int j = 0; j < n; ++j) {
    probs[j] = exp(probs[j] - mx);
    sum += probs[j];
  }
  for (int j = 0; j < n; ++j) probs[j] /= sum;
  for (int i = 0; i < hd; ++i) {
    double acc = 0.0;
    for (int j = 0; j < n; ++j) acc += probs[j] * V[(size_t)j * hd + i];
    out[i] = acc;
  }
}

/*
 * Run T tokens at positions pos0..pos0+T-1 through layers [0, l_end).  K/V of
 * these positions are written to the cache for those layers.  hidden_out
 * [T][d] receives the residual stream after layer l_end-1 (the embedding if
 * l_end = 0).  Returns 0, or -1 on bad arguments / allocation failure.
 */
int oracle_forward(const OracleModel* M, const int32_t* tokens, int T, int pos0, int l_end,
                   double* hidden_out) {
  const int d = M->d, nq = M->nq, nkv = M->nkv, hd = M->hd, F = M->ffn;
  const int qd = nq * hd, kvd = nkv * hd, group = nq / nkv;
  if (T <= 0 || pos0 < 0 || pos0 + T > M->max_ctx || l_end < 0 || l_end > M->n_layers) return -1;
  for (int t = 0; t < T; ++t)
    if (tokens[t] < 0 || tokens[t] >= M->vocab) return -1;

  double* x = hidden_out;
  double* u = malloc(sizeof(double) * (size_t)T * d);
  double* q = malloc(sizeof(double) * (size_t)T * qd);
  double* k = malloc(sizeof(double) * (size_t)T * kvd);
  double* v = malloc(sizeof(double) * (size_t)T * kvd);
  double* o = malloc(sizeof(double) * (size_t)T * qd);
  double* y = malloc(sizeof(double) * (size_t)T * (d > F ? d : F));
  double* g = malloc(sizeof(double) * (size_t)T * F);
  double* up = malloc(sizeof(double) * (size_t)T * F);
  if (!u || !q || !k || !v || !o || !y || !g || !up) {
    free(u); free(q); free(k); free(v); free(o); free(y); free(g); free(up);
    return -1;
  }

  for (int t = 0; t < T; ++t)
    for (int i = 0; i < d; ++i) x[(size_t)t * d + i] = wget(M, M->embed, (size_t)tokens[t] * d + i);

  for (int l = 0; l < l_end; ++l) {
    /* attention block */
    for (int t = 0; t < T; ++t) {
      rmsnorm(M, x + (size_t)t * d, M->attn_norm[l], d, M->eps, u + (size_t)t * d);
      for (int i = 0; i < d; ++i) u[(size_t)t * d + i] = act_round(M, u[(size_t)t * d + i]);
    }
    matvec_rows(M, M->wq[l], qd, d, u, T, q);
    matvec_rows(M, M->wk[l], kvd, d, u, T, k);
    matvec_rows(M, M->wv[l], kvd, d, u, T, v);
    for (int t = 0; t < T; ++t) {
      int pos = pos0 + t;
      for (int h = 0; h < nq; ++h) rope(q + (size_t)t * qd + (size_t)h * hd, hd, pos, M->rope_base);
      for (int h = 0; h < nkv; ++h) rope(k + (size_t)t * kvd + (size_t)h * hd, hd, pos, M->rope_base);
      double* kc = M->kcache + ((size_t)l * M->max_ctx + pos) * kvd;
      double* vc = M->vcache + ((size_t)l * M->max_ctx + pos) * kvd;
      for (int i = 0; i < kvd; ++i) {
        kc[i] = act_round(M, k[(size_t)t * kvd + i]);
        vc[i] = act_round(M, v[(size_t)t * kvd + i]);
      }
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int t = 0; t < T; ++t) {
      for (int h = 0; h < nq; ++h) {
        int pos = pos0 + t, kvh = h / group, n = pos + 1;
        double* Kh = malloc(sizeof(double) * (size_t)n * hd);
        double* Vh = malloc(sizeof(double) * (size_t)n * hd);
        double* pr = malloc(sizeof(double) * (size_t)n);
        for (int j = 0; j < n; ++j) {
          const double* kc = M->kcache + ((size_t)l * M->max_ctx + j) * kvd + (size_t)kvh * hd;
          const double* vc = M->vcache + ((size_t)l * M->max_ctx + j) * kvd + (size_t)kvh * hd;
          memcpy(Kh + (size_t)j * hd, kc, sizeof(double) * hd);
          memcpy(Vh + (size_t)j * hd, vc, sizeof(double) * hd);
        }
        oracle_attend(q + (size_t)t * qd + (size_t)h * hd, Kh, Vh, n, hd, o + (size_t)t * qd + (size_t)h * hd, pr);
        free(Kh); free(Vh); free(pr);
      }
    }
    for (size_t i = 0; i < (size_t)T * qd; ++i) o[i] = act_round(M, o[i]);
    matvec_rows(M, M->wo[l], d, qd, o, T, y);
    for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];

    /* feed-forward block */
    for (int t = 0; t < T; ++t) {
      rmsnorm(M, x + (size_t)t * d, M->ffn_norm[l], d, M->eps, u + (size_t)t * d);
      for (int i = 0; i < d; ++i) u[(size_t)t * d + i] = act_round(M, u[(size_t)t * d + i]);
    }
    matvec_rows(M, M->wg[l], F, d, u, T, g);
    matvec_rows(M, M->wu[l], F, d, u, T, up);
    for (size_t i = 0; i < (size_t)T * F; ++i) {
      double z = g[i];
      g[i] = act_round(M, z / (1.0 + exp(-z)) * up[i]);
    }
    matvec_rows(M, M->wd[l], d, F, g, T, y);
    for (size_t i = 0; i < (size_t)T * d; ++i) x[i] += y[i];
  }
  free(u); free(q); free(k); free(v); free(o); free(y); free(g); free(up);
  return 0;
}

/*
 * Early-exit / final head on T hidden rows: logits[t] = W_head RMSNorm(h_t; g_f)
 * (the normalised vector is a linear-layer input, so it is rounded to bf16 for
 * bf16 models).  normed_out (nullable) receives the normalised rows [T][d]
 * before that rounding.
 */
int oracle_head(const OracleModel* M, const double* hidden, int T, double* logits, double* normed_out) {
  const int d = M->d;
  double* u = malloc(sizeof(double) * (size_t)T * d);
  if (!u) return -1;
  for (int t = 0; t < T; ++t) {
    rmsnorm(M, hidden + (size_t)t * d, M->final_norm, d, M->eps, u + (size_t)t * d);
    if (normed_out) memcpy(normed_out + (size_t)t * d, u + (size_t)t * d, sizeof(double) * d);
    for (int i = 0; i < d; ++i) u[(size_t)t * d + i] = act_round(M, u[(size_t)t * d + i]);
  }
  matvec_rows(M, M->head, M->vocab, d, u, T, logits);
  free(u);
  return 0;
}

/* Plain fp64 y = W x (+ b) for float32 W [N][K] (the Q-network layers). */
void oracle_linear_f32(const float* W, const float* b, int N, int K, const double* x, double* y) {
  for (int n = 0; n < N; ++n) {
    double acc = 0.0;
    for (int k = 0; k < K; ++k) acc += (double)W[(size_t)n * K + k] * x[k];
    y[n] = acc + (b ? (double)b[n] : 0.0);
  }
}

/* y[t][n] = sum_k W[n][k] x[t][k] for a bf16 (is_bf16) or float32 W [N][K]. */
void oracle_matvec(const void* W, int is_bf16, int N, int K, const double* x, int T, double* y) {
  OracleModel M;
  memset(&M, 0, sizeof M);
  M.is_bf16 = is_bf16;
  matvec_rows(&M, W, N, K, x, T, y);
}
