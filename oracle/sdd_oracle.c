/*
 * CPU oracle for verifier-skipped speculative diffusion decoding.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by tests/, the smoke entry and the
 * benchmark's CPU-baseline leg, never by the GPU product path.  It shares no
 * code with the HIP library.  Plain loops, IEEE double precision for every
 * quantity of the method; the acceptance/confidence decisions that the paper
 * takes on FP32 log-probabilities are taken in fp32 here as well.
 *
 * Parts and the passages they follow:
 *   - decoder forward (target model): the paper names the verifier
 *     (Qwen3-32B, Sec. 5.1 "Experimental Setup") but prints no architecture;
 *     the textbook pre-norm decoder (RMSNorm, GQA attention with rotate-half
 *     RoPE, optional per-head QK RMSNorm, SwiGLU FFN, untied LM head) is written
 *     out literally.  Two independent routes: full recomputation over the whole
 *     sequence with no cache (the paper's measured verifier, Appendix
 *     "Evaluation and Throughput") and a cached block verify.
 *   - strict greedy acceptance and the accepted length L (Sec. 3.1), lenience
 *     (lenience equation, Appendix "Baselines and Sweep Settings"), top-k
 *     membership (same appendix), and the distribution-preserving ratio test
 *     min(1, p/q) that Sec. 3.1 cites.
 *   - raw confidence q_j = max softmax and the local gate B_k = min_{j<=k} q_j
 *     with K = max{k : B_k >= tau} (Sec. 4.1 candidate skip length, Sec. 4.2
 *     raw confidence).
 *   - the survival predictor MLP (Appendix "Predictor Details") whose sigmoid
 *     output is the marginal or conditional survival score (Sec. 4.2).
 *   - agreement with strict verification, StrictToken and FullPrefix over
 *     the rounds that commit an unverified prefix (Sec. 3.2).
 *   - the two-gate skip scheduler with its three confidence signals, the
 *     guards and the staleness counter D (Sec. 4.1 candidate skip length and
 *     commit rule, Sec. 4.2 signals, Appendix "Baselines and Sweep Settings").
 */
#include "sdd_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Synthetic weights.  SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) as a
 * counter-based generator; the normal variate is the Irwin-Hall sum of four
 * 16-bit uniforms, scaled to standard deviation sigma.  Integer arithmetic up
 * to one fp32 multiply, so any IEEE implementation reproduces it bit for bit. */

uint64_t orc_splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

int orc_tensor_id(int kind, int layer) {
  switch (kind) {
    case ORC_EMBED: return 1;
    case ORC_LM_HEAD: return 2;
    case ORC_FINAL_NORM: return 3;
    case ORC_WQ: return 16 + 16 * layer + 0;
    case ORC_WK: return 16 + 16 * layer + 1;
    case ORC_WV: return 16 + 16 * layer + 2;
    case ORC_WO: return 16 + 16 * layer + 3;
    case ORC_WGATE: return 16 + 16 * layer + 4;
    case ORC_WUP: return 16 + 16 * layer + 5;
    case ORC_WDOWN: return 16 + 16 * layer + 6;
    case ORC_ATTN_NORM: return 16 + 16 * layer + 7;
    case ORC_FFN_NORM: return 16 + 16 * layer + 8;
    case ORC_Q_NORM: return 16 + 16 * layer + 9;
    case ORC_K_NORM: return 16 + 16 * layer + 10;
  }
  return -1;
}

static float orc_round_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return f; /* inf/nan untouched */
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb; /* round to nearest, ties to even */
  u &= 0xffff0000u;
  memcpy(&f, &u, 4);
  return f;
}

void orc_weight_values(uint64_t seed, int tensor_id, uint64_t start, uint64_t count,
                       double sigma, int bf16, float* out) {
  const uint64_t gamma = 0x9E3779B97F4A7C15ULL;
  uint64_t key = orc_splitmix64(orc_splitmix64(seed) + (uint64_t)tensor_id);
  float scale = (float)(sigma * 1.7320508075688772 / 65536.0);
  for (uint64_t i = 0; i < count; ++i) {
    uint64_t r = orc_splitmix64(key + (start + i) * gamma);
    int32_t s = (int32_t)(r & 0xffff) + (int32_t)((r >> 16) & 0xffff) +
                (int32_t)((r >> 32) & 0xffff) + (int32_t)(r >> 48) - 131070;
    float w = (float)s * scale;
    out[i] = bf16 ? orc_round_bf16(w) : w;
  }
}

/* ------------------------------------------------------------------------ */
/* Model */

struct orc_model {
  orc_config c;
  float* embed;   /* [V][d] */
  float* lm_head; /* [V][d] */
  float* final_norm;
  struct {
    float *wq, *wk, *wv, *wo, *wg, *wu, *wd;
    float *attn_norm, *ffn_norm, *q_norm, *k_norm;
  } * L;
  /* Layer streaming (orc_model_create_streamed): the layers' tensors are not
   * held; a forward generates a layer's tensors when it reaches the layer and
   * frees them after it, so a model whose fp32 copy exceeds host memory (the
   * 64-layer Qwen3-32B shape: 131 GB) can still be run.  The values are the
   * ones a materialized model holds (same generator, same indices). */
  int streamed;
  uint64_t seed;
  double sigma;
  float* stream_buf[ORC_K_NORM + 1]; /* one layer's tensors, reused by every layer (indexed by kind) */
};

int orc_tensor_shape(const orc_config* c, int kind, int64_t* rows, int64_t* cols) {
  int64_t d = c->d_model, hq = (int64_t)c->n_q_heads * c->head_dim,
          hk = (int64_t)c->n_kv_heads * c->head_dim;
  switch (kind) {
    case ORC_EMBED: case ORC_LM_HEAD: *rows = c->vocab; *cols = d; return 0;
    case ORC_FINAL_NORM: case ORC_ATTN_NORM: case ORC_FFN_NORM: *rows = 1; *cols = d; return 0;
    case ORC_Q_NORM: case ORC_K_NORM: *rows = 1; *cols = c->head_dim; return 0;
    case ORC_WQ: *rows = hq; *cols = d; return 0;
    case ORC_WK: case ORC_WV: *rows = hk; *cols = d; return 0;
    case ORC_WO: *rows = d; *cols = hq; return 0;
    case ORC_WGATE: case ORC_WUP: *rows = c->d_ff; *cols = d; return 0;
    case ORC_WDOWN: *rows = d; *cols = c->d_ff; return 0;
  }
  return -1;
}

static float** orc_slot(orc_model* m, int kind, int layer) {
  switch (kind) {
    case ORC_EMBED: return &m->embed;
    case ORC_LM_HEAD: return &m->lm_head;
    case ORC_FINAL_NORM: return &m->final_norm;
    case ORC_WQ: return &m->L[layer].wq;
    case ORC_WK: return &m->L[layer].wk;
    case ORC_WV: return &m->L[layer].wv;
    case ORC_WO: return &m->L[layer].wo;
    case ORC_WGATE: return &m->L[layer].wg;
    case ORC_WUP: return &m->L[layer].wu;
    case ORC_WDOWN: return &m->L[layer].wd;
    case ORC_ATTN_NORM: return &m->L[layer].attn_norm;
    case ORC_FFN_NORM: return &m->L[layer].ffn_norm;
    case ORC_Q_NORM: return &m->L[layer].q_norm;
    case ORC_K_NORM: return &m->L[layer].k_norm;
  }
  return NULL;
}

static int orc_is_norm(int kind) {
  return kind == ORC_FINAL_NORM || kind == ORC_ATTN_NORM || kind == ORC_FFN_NORM ||
         kind == ORC_Q_NORM || kind == ORC_K_NORM;
}

/* Writes tensor (kind, layer)'s synthetic values into t. */
static void orc_fill_tensor(const orc_config* c, int kind, int layer, uint64_t seed, double sigma, float* t) {
  int64_t rows, cols;
  orc_tensor_shape(c, kind, &rows, &cols);
  int64_t n = rows * cols;
  if (orc_is_norm(kind)) { /* RMSNorm gains start at one */
    for (int64_t i = 0; i < n; ++i) t[i] = 1.0f;
    return;
  }
  int id = orc_tensor_id(kind, layer);
  const int64_t chunk = 1 << 16;
#pragma omp parallel for schedule(static)
  for (int64_t s = 0; s < n; s += chunk) {
    int64_t cnt = (n - s < chunk) ? n - s : chunk;
    orc_weight_values(seed, id, (uint64_t)s, (uint64_t)cnt, sigma, c->bf16_weights, t + s);
  }
}

static float* orc_make_tensor(const orc_config* c, int kind, int layer, uint64_t seed,
                              double sigma) {
  int64_t rows, cols;
  orc_tensor_shape(c, kind, &rows, &cols);
  float* t = (float*)malloc((size_t)(rows * cols) * sizeof(float));
  if (t) orc_fill_tensor(c, kind, layer, seed, sigma, t);
  return t;
}

void orc_model_free(orc_model* m) {
  if (!m) return;
  for (int kind = 0; kind <= ORC_K_NORM; ++kind) free(m->stream_buf[kind]);
  free(m->embed);
  free(m->lm_head);
  free(m->final_norm);
  if (m->L && !m->streamed) {
    for (int l = 0; l < m->c.n_layers; ++l) {
      free(m->L[l].wq); free(m->L[l].wk); free(m->L[l].wv); free(m->L[l].wo);
      free(m->L[l].wg); free(m->L[l].wu); free(m->L[l].wd);
      free(m->L[l].attn_norm); free(m->L[l].ffn_norm);
      free(m->L[l].q_norm); free(m->L[l].k_norm);
    }
    free(m->L);
  }
  free(m);
}

orc_model* orc_model_create(const orc_config* cfg, uint64_t seed, double sigma) {
  if (!cfg || cfg->n_layers < 0 || cfg->d_model <= 0 || cfg->n_q_heads <= 0 ||
      cfg->n_kv_heads <= 0 || cfg->n_q_heads % cfg->n_kv_heads || cfg->head_dim <= 0 ||
      cfg->head_dim % 2 || cfg->d_ff <= 0 || cfg->vocab <= 0)
    return NULL;
  orc_model* m = (orc_model*)calloc(1, sizeof(orc_model));
  if (!m) return NULL;
  m->c = *cfg;
  m->L = calloc((size_t)(cfg->n_layers > 0 ? cfg->n_layers : 1), sizeof(*m->L));
  int ok = m->L != NULL;
  for (int kind = ORC_EMBED; ok && kind <= ORC_FINAL_NORM; ++kind) {
    float** s = orc_slot(m, kind, 0);
    *s = orc_make_tensor(cfg, kind, 0, seed, sigma);
    ok = *s != NULL;
  }
  for (int l = 0; ok && l < cfg->n_layers; ++l)
    for (int kind = ORC_WQ; ok && kind <= ORC_K_NORM; ++kind) {
      float** s = orc_slot(m, kind, l);
      *s = orc_make_tensor(cfg, kind, l, seed, sigma);
      ok = *s != NULL;
    }
  if (!ok) {
    orc_model_free(m);
    return NULL;
  }
  return m;
}

orc_model* orc_model_create_streamed(const orc_config* cfg, uint64_t seed, double sigma) {
  if (!cfg || cfg->n_layers < 0 || cfg->d_model <= 0 || cfg->n_q_heads <= 0 ||
      cfg->n_kv_heads <= 0 || cfg->n_q_heads % cfg->n_kv_heads || cfg->head_dim <= 0 ||
      cfg->head_dim % 2 || cfg->d_ff <= 0 || cfg->vocab <= 0)
    return NULL;
  orc_model* m = (orc_model*)calloc(1, sizeof(orc_model));
  if (!m) return NULL;
  m->c = *cfg;
  m->streamed = 1;
  m->seed = seed;
  m->sigma = sigma;
  m->L = calloc((size_t)(cfg->n_layers > 0 ? cfg->n_layers : 1), sizeof(*m->L));
  int ok = m->L != NULL;
  for (int kind = ORC_EMBED; ok && kind <= ORC_FINAL_NORM; ++kind) {
    float** s = orc_slot(m, kind, 0);
    *s = orc_make_tensor(cfg, kind, 0, seed, sigma);
    ok = *s != NULL;
  }
  if (!ok) {
    orc_model_free(m);
    return NULL;
  }
  return m;
}

/* Layer l's tensors for a forward: present in a materialized model, generated
 * now in a streamed one (0 on success). */
static int layer_acquire(const orc_model* cm, int l) {
  if (!cm->streamed) return 0;
  orc_model* m = (orc_model*)cm; /* a streamed model's layer slots are a per-forward cache */
  for (int kind = ORC_WQ; kind <= ORC_K_NORM; ++kind) {
    if (!m->stream_buf[kind]) { /* every layer has the same shapes: one buffer per kind */
      int64_t rows, cols;
      orc_tensor_shape(&m->c, kind, &rows, &cols);
      m->stream_buf[kind] = (float*)malloc((size_t)(rows * cols) * sizeof(float));
      if (!m->stream_buf[kind]) return -1;
    }
    orc_fill_tensor(&m->c, kind, l, m->seed, m->sigma, m->stream_buf[kind]);
    *orc_slot(m, kind, l) = m->stream_buf[kind];
  }
  return 0;
}

static void layer_release(const orc_model* cm, int l) {
  if (!cm->streamed) return;
  orc_model* m = (orc_model*)cm;
  for (int kind = ORC_WQ; kind <= ORC_K_NORM; ++kind) *orc_slot(m, kind, l) = NULL;
}

int orc_model_set_tensor(orc_model* m, int kind, int layer, const float* src) {
  if (!m || !src || kind < ORC_EMBED || kind > ORC_K_NORM) return -1;
  if (kind >= ORC_WQ && (layer < 0 || layer >= m->c.n_layers)) return -1;
  if (kind >= ORC_WQ && m->streamed) return -1; /* a streamed model regenerates its layers */
  int64_t rows, cols;
  orc_tensor_shape(&m->c, kind, &rows, &cols);
  memcpy(*orc_slot(m, kind, layer), src, (size_t)(rows * cols) * sizeof(float));
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Decoder building blocks, fp64 */

/* Y[r][n] = sum_k X[r][k] * W[n][k]  (PyTorch Linear convention W[out][in]) */
/* Every Y[r][n] is one running sum over k = 0..K-1 in increasing order.  Four
 * rows walk W's row n together (four independent running sums: the same
 * additions, in the same order, as one row at a time; it only keeps the
 * processor's adders busy). */
static void linear(const float* W, int N, int K, const double* X, int R, double* Y) {
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n) {
    const float* w = W + (size_t)n * K;
    int r = 0;
    for (; r + 4 <= R; r += 4) {
      const double *x0 = X + (size_t)r * K, *x1 = x0 + K, *x2 = x1 + K, *x3 = x2 + K;
      double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
      for (int k = 0; k < K; ++k) {
        const double wk = (double)w[k];
        a0 += x0[k] * wk;
        a1 += x1[k] * wk;
        a2 += x2[k] * wk;
        a3 += x3[k] * wk;
      }
      Y[(size_t)r * N + n] = a0;
      Y[(size_t)(r + 1) * N + n] = a1;
      Y[(size_t)(r + 2) * N + n] = a2;
      Y[(size_t)(r + 3) * N + n] = a3;
    }
    for (; r < R; ++r) {
      const double* x = X + (size_t)r * K;
      double acc = 0.0;
      for (int k = 0; k < K; ++k) acc += x[k] * (double)w[k];
      Y[(size_t)r * N + n] = acc;
    }
  }
}

/* RMSNorm: y = x / sqrt(mean(x^2) + eps) * g */
static void rmsnorm(const double* x, int d, const float* g, double eps, double* y) {
  double ss = 0.0;
  for (int i = 0; i < d; ++i) ss += x[i] * x[i];
  double inv = 1.0 / sqrt(ss / d + eps);
  for (int i = 0; i < d; ++i) y[i] = x[i] * inv * (double)g[i];
}

/* BF16-operand mode (orc_config.bf16_operands).  The paper runs its verifier
 * as a BF16 model (Appendix "Evaluation and Throughput": BF16 weights, logits
 * converted to FP32).  Taken literally for the matrix products: every operand
 * of a product is a BF16 value (the weights already are; the activations are
 * rounded to BF16 where they enter a product: the gained input x * g of every
 * projection, q, k and v, the attention output, the FFN hidden state), every
 * sum is exact (fp64 here), and RMSNorm's row scale r = 1/sqrt(mean x^2 + eps)
 * multiplies the product, (r x * g) W = r ((x * g) W).  Softmax, norms, RoPE
 * and the residual stream stay exact.  Off (0), the oracle is exact fp64. */

/* Nearest BF16 value (8 significant bits, ties to even) of a finite double. */
static double round_bf16(double x) {
  if (!isfinite(x) || x == 0.0) return x;
  int e;
  frexp(x, &e); /* |x| = f 2^e, f in [0.5, 1) */
  if (e < -125) e = -125; /* BF16 subnormals: spacing 2^-133 */
  const double s = ldexp(1.0, 8 - e);
  return nearbyint(x * s) / s; /* default rounding mode: ties to even */
}

/* Rounds the n values of an operand to BF16 in BF16-operand mode. */
static void bf16_operand(const orc_model* m, double* a, size_t n) {
  if (!m->c.bf16_operands) return;
  for (size_t i = 0; i < n; ++i) a[i] = round_bf16(a[i]);
}

/* Operand of the projections that follow an RMSNorm with gain g, for R rows of
 * x: exact mode h = RMSNorm(x) * g and rs = 1; BF16-operand mode h = BF16(x * g)
 * and rs = the row scales, applied to the products by scale_rows. */
static void norm_operand(const orc_model* m, const double* x, int R, const float* g, double* h, double* rs) {
  const orc_config* c = &m->c;
  int d = c->d_model;
  for (int r = 0; r < R; ++r) {
    const double* xr = x + (size_t)r * d;
    double* hr = h + (size_t)r * d;
    if (!c->bf16_operands) {
      rmsnorm(xr, d, g, c->rms_eps, hr);
      rs[r] = 1.0;
    } else {
      double ss = 0.0;
      for (int i = 0; i < d; ++i) ss += xr[i] * xr[i];
      rs[r] = 1.0 / sqrt(ss / d + c->rms_eps);
      for (int i = 0; i < d; ++i) hr[i] = round_bf16(xr[i] * (double)g[i]);
    }
  }
}

/* Y[r][n] *= rs[r] */
static void scale_rows(double* Y, int R, int N, const double* rs) {
  for (int r = 0; r < R; ++r)
    for (int n = 0; n < N; ++n) Y[(size_t)r * N + n] *= rs[r];
}

/* Rotate-half RoPE at absolute position pos: pairs (i, i + hd/2) rotate by
 * pos * theta^(-2i/hd). */
static void rope(double* v, int hd, int pos, double theta) {
  int h = hd / 2;
  for (int i = 0; i < h; ++i) {
    double inv_freq = pow(theta, -2.0 * i / hd);
    double a = pos * inv_freq, c = cos(a), s = sin(a);
    double x0 = v[i], x1 = v[i + h];
    v[i] = x0 * c - x1 * s;
    v[i + h] = x1 * c + x0 * s;
  }
}

static double silu(double g) { return g / (1.0 + exp(-g)); }

/* q/k projections of R rows at positions pos0.., with optional QK-norm and
 * RoPE applied in place. */
static void qk_post(const orc_model* m, int l, double* q, double* k, int R, int pos0) {
  const orc_config* c = &m->c;
  int hd = c->head_dim, hq = c->n_q_heads, hk = c->n_kv_heads;
  double* tmp = (double*)malloc(sizeof(double) * hd);
  for (int r = 0; r < R; ++r) {
    for (int h = 0; h < hq; ++h) {
      double* v = q + ((size_t)r * hq + h) * hd;
      if (c->qk_norm) {
        rmsnorm(v, hd, m->L[l].q_norm, c->rms_eps, tmp);
        memcpy(v, tmp, sizeof(double) * hd);
      }
      rope(v, hd, pos0 + r, c->rope_theta);
    }
    for (int h = 0; h < hk; ++h) {
      double* v = k + ((size_t)r * hk + h) * hd;
      if (c->qk_norm) {
        rmsnorm(v, hd, m->L[l].k_norm, c->rms_eps, tmp);
        memcpy(v, tmp, sizeof(double) * hd);
      }
      rope(v, hd, pos0 + r, c->rope_theta);
    }
  }
  free(tmp);
}

/* Residual FFN block on R rows: x += down(silu(gate(h)) * up(h)), h = RMSNorm(x). */
static void ffn_block(const orc_model* m, int l, double* x, int R) {
  const orc_config* c = &m->c;
  int d = c->d_model, f = c->d_ff;
  double* h = (double*)malloc(sizeof(double) * (size_t)R * d);
  double* g = (double*)malloc(sizeof(double) * (size_t)R * f);
  double* u = (double*)malloc(sizeof(double) * (size_t)R * f);
  double* y = (double*)malloc(sizeof(double) * (size_t)R * d);
  double* rs = (double*)malloc(sizeof(double) * (size_t)R);
  norm_operand(m, x, R, m->L[l].ffn_norm, h, rs);
  linear(m->L[l].wg, f, d, h, R, g);
  linear(m->L[l].wu, f, d, h, R, u);
  scale_rows(g, R, f, rs);
  scale_rows(u, R, f, rs);
  for (size_t i = 0; i < (size_t)R * f; ++i) g[i] = silu(g[i]) * u[i];
  bf16_operand(m, g, (size_t)R * f);
  linear(m->L[l].wd, d, f, g, R, y);
  for (size_t i = 0; i < (size_t)R * d; ++i) x[i] += y[i];
  free(h); free(g); free(u); free(y); free(rs);
}

/* final RMSNorm + LM head on R rows */
static void lm_head(const orc_model* m, const double* x, int R, double* logits) {
  const orc_config* c = &m->c;
  int d = c->d_model;
  double* h = (double*)malloc(sizeof(double) * (size_t)R * d);
  double* rs = (double*)malloc(sizeof(double) * (size_t)R);
  norm_operand(m, x, R, m->final_norm, h, rs);
  linear(m->lm_head, c->vocab, d, h, R, logits);
  scale_rows(logits, R, c->vocab, rs);
  free(h);
  free(rs);
}

static void embed_rows(const orc_model* m, const int32_t* tok, int R, double* x) {
  int d = m->c.d_model;
  for (int r = 0; r < R; ++r)
    for (int i = 0; i < d; ++i) x[(size_t)r * d + i] = (double)m->embed[(size_t)tok[r] * d + i];
}

static int tokens_ok(const orc_model* m, const int32_t* tok, int n) {
  for (int i = 0; i < n; ++i)
    if (tok[i] < 0 || tok[i] >= m->c.vocab) return 0;
  return 1;
}

/* ------------------------------------------------------------------------ */
/* Route 1: full recomputation, no cache.  Every row attends to rows 0..i of
 * the same pass (causal mask). */

/* Layer l of the full recomputation applied to the n rows x in place. */
static int layer_full(const orc_model* m, int l, int n, double* x) {
  const orc_config* c = &m->c;
  int d = c->d_model, hd = c->head_dim, hq = c->n_q_heads, hk = c->n_kv_heads;
  int grp = hq / hk;
  size_t nq = (size_t)hq * hd, nk = (size_t)hk * hd;
  int rc = layer_acquire(m, l);
  if (rc) return rc;
  double* h = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* q = (double*)malloc(sizeof(double) * (size_t)n * nq);
  double* k = (double*)malloc(sizeof(double) * (size_t)n * nk);
  double* v = (double*)malloc(sizeof(double) * (size_t)n * nk);
  double* o = (double*)malloc(sizeof(double) * (size_t)n * nq);
  double* y = (double*)malloc(sizeof(double) * (size_t)n * d);
  double* rs = (double*)malloc(sizeof(double) * (size_t)n);
  double scale = 1.0 / sqrt((double)hd);
  norm_operand(m, x, n, m->L[l].attn_norm, h, rs);
  linear(m->L[l].wq, (int)nq, d, h, n, q);
  linear(m->L[l].wk, (int)nk, d, h, n, k);
  linear(m->L[l].wv, (int)nk, d, h, n, v);
  scale_rows(q, n, (int)nq, rs);
  scale_rows(k, n, (int)nk, rs);
  scale_rows(v, n, (int)nk, rs);
  qk_post(m, l, q, k, n, 0);
  bf16_operand(m, q, (size_t)n * nq);
  bf16_operand(m, k, (size_t)n * nk);
  bf16_operand(m, v, (size_t)n * nk);
#pragma omp parallel for schedule(dynamic)
  for (int i = 0; i < n; ++i) {
    double* s = (double*)malloc(sizeof(double) * (size_t)(i + 1));
    for (int hh = 0; hh < hq; ++hh) {
      int kh = hh / grp;
      const double* qi = q + ((size_t)i * hq + hh) * hd;
      double mx = -INFINITY;
      for (int j = 0; j <= i; ++j) {
        const double* kj = k + ((size_t)j * hk + kh) * hd;
        double dot = 0.0;
        for (int t = 0; t < hd; ++t) dot += qi[t] * kj[t];
        s[j] = dot * scale;
        if (s[j] > mx) mx = s[j];
      }
      double den = 0.0;
      for (int j = 0; j <= i; ++j) { s[j] = exp(s[j] - mx); den += s[j]; }
      /* o_t = sum_j s_j v_j,t / den: every o_t sums over j = 0..i in order (the
       * loops are interchanged only so that V is read row by row) */
      double* oi = o + ((size_t)i * hq + hh) * hd;
      for (int t = 0; t < hd; ++t) oi[t] = 0.0;
      for (int j = 0; j <= i; ++j) {
        const double* vj = v + ((size_t)j * hk + kh) * hd;
        for (int t = 0; t < hd; ++t) oi[t] += s[j] * vj[t];
      }
      for (int t = 0; t < hd; ++t) oi[t] /= den;
    }
    free(s);
  }
  bf16_operand(m, o, (size_t)n * nq);
  linear(m->L[l].wo, d, (int)nq, o, n, y);
  for (size_t i = 0; i < (size_t)n * d; ++i) x[i] += y[i];
  ffn_block(m, l, x, n);
  layer_release(m, l);
  free(h); free(q); free(k); free(v); free(o); free(y); free(rs);
  return 0;
}

static int forward_full_x(const orc_model* m, const int32_t* tokens, int n, double* x) {
  embed_rows(m, tokens, n, x);
  for (int l = 0; l < m->c.n_layers; ++l) {
    int rc = layer_full(m, l, n, x);
    if (rc) return rc;
  }
  return 0;
}

/* The full recomputation in steps (the same functions orc_forward_full runs),
 * so that a caller can follow a long forward layer by layer. */
int orc_embed(const orc_model* m, const int32_t* tokens, int n, double* x) {
  if (!m || !tokens || !x || n <= 0 || !tokens_ok(m, tokens, n)) return -1;
  embed_rows(m, tokens, n, x);
  return 0;
}

int orc_layer_full(const orc_model* m, int layer, int n, double* x) {
  if (!m || !x || n <= 0 || layer < 0 || layer >= m->c.n_layers) return -1;
  return layer_full(m, layer, n, x);
}

int orc_final_logits(const orc_model* m, const double* x, int R, double* logits) {
  if (!m || !x || !logits || R <= 0) return -1;
  lm_head(m, x, R, logits);
  return 0;
}

int orc_forward_full(const orc_model* m, const int32_t* tokens, int n, int row0, double* logits) {
  if (!m || !tokens || !logits || n <= 0 || row0 < 0 || row0 >= n || !tokens_ok(m, tokens, n)) return -1;
  int d = m->c.d_model;
  double* x = (double*)malloc(sizeof(double) * (size_t)n * d);
  int rc = forward_full_x(m, tokens, n, x);
  if (rc == 0) lm_head(m, x + (size_t)row0 * d, n - row0, logits);
  free(x);
  return rc;
}

int orc_forward_full_hidden(const orc_model* m, const int32_t* tokens, int n, int row0, double* hidden) {
  if (!m || !tokens || !hidden || n <= 0 || row0 < 0 || row0 >= n || !tokens_ok(m, tokens, n)) return -1;
  int d = m->c.d_model;
  double* x = (double*)malloc(sizeof(double) * (size_t)n * d);
  int rc = forward_full_x(m, tokens, n, x);
  if (rc == 0) memcpy(hidden, x + (size_t)row0 * d, sizeof(double) * (size_t)(n - row0) * d);
  free(x);
  return rc;
}

/* ------------------------------------------------------------------------ */
/* Route 2: cached.  The cache holds K (after QK-norm and RoPE) and V of every
 * committed position; a block of R rows at positions len..len+R-1 appends its
 * own K/V and attends to positions 0..its own. */

struct orc_kv {
  const orc_model* m;
  int max_len, len, pending;
  double* k; /* [layers][max_len][Hkv*hd] */
  double* v;
};

orc_kv* orc_kv_create(const orc_model* m, int max_len) {
  if (!m || max_len <= 0) return NULL;
  orc_kv* kv = (orc_kv*)calloc(1, sizeof(orc_kv));
  size_t per = (size_t)m->c.n_kv_heads * m->c.head_dim;
  size_t nl = (size_t)(m->c.n_layers > 0 ? m->c.n_layers : 1);
  kv->m = m;
  kv->max_len = max_len;
  kv->k = (double*)calloc(nl * max_len * per, sizeof(double));
  kv->v = (double*)calloc(nl * max_len * per, sizeof(double));
  if (!kv->k || !kv->v) {
    orc_kv_free(kv);
    return NULL;
  }
  return kv;
}

void orc_kv_free(orc_kv* kv) {
  if (!kv) return;
  free(kv->k);
  free(kv->v);
  free(kv);
}

int orc_kv_len(const orc_kv* kv) { return kv ? kv->len : -1; }
int orc_kv_pending(const orc_kv* kv) { return kv ? kv->pending : -1; }

int orc_kv_read(const orc_kv* kv, int layer, int pos, double* k, double* v) {
  if (!kv || layer < 0 || layer >= kv->m->c.n_layers || pos < 0 || pos >= kv->max_len) return -1;
  size_t per = (size_t)kv->m->c.n_kv_heads * kv->m->c.head_dim;
  size_t off = ((size_t)layer * kv->max_len + pos) * per;
  if (k) memcpy(k, kv->k + off, per * sizeof(double));
  if (v) memcpy(v, kv->v + off, per * sizeof(double));
  return 0;
}

/* Runs R rows at positions pos0.. through all layers, appending K/V. */
static int block_forward(orc_kv* kv, const int32_t* tok, int R, int pos0, double* x) {
  const orc_model* m = kv->m;
  const orc_config* c = &m->c;
  int d = c->d_model, hd = c->head_dim, hq = c->n_q_heads, hk = c->n_kv_heads;
  int grp = hq / hk;
  size_t nq = (size_t)hq * hd, nk = (size_t)hk * hd;
  double* h = (double*)malloc(sizeof(double) * (size_t)R * d);
  double* q = (double*)malloc(sizeof(double) * (size_t)R * nq);
  double* k = (double*)malloc(sizeof(double) * (size_t)R * nk);
  double* v = (double*)malloc(sizeof(double) * (size_t)R * nk);
  double* o = (double*)malloc(sizeof(double) * (size_t)R * nq);
  double* y = (double*)malloc(sizeof(double) * (size_t)R * d);
  double* rs = (double*)malloc(sizeof(double) * (size_t)R);
  embed_rows(m, tok, R, x);
  double scale = 1.0 / sqrt((double)hd);
  int rc = 0;
  for (int l = 0; l < c->n_layers; ++l) {
    if ((rc = layer_acquire(m, l))) break;
    double* K = kv->k + (size_t)l * kv->max_len * nk;
    double* V = kv->v + (size_t)l * kv->max_len * nk;
    norm_operand(m, x, R, m->L[l].attn_norm, h, rs);
    linear(m->L[l].wq, (int)nq, d, h, R, q);
    linear(m->L[l].wk, (int)nk, d, h, R, k);
    linear(m->L[l].wv, (int)nk, d, h, R, v);
    scale_rows(q, R, (int)nq, rs);
    scale_rows(k, R, (int)nk, rs);
    scale_rows(v, R, (int)nk, rs);
    qk_post(m, l, q, k, R, pos0);
    bf16_operand(m, q, (size_t)R * nq);
    bf16_operand(m, k, (size_t)R * nk);
    bf16_operand(m, v, (size_t)R * nk);
    memcpy(K + (size_t)pos0 * nk, k, sizeof(double) * (size_t)R * nk);
    memcpy(V + (size_t)pos0 * nk, v, sizeof(double) * (size_t)R * nk);
#pragma omp parallel for schedule(dynamic)
    for (int r = 0; r < R; ++r) {
      int last = pos0 + r;
      double* s = (double*)malloc(sizeof(double) * (size_t)(last + 1));
      for (int hh = 0; hh < hq; ++hh) {
        int kh = hh / grp;
        const double* qi = q + ((size_t)r * hq + hh) * hd;
        double mx = -INFINITY;
        for (int j = 0; j <= last; ++j) {
          const double* kj = K + (size_t)j * nk + (size_t)kh * hd;
          double dot = 0.0;
          for (int t = 0; t < hd; ++t) dot += qi[t] * kj[t];
          s[j] = dot * scale;
          if (s[j] > mx) mx = s[j];
        }
        double den = 0.0;
        for (int j = 0; j <= last; ++j) { s[j] = exp(s[j] - mx); den += s[j]; }
        /* every o_t sums over j = 0..last in order (loops interchanged to read V row by row) */
        double* oi = o + ((size_t)r * hq + hh) * hd;
        for (int t = 0; t < hd; ++t) oi[t] = 0.0;
        for (int j = 0; j <= last; ++j) {
          const double* vj = V + (size_t)j * nk + (size_t)kh * hd;
          for (int t = 0; t < hd; ++t) oi[t] += s[j] * vj[t];
        }
        for (int t = 0; t < hd; ++t) oi[t] /= den;
      }
      free(s);
    }
    bf16_operand(m, o, (size_t)R * nq);
    linear(m->L[l].wo, d, (int)nq, o, R, y);
    for (size_t i = 0; i < (size_t)R * d; ++i) x[i] += y[i];
    ffn_block(m, l, x, R);
    layer_release(m, l);
  }
  free(h); free(q); free(k); free(v); free(o); free(y); free(rs);
  return rc;
}

int orc_kv_prefill(orc_kv* kv, const int32_t* tokens, int n) {
  if (!kv || !tokens || n <= 0 || n > kv->max_len || !tokens_ok(kv->m, tokens, n)) return -1;
  int d = kv->m->c.d_model;
  if (n > 1) {
    double* x = (double*)malloc(sizeof(double) * (size_t)(n - 1) * d);
    int rc = block_forward(kv, tokens, n - 1, 0, x);
    free(x);
    if (rc) return rc;
  }
  kv->len = n - 1;
  kv->pending = tokens[n - 1];
  return 0;
}

int orc_verify(orc_kv* kv, const int32_t* drafts, int gamma, double* logits) {
  if (!kv || gamma < 0 || !logits || (gamma > 0 && !drafts)) return -1;
  if (kv->len + gamma + 1 > kv->max_len) return -4;
  if (!tokens_ok(kv->m, drafts, gamma)) return -1;
  int R = gamma + 1, d = kv->m->c.d_model;
  int32_t* tok = (int32_t*)malloc(sizeof(int32_t) * R);
  tok[0] = kv->pending;
  for (int j = 0; j < gamma; ++j) tok[j + 1] = drafts[j];
  double* x = (double*)malloc(sizeof(double) * (size_t)R * d);
  int rc = block_forward(kv, tok, R, kv->len, x);
  if (rc == 0) lm_head(kv->m, x, R, logits);
  free(x);
  free(tok);
  return rc;
}

int orc_commit(orc_kv* kv, int accepted_len, int next_token) {
  if (!kv || accepted_len < 0 || next_token < 0 || next_token >= kv->m->c.vocab) return -1;
  if (kv->len + accepted_len + 1 > kv->max_len) return -4;
  kv->len += accepted_len + 1;
  kv->pending = next_token;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Acceptance */

static int row_finite(const float* z, int V) {
  for (int v = 0; v < V; ++v)
    if (!isfinite(z[v])) return 0;
  return 1;
}

/* argmax with the lowest index among equal maxima; NaN never wins */
static int row_argmax(const float* z, int V) {
  int best = -1;
  for (int v = 0; v < V; ++v) {
    if (isnan(z[v])) continue;
    if (best < 0 || z[v] > z[best]) best = v;
  }
  return best < 0 ? 0 : best;
}

static double row_lse(const float* z, int V) {
  double mx = -INFINITY;
  for (int v = 0; v < V; ++v)
    if ((double)z[v] > mx) mx = z[v];
  double s = 0.0;
  for (int v = 0; v < V; ++v) s += exp((double)z[v] - mx);
  return mx + log(s);
}

/* largest value among v != x */
static double max_excluding(const float* z, int V, int x) {
  double mx = -INFINITY;
  for (int v = 0; v < V; ++v)
    if (v != x && (double)z[v] > mx) mx = z[v];
  return mx;
}

/* k-th largest (1-based) value among v != x; -inf if fewer than k values */
static int cmp_desc(const void* a, const void* b) {
  double x = *(const double*)a, y = *(const double*)b;
  return (x < y) - (x > y);
}
static double kth_excluding(const float* z, int V, int x, int k) {
  if (k > V - 1) return -INFINITY;
  double* t = (double*)malloc(sizeof(double) * (size_t)V);
  int n = 0;
  for (int v = 0; v < V; ++v)
    if (v != x) t[n++] = z[v];
  qsort(t, (size_t)n, sizeof(double), cmp_desc);
  double r = t[k - 1];
  free(t);
  return r;
}

/* Residual draw of the distribution-preserving ratio rule: weights
 * r(v) = max(0, p(v) - q(v)) (q = NULL: r = p), total R, target t = u R; the
 * draw is the first v with r(v) > 0 whose cumulative weight exceeds t.  R <= 0
 * (p and q equal to rounding) draws from p.  *margin = distance of t from the
 * drawn interval's edges over R. */
static int residual_draw(const float* zp, const float* zq, int V, double u, double* margin) {
  const double lp = row_lse(zp, V), lq = zq ? row_lse(zq, V) : 0.0;
  double R = 0.0;
  for (int v = 0; v < V; ++v) {
    const double r = exp((double)zp[v] - lp) - (zq ? exp((double)zq[v] - lq) : 0.0);
    if (r > 0.0) R += r;
  }
  if (!(R > 0.0)) {
    zq = NULL;
    R = 0.0;
    for (int v = 0; v < V; ++v) R += exp((double)zp[v] - lp);
  }
  const double t = u * R;
  double c = 0.0;
  int last = -1;
  for (int v = 0; v < V; ++v) {
    const double r = exp((double)zp[v] - lp) - (zq ? exp((double)zq[v] - lq) : 0.0);
    if (!(r > 0.0)) continue;
    last = v;
    if (c + r > t) {
      const double lo = t - c, hi = c + r - t;
      *margin = (lo < hi ? lo : hi) / R;
      return v;
    }
    c += r;
  }
  *margin = 0.0; /* t at or beyond the total: rounding; the last positive weight */
  return last;
}

int orc_accept(int mode, const int32_t* draft, const float* p, const float* q,
               size_t q_seq_stride, const float* u, int B, int gamma, int V, int k,
               double lenience, int32_t* accepted_len, int32_t* next_token,
               double* dec_margin, double* argmax_gap, int32_t* flags, double* sample_margin) {
  if (!p || !accepted_len || !next_token || B <= 0 || gamma < 0 || V <= 0) return -1;
  if (gamma > 0 && !draft) return -1;
  if (mode == ORC_TOPK && k < 1) return -1;
  if (mode == ORC_LENIENT && !(lenience > 0.0 && lenience <= 1.0)) return -1;
  const int ratio = mode == ORC_RATIO || mode == ORC_RATIO_SAMPLE;
  if (ratio && (!u || (gamma > 0 && !q))) return -1; /* no drafter row is read when gamma = 0 */
  if (mode < ORC_GREEDY || mode > ORC_RATIO_SAMPLE) return -1;
  const int u_stride = mode == ORC_RATIO_SAMPLE ? gamma + 1 : gamma;
  const float log_len32 = (float)log(lenience);
  for (int b = 0; b < B; ++b) {
    int L = gamma, fl = 0;
    for (int j = 0; j < gamma; ++j) {
      const float* z = p + ((size_t)b * (gamma + 1) + j) * V;
      int x = draft[(size_t)b * gamma + j];
      int pass;
      double margin = INFINITY;
      if (x < 0 || x >= V) {
        pass = 0;
        fl |= 2;
      } else if (!row_finite(z, V) ||
                 (ratio && !row_finite(q + (size_t)b * q_seq_stride + (size_t)j * V, V))) {
        pass = 0;
        fl |= 1;
      } else if (mode == ORC_GREEDY || (mode == ORC_LENIENT && lenience == 1.0)) {
        /* strict: the draft token must be the target argmax (lowest index) */
        pass = row_argmax(z, V) == x;
        margin = fabs((double)z[x] - max_excluding(z, V, x));
      } else if (mode == ORC_TOPK) {
        /* rank of x: strictly larger values, plus equal values at lower index */
        long rank = 0;
        for (int v = 0; v < V; ++v)
          if (z[v] > z[x] || (z[v] == z[x] && v < x)) ++rank;
        pass = rank < k;
        margin = fabs((double)z[x] - kth_excluding(z, V, x, k));
      } else if (mode == ORC_LENIENT) {
        /* z(x) - max_v z(v) >= log(lenience), decided in fp32 */
        float zmax = z[row_argmax(z, V)];
        float diff = z[x] - zmax;
        pass = diff >= log_len32;
        margin = fabs((double)diff - (double)log_len32);
      } else {
        /* ratio: accept iff u < p(x)/q(x), i.e. log u < lp - lq */
        const float* zq = q + (size_t)b * q_seq_stride + (size_t)j * V;
        double lp = (double)z[x] - row_lse(z, V);
        double lq = (double)zq[x] - row_lse(zq, V);
        double uu = u[(size_t)b * u_stride + j];
        double lu = uu > 0.0 ? log(uu) : -INFINITY;
        pass = lu < lp - lq;
        margin = fabs(lu - (lp - lq));
      }
      if (dec_margin) dec_margin[(size_t)b * gamma + j] = margin;
      if (!pass) {
        L = j;
        break;
      }
    }
    if (dec_margin)
      for (int j = L + 1; j < gamma; ++j) dec_margin[(size_t)b * gamma + j] = INFINITY;
    const float* zL = p + ((size_t)b * (gamma + 1) + L) * V;
    if (!row_finite(zL, V)) fl |= 1;
    accepted_len[b] = L;
    next_token[b] = row_argmax(zL, V);
    double sm = INFINITY;
    if (mode == ORC_RATIO_SAMPLE && row_finite(zL, V)) {
      const float* zqL = L < gamma ? q + (size_t)b * q_seq_stride + (size_t)L * V : NULL;
      if (!zqL || row_finite(zqL, V)) next_token[b] = residual_draw(zL, zqL, V, u[(size_t)b * u_stride + gamma], &sm);
    }
    if (sample_margin) sample_margin[b] = sm;
    if (flags) flags[b] = fl;
    if (argmax_gap)
      for (int j = 0; j <= gamma; ++j) {
        const float* z = p + ((size_t)b * (gamma + 1) + j) * V;
        int a = row_argmax(z, V);
        argmax_gap[(size_t)b * (gamma + 1) + j] = (double)z[a] - max_excluding(z, V, a);
      }
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Confidence prefix */

int orc_confidence_prefix(const float* logits, size_t seq_stride, int B, int gamma, int V,
                          double tau, int32_t* skip_len, double* log_conf,
                          const int32_t* draft, double* log_p_draft) {
  if (!logits || !skip_len || B <= 0 || gamma < 0 || V <= 0 || isnan(tau)) return -1;
  /* q_j >= tau  <=>  log q_j >= log tau; decided on fp32 values */
  const float log_tau32 = tau > 0.0 ? (float)log(tau) : -INFINITY;
  for (int b = 0; b < B; ++b) {
    int K = gamma;
    for (int j = 0; j < gamma; ++j) {
      const float* z = logits + (size_t)b * seq_stride + (size_t)j * V;
      double lc = NAN;
      if (row_finite(z, V)) lc = (double)z[row_argmax(z, V)] - row_lse(z, V);
      if (log_conf) log_conf[(size_t)b * gamma + j] = lc;
      if (draft && log_p_draft) {
        int x = draft[(size_t)b * gamma + j];
        log_p_draft[(size_t)b * gamma + j] =
            (x >= 0 && x < V && row_finite(z, V)) ? (double)z[x] - row_lse(z, V) : NAN;
      }
      /* the local gate B_k = min_{j<=k} q_j first falls below tau at the
       * first position whose own score does */
      if (K == gamma && !((float)lc >= log_tau32)) K = j;
    }
    skip_len[b] = K;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Skip scheduler (Sec. 4.1 - 4.2) */

static float log_threshold(double eta) { return eta > 0.0 ? (float)log(eta) : -INFINITY; }

int orc_schedule(const float* log_q, const int32_t* draft, int B, int gamma, int signal, double eta_b,
                 double eta_c, int k_min, int s_max, const int32_t* block_len, const int32_t* special,
                 int n_special, int rep_max, int32_t* D, int32_t* K, int32_t* K_hat, int32_t* reason) {
  if (!log_q || !D || !K || B <= 0 || gamma < 0 || gamma > 64 || signal < 0 || signal > 2 || isnan(eta_b) ||
      isnan(eta_c) || n_special < 0 || (n_special > 0 && !special) || ((n_special > 0 || rep_max >= 2) && !draft))
    return -1;
  const float lb = log_threshold(eta_b), lc = log_threshold(eta_c);
  for (int b = 0; b < B; ++b) {
    const float* lq = log_q + (size_t)b * gamma;
    /* Eq. (candidate skip length): the largest k whose prefix passes both gates */
    int khat = 0;
    float Bk = INFINITY, S = 0.0f;
    for (int k = 1; k <= gamma; ++k) {
      const float x = lq[k - 1];
      if (isnan(x) || x == INFINITY) break; /* invalid score: no longer prefix passes */
      Bk = x < Bk ? x : Bk;
      S = S + x;
      float C;
      if (signal == ORC_SIG_RAW) C = S / (float)k;
      else if (signal == ORC_SIG_MARGINAL) C = Bk;
      else C = S;
      if (Bk >= lb && C >= lc) khat = k;
    }
    int r;
    if (D[b] >= s_max) r = ORC_R_STALE;
    else if (khat == 0) r = ORC_R_NO_CANDIDATE;
    else if (khat < k_min) r = ORC_R_SHORT;
    else if (block_len && block_len[b] < gamma) r = ORC_R_SHORT_BLOCK;
    else {
      r = ORC_R_SKIP;
      const int32_t* x = draft ? draft + (size_t)b * gamma : NULL;
      for (int j = 0; j < khat && r == ORC_R_SKIP && n_special > 0; ++j)
        for (int s = 0; s < n_special; ++s)
          if (x[j] == special[s]) r = ORC_R_SPECIAL;
      if (r == ORC_R_SKIP && rep_max >= 2) {
        int run = 1;
        for (int j = 1; j < khat; ++j) {
          run = x[j] == x[j - 1] ? run + 1 : 1;
          if (run >= rep_max) { r = ORC_R_REPEAT; break; }
        }
      }
    }
    K[b] = r == ORC_R_SKIP ? khat : 0;
    if (K_hat) K_hat[b] = khat;
    if (reason) reason[b] = r;
    D[b] = K[b] > 0 ? D[b] + K[b] : 0;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Survival predictor MLP */

static double gelu_erf(double x) { return 0.5 * x * (1.0 + erf(x / sqrt(2.0))); }

static double bf16_bits_value(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* log sigmoid(z) = -log(1 + exp(-z)), evaluated without overflow */
static double log_sigmoid(double z) { return z >= 0.0 ? -log1p(exp(-z)) : z - log1p(exp(z)); }

static void dense(const double* x, int din, const float* W, const float* b, int dout, double* y, int act) {
  for (int o = 0; o < dout; ++o) {
    double acc = b ? (double)b[o] : 0.0;
    for (int i = 0; i < din; ++i) acc += (double)W[(size_t)o * din + i] * x[i];
    y[o] = act ? gelu_erf(acc) : acc;
  }
}

int orc_survival_mlp(const uint16_t* hidden, const float* scalars, int n, int d_hid, int n_sc, int H,
                     const float* mu, const float* sigma, const float* W1, const float* b1, const float* W2,
                     const float* b2, const float* W3, const float* b3, const float* w4, float b4,
                     double* log_score, double* logit) {
  if (!hidden || (n_sc > 0 && !scalars) || !mu || !sigma || !W1 || !W2 || !W3 || !w4 || !log_score || n < 0 ||
      d_hid < 0 || n_sc < 0 || d_hid + n_sc <= 0 || H <= 0)
    return -1;
  const int din = d_hid + n_sc;
  int rc = 0;
#pragma omp parallel for schedule(static) reduction(| : rc)
  for (int r = 0; r < n; ++r) {
    double* x = (double*)malloc(sizeof(double) * (size_t)(din + 3 * H));
    if (!x) { rc |= 1; continue; }
    double *h1 = x + din, *h2 = h1 + H, *h3 = h2 + H;
    for (int i = 0; i < din; ++i) {
      const double raw = i < d_hid ? bf16_bits_value(hidden[(size_t)r * d_hid + i])
                                   : (double)scalars[(size_t)r * n_sc + (i - d_hid)];
      x[i] = (raw - (double)mu[i]) / (double)sigma[i];
    }
    dense(x, din, W1, b1, H, h1, 1);
    dense(h1, H, W2, b2, H, h2, 1);
    dense(h2, H, W3, b3, H, h3, 1);
    double z;
    dense(h3, H, w4, NULL, 1, &z, 0);
    z += (double)b4;
    log_score[r] = log_sigmoid(z);
    if (logit) logit[r] = z;
    free(x);
  }
  return rc ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* Agreement accounting */

int orc_audit_accumulate(const int32_t* K, const int32_t* L, int B, int64_t* acc) {
  if (!K || !L || !acc || B < 0) return -1;
  for (int b = 0; b < B; ++b) {
    if (K[b] <= 0) continue; /* strict round: not in A */
    acc[0] += 1;
    acc[1] += K[b];
    acc[2] += K[b] < L[b] ? K[b] : L[b];
    acc[3] += K[b] <= L[b] ? 1 : 0;
  }
  return 0;
}
