/*
 * CPU oracle for verifier-skipped speculative diffusion decoding.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke entry and the CPU-baseline
 * leg of the benchmark may load this library.  The GPU product path never
 * links, imports or calls it, and it shares no code with the GPU path.
 *
 * Plain, slow, obviously correct: every floating-point quantity of the method
 * is computed in IEEE double precision, except where the paper fixes fp32 (the
 * acceptance and confidence decisions are taken in fp32, the precision the
 * paper uses for target log-probabilities, Appendix "Evaluation and
 * Throughput").  Weights are synthetic bf16 (or fp32) values held exactly in
 * float storage.
 *
 * Paper: "From Positionwise Confidence to Prefix Scheduling: Verifier Skipping
 * in Speculative Decoding".
 */
#ifndef SDD_ORACLE_H
#define SDD_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Decoder shape (the paper names Qwen3-32B / Qwen2.5-7B-class targets but
 * prints no architecture; the textbook pre-norm decoder is written out). */
typedef struct {
  int n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab;
  double rms_eps, rope_theta;
  int qk_norm;      /* 1: per-head RMSNorm of q and k before RoPE */
  int bf16_weights; /* 1: weights are bf16 values; 0: fp32 values */
  /* 1: BF16-operand mode (the verifier as a BF16 model, Appendix "Evaluation
   * and Throughput"): every activation that enters a matrix product (x * g of
   * each projection with the RMSNorm row scale applied to the product, q, k,
   * v, the attention output, the FFN hidden state) is rounded to BF16 (ties to
   * even); sums, softmax, norms, RoPE and the residual stream stay exact.
   * 0: exact fp64 throughout. */
  int bf16_operands;
} orc_config;

/* Tensor kinds for orc_model_set_tensor / orc_weight_values. */
enum {
  ORC_EMBED = 0, ORC_LM_HEAD = 1, ORC_FINAL_NORM = 2,
  ORC_WQ = 3, ORC_WK = 4, ORC_WV = 5, ORC_WO = 6,
  ORC_WGATE = 7, ORC_WUP = 8, ORC_WDOWN = 9,
  ORC_ATTN_NORM = 10, ORC_FFN_NORM = 11, ORC_Q_NORM = 12, ORC_K_NORM = 13
};

/* Acceptance modes (Appendix "Baselines and Sweep Settings"; Sec. 3.1). */
enum { ORC_GREEDY = 0, ORC_RATIO = 1, ORC_TOPK = 2, ORC_LENIENT = 3, ORC_RATIO_SAMPLE = 4 };

/* Threads the oracle's parallel loops use. */
int orc_num_threads(void);

/* Counter-based synthetic weight generator (SplitMix64 + Irwin-Hall(4)). */
uint64_t orc_splitmix64(uint64_t x);
int orc_tensor_id(int kind, int layer);
void orc_weight_values(uint64_t seed, int tensor_id, uint64_t start, uint64_t count,
                       double sigma, int bf16, float* out);

typedef struct orc_model orc_model;
orc_model* orc_model_create(const orc_config* cfg, uint64_t seed, double sigma);
void orc_model_free(orc_model* m);
/* The same model with layer streaming: only the embedding, LM head and final
 * norm are held; every forward (full or cached route) generates a layer's
 * tensors when it reaches the layer and frees them after it.  Same values as
 * orc_model_create; norm gains are 1 and cannot be replaced
 * (orc_model_set_tensor refuses layer tensors). */
orc_model* orc_model_create_streamed(const orc_config* cfg, uint64_t seed, double sigma);
/* shape of a tensor kind: rows x cols (row-major, PyTorch Linear [out][in]) */
int orc_tensor_shape(const orc_config* cfg, int kind, int64_t* rows, int64_t* cols);
int orc_model_set_tensor(orc_model* m, int kind, int layer, const float* src);

/* Full recompute (the paper's verifier: no KV cache).  Causal forward over
 * tokens[0..n); writes logits of rows [row0, n) to logits[(n-row0) * V]. */
int orc_forward_full(const orc_model* m, const int32_t* tokens, int n, int row0, double* logits);
/* Same, but returns the final hidden rows (after the last layer, before the
 * final norm) for rows [row0, n): hidden[(n-row0) * d]. */
int orc_forward_full_hidden(const orc_model* m, const int32_t* tokens, int n, int row0, double* hidden);

/* orc_forward_full in steps: x[n][d] (fp64) = embedding rows of tokens;
 * orc_layer_full applies layer `layer` to all n rows in place (causal
 * attention among them); orc_final_logits applies the final norm and the LM
 * head to R rows.  Embedding, layers 0..n_layers-1 in order, then the rows
 * from row0 give exactly orc_forward_full's logits. */
int orc_embed(const orc_model* m, const int32_t* tokens, int n, double* x);
int orc_layer_full(const orc_model* m, int layer, int n, double* x);
int orc_final_logits(const orc_model* m, const double* x, int R, double* logits);

/* Cached mode: one sequence, K/V of every layer kept in fp64. */
typedef struct orc_kv orc_kv;
orc_kv* orc_kv_create(const orc_model* m, int max_len);
void orc_kv_free(orc_kv* kv);
int orc_kv_len(const orc_kv* kv);
int orc_kv_pending(const orc_kv* kv);
/* K/V of the cache: layer, position -> k[Hkv*hd], v[Hkv*hd] (fp64). */
int orc_kv_read(const orc_kv* kv, int layer, int pos, double* k, double* v);
/* Prefill: caches tokens[0..n-1), len = n-1, pending = tokens[n-1]. */
int orc_kv_prefill(orc_kv* kv, const int32_t* tokens, int n);
/* Verify: rows [pending, drafts[0..gamma)] at positions len..len+gamma;
 * logits[(gamma+1) * V].  K/V rows are written but len is unchanged. */
int orc_verify(orc_kv* kv, const int32_t* drafts, int gamma, double* logits);
/* Commit: len += L + 1, pending = next. */
int orc_commit(orc_kv* kv, int accepted_len, int next_token);

/* Acceptance test over target rows p[B][gamma+1][V] (fp32 values).
 * Ratio modes also read drafter rows q (row j of sequence b at
 * q + b*q_seq_stride + j*V) and uniforms: u[B][gamma] (RATIO) or
 * u[B][gamma+1] (RATIO_SAMPLE, column gamma is the draw of the next token).
 * RATIO_SAMPLE is the distribution-preserving rule of the min(1, p/q) test
 * that Sec. 3.1 cites: after the first rejection at row L the next token is
 * drawn from norm(max(0, p_L - q_L)), after a fully accepted block from
 * p_gamma, by inverse CDF in vocabulary order (first v whose cumulative
 * weight exceeds u * R, R the total weight; R <= 0 draws from p_L); p and q
 * are softmax of the rows, in fp64.  The other modes take next = argmax of
 * row L (lowest index), as does RATIO_SAMPLE when row L is non-finite.
 * Outputs accepted_len[B], next_token[B]; optional margins:
 *   dec_margin[B][gamma]   distance of each decision from its threshold
 *   argmax_gap[B][gamma+1] top-1 minus top-2 value of each target row
 *   flags[B]               bit0: a non-finite value was seen in a decisive row
 *                          bit1: a draft token outside [0, V)
 *   sample_margin[B]       RATIO_SAMPLE: distance of u * R from the edges of
 *                          the drawn token's interval, divided by R */
int orc_accept(int mode, const int32_t* draft, const float* p, const float* q,
               size_t q_seq_stride, const float* u, int B, int gamma, int V, int k,
               double lenience, int32_t* accepted_len, int32_t* next_token,
               double* dec_margin, double* argmax_gap, int32_t* flags, double* sample_margin);

/* Raw-confidence prefix (Sec. 4.1-4.2): log conf_j = max_v z_j - LSE(z_j);
 * skip_len = first j with conf_j < tau (gamma if none).  Rows of sequence b
 * start at logits + b*seq_stride, row j at +j*V.  log_conf[B][gamma] and
 * p_draft[B][gamma] (probability of draft[b][j] if draft != NULL) optional. */
int orc_confidence_prefix(const float* logits, size_t seq_stride, int B, int gamma, int V,
                          double tau, int32_t* skip_len, double* log_conf,
                          const int32_t* draft, double* log_p_draft);

/* Skip scheduler (Sec. 4.1 candidate skip length and guards; Sec. 4.2
 * confidence signals; Appendix "Baselines and Sweep Settings" guard list).
 * log_q[b][j] (fp32) is log q_{j+1}, the position score of draft j.  Gates
 * for a prefix of length k, decided in fp32 on fp32 values:
 *   local gate  B_k = min_{j<=k} log q_j            >= fl(log eta_b)
 *   prefix gate C_k >= fl(log eta_c), with C_k (log) for the signal:
 *     RAW          mean of log q_1..k  (geometric mean)  = S_k / k
 *     MARGINAL     B_k                                  (running minimum)
 *     CONDITIONAL  S_k = sum of log q_1..k              (product, log space)
 *   where S_k = fl(S_{k-1} + log q_k) in position order.
 * K_hat = max{k in 1..gamma : both gates}, 0 if none; a non-finite score
 * (NaN, +inf) is invalid and no prefix reaching it passes.  Guards, in order
 * (reason code when the round is strict): D >= s_max (STALE); K_hat = 0
 * (NO_CANDIDATE); K_hat < k_min (SHORT); block_len[b] < gamma (SHORT_BLOCK;
 * block_len may be NULL: every block is whole);
 * a draft in x_1..x_{K_hat} in special[] (SPECIAL); rep_max >= 2 and
 * rep_max equal consecutive drafts in x_1..x_{K_hat} (REPEAT).  Otherwise
 * K = K_hat (SKIP).  Then D += K if K > 0, else D = 0 (a strict round calls
 * the verifier).  draft may be NULL when n_special = 0 and rep_max < 2. */
enum { ORC_SIG_RAW = 0, ORC_SIG_MARGINAL = 1, ORC_SIG_CONDITIONAL = 2 };
enum { ORC_R_SKIP = 0, ORC_R_STALE = 1, ORC_R_NO_CANDIDATE = 2, ORC_R_SHORT = 3, ORC_R_SHORT_BLOCK = 4,
       ORC_R_SPECIAL = 5, ORC_R_REPEAT = 6 };
int orc_schedule(const float* log_q, const int32_t* draft, int B, int gamma, int signal, double eta_b,
                 double eta_c, int k_min, int s_max, const int32_t* block_len, const int32_t* special,
                 int n_special, int rep_max, int32_t* D, int32_t* K, int32_t* K_hat, int32_t* reason);

/* Survival predictor (Appendix "Predictor Details"): per draft position, the
 * drafter's LM-head input h (d_hid values, bf16 bits) and n_sc scalar
 * features form x = [h, s] (d_in = d_hid + n_sc); x is normalized as
 * (x - mu) / sigma; then an MLP d_in -> H -> H -> H -> 1 with GELU (erf
 * form) after each hidden layer (dropout is off at inference):
 *   h1 = GELU(W1 x~ + b1), h2 = GELU(W2 h1 + b2), h3 = GELU(W3 h2 + b3),
 *   z = w4 . h3 + b4,  log score = log sigmoid(z)
 * (the marginal a_j or conditional s_j survival estimate, Sec. 4.2).  Weights
 * are PyTorch Linear layouts [out][in], fp32.  Everything in fp64.
 * Outputs log_score[n] and (optional) logit[n]. */
int orc_survival_mlp(const uint16_t* hidden, const float* scalars, int n, int d_hid, int n_sc, int H,
                     const float* mu, const float* sigma, const float* W1, const float* b1, const float* W2,
                     const float* b2, const float* W3, const float* b3, const float* w4, float b4,
                     double* log_score, double* logit);

/* Agreement with strict verification (Sec. 3.2, strict token agreement and
 * full prefix acceptance equations): over the rounds b with K_b > 0 (the set
 * A of rounds that commit a nonempty unverified prefix), accumulate
 * acc[0] += |A|, acc[1] += sum K_b, acc[2] += sum min(K_b, L_b),
 * acc[3] += sum 1{K_b <= L_b}.  StrictToken = acc[2] / acc[1],
 * FullPrefix = acc[3] / acc[0] (both 1 when A is empty, as for Strict SDD). */
int orc_audit_accumulate(const int32_t* K, const int32_t* L, int B, int64_t* acc);

#ifdef __cplusplus
}
#endif
#endif
