/*
 * sdd.h -- C ABI of the MI355X (gfx950) hot path of verifier-skipped
 * speculative diffusion decoding.
 *
 * Paper: "From Positionwise Confidence to Prefix Scheduling: Verifier Skipping
 * in Speculative Decoding".  A diffusion drafter proposes a block
 * x^_1..x^_gamma; the target model verifies it in one call and accepts a prefix
 * of length L in {0..gamma} (Sec. 3.1 "Strict Decoding and Verifier
 * Skipping"); a confidence scheduler may instead commit a prefix of length K
 * without calling the target (Sec. 4.1 "Skip Policy", candidate skip length
 * equation).
 *
 * Conventions for every function:
 *  - returns SDD_OK (0) or a negative SDD_E* code; sdd_last_error() gives a
 *    human-readable message for the last failure on the calling thread;
 *  - argument errors are detected synchronously, before anything is launched;
 *  - pointers documented as "device" are caller-owned device allocations
 *    (e.g. from torch); the library never allocates device memory;
 *  - work is enqueued on the given HIP stream and completes asynchronously;
 *    the caller synchronizes before reading outputs;
 *  - integer outputs are deterministic: reductions use fixed orders and no
 *    floating-point atomics, so repeated calls give bit-identical results.
 */
#ifndef SDD_H
#define SDD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* sdd_stream_t; /* a hipStream_t; NULL = default stream */

/* status codes */
#define SDD_OK 0
#define SDD_EINVAL (-1)       /* bad argument */
#define SDD_ENOMEM (-2)       /* buffer too small / host allocation failed */
#define SDD_EHIP (-3)         /* a HIP call or kernel launch failed */
#define SDD_ECAPACITY (-4)    /* KV cache or workspace capacity exceeded */
#define SDD_EUNSUPPORTED (-5) /* shape/dtype/mode combination not built */

/* element types */
#define SDD_F32 0
#define SDD_BF16 1

/* acceptance modes (Sec. 3.1; Appendix "Baselines and Sweep Settings") */
#define SDD_GREEDY 0  /* accept x^_j iff it is the target argmax (lowest index on ties) */
#define SDD_RATIO 1   /* accept iff u_j < p(x^_j)/q(x^_j) (min(1, p/q) test of [Leviathan 2023]) */
#define SDD_TOPK 2    /* accept iff x^_j is among the k largest target logits */
#define SDD_LENIENT 3 /* accept iff z(x^_j) - max_v z(v) >= log(lenience); lenience 1 = greedy */
#define SDD_RATIO_SAMPLE 4 /* RATIO, and the next token is drawn (distribution-preserving rule, below) */

/* tensor kinds for sdd_model_load_tensor (row-major, PyTorch Linear [out][in]) */
#define SDD_T_EMBED 0      /* [vocab][d_model] */
#define SDD_T_LM_HEAD 1    /* [vocab][d_model] */
#define SDD_T_FINAL_NORM 2 /* [d_model], fp32 */
#define SDD_T_WQ 3         /* [n_q_heads*head_dim][d_model] */
#define SDD_T_WK 4         /* [n_kv_heads*head_dim][d_model] */
#define SDD_T_WV 5         /* [n_kv_heads*head_dim][d_model] */
#define SDD_T_WO 6         /* [d_model][n_q_heads*head_dim] */
#define SDD_T_WGATE 7      /* [d_ff][d_model] */
#define SDD_T_WUP 8        /* [d_ff][d_model] */
#define SDD_T_WDOWN 9      /* [d_model][d_ff] */
#define SDD_T_ATTN_NORM 10 /* [d_model], fp32 */
#define SDD_T_FFN_NORM 11  /* [d_model], fp32 */
#define SDD_T_Q_NORM 12    /* [head_dim], fp32 */
#define SDD_T_K_NORM 13    /* [head_dim], fp32 */

/* Target decoder shape.  The paper names its verifier (Qwen3-32B, Sec. 5.1)
 * but not its architecture; this is the pre-norm decoder of that family:
 * RMSNorm, GQA attention with rotate-half RoPE (optionally per-head QK
 * RMSNorm before RoPE), SwiGLU FFN, untied LM head, no biases. */
typedef struct {
  int n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rms_eps, rope_theta;
  int qk_norm; /* 1: per-head RMSNorm on q and k before RoPE */
  int dtype;   /* SDD_F32 or SDD_BF16: weights, KV cache and GEMM inputs */
} sdd_model_config;

typedef struct sdd_model sdd_model;
typedef struct sdd_kv sdd_kv;

const char* sdd_status_string(int status);
const char* sdd_last_error(void);
/* 1 if the library was built for gfx950 and a gfx950 device is current. */
int sdd_device_ok(void);

/* ---- model ------------------------------------------------------------ */

/* Bytes of the device weight buffer for cfg on the current device.  Weights
 * are stored in the library's MFMA-tiled layout, not row-major, in an order
 * that depends on the device's compute-unit count (sdd_model_matrix_layout). */
int sdd_weights_bytes(const sdd_model_config* cfg, size_t* bytes);

/* Wraps a caller-owned device buffer of at least sdd_weights_bytes() bytes.
 * The handle is host memory; destroy with sdd_model_destroy (the buffer stays
 * the caller's).  Supported: head_dim 64 or 128, n_q_heads % n_kv_heads == 0,
 * d_model and vocab multiples of 32, d_ff a multiple of 32 (bf16) or 16 (fp32). */
int sdd_model_create(const sdd_model_config* cfg, void* weights, size_t bytes, sdd_model** out);
int sdd_model_destroy(sdd_model* m);

/* Fills every weight with the synthetic counter-based generator:
 * w = round(sigma * sqrt(3)/65536 * S) with S the Irwin-Hall sum of the four
 * 16-bit lanes of SplitMix64(key(seed, tensor) + index * golden), index the
 * row-major position in the [out][in] matrix; norm gains are set to 1. */
int sdd_model_init_random(sdd_model* m, uint64_t seed, float sigma, sdd_stream_t stream);

/* Copies one row-major tensor (device pointer; model dtype for matrices and
 * embeddings, fp32 for norm gains) into the tiled layout. */
int sdd_model_load_tensor(sdd_model* m, int kind, int layer, const void* src, sdd_stream_t stream);

/* Layout of one tiled weight matrix (kind SDD_T_LM_HEAD, or SDD_T_WQ..SDD_T_WDOWN
 * of `layer`; q/k/v share one fused matrix [Wq; Wk; Wv], gate/up one matrix whose
 * 16-row tiles alternate gate, up).  A tile is 1 KiB: 16 rows x kt columns
 * (kt 32 for bf16, 16 for fp32), lane l's 16 bytes holding row l % 16 and the
 * 16 / elem columns from (l / 16) * 16 / elem.  Row tiles form column groups
 * of *ng; unit (g, k) is the ng tiles of group g at k-step k (u = g KT + k),
 * and the plan splits the G * KT units over *n_wg workgroups by cost: each
 * group counts as KT + c units (c = *seg_units, the cost of a workgroup's
 * entering one more group; 0 gives equal shares), and workgroup w owns units
 * [start(w), start(w + 1)) with start(w) = g KT + max(0, o - c) for
 * x = w G (KT + c) / n_wg, g = x / (KT + c), o = x mod (KT + c) (integer
 * division).  The i-th unit of workgroup w is stored at slot i * n_wg + w, its
 * tile j (row tile g * ng + j) at byte *offset + (slot * ng + j) * 1024 of the
 * weight buffer; the matrix holds n_wg times the longest share of slots, and
 * slots past a shorter share are zero.  *bytes is the matrix's extent.
 * Host-only (no device access).  Errors: SDD_EINVAL for a NULL pointer, a bad
 * kind or layer. */
int sdd_model_matrix_layout(const sdd_model* m, int kind, int layer, size_t* offset, size_t* bytes, int* KT,
                            int* G, int* ng, int* n_wg, int* seg_units);

/* ---- KV cache ---------------------------------------------------------- */

/* Bytes of a KV cache for max_batch sequences of up to max_len positions. */
int sdd_kv_bytes(const sdd_model_config* cfg, int max_batch, int max_len, size_t* bytes);
/* Wraps a caller-owned device buffer and resets every sequence to empty
 * (length 0, pending token 0) with a kernel on stream. */
int sdd_kv_create(sdd_model* m, int max_batch, int max_len, void* buf, size_t bytes,
                  sdd_stream_t stream, sdd_kv** out);
int sdd_kv_destroy(sdd_kv* kv);
/* Synchronous read of per-sequence state: len[max_batch], pending[max_batch]
 * (host pointers, either may be NULL) and the sticky error word (bit0: a
 * capacity overflow was refused on the device, bit1: a token outside
 * [0, vocab) was replaced by 0, bit2: a sequence id outside [0, max_batch)
 * was refused, bit3: a GEMM workgroup's internal hand-off between its waves
 * gave up after its bounded wait, so that call's outputs are invalid). */
int sdd_kv_state(sdd_kv* kv, int32_t* len, int32_t* pending, int32_t* error_bits,
                 sdd_stream_t stream);

/* Device pointers to the per-sequence length and pending-token arrays
 * (int32[max_batch] each), valid while kv exists; lets callers build the next
 * block on the device without a host round trip.  Read-only for callers. */
int sdd_kv_device_state(sdd_kv* kv, const int32_t** len, const int32_t** pending);

/* Workspace for prefill/verify of up to max_rows rows per call. */
int sdd_workspace_bytes(const sdd_model* m, int max_rows, size_t* bytes);
/* Prepares a caller-owned device workspace (zeroes its counters with a
 * kernel); needed once after allocation.  Every call leaves the counters zero
 * again, so the workspace may be reused by any number of later calls on the
 * same stream. */
int sdd_workspace_init(void* ws, size_t bytes, sdd_stream_t stream);

/* Prefill of sequence seq with tokens[0..n) (device int32): caches positions
 * 0..n-2, sets len = n-1 and pending = tokens[n-1].  The prompt is processed
 * in row chunks of at most max_rows of the workspace.
 * The verifier KV cache is this library's reading of the verify call: the
 * paper's own verifier keeps no cache and recomputes the whole sequence every
 * call (Appendix "Evaluation and Throughput"; sdd_verify_full is that mode).
 * Caching the committed prefix leaves the call's result unchanged: attention
 * of a position depends only on the positions before it (the causal decoder
 * the target is).  Errors: SDD_EINVAL (NULL pointer, seq outside
 * [0, max_batch), n < 1), SDD_ECAPACITY (n - 1 > max_len, workspace too
 * small for a 16-row chunk); a token outside [0, vocab) is replaced by 0 on
 * the device and sets sticky error bit1. */
int sdd_kv_prefill(sdd_model* m, sdd_kv* kv, int seq, const int32_t* tokens, int n,
                   void* ws, size_t ws_bytes, sdd_stream_t stream);

/* Block verification (Sec. 3.1): for each of n_seq sequences (seq_ids,
 * device int32[n_seq]) runs the causal decoder over the gamma+1 rows
 * [pending, drafts[s][0..gamma)] at positions len..len+gamma against the
 * sequence's cache.  Row j < gamma scores draft j; row gamma is the bonus
 * position.  Outputs (device): logits fp32 [n_seq][gamma+1][vocab] and
 * argmax int32 [n_seq][gamma+1] (lowest index on ties; may be NULL).  K/V of
 * the rows are written at len..len+gamma but len is unchanged until
 * sdd_kv_commit.  gamma = 0 is a plain decode step.  Sequences whose cache
 * cannot hold the block are refused on the device (sticky error bit0; their
 * outputs are left unwritten).  Requires n_seq*(gamma+1) <= max_rows of ws. */
int sdd_verify_block(sdd_model* m, sdd_kv* kv, const int32_t* seq_ids, int n_seq,
                     const int32_t* drafts, int gamma, float* logits, int32_t* argmax,
                     void* ws, size_t ws_bytes, sdd_stream_t stream);

/* Full-recompute verification (the verifier the paper measures: no verifier
 * KV cache, Appendix "Evaluation and Throughput"; rows as in Sec. 3.1).
 * tokens (device int32 [n]) is one sequence's context followed by its gamma
 * drafts; every position's K/V is recomputed from scratch into slot 0 of the
 * caller's scratch cache (max_len >= n; its slot-0 contents are overwritten,
 * other slots untouched).  Outputs as sdd_verify_block for that one sequence:
 * logits fp32 [gamma+1][vocab] of positions n-gamma-1 .. n-1 (row j < gamma
 * scores draft j, row gamma is the bonus position), argmax int32 [gamma+1]
 * (may be NULL).  The same kernels as the cached call, so the logits equal
 * those of sdd_verify_block on a cache prefilled with the context.
 * Errors: SDD_EINVAL (NULL pointer, gamma outside [0, 64], n < gamma + 1),
 * SDD_ECAPACITY (n > max_len, small workspace). */
int sdd_verify_full(sdd_model* m, sdd_kv* scratch, const int32_t* tokens, int n, int gamma, float* logits,
                    int32_t* argmax, void* ws, size_t ws_bytes, sdd_stream_t stream);

/* Commit after acceptance (Sec. 3.1: the target accepts the prefix
 * x^_1..x^_L and supplies one more token, its correction at L or the bonus
 * token after a fully accepted block; Sec. 4.1 commit rule, a strict round
 * advances by the verified prefix plus that token).  Device int32 arrays
 * [n_seq]: for sequence seq_ids[i], len += accepted_len[i] + 1 and pending =
 * next_token[i]; the cache rows len..len+L written by the verify call become
 * committed, later rows are overwritten by the next call.  Errors: SDD_EINVAL
 * (NULL pointer, n_seq outside [1, max_batch]); on the device a sequence id
 * out of range (sticky bit2), a negative length, an overflow of max_len or a
 * token outside [0, vocab) (sticky bit0) leave that sequence unchanged. */
int sdd_kv_commit(sdd_kv* kv, const int32_t* seq_ids, int n_seq, const int32_t* accepted_len,
                  const int32_t* next_token, sdd_stream_t stream);
/* ---- acceptance and confidence ---------------------------------------- */

/* Workspace bytes for sdd_accept / sdd_confidence_prefix at these shapes
 * (zeroed once by sdd_workspace_init; the calls leave it reusable). */
int sdd_rowstats_workspace_bytes(int B, int gamma, int V, size_t* bytes);

/* Acceptance test (Sec. 3.1; lenience equation and top-k rule, Appendix
 * "Baselines and Sweep Settings").  Device inputs:
 *   draft     int32 [B][gamma]
 *   p_logits  target logits [B][gamma+1][V], dtype p_dtype, contiguous
 *   q_logits  drafter logits, ratio modes only: row j of sequence b at
 *             q_logits + b*q_seq_stride + j*V elements (dtype q_dtype)
 *   uniforms  fp32 in [0,1): [B][gamma] (RATIO) or [B][gamma+1]
 *             (RATIO_SAMPLE; column gamma draws the next token)
 * For j < gamma, row j decides draft j; L = first failing j (gamma if none);
 * next_token = argmax of target row L (lowest index on ties).  RATIO_SAMPLE
 * (the distribution-preserving form of the min(1, p/q) rule that Sec. 3.1
 * cites) instead draws next_token from norm(max(0, p_L - q_L)) when L <
 * gamma and from p_gamma when every draft passed, p and q being the softmax
 * of the rows: inverse CDF in vocabulary order, the first v whose running
 * weight exceeds u * W (W the total weight), with fp32 weights summed in one
 * fixed order (bit-reproducible); if the residual total is not positive the
 * draw is from p_L; a non-finite row L keeps the argmax.  A non-finite
 * value in a deciding row, or a draft token outside [0,V), fails that
 * position.  Outputs (device int32 [B]): accepted_len, next_token, and flags
 * (may be NULL; bit0 non-finite value seen, bit1 draft token out of range).
 * Errors: SDD_EINVAL for NULL required pointers (uniforms in the ratio
 * modes, drafter logits in the ratio modes when gamma > 0), B <= 0, gamma < 0
 * or > 64, V <= 0, k < 1 (TOPK), lenience not in (0,1] (LENIENT), drafter and
 * target logits of different dtypes (ratio modes). */
int sdd_accept(const int32_t* draft, const void* p_logits, int p_dtype, const void* q_logits,
               int q_dtype, size_t q_seq_stride, const float* uniforms, int B, int gamma, int V,
               int mode, int k, float lenience, int32_t* accepted_len, int32_t* next_token,
               int32_t* flags, void* ws, size_t ws_bytes, sdd_stream_t stream);

/* sdd_accept for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments and results as sdd_accept without the workspace.  Its
 * workspace is a 256 KiB array inside the library, one per GPU, held until the
 * process ends; the call allocates nothing.  Calls on one GPU share that
 * array: calls that overlap in time on one GPU (other streams, other host
 * threads) race and must be serialized by the caller.  The first call on a
 * device looks up the array's address and enqueues a kernel that clears it
 * on the stream.  Errors: those of sdd_accept, and SDD_ECAPACITY when the
 * shape needs more than 256 KiB of workspace (sdd_rowstats_workspace_bytes;
 * e.g. B = 64 with gamma = 64 fits, about B * (gamma + 1) <= 7000 rows). */
int sdd_accept_noalloc(const int32_t* draft, const void* p_logits, int p_dtype, const void* q_logits,
                       int q_dtype, size_t q_seq_stride, const float* uniforms, int B, int gamma, int V,
                       int mode, int k, float lenience, int32_t* accepted_len, int32_t* next_token,
                       int32_t* flags, sdd_stream_t stream);

/* Raw-confidence prefix (Sec. 4.1 local gate B_k = min_{j<=k} q_j; Sec. 4.2
 * raw confidence = max softmax of the drafter row).  Row j < gamma of
 * sequence b at logits + b*seq_stride + j*V elements.  skip_len[b] =
 * max{k : B_k >= tau} = first j with q_j < tau (gamma if none), decided as
 * fp32 log q_j >= fp32 log tau.  Optional outputs: log_conf fp32 [B][gamma];
 * with draft != NULL, log_p_draft fp32 [B][gamma] = log softmax at the draft
 * token.  A row with a non-finite value has log q = NaN and stops the prefix.
 * Errors: SDD_EINVAL for NULL required pointers, B <= 0, gamma < 0 or > 64,
 * V <= 0, tau NaN. */
int sdd_confidence_prefix(const void* logits, int dtype, size_t seq_stride, int B, int gamma,
                          int V, float tau, int32_t* skip_len, float* log_conf,
                          const int32_t* draft, float* log_p_draft, void* ws, size_t ws_bytes,
                          sdd_stream_t stream);

/* ---- skip scheduler ------------------------------------------------------ */

/* confidence signals for the prefix gate (Sec. 4.2) */
#define SDD_SIG_RAW 0         /* C_k = geometric mean of q_1..q_k (raw confidence) */
#define SDD_SIG_MARGINAL 1    /* C_k = min_{j<=k} a_j (marginal survival; both gates become eta_m) */
#define SDD_SIG_CONDITIONAL 2 /* C_k = prod_{j<=k} s_j (conditional survival, chain rule) */

/* why a round is a skip (K > 0) or strict (K = 0) */
#define SDD_SKIP_OK 0           /* all conditions hold: K = K_hat tokens are committed unverified */
#define SDD_SKIP_STALE 1        /* D >= s_max: staleness forces a strict round */
#define SDD_SKIP_NO_CANDIDATE 2 /* K_hat = 0 */
#define SDD_SKIP_SHORT 3        /* K_hat < k_min */
#define SDD_SKIP_SHORT_BLOCK 4  /* the block is a shortened final block */
#define SDD_SKIP_SPECIAL 5      /* a special (e.g. end-of-sequence) token in x^_1..x^_K_hat */
#define SDD_SKIP_REPEAT 6       /* rep_max equal consecutive drafts in x^_1..x^_K_hat */

/* Skip decision for B sequences (Sec. 4.1 candidate skip length, commit rule
 * and staleness; Sec. 4.2 signals; Appendix "Baselines and Sweep Settings"
 * guard list).  Device inputs:
 *   log_q      fp32 [B][gamma]: log of the position score of draft j (raw
 *              confidence, marginal survival a_j or conditional survival s_j;
 *              sdd_confidence_prefix's log_conf is the raw one)
 *   draft      int32 [B][gamma]; needed when n_special > 0 or rep_max >= 2
 *   block_len  int32 [B] drafted block length (< gamma: shortened final
 *              block); NULL = every block is whole
 *   special    int32 [n_special] tokens a skipped prefix may not contain
 *   D          int32 [B] unverified tokens committed since the last verifier
 *              call; read and updated in place
 * For a prefix of length k the local gate is B_k = min_{j<=k} log q_j >=
 * log eta_b and the prefix gate is C_k >= log eta_c (C_k per signal, in log
 * space; the raw mean is S_k / k with S_k = S_{k-1} + log q_k summed in
 * position order in fp32).  Thresholds are rounded to fp32 as
 * (float)log(eta) (eta <= 0: -inf) and every comparison is an fp32 >=.
 * K_hat = the largest k passing both gates (0 if none); a NaN or +inf score
 * ends the search.  Guards in order: D >= s_max, K_hat = 0, K_hat < k_min,
 * block_len < gamma, special token, repetition; the first that applies sets
 * reason and K = 0, otherwise K = K_hat.  D becomes D + K after a skip and 0
 * after a strict round.  Outputs (device int32 [B]): K, and optionally K_hat
 * and reason (may be NULL).
 * Errors: SDD_EINVAL for NULL required pointers, B <= 0, gamma outside
 * [0, 64], a bad signal, a NaN threshold, n_special outside [0, 256]. */
int sdd_schedule(const float* log_q, const int32_t* draft, const int32_t* block_len, int B, int gamma,
                 int signal, double eta_b, double eta_c, int k_min, int s_max, const int32_t* special,
                 int n_special, int rep_max, int32_t* D, int32_t* K, int32_t* K_hat, int32_t* reason,
                 sdd_stream_t stream);

/* Agreement with strict verification (Sec. 3.2, strict token agreement and
 * full prefix acceptance): for the rounds b with K[b] > 0, acc (device int64
 * [4], caller-zeroed, accumulated across calls) gains |A| += 1, acc[1] += K,
 * acc[2] += min(K, L), acc[3] += [K <= L]; K is the committed skip length and
 * L what strict verification accepts from the same block (a shadow verifier
 * call).  StrictToken = acc[2] / acc[1], FullPrefix = acc[3] / acc[0].
 * Errors: SDD_EINVAL for NULL pointers or B < 0. */
int sdd_audit_accumulate(const int32_t* K, const int32_t* L, int B, int64_t* acc, sdd_stream_t stream);

/* ---- survival predictor ------------------------------------------------- */

/* Weights of the learned survival predictor (Appendix "Predictor Details"):
 * inputs x = [h, s], h the drafter's LM-head input (d_hid values, bf16), s
 * the n_sc scalar features (fp32), normalized as (x - mu) / sigma; MLP
 * d_in -> H -> H -> H -> 1 (d_in = d_hid + n_sc; the paper: 3584 + 19 = 3603
 * and H = 256) with GELU (erf form) after each hidden layer.  Device fp32
 * tensors in PyTorch Linear layout [out][in]: W1 [H][d_in], W2 and W3 [H][H],
 * w4 [H]; biases b1..b3 [H]; mu, sigma [d_in].  Caller-owned; read only. */
typedef struct {
  int d_hid, n_sc, H; /* H a multiple of 16, at most 256 */
  const float *mu, *sigma, *W1, *b1, *W2, *b2, *W3, *b3, *w4;
  float b4;
} sdd_mlp;

/* Workspace bytes for sdd_survival_mlp over n positions. */
int sdd_survival_workspace_bytes(const sdd_mlp* m, int n, size_t* bytes);

/* Survival scores of n draft positions (Sec. 4.2: the marginal a_j or the
 * conditional s_j estimate, depending on which targets the weights were
 * trained on): log_score[i] = log sigmoid(z_i) fp32 [n] (device), the log
 * position score that sdd_schedule takes (SDD_SIG_MARGINAL or
 * SDD_SIG_CONDITIONAL); logit (may be NULL) receives z_i.  Inputs (device):
 * hidden bf16 [n][d_hid], scalars fp32 [n][n_sc].  Sums run in a fixed order
 * in fp32 (MFMA), so results are bit-reproducible.  The workspace (zeroed
 * once by sdd_workspace_init, 256-byte aligned) is left reusable.
 * Errors: SDD_EINVAL for a bad shape or NULL pointer, SDD_ENOMEM for a small
 * workspace. */
int sdd_survival_mlp(const sdd_mlp* m, const uint16_t* hidden, const float* scalars, int n, float* log_score,
                     float* logit, void* ws, size_t ws_bytes, sdd_stream_t stream);

/* ---- launch timing (benchmarks) ----------------------------------------- */

/* Kernel classes */
#define SDD_PROF_EMBED 1u
#define SDD_PROF_GEMM_QKV 2u
#define SDD_PROF_ATTN 4u
#define SDD_PROF_GEMM_O 8u
#define SDD_PROF_GEMM_GATEUP 16u
#define SDD_PROF_GEMM_DOWN 32u
#define SDD_PROF_GEMM_LM 64u
#define SDD_PROF_ACCEPT 128u
#define SDD_PROF_CONF 256u
#define SDD_PROF_SCHED 512u
#define SDD_PROF_MLP 1024u

/* Starts timing: until sdd_profile_stop, every every-th launch (1: each) of
 * the classes in class_mask is bracketed by two HIP events on its own stream
 * (at most max_launches launches are recorded; events are allocated here, on
 * the host thread, not during the launches).  SDD_EINVAL for max_launches
 * outside [1, 2^20] or every < 1.  Not thread-safe: one profiling session per
 * process. */
int sdd_profile_start(unsigned class_mask, int max_launches, int every);
/* Waits for the recorded events and returns, over the launches of the
 * classes in cls: count, total, min and max duration in ms (min/max may be
 * NULL). */
int sdd_profile_read(unsigned cls, int* launches, double* total_ms, double* min_ms, double* max_ms);
/* Stops timing and releases the events. */
int sdd_profile_stop(void);

#ifdef __cplusplus
}
#endif
#endif /* SDD_H */
