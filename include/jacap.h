/*
 * jacap.h -- C ABI of libjacap.so: Jacap KV-cache eviction scoring, top-B
 * selection and compaction on AMD Instinct MI355X (gfx950).
 *
 * The method is Algorithm 1 of the Jacap paper (Sec. 3.4): for every cached
 * token i of one (sequence, layer, KV head) -- a "unit" --
 *
 *   bar-alpha_i = softmax_i( k_i . mu_Q / (tau sqrt(d)) )      centre attention
 *   kappa_i     = k_i^T Lambda_Q k_i                           query response
 *   w_i         = bar-alpha_i^2 (1 - bar-alpha_i)^2 kappa_i / d   (Eq. 8)
 *   A           = ridge I + sum_j w_j v_j v_j^T                (Eq. 9)
 *   score_i     = w_i v_i^T A^{-1} v_i                         (Eq. 10)
 *
 * then keeps the B highest-scoring tokens (Algorithm 1, TOP-B) and gathers
 * the retained cache Z_C = {(k_i, v_i)}_{i in C} (Sec. 3.1). The query
 * statistics (mu_Q, Lambda_Q) are the sample mean and 1/N covariance of the
 * observation-window queries (Sec. 3.4, last paragraph); the G = H_q / H_kv
 * query heads that share a KV head are pooled into one sample of G*w queries.
 * u_i = v_i is the output-direction proxy the paper uses when W_O is not
 * applied (Sec. 3.4).
 *
 * ridge: ridge = 1 is Eq. 9 as printed; ridge = 1/d gives exactly the scores
 * of Algorithm 1 as printed (whose weight omits the 1/d of Eq. 8); ridge = 0
 * is the plain statistical leverage score of App. B.1/B.2.
 *
 * Output-projection variant (cfg->ridge_mode = JACAP_RIDGE_MATRIX): with
 * u_i = W~ v_i in place of the proxy v_i (Sec. 3.1, Preliminary, defines u_i = W_O v_i;
 * W~ is the sum of the output-projection column slices of the G query heads
 * of the KV head, whose outputs the layer adds), Eq. 9 / Eq. 10 in output
 * space equal, by the push-through identity,
 *   score_i = w_i v_i^T (R + sum_j w_j v_j v_j^T)^{-1} v_i,  R = (W~^T W~)^{-1},
 * so the caller supplies the d x d matrices R per (layer, KV head) in
 * batch->ridge_mat and they replace ridge * I.
 *
 * GQA (the paper is single-head): by default the G query heads of a KV head
 * are pooled into one window of G*w queries. With cfg->gqa_mode =
 * JACAP_GQA_PER_HEAD each query head g is scored alone (its own w queries give
 * its mu_Q, Lambda_Q, weights and capacity matrix) and a token's score is the
 * mean over the G heads.
 *
 * Protected tokens (Algorithm 1 ranks every token; cfg->protect_last = 0 keeps
 * that): with protect_last = P > 0 the last min(P, n_b) positions of every
 * sequence are always kept and the rest of the budget is filled by score
 * from the earlier positions (budget <= P keeps the last `budget` positions).
 *
 * Conventions common to every entry point
 * ---------------------------------------
 * - All data pointers are DEVICE pointers on the current HIP device, except
 *   the two descriptor structs and `flags` of jacap_read_status, which are
 *   host pointers read (or written) during the call only.
 * - The caller owns every buffer. The library allocates no memory, keeps no
 *   pointer after returning and holds no global state (apart from the
 *   optional timing records of jacap_timing_* and the static scratch array of
 *   jacap_evict_noalloc, on each device that call uses); all work is enqueued
 *   asynchronously on `stream` (a hipStream_t; NULL = the null stream).
 *   Calls on different streams are independent if they use distinct
 *   workspaces.
 * - A batch without tokens (total_tokens = 0) is a no-op that still writes
 *   the padding of the outputs (idx, slots: -1); its K, V, query and score
 *   pointers may then be null (empty arrays), as may k_out / v_out.
 * - Host-detectable errors (null or misaligned pointers, bad shapes or
 *   strides, unsupported head_dim or dtype, too small a workspace) return an
 *   error code and enqueue nothing. K and V token strides above 2^24
 *   elements, and batches with units x ceil(max_seq_len / 1024) above 2^31 - 1
 *   (units x G with per-query-head GQA, plus a padding of 8 G), give
 *   JACAP_ERR_UNSUPPORTED. A failed launch returns JACAP_ERR_HIP.
 * - Data-dependent problems are reported through sticky device flags in the
 *   workspace (read with jacap_read_status): JACAP_FLAG_NONFINITE when a
 *   query, key or value is NaN/Inf, JACAP_FLAG_SINGULAR when A is not
 *   numerically positive definite (only possible at ridge 0). The scores of
 *   an affected unit are NaN, and NaN ranks lowest in selection.
 *
 * Layouts (element strides, head_dim contiguous, base pointers 16-byte
 * aligned, every stride a multiple of 8 elements):
 *   K, V      : element (layer l, kv head h, packed token t, channel c) at
 *               l*kv_stride_layer + h*kv_stride_head + t*kv_stride_token + c.
 *               Sequence b owns packed tokens seq_offsets[b] .. seq_offsets[b+1]-1.
 *               Default [L][H_kv][T_total][d].
 *   Q window  : element (seq b, layer l, query head g, position p, channel c)
 *               at b*q_stride_seq + l*q_stride_layer + g*q_stride_head +
 *               p*q_stride_pos + c. Default [B][L][H_q][w][d]. Query heads
 *               h*G .. h*G+G-1 serve KV head h.
 *   scores    : float32 [L][H_kv][T_total] (dense), the per-token scores.
 *   idx       : int32 [B][L][H_kv][budget_k] (dense): kept token positions
 *               (0-based within the sequence), ascending; slots past
 *               min(budget_k, n_b) hold -1.
 *   K', V'    : row j of unit (b, l, h) at b*out_stride_seq +
 *               l*out_stride_layer + h*out_stride_head + j*out_stride_row.
 *               Default [B][L][H_kv][budget_k][d]. Rows past min(budget_k, n_b)
 *               are left untouched.
 */
#ifndef JACAP_H
#define JACAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum jacap_status {
  JACAP_OK = 0,
  JACAP_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad shape/stride/parameter */
  JACAP_ERR_UNSUPPORTED = 2, /* head_dim not in {64, 128}, or an unknown dtype / mode */
  JACAP_ERR_WORKSPACE = 3,   /* workspace smaller than jacap_workspace_size() */
  JACAP_ERR_HIP = 4          /* a HIP launch or runtime call failed */
} jacap_status;

enum jacap_cov_mode {
  JACAP_COV_DIAG = 0, /* Lambda_Q = per-channel variances (App. B.2 "in practice") */
  JACAP_COV_FULL = 1  /* Lambda_Q = full d x d covariance (Algorithm 1 input) */
};

enum jacap_ridge_mode {
  JACAP_RIDGE_SCALAR = 0, /* A = cfg->ridge * I + M (Eq. 9) */
  JACAP_RIDGE_MATRIX = 1  /* A = R + M with R from batch->ridge_mat (output-projection variant) */
};

enum jacap_gqa_mode {
  JACAP_GQA_POOLED = 0,   /* one sample of G*w window queries per KV head */
  JACAP_GQA_PER_HEAD = 1  /* score per query head, average over the group */
};

enum jacap_dtype {
  JACAP_DTYPE_FP32 = 0, /* K, V, Q stored as float32 */
  JACAP_DTYPE_BF16 = 1  /* K, V, Q stored as bfloat16 */
};

enum jacap_flags {
  JACAP_FLAG_NONFINITE = 1u << 0, /* a NaN/Inf input reached a unit's statistics */
  JACAP_FLAG_SINGULAR = 1u << 1,  /* A = ridge I + M numerically singular at the score
                                     tolerance: the fp64 Cholesky factorisation of the
                                     fp64-accumulated A met a pivot at or below 1e-10
                                     (bf16 inputs) / 1e-8 (fp32 inputs) of its diagonal
                                     entry, so cond(A) > 1e10 / 1e8 and fp64 rounding
                                     alone moves the scores by more than the 1e-3 / 1e-5
                                     tolerance; in practice ridge 0 with a rank-deficient
                                     weighted Gram (fewer tokens than d) or weights of a
                                     saturated softmax spanning tens of decades */
  JACAP_FLAG_BAD_OFFSETS = 1u << 2 /* a sequence's offsets contradict max_seq_len /
                                      total_tokens; it was treated as empty */
};

/* Method and shape parameters (host struct). */
typedef struct jacap_config {
  int32_t num_layers;   /* L >= 1 */
  int32_t num_kv_heads; /* H_kv >= 1 */
  int32_t num_q_heads;  /* H_q, a positive multiple of H_kv */
  int32_t head_dim;     /* d: 64 or 128 */
  int32_t window;       /* w >= 1 observation-window queries per query head */
  int32_t budget_k;     /* B >= 0 tokens kept per unit (Algorithm 1 budget) */
  float temperature;    /* tau > 0 (the paper's best value is 10, Sec. 4.4) */
  float ridge;          /* ridge >= 0 (see the header comment) */
  int32_t cov_mode;     /* enum jacap_cov_mode */
  int32_t dtype;        /* enum jacap_dtype */
  int32_t ridge_mode;   /* enum jacap_ridge_mode (0 = scalar ridge) */
  int32_t gqa_mode;     /* enum jacap_gqa_mode (0 = pooled) */
  int32_t protect_last; /* >= 0: most recent positions of each sequence always kept */
} jacap_config;

/* Batch geometry and strides (host struct; seq_offsets is a device pointer). */
typedef struct jacap_batch {
  int32_t num_seqs;           /* B >= 1 */
  int32_t max_seq_len;        /* >= every n_b = seq_offsets[b+1]-seq_offsets[b] */
  int64_t total_tokens;       /* T_total = seq_offsets[B] */
  const int32_t* seq_offsets; /* device int32 [B+1], non-decreasing, [0] = 0 */
  int64_t k_stride_layer, k_stride_head, k_stride_token;
  int64_t v_stride_layer, v_stride_head, v_stride_token;
  int64_t q_stride_seq, q_stride_layer, q_stride_head, q_stride_pos;
  int64_t out_stride_seq, out_stride_layer, out_stride_head, out_stride_row;
  const double* ridge_mat;    /* device fp64 [L][H_kv][d][d], row-major, symmetric positive
                                 definite; read only when cfg->ridge_mode is
                                 JACAP_RIDGE_MATRIX (then non-null, 8-byte aligned) */
} jacap_batch;

/* Bytes of device workspace that jacap_score / jacap_select / jacap_evict /
 * jacap_select_evicted / jacap_evict_slots
 * need for this configuration and batch (an upper bound that depends only on
 * the host fields). Returns JACAP_ERR_INVALID_ARG / _UNSUPPORTED for an
 * invalid configuration. Workspace base pointers must be 256-byte aligned.
 * Per-query-head GQA scores every query head as a unit of its own, so its
 * per-unit and per-token storage is G times the pooled one (about 16 G bytes
 * per cached token and KV head). */
jacap_status jacap_workspace_size(const jacap_config* cfg, const jacap_batch* batch,
                                  size_t* bytes);

/* Algorithm 1 steps 1-4 (centre attention, Eq. 8 weights, Eq. 9 capacity
 * matrix, Eq. 10 leverage scores) for every unit: writes scores[L][H_kv][T]
 * (float32). q_win, k, v are in cfg->dtype. Resets the workspace status
 * flags first. Precision: with bf16 inputs A is accumulated in fp32 from
 * exact bf16 products of a two-term split of w_i v_i, and the leverage
 * products use a two-term bf16 L^{-1}; a unit whose capacity matrix the fp64
 * factorisation finds ill-conditioned (a bound on cond(A) above 2e4, or a
 * pivot below 1e-4 of its diagonal entry) is recomputed in fp64 throughout
 * (Gram, Cholesky, L^{-1} v). fp32 inputs take the fp64 path for every unit.
 * FULL covariance with bf16 keys: kappa_i = k_i^T Lambda_Q k_i comes either
 * from the bf16 MFMA tile of the keys against the window queries (exact
 * products, fp32 sums) or, for units of at least 8192 tokens with at least
 * 2d window queries, as ||X k_i||^2 with Lambda_Q = X^T X factored in fp64 and
 * X held in two bf16 terms; a numerically rank-deficient Lambda_Q (a pivot
 * at most 1e-3 of its diagonal entry) keeps the tile. */
jacap_status jacap_score(const jacap_config* cfg, const jacap_batch* batch,
                         const void* q_win, const void* k, const void* v, float* scores,
                         void* ws, size_t ws_bytes, void* stream);

/* jacap_score with the literal inputs of Algorithm 1: the query statistics
 * (mu_Q, Lambda_Q) of every unit are given instead of the observation window.
 *   mu     : device float64 [U][d], U = num_seqs * num_layers * num_kv_heads
 *            in unit order (seq, layer, kv head) -- the order of idx;
 *   lambda : device float64, cfg->cov_mode = JACAP_COV_DIAG: [U][d]
 *            per-channel variances; JACAP_COV_FULL: [U][d][d] row-major,
 *            symmetric positive semi-definite (not checked; it enters the
 *            K pass rounded to float32, as jacap_score's own estimate does).
 * Both 8-byte aligned, read during the call's kernels only. The batch's Q
 * strides are ignored; cfg->window must still be >= 1. Per-query-head GQA
 * (cfg->gqa_mode = JACAP_GQA_PER_HEAD with num_q_heads > num_kv_heads) gives
 * JACAP_ERR_UNSUPPORTED: the statistics are per unit. A non-finite mu or
 * lambda entry raises JACAP_FLAG_NONFINITE for its unit. */
jacap_status jacap_score_from_stats(const jacap_config* cfg, const jacap_batch* batch,
                                    const double* mu, const double* lambda, const void* k,
                                    const void* v, float* scores, void* ws, size_t ws_bytes,
                                    void* stream);

/* Algorithm 1 step 5 (TOP-B): for each unit keeps min(budget_k, n_b) tokens
 * ordered by (score descending, position ascending), NaN lowest and -0 equal
 * to +0, and writes their positions in ascending order to idx (-1 padding).
 * With cfg->protect_last = P > 0 the last min(P, n_b) positions are kept
 * first and the ranking fills the rest from the earlier positions.
 * Bit-exact and deterministic for given scores. */
jacap_status jacap_select(const jacap_config* cfg, const jacap_batch* batch,
                          const float* scores, int32_t* idx, void* ws, size_t ws_bytes,
                          void* stream);

/* Retained cache Z_C (Sec. 3.1): K'[j] = K[idx[j]], V'[j] = V[idx[j]], exact
 * copies in cfg->dtype, for every idx[j] >= 0. */
jacap_status jacap_compact(const jacap_config* cfg, const jacap_batch* batch,
                           const int32_t* idx, const void* k, const void* v, void* k_out,
                           void* v_out, void* stream);

/* jacap_score, jacap_select and jacap_compact enqueued as one launch
 * sequence on `stream`. */
jacap_status jacap_evict(const jacap_config* cfg, const jacap_batch* batch,
                         const void* q_win, const void* k, const void* v, float* scores,
                         int32_t* idx, void* k_out, void* v_out, void* ws, size_t ws_bytes,
                         void* stream);

/* jacap_evict for callers that cannot allocate device memory -- code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc: the
 * same launch sequence and results, with the library's own workspace instead
 * of the caller's. That workspace is a static device array of 64 MiB which
 * every GPU the library runs on holds until the process ends (looked up on
 * the call's first use of a device; nothing is allocated by any call). It
 * serves problems whose jacap_workspace_size() is at most 64 MiB (one
 * Llama-3-8B layer of 8 KV heads x 8192 tokens needs about 20 MiB, 32 layers
 * of one 1024-token sequence about 50 MiB); larger ones return
 * JACAP_ERR_WORKSPACE and enqueue nothing. All calls on one GPU share the
 * array: calls that overlap on one GPU (several streams or host threads)
 * race, so they must be ordered by the caller. Per-phase timing is never
 * recorded for this call.
 *   status : optional (NULL = not written) device uint32, 4-byte aligned: the
 *            call's sticky flags (enum jacap_flags), written by its last
 *            kernel; jacap_read_status does not apply to this call.
 * Other arguments and errors as jacap_evict. */
jacap_status jacap_evict_noalloc(const jacap_config* cfg, const jacap_batch* batch,
                                 const void* q_win, const void* k, const void* v, float* scores,
                                 int32_t* idx, void* k_out, void* v_out, uint32_t* status,
                                 void* stream);

/* The complement of jacap_select, for caches refilled in place during
 * decoding (the periodic re-eviction of the decoding-stage setting, Sec. 4.3):
 * for each unit, the positions of the n_b - min(budget_k, n_b) tokens that
 * TOP-B evicts (the same kept set as jacap_select, protect_last included),
 * in ascending order, written to slots[u][0 ..) with -1 in the rest. A caller
 * overwrites those cache rows with its next tokens instead of compacting the
 * kept ones: the positions then no longer follow arrival order, and the ties
 * of the ranking resolve by slot. budget_k = 0 evicts every position.
 *   slots    : int32 [B][L][H_kv][slot_cap], 16-byte aligned, owned by the
 *              caller; slot_cap >= max(0, max_seq_len - budget_k), else
 *              JACAP_ERR_INVALID_ARG.
 *   ws       : required (jacap_workspace_size() bytes): the kept positions are
 *              staged in it. */
jacap_status jacap_select_evicted(const jacap_config* cfg, const jacap_batch* batch,
                                  const float* scores, int32_t* slots, int32_t slot_cap, void* ws,
                                  size_t ws_bytes, void* stream);

/* jacap_score and jacap_select_evicted enqueued as one launch sequence on
 * `stream`: one decoding-stage eviction round without the copy of the kept
 * rows. */
jacap_status jacap_evict_slots(const jacap_config* cfg, const jacap_batch* batch,
                               const void* q_win, const void* k, const void* v, float* scores,
                               int32_t* slots, int32_t slot_cap, void* ws, size_t ws_bytes,
                               void* stream);

/* ------------------------------------------------------------------------
 * Exact greedy log-det selection (App. B.1): the sequential selection that
 * the one-shot leverage score of Eq. 10 approximates, for comparing the
 * quality of TOP-B. With the same Eq. 8 weights w_i and u_i = v_i, for each
 * unit, B = min(budget_k, n_b) times: add the token with the largest gain
 * w_i u_i^T A_C^{-1} u_i, A_C = ridge I + sum_{j in C} w_j u_j u_j^T (its
 * log-det increase is log(1 + gain)), ties to the lower position. C starts
 * empty; with cfg->protect_last = P > 0 it starts with the last min(P, B)
 * positions (taken first, in position order) and the search covers the rest.
 *
 * Outputs (device pointers):
 *   idx    : int32 [B][L][H_kv][budget_k], the chosen positions ascending,
 *            -1 padding (the jacap_select layout; jacap_compact accepts it).
 *   order  : optional (NULL = not written) int32 [B][L][H_kv][budget_k], the
 *            positions in the order they were added, -1 padding.
 *   logdet : optional (NULL = not written) double [B][L][H_kv], the objective
 *            log det(ridge I + sum_{i in C} w_i u_i u_i^T) of the chosen set,
 *            accumulated as d log(ridge) + sum_t log(1 + gain_t).
 *
 * Requirements beyond jacap_score's: cfg->ridge_mode = JACAP_RIDGE_SCALAR
 * with ridge > 0 (JACAP_ERR_INVALID_ARG for ridge 0: A_0 would be singular),
 * pooled GQA (cfg->gqa_mode = JACAP_GQA_PER_HEAD with H_q > H_kv and the
 * matrix ridge give JACAP_ERR_UNSUPPORTED), max_seq_len <= 524288
 * (JACAP_ERR_UNSUPPORTED), and a workspace of jacap_greedy_workspace_size()
 * bytes (256-byte aligned). Runs the weight steps of jacap_score (status
 * flags reset first), then one workgroup per unit; the work is sequential in
 * the picks, so it takes far longer than jacap_evict. Deterministic. */
jacap_status jacap_greedy_workspace_size(const jacap_config* cfg, const jacap_batch* batch,
                                         size_t* bytes);

jacap_status jacap_greedy(const jacap_config* cfg, const jacap_batch* batch, const void* q_win,
                          const void* k, const void* v, int32_t* idx, int32_t* order,
                          double* logdet, void* ws, size_t ws_bytes, void* stream);

/* Synchronises `stream` and returns the sticky device flags (enum
 * jacap_flags, OR-ed) written by the last jacap_score / jacap_evict that used
 * this workspace. */
jacap_status jacap_read_status(const void* ws, void* stream, uint32_t* flags);

/* Static, human-readable name of a status code. */
const char* jacap_status_string(jacap_status s);

/* ------------------------------------------------------------------------
 * Per-phase GPU timing, for measurement tools (off by default; nothing here
 * is needed to use the entry points above).
 *
 * While timing is on, every jacap_score / jacap_select / jacap_compact /
 * jacap_evict / jacap_greedy call records a HIP event before and after each phase whose bit
 * (1u << phase) is set in the mask, on the stream the phase's kernels are
 * launched on; the elapsed time between the two events is that phase's GPU
 * duration. Events are created on the device that is current when the call
 * is made. Timing state is process-wide and guarded by a lock; calls that
 * overlap on several host threads are all recorded.
 * ------------------------------------------------------------------------ */
enum jacap_phase {
  JACAP_PHASE_INIT = 0,        /* status/flag reset */
  JACAP_PHASE_QSTATS = 1,      /* window statistics mu, Lambda (Sec. 3.3, local query model) */
  JACAP_PHASE_KPASS = 2,       /* centre logits and query response per token */
  JACAP_PHASE_WEIGHTS = 3,     /* softmax normaliser and Eq. 8 weights */
  JACAP_PHASE_GRAM = 4,        /* weighted Gram partials (Eq. 9) */
  JACAP_PHASE_GRAM_REDUCE = 5, /* fixed-order sum of the Gram partials (units of many chunks) */
  JACAP_PHASE_FACTOR = 6,      /* Cholesky factor and L^{-1} */
  JACAP_PHASE_REFINE = 7,      /* fp64 Gram, factor and leverage of ill-conditioned units */
  JACAP_PHASE_LEVERAGE = 8,    /* leverage scores (Eq. 10) */
  JACAP_PHASE_SELECT = 9,      /* TOP-B selection */
  JACAP_PHASE_COMPACT = 10,    /* K/V compaction */
  JACAP_PHASE_GREEDY_INIT = 11, /* greedy selection: initial c_i and block maxima */
  JACAP_PHASE_GREEDY = 12,     /* greedy selection: the sequential picks */
  JACAP_NUM_PHASES = 13
};

/* Clears the accumulated times and starts recording the phases in
 * phase_mask (0 stops recording). Returns JACAP_ERR_INVALID_ARG for bits at
 * or above JACAP_NUM_PHASES. */
jacap_status jacap_timing_start(uint32_t phase_mask);

/* Stops recording, waits for every recorded event, and writes per phase the
 * summed GPU milliseconds (ms[JACAP_NUM_PHASES]) and the number of recorded
 * calls (calls[JACAP_NUM_PHASES]); either pointer may be NULL. The records
 * are cleared. Returns JACAP_ERR_HIP if an event query failed. */
jacap_status jacap_timing_stop(double* ms, int32_t* calls);

/* Static name of a phase ("gram", "leverage", "greedy", ...), or "unknown". */
const char* jacap_phase_name(int32_t phase);

/* Streaming-read probe, for measurement tools: the HBM read bandwidth the
 * streaming kernels can be compared with. Reads the `bytes` bytes at device
 * pointer `src` once (16-byte loads, whole 128-byte lines per wave
 * instruction, the non-temporal hint, 1 MiB per workgroup) on `stream`, and
 * writes nothing except, in the practically impossible case that the XOR of
 * all words equals 0x9E3779B9, that value to *sink (device, 4 bytes). src
 * and bytes must be multiples of 16 (else JACAP_ERR_INVALID_ARG). */
jacap_status jacap_stream_read(const void* src, size_t bytes, uint32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* JACAP_H */
