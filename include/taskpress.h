/*
 * taskpress.h — C ABI of the task-guided prefill-time KV-cache eviction path
 * (TaskPress, arXiv 2608.03276) for AMD Instinct MI355X (gfx950).
 *
 * The path, per (sequence, layer, KV head) "segment":
 *   1. tp_guide_scores        key score s_key of Eq. 1 (Sec. 3.2): softmax attention
 *                             of the task-guide queries on the context keys, summed
 *                             over guide tokens, averaged over the GQA group, pooled.
 *   2. tp_quantize_v_scales   value score gamma of Eq. 2 (Sec. 3.3): the per-token
 *                             quantisation scale, fused with quantising V.
 *   3. tp_combine_select_topk combined score of Eq. 3 (Sec. 3.4) and the top-k kept
 *                             index set I per KV head (uniform budget, Sec. 4 setup).
 *   4. tp_compact_kv          gather of the kept K rows, quantised V rows and scales
 *                             (the evicted tokens and the guide's KV are dropped).
 *
 * Conventions (every entry point):
 *  - Returns tp_status.  All arguments are validated on the host before any GPU
 *    work is enqueued; on error nothing is enqueued and tp_last_error() describes
 *    the problem (thread-local, valid until the next call on the same thread).
 *  - Tensor pointers are DEVICE pointers; shape / offset arrays are HOST pointers.
 *    `stream` is a hipStream_t (NULL = the default stream).
 *  - Ownership: the caller allocates every input, output and workspace buffer.
 *    The library allocates no memory and keeps no pointer after returning; buffers
 *    must stay valid until the enqueued work has completed.  (tp_evict keeps one
 *    stream and four events of its own per device: see tp_evict.)
 *  - Execution is asynchronous and stream-ordered; nothing synchronises inside a
 *    call.  Calls are re-entrant.  Results are bit-identical from run to run (no
 *    floating-point atomics; fixed reduction orders).
 *  - Layouts are row-major and contiguous, head-major, so each segment is one
 *    contiguous block; sequences of a batch sit back to back along the token axis:
 *      q_guide   bf16 [L][Hq][G_tot][d]
 *      k, v      bf16 [L][Hkv][N_tot][d]
 *      per-token fp32 [L][Hkv][N_tot]            (s_key, scales, combined score)
 *      v_q       bytes [L][Hkv][N_tot][row_bytes] (row_bytes = d, or d/2 for int b<=4)
 *      kept      int32 [L][Hkv][K_tot]  and  [L][Hkv][K_tot][d] / [..][row_bytes]
 *    Query head r belongs to KV head r / (Hq/Hkv) (grouped-query attention).
 *  - Inputs are finite (no NaN/Inf).  bf16 values are raw bit patterns (uint16).
 */
#ifndef TASKPRESS_H
#define TASKPRESS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tp_status;
enum {
  TP_OK = 0,
  TP_ERR_NULL = 1,        /* a required pointer is NULL */
  TP_ERR_SHAPE = 2,       /* inconsistent dims, offsets or sizes */
  TP_ERR_PARAM = 3,       /* a scalar parameter is out of its domain */
  TP_ERR_UNSUPPORTED = 4, /* valid but not implemented here (e.g. head_dim, batch size) */
  TP_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than tp_workspace_size() */
  TP_ERR_HIP = 6          /* a HIP runtime call or kernel launch failed */
};

/* Quantisation format of V (Eq. 2 and Sec. 4 setup). */
enum {
  TP_QFMT_INT = 0,     /* symmetric b-bit integers, qmax = 2^(b-1)-1, b in [2, 8];
                          b <= 4 packs two values per byte (even element in the low nibble,
                          4-bit two's complement), otherwise one int8 per value */
  TP_QFMT_FP8_E4M3 = 1 /* OCP E4M3 codes, qmax = 448; `bits` is ignored */
};

/* Combination rule of the key and value scores. */
enum {
  TP_COMBINE_MUL = 0,      /* s = s_key * gamma (Eq. 3, the method's rule) */
  TP_COMBINE_NORM_ADD = 1, /* s = s_key/||s_key||_2 + gamma/||gamma||_2 (aggregation table, Sec. 4.4) */
  TP_COMBINE_HARMONIC = 2, /* s = 2 s_key gamma / (s_key + gamma), 0 if both are 0 (same table) */
  TP_COMBINE_KEY_ONLY = 3  /* s = s_key (key-score-only ablation, Sec. 4.3) */
};

/* Entry points that take a workspace (argument of tp_workspace_size). */
enum { TP_FN_GUIDE_SCORES = 0, TP_FN_COMBINE_SELECT_TOPK = 1, TP_FN_EVICT = 2, TP_FN_GUIDE_ATTENTION = 3 };

typedef struct tp_dims {
  int32_t num_layers;   /* L   >= 1 */
  int32_t num_q_heads;  /* Hq  >= 1, a multiple of Hkv */
  int32_t num_kv_heads; /* Hkv >= 1 */
  int32_t head_dim;     /* d: 64 or 128 */
} tp_dims;

#define TP_MAX_BATCH 64

typedef struct tp_batch {
  int32_t batch;                /* B in [1, TP_MAX_BATCH] */
  const int64_t* ctx_offsets;   /* host [B+1]: sequence b owns context tokens
                                   [ctx_offsets[b], ctx_offsets[b+1]); ctx_offsets[0] = 0,
                                   N_b = difference >= 1, N_tot = ctx_offsets[B] */
  const int64_t* guide_offsets; /* host [B+1]: guide tokens of sequence b, G_b >= 1 (for
                                   tp_guide_scores; may be NULL for the other calls) */
} tp_batch;
/* Size limits (TP_ERR_UNSUPPORTED beyond them; far above what one GPU holds): N_tot <= 2^30;
 * with guides G_tot <= 2^31 - 1, L * Hq * G_tot <= 2^32 and L * Hq * G_b <= 2^26 for every b. */

/* Version string of the library. */
const char* tp_version(void);

/* Human-readable name of a status code. */
const char* tp_status_string(tp_status s);

/* Detail message of the last error on this thread ("" after a successful call). */
const char* tp_last_error(void);

/*
 * Size of the kept set of one KV head (problem statement, Sec. 3.1; uniform
 * per-head budget, Sec. 4 setup).  Exactly one of keep_ratio / keep_budget is
 * used: keep_ratio in (0, 1] (= 1 - eviction ratio) gives
 * k = max(1, floor(n * keep_ratio)) computed in binary64; keep_ratio <= 0 selects
 * the budget, k = min(keep_budget, n).  Returns -1 if n < 1 or neither / both
 * are valid.  Host only.
 */
int64_t tp_keep_count(int64_t n, double keep_ratio, int64_t keep_budget);

/*
 * Bytes of device workspace `fn` needs for these dims / batch (host only).
 * TP_FN_GUIDE_SCORES needs guide_offsets; TP_FN_COMBINE_SELECT_TOPK does not.
 */
tp_status tp_workspace_size(int32_t fn, const tp_dims* dims, const tp_batch* batch, size_t* bytes);

/*
 * Step 1 — key score of Eq. 1 (Sec. 3.2), for every (sequence b, layer l, KV head h):
 *   A^(r)[j][i] = exp(x_ji) / Z_j with x_ji = softmax_scale * <q_guide[l][r][g0+j], k[l][h][n0+i]>
 *                 (softmax-normalised as stated in Sec. 6), where the normaliser Z_j is
 *                 - k_guide == NULL: sum_i exp(x_ji) over the N_b context tokens of sequence b;
 *                 - k_guide != NULL: that sum plus sum_{t<=j} exp(softmax_scale *
 *                   <q_guide[l][r][g0+j], k_guide[l][h][g0+t]>), i.e. A is the context slice
 *                   of the causal attention over the context with the guide appended after
 *                   it (the slice of the full attention map described in Sec. 3.2),
 *   raw[i]      = (1/R) * sum over the R query heads r of KV head h, sum_{j<G_b} A^(r)[j][i],
 *   s_key[l][h][n0+i] = (1/pool_k) * sum_{|t| <= pool_k/2} raw[i+t], raw = 0 outside [0, N_b).
 * q_guide bf16 [L][Hq][G_tot][d], k bf16 [L][Hkv][N_tot][d], k_guide bf16 [L][Hkv][G_tot][d]
 * (the guide tokens' keys) or NULL, s_key fp32 [L][Hkv][N_tot] (out).
 * softmax_scale > 0 (callers pass 1/sqrt(d)); pool_k odd, >= 1.
 * workspace: device, >= tp_workspace_size(TP_FN_GUIDE_SCORES, ...) bytes, 256-byte aligned.
 * Errors: TP_ERR_NULL, TP_ERR_SHAPE, TP_ERR_PARAM, TP_ERR_UNSUPPORTED, TP_ERR_WORKSPACE,
 * TP_ERR_HIP.
 */
tp_status tp_guide_scores(const tp_dims* dims, const tp_batch* batch, const void* q_guide,
                          const void* k, const void* k_guide, float softmax_scale, int32_t pool_k,
                          float* s_key, void* workspace, size_t ws_bytes, void* stream);

/*
 * Step 1 with the row normalisers supplied by the caller.  Sec. 3.2 takes A from the
 * attention map of the prefill over the context with the guide appended; the prefill
 * attention kernel already holds, for every guide row, the log-sum-exp of its scaled logits
 * over the keys it attended to.  Given those, the score needs one pass over K instead of two:
 *   A^(r)[j][i] = exp(softmax_scale * <q_guide[l][r][g0+j], k[l][h][n0+i]> - guide_lse[l][r][g0+j])
 * and raw, s_key exactly as for tp_guide_scores.  With guide_lse equal to
 * ln Z_j of tp_guide_scores (either normaliser) the results agree with it to rounding.
 * guide_lse: device fp32 [L][Hq][G_tot], natural log, finite, 4-byte aligned; it must
 * include softmax_scale in the logits (the convention of flash-attention's exported
 * log-sum-exp).  Other arguments and errors as for tp_guide_scores (same workspace size).
 */
tp_status tp_guide_scores_lse(const tp_dims* dims, const tp_batch* batch, const void* q_guide,
                              const void* k, const float* guide_lse, float softmax_scale,
                              int32_t pool_k, float* s_key, void* workspace, size_t ws_bytes,
                              void* stream);

/*
 * The prefill's attention for the appended guide rows (Sec. 3.2: the guide follows the
 * context and attends causally), whose normalisers feed step 1 (tp_guide_scores_lse,
 * tp_evict's guide_lse), so the eviction adds one sweep over K to this one:
 *   x_jt = softmax_scale * <q_guide[l][r][g0+j], key_t> over the keys row j sees: the N_b
 *          context keys k[l][h][n0+i], and, when k_guide is given, the guide keys
 *          k_guide[l][h][g0+t] for t <= j;
 *   o_guide[l][r][g0+j][:] = sum_t exp(x_jt) value_t / sum_t exp(x_jt)   (values v, v_guide),
 *   guide_lse[l][r][g0+j]  = ln sum_t exp(x_jt),
 * for query head r of KV head h = r / (Hq/Hkv) and every guide token j of sequence b.
 * q_guide bf16 [L][Hq][G_tot][d]; k, v bf16 [L][Hkv][N_tot][d]; k_guide, v_guide bf16
 * [L][Hkv][G_tot][d], both NULL (the context only) or both given; o_guide fp32
 * [L][Hq][G_tot][d] (out); guide_lse fp32 [L][Hq][G_tot] (out).  softmax_scale > 0.
 * workspace: device, >= tp_workspace_size(TP_FN_GUIDE_ATTENTION, ...) bytes, 256-byte
 * aligned (per chunk of context tokens and guide row, a partial maximum, sum and output).
 * The probabilities are rounded to bf16 for the value product (as flash attention does);
 * the normalisers are fp32 sums of the unrounded ones.
 * Errors: TP_ERR_NULL, TP_ERR_SHAPE, TP_ERR_PARAM, TP_ERR_UNSUPPORTED, TP_ERR_WORKSPACE,
 * TP_ERR_HIP.
 */
tp_status tp_guide_attention(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                             const void* v, const void* k_guide, const void* v_guide, float softmax_scale,
                             float* o_guide, float* guide_lse, void* workspace, size_t ws_bytes, void* stream);

/*
 * tp_guide_attention together with step 2 (Eq. 2, Sec. 3.3) from the one sweep over V: the
 * V tiles the attention stages are also quantised, so the prefill's quantised cache and the
 * value scores come from the attention's own read of V (the paper takes the scales as
 * already computed by the cache's quantisation).  Outputs o_guide and guide_lse exactly as
 * tp_guide_attention; scales and v_q exactly (bit for bit) as tp_quantize_v_scales with the
 * same qfmt and bits, for every context token of the batch.  v_q must be non-NULL
 * (TP_ERR_NULL otherwise).  tp_evict then takes v = NULL with these scales and codes.
 * Same workspace as tp_guide_attention.  Errors as for tp_guide_attention and
 * tp_quantize_v_scales.
 */
tp_status tp_guide_attention_quantize(const tp_dims* dims, const tp_batch* batch, const void* q_guide,
                                      const void* k, const void* v, const void* k_guide, const void* v_guide,
                                      float softmax_scale, int32_t qfmt, int32_t bits, float* o_guide,
                                      float* guide_lse, float* scales, void* v_q, void* workspace, size_t ws_bytes,
                                      void* stream);

/*
 * Step 2 — value score of Eq. 2 (Sec. 3.3), fused with per-token quantisation of V
 * (KIVI-style per-token scheme cited in Sec. 3.3; int4 cache of Sec. 4 setup):
 *   gamma[l][h][t] = fl32( max_c |v[l][h][t][c]| / qmax )
 *   q[l][h][t][c]  = clamp(RNE(fl32(v / gamma)), -qmax, qmax)   (TP_QFMT_INT), or the OCP E4M3
 *                    code of fl32(v / gamma), round-to-nearest-even, saturating at 448
 *                    (TP_QFMT_FP8_E4M3); rows with gamma = 0 give q = 0.
 * Independent of the batch split (every token of N_tot is processed); `batch` only
 * provides N_tot.  v bf16 [L][Hkv][N_tot][d]; scales fp32 [L][Hkv][N_tot] (out);
 * v_q bytes [L][Hkv][N_tot][row_bytes] (out) or NULL to compute the scales only.
 * Errors: TP_ERR_NULL, TP_ERR_SHAPE, TP_ERR_PARAM (qfmt, bits), TP_ERR_UNSUPPORTED, TP_ERR_HIP.
 */
tp_status tp_quantize_v_scales(const tp_dims* dims, const tp_batch* batch, const void* v,
                               int32_t qfmt, int32_t bits, float* scales, void* v_q,
                               void* stream);

/*
 * Step 3 — combined score (Eq. 3, or a variant from the aggregation table) and the
 * kept index set I of every (sequence, layer, KV head) (Sec. 3.4; uniform budget,
 * selected per head independently, Sec. 4 setup):
 *   S[i] = combine(s_key[i], scales[i]) stored as fp32 (TP_COMBINE_*),
 *   k_b  = tp_keep_count(N_b, keep_ratio, keep_budget),
 *   I    = the k_b indices with the largest S, ties broken towards the lower index,
 *          written in ascending order as sequence-local token indices in [0, N_b).
 * s_key, scales fp32 [L][Hkv][N_tot], all finite and >= 0.
 * kept_offsets: host [B+1], must equal the prefix sums of k_b (TP_ERR_SHAPE otherwise);
 * kept_idx int32 [L][Hkv][K_tot] (out), K_tot = kept_offsets[B];
 * s_out fp32 [L][Hkv][N_tot] (out, optional): the combined scores S.
 * workspace: device, >= tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, ...) bytes, 256-byte
 * aligned, always required: the combined scores when s_out is NULL, and the per-part counts
 * of the selection (each segment's tokens are ranked in parts of 8192 by several workgroups).
 * Exactly one of keep_ratio in (0, 1] / keep_budget >= 1 must be given (the other
 * <= 0), otherwise TP_ERR_PARAM.
 */
tp_status tp_combine_select_topk(const tp_dims* dims, const tp_batch* batch, const float* s_key,
                                 const float* scales, int32_t rule, double keep_ratio,
                                 int64_t keep_budget, const int64_t* kept_offsets,
                                 int32_t* kept_idx, float* s_out, void* workspace,
                                 size_t ws_bytes, void* stream);

/*
 * Step 3 for callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): tp_combine_select_topk with s_out = NULL
 * and no workspace argument.  The combined scores and the selection's counts are staged in a
 * buffer of TP_STATIC_SCRATCH_BYTES that the library holds as a static device array, one per
 * GPU its code is loaded on, kept until the process ends; the call allocates nothing.
 * Arguments, results and errors as for tp_combine_select_topk, plus TP_ERR_WORKSPACE when
 * the selection's workspace (tp_workspace_size(TP_FN_COMBINE_SELECT_TOPK, ...), about
 * 5 bytes per token and segment plus 32 KB per segment and sequence) exceeds TP_STATIC_SCRATCH_BYTES (validated before
 * anything is enqueued), and TP_ERR_HIP if the buffer's address on the stream's device
 * cannot be resolved (done once per device, on the first call there).
 * Every call on one GPU uses that GPU's one buffer: calls whose work overlaps on a GPU (other
 * streams, other threads) race and must be ordered by the caller.  The buffer keeps the last
 * call's contents; each call writes every value it reads.
 */
#define TP_STATIC_SCRATCH_BYTES (64u << 20)
tp_status tp_combine_select_topk_static(const tp_dims* dims, const tp_batch* batch, const float* s_key,
                                        const float* scales, int32_t rule, double keep_ratio,
                                        int64_t keep_budget, const int64_t* kept_offsets,
                                        int32_t* kept_idx, void* stream);

/*
 * Step 4 — compaction (Sec. 3.1: only I is kept; Sec. 4 setup: eviction after
 * prefill, the guide's KV discarded — it is not part of k / v here):
 *   k_out[l][h][ko_b + t][:]      = k[l][h][n0_b + kept_idx[l][h][ko_b + t]][:]
 *   v_q_out[l][h][ko_b + t][:]    = v_q[l][h][n0_b + idx][:]       (row_bytes bytes)
 *   scales_out[l][h][ko_b + t]    = scales[l][h][n0_b + idx]
 * for t < kept_offsets[b+1] - kept_offsets[b] (= ko_{b+1} - ko_b <= N_b).  qfmt/bits give
 * row_bytes.  An index outside [0, N_b) yields a zero row and zero scale (no fault).
 * v_q/v_q_out and scales/scales_out may be NULL pairwise to skip that output.
 */
tp_status tp_compact_kv(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                        const int32_t* kept_idx, const void* k, const void* v_q,
                        const float* scales, int32_t qfmt, int32_t bits, void* k_out,
                        void* v_q_out, float* scales_out, void* stream);

/*
 * Step 4 fused with step 2 for the kept rows only: the kept V rows are read in bf16 and
 * quantised (Eq. 2, Sec. 3.3; per-token scale and codes exactly as tp_quantize_v_scales)
 * while they are gathered, so the codes of evicted rows are never written:
 *   k_out[l][h][ko_b + t][:]   = k[l][h][n0_b + idx][:]
 *   v_q_out[l][h][ko_b + t][:] = codes of v[l][h][n0_b + idx][:]
 *   scales_out[l][h][ko_b + t] = gamma of that row
 * with idx = kept_idx[l][h][ko_b + t]; results bit-identical to tp_quantize_v_scales followed
 * by tp_compact_kv.  v bf16 [L][Hkv][N_tot][d]; every output required.  An index outside
 * [0, N_b) yields a zero row, zero codes and a zero scale.
 */
tp_status tp_compact_quantize_kv(const tp_dims* dims, const tp_batch* batch, const int64_t* kept_offsets,
                                 const int32_t* kept_idx, const void* k, const void* v, int32_t qfmt,
                                 int32_t bits, void* k_out, void* v_q_out, float* scales_out,
                                 void* stream);

/*
 * Optional timing hooks of tp_evict, for callers that profile the path.  With num_events
 * = TP_EVICT_EVENTS, tp_evict records events[i] (hipEvent_t created by the caller) on the
 * stream, in launch order: [0] before the work, [1] after score pass 1, [2] after the row
 * normalisers, [3] after the V quantisation, [4] after score pass 2, [5] after pooling,
 * [6] after the selection, [7] after the compaction; one kernel runs between consecutive
 * events (with guide_lse, none between [0] and [1], and [1]..[2] converts the supplied
 * normalisers).
 * num_events = 0 (or a NULL profile) records none.
 */
#define TP_EVICT_EVENTS 8
typedef struct tp_profile {
  int32_t num_events;
  void* events[TP_EVICT_EVENTS];
} tp_profile;

/*
 * The whole path in one call: steps 1-4 above with the same arguments and results as
 * tp_guide_scores + tp_quantize_v_scales + tp_combine_select_topk + tp_compact_kv
 * (bit-identical outputs; Sec. 3.2-3.4 as for the separate calls), validated as a whole
 * before anything is enqueued, with optional per-kernel timing events.
 * guide_lse: NULL, or the guide rows' log-normalisers as for tp_guide_scores_lse (then score
 * pass 1 is skipped); k_guide and guide_lse may not both be given (TP_ERR_PARAM).
 * Outputs: s_key, scales, v_q (optional), s_out (optional), kept_idx, k_out, v_q_out,
 * scales_out.  With v_q == NULL step 2 computes the scales only and the compaction
 * quantises the kept V rows itself (tp_compact_quantize_kv): the compact cache is the same
 * and the codes of the evicted rows are never written.
 * v == NULL: step 2 has been done (tp_guide_attention_quantize, or tp_quantize_v_scales):
 * scales and v_q are inputs holding its results for qfmt and bits (both non-NULL, else
 * TP_ERR_NULL), and everything runs on `stream` (no second stream, no library state).
 * workspace: >= tp_workspace_size(TP_FN_EVICT, ...) bytes, 256-byte aligned (the score
 * pass's workspace followed by the selection's).
 * Step 2 of most V rows runs on a second stream of the library's: 2/5 concurrently with each
 * score pass (half with each when v_q is NULL), or, with guide_lse given, the first half
 * (3/5 when v_q is NULL) concurrently with the rest of the step; the arithmetic is the same,
 * so the results are as for the separate calls.  That stream and four events are created, with default priority, by the first
 * tp_evict call on a device and kept until the process ends (TP_ERR_HIP if that fails); the
 * work is forked from and joined back to `stream`, so the call stays stream-ordered and may
 * be captured into a graph (once the first call on the device, which creates the stream,
 * has been made outside capture).  Calls on one device enqueue one at a time (a lock held while
 * enqueueing, not while the work runs).
 * Every argument is validated before anything is enqueued.  Errors as for the four calls.
 */
tp_status tp_evict(const tp_dims* dims, const tp_batch* batch, const void* q_guide, const void* k,
                   const void* k_guide, const float* guide_lse, const void* v, float softmax_scale,
                   int32_t pool_k,
                   int32_t qfmt, int32_t bits, int32_t rule, double keep_ratio, int64_t keep_budget,
                   const int64_t* kept_offsets,
                   float* s_key, float* scales, void* v_q, float* s_out, int32_t* kept_idx,
                   void* k_out, void* v_q_out, float* scales_out, void* workspace, size_t ws_bytes,
                   const tp_profile* profile, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* TASKPRESS_H */
