/*
 * sx.h - C ABI of the SparseX per-layer Sparse-KV Recomputation step on AMD Instinct MI355X
 * (gfx950).
 *
 * The step (paper: "SparseX: Efficient Segment-Level KV Cache Sharing for Interleaved LLM
 * Serving", Section 3 and Algorithm 1) has these parts, each one entry point below:
 *
 *   sx_rope_realign   RoPE re-alignment of reused cached segments into the request's paged
 *                     cache: K rotated by R_{p'-p}, V copied (Section 3.1; Algorithm 1 step 6).
 *   sx_sparseq_score  Sparse-Q attention of the non-reused query rows over all visible keys,
 *                     summed per key over rows and heads (Eq. sparseq-attn, Eq. sparseq-score,
 *                     cross-head aggregation of Section 3.2; Algorithm 1 steps 11-13).
 *   sx_topk_select    top-k key selection, overflow and tail fallback, giving the recompute set
 *                     R (Eq. topk, Section 3.3; Algorithm 1 steps 14-17).
 *   sx_kv_scatter     write of freshly computed K/V rows into the paged cache
 *                     (Algorithm 1 steps 19-20).
 *   sx_sparse_attn    causal attention of the rows of R over the mixed paged cache
 *                     (Algorithm 1 step 21).
 *   sx_full_attn      plain causal prefill attention of the layers before the full+sparse
 *                     hybrid threshold (Section 3.4; Algorithm 1 steps 7-10).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Status: every function returns SX_OK (0) or a negative sx_status; it never aborts and never
 *   throws.  sx_last_error() gives a text for the last failure of the calling thread.
 * Validation: arguments the host can see (descriptors, segment and block tables, sizes) are checked
 *   on the host.  Index arrays in device memory (row lists, n_rows, cu_seqlens) are trusted by the
 *   release library, libsx.so; the checked library, libsx_checked.so (same ABI, built alongside),
 *   validates them on the device before any compute kernel reads them, synchronising the call's
 *   stream, and returns SX_EDEVICE for an invalid one.
 * Memory: every tensor argument is device memory allocated and owned by the caller; the library
 *   never frees or keeps it.  The plan owns only its own metadata and scratch (device memory it
 *   allocates in sx_plan_create and frees in sx_plan_destroy).
 * Streams: `stream` is a hipStream_t (NULL = the default stream).  All compute calls are
 *   asynchronous and stream-ordered; none synchronises the host.  Calls sharing one plan must
 *   be issued on one stream (or ordered by the caller), because they share the plan's scratch.
 * Element types: desc.dtype selects float32 or bfloat16 for Q, K, V, caches and attention
 *   outputs.  Scores are float32.  Index arrays are int32.
 * Layouts (row-major, innermost last):
 *   q                     [sum T][Hq][d]      fresh queries of every token, requests concatenated
 *   k_new, v_new          [sum T][Hkv][d]     fresh keys / values of every token
 *   k_cache, v_cache      [n_dst_blocks][Hkv][b][d]   destination (request) pool; token t of
 *                         request r lives in block block_table_r[t / b], slot t % b
 *   src_k, src_v          [n_src_blocks][Hkv][b][d]   source pool of cached segments; token j of
 *                         a cached segment lives in block src_block_ids[src_block_start + j / b],
 *                         slot j % b (segments start at slot 0 of their first block)
 *   scores                [sum T] float32
 *   row lists             `rows` [sum T] int32 and `n_rows` [n_req] int32: the rows of request
 *                         r are rows[off_r .. off_r + n_rows[r]) in ascending order, where off_r
 *                         is the request's first token in the concatenation; values are
 *                         request-local token indices.
 *   out (sparse)          [sum T][Hq][d]: out[off_r + n] belongs to rows[off_r + n]
 *   out (full)            [sum T][Hq][d]
 * Query head h reads KV head h / (Hq / Hkv).  Causality is by token index; RoPE positions
 * (old_pos/new_pos) are used only by the re-alignment.
 */
#ifndef SX_H
#define SX_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t sx_status;

enum {
  SX_OK = 0,
  SX_EINVAL = -1,        /* bad argument: NULL pointer, bad segment table, bad ratio, ... */
  SX_ESHAPE = -2,        /* inconsistent sizes (heads, block ids out of range, ...) */
  SX_EUNSUPPORTED = -3,  /* valid but not implemented (head_dim, block_size, dtype) */
  SX_EHIP = -4,          /* a HIP runtime call failed */
  SX_EDEVICE = -5,       /* checked library only: an index array in device memory is invalid (a row
                            list out of range or not ascending, n_rows > T, bad cu_seqlens); nothing
                            was computed */
  SX_ENOMEM = -6,        /* device allocation failed */
  SX_EFULL = -7          /* the block pool cannot hold the request (sx_cache_schedule) */
};

enum { SX_F32 = 0, SX_BF16 = 1 };
/* RoPE pair layout: NEOX rotates (i, i + d/2), GPTJ rotates (2i, 2i + 1), frequency
 * theta_i = rope_base^(-2i/d) for i in [0, d/2). */
enum { SX_ROPE_NEOX = 0, SX_ROPE_GPTJ = 1 };

typedef struct sx_layer_desc {
  int32_t n_q_heads;      /* Hq >= 1 */
  int32_t n_kv_heads;     /* Hkv >= 1, Hq % Hkv == 0, Hq / Hkv <= 64 */
  int32_t head_dim;       /* d: 64 or 128 */
  int32_t block_size;     /* b: 16 */
  int32_t dtype;          /* SX_F32 or SX_BF16 */
  int32_t rope_style;     /* SX_ROPE_NEOX or SX_ROPE_GPTJ */
  double rope_base;       /* > 0 */
  float softmax_scale;    /* 0 -> 1/sqrt(head_dim) */
  int32_t flags;          /* 0, or SX_TOPK_ALL_POSITIONS */
} sx_layer_desc;

/* sx_layer_desc.flags.  SX_TOPK_ALL_POSITIONS: the top-k of Eq. topk ranges over every position of
 * the request (the equation as printed) instead of the reused positions only; the budget becomes
 * k = min(T, floor(ratio * T + 1/2)).  I_nr, the overflow and the tail-fallback rows are unchanged
 * and still always in R, so a selected uncached position spends budget without adding a row. */
#define SX_TOPK_ALL_POSITIONS 1

/* One contiguous segment of a request (Section 3.1 segment-level cache; Algorithm 1 input:
 * original positions p_m and current positions p'_m). */
typedef struct sx_segment {
  int32_t seq_start;        /* first token index of the segment in the new sequence */
  int32_t length;           /* > 0 tokens; segments tile [0, n_tokens) in order */
  int32_t cached;           /* 1: reused (I_reuse); 0: computed now (I_nr, Sparse-Q rows) */
  int32_t old_pos;          /* RoPE position of the first token where it was cached (>= 0) */
  int32_t new_pos;          /* RoPE position of the first token in the new sequence (>= 0) */
  int32_t src_block_start;  /* cached only: index into src_block_ids of its first block */
} sx_segment;

/* One request.  All pointers are HOST memory, read only during sx_plan_create. */
typedef struct sx_request {
  int32_t n_tokens;                /* T > 0 */
  int32_t n_segments;
  const sx_segment* segments;      /* [n_segments] */
  const int32_t* block_table;      /* [ceil(T / b)] destination-pool block ids, all distinct
                                      across every request of the plan */
  const int32_t* src_block_ids;    /* [n_src_block_ids] source-pool block ids */
  int32_t n_src_block_ids;
} sx_request;

typedef struct sx_plan sx_plan;

typedef struct sx_plan_info {
  int64_t total_tokens;     /* sum T */
  int32_t n_requests;
  int32_t max_tokens;       /* max T */
  int64_t n_reused;         /* sum of top-k candidates: |I_reuse| (T with SX_TOPK_ALL_POSITIONS) */
  int64_t n_nonreused;      /* sum |I_nr| */
  int64_t n_probes;         /* sum |I_nr U S_tail| (Sparse-Q rows that score) */
  int64_t n_base;           /* sum |I_nr U S_ov U S_tail| (rows of R whatever the scores) */
  int32_t max_nonreused;    /* max over requests of |I_nr| */
  int32_t max_probes;       /* max over requests of |I_nr U S_tail| */
  int64_t device_bytes;     /* device memory held by the plan */
} sx_plan_info;

/* Builds the per-batch metadata of the step: validates the segment tables and block tables,
 * derives I_nr, I_reuse, the probe rows, the overflow rows S_ov (b positions on each side of
 * every maximal run of I_nr, Section 3.3) and the tail-fallback rows S_tail (the last
 * min(64, len) tokens of the final segment when that segment is reused, Section 3.2), and the
 * float64 cos/sin tables of every cached segment's shift (rounded to float32).
 * n_dst_blocks / n_src_blocks are the pool sizes used to range-check block ids.
 * Limits (SX_EUNSUPPORTED beyond them): at most 2^31 - 1 tokens in one plan and 2^21 tokens
 * in one request.
 * Allocates device memory (owned by the plan).  *out is set only on success. */
sx_status sx_plan_create(const sx_layer_desc* desc, const sx_request* requests, int32_t n_requests,
                         int64_t n_dst_blocks, int64_t n_src_blocks, sx_plan** out);
sx_status sx_plan_destroy(sx_plan* plan);  /* NULL is allowed; waits for the device first */
sx_status sx_plan_get_info(const sx_plan* plan, sx_plan_info* info);

/* Top-k budget of a recompute ratio r in [0, 1]: per request k_r = min(n_r, floor(r*n_r + 1/2))
 * with n_r = |I_reuse of request r| (float64 arithmetic).  *k_total = sum k_r; *max_rows =
 * max over requests of |I_nr U S_ov U S_tail| + k_r, an upper bound on every |R_r| and the
 * `max_rows` to pass to sx_kv_scatter / sx_sparse_attn for rows produced with this ratio. */
sx_status sx_plan_budget(const sx_plan* plan, double ratio, int64_t* k_total, int32_t* max_rows);

/* Device row list of I_nr owned by the plan (row-list layout above), and its bound max_rows.
 * Valid until sx_plan_destroy. */
sx_status sx_plan_nonreused_rows(const sx_plan* plan, const int32_t** rows, const int32_t** n_rows,
                                 int32_t* max_rows);

/* Section 3.1 / Algorithm 1 step 6: for every token of every cached segment (shift
 * delta = new_pos - old_pos), k_cache[dst slot] = R_delta src_k[src slot] and
 * v_cache[dst slot] = src_v[src slot].  The rotation of pair (x1, x2) with frequency theta_i is
 * x1' = x1*c - x2*s, x2' = x2*c + x1*s with c, s the float32 roundings of cos/sin(delta*theta_i)
 * (angle in float64), each product and sum rounded once in float32, then stored in the cache
 * type (bfloat16: round to nearest even).  Slots of non-cached tokens are not touched.
 * Source slots and destination slots must not overlap.  One pool may serve as both the source
 * pool and the cache (src_k == k_cache, the layout the segment cache manager produces) as long as
 * the segments' source blocks and the request's destination blocks are distinct blocks. */
sx_status sx_rope_realign(const sx_plan* plan, const void* src_k, const void* src_v, void* k_cache,
                          void* v_cache, void* stream);

/* Algorithm 1 steps 19-20: copies k_new/v_new row t of request r into the cache slot of t for
 * every listed row (bit-exact).  rows == NULL writes every token of every request (n_rows and
 * max_rows are then ignored).  Otherwise rows/n_rows use the row-list layout and max_rows should
 * be >= every n_rows[r] (sx_plan_budget gives it): only the first min(n_rows[r], max_rows) rows of
 * each request are written, so an undersized bound drops the last rows of a list.  Every other
 * entry point that takes rows/n_rows/max_rows processes the same first min(n_rows[r], max_rows)
 * rows. */
sx_status sx_kv_scatter(const sx_plan* plan, const void* k_new, const void* v_new, const int32_t* rows,
                        const int32_t* n_rows, int32_t max_rows, void* k_cache, void* v_cache,
                        void* stream);

/* Algorithm 1 steps 6 and 19-20 in one pass for a layer whose recompute set R is known (the
 * sparse layers of a hybrid stack reuse the boundary layer's R, Section 3.4): the cache slot of
 * every listed row of request r gets k_new/v_new (bit-exact, as sx_kv_scatter), the slot of every
 * other reused token gets its re-aligned cached K and V (as sx_rope_realign); other tokens are not
 * touched.  Same result as sx_rope_realign followed by sx_kv_scatter with the same rows, but each
 * slot is read and written once.  rows/n_rows/max_rows as in sx_kv_scatter (rows required);
 * src_k/src_v may be NULL only when no segment is cached.  Keeps a row-set mark per token in plan
 * scratch, so calls sharing a plan must be stream-ordered. */
sx_status sx_realign_scatter(const sx_plan* plan, const void* src_k, const void* src_v, const void* k_new,
                             const void* v_new, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             void* k_cache, void* v_cache, void* stream);

/* Device buffers of one layer for sx_realign_scatter_layers (same meaning as the arguments of
 * sx_realign_scatter). */
typedef struct {
  const void* src_k;
  const void* src_v;
  const void* k_new;
  const void* v_new;
  void* k_cache;
  void* v_cache;
} sx_layer_kv;

/* sx_realign_scatter for n_layers layers that share the plan and the row set R (the sparse layers
 * of a hybrid stack after the boundary selection, Section 3.4), batched into as few launches as
 * possible, as the paper re-aligns a whole batch's reused blocks at once (Section 3.1, Algorithm 1
 * step 6).  `layers` is a HOST array of n_layers entries, read during the call only; the buffers
 * it names are device memory.  Each entry is validated as in sx_realign_scatter; n_layers == 0 is
 * a no-op. */
sx_status sx_realign_scatter_layers(const sx_plan* plan, int32_t n_layers, const sx_layer_kv* layers,
                                    const int32_t* rows, const int32_t* n_rows, int32_t max_rows, void* stream);

/* Per-token byte mask of a row list (the recompute set R that sx_topk_select writes), for
 * sx_realign_scatter_masked: mask[off_r + t] = 1 for every listed row t of request r
 * (rows[off_r .. off_r + min(n_rows[r], max_rows))), 0 for every other token of the plan.
 * mask is caller-owned DEVICE memory of sum T bytes; rows/n_rows/max_rows as in sx_kv_scatter.
 * Listed values outside [0, T_r) are ignored.  Two kernels on `stream`, no host sync.  bfloat16
 * plans: a third kernel plans, in the plan's scratch, the order in which sx_sparse_attn takes its
 * row tiles (Multifit over their estimated costs); sx_sparse_attn uses it when called with the
 * same rows, n_rows and max_rows, as the sparse layers that share R are (Section 3.4).  The order
 * changes only which workgroup computes a row tile, never a result. */
sx_status sx_rows_mask(const sx_plan* plan, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                       uint8_t* mask, void* stream);

/* sx_realign_scatter with R given as a per-token byte mask (sx_rows_mask): the slot of every token
 * with mask[off_r + t] != 0 gets k_new/v_new (bit-exact), the slot of every other reused token its
 * re-aligned cached K and V (Section 3.1, Algorithm 1 steps 6 and 19-20); other tokens are not
 * touched.  One kernel, each slot read and written once.  The mask is built once for the sparse
 * layers that share R (Section 3.4), so no per-layer marking pass is needed, and nothing of the
 * plan is written: calls sharing a plan may run concurrently on different streams when their
 * caches differ.  mask: DEVICE [sum T] bytes; src_k/src_v may be NULL only when no segment is
 * cached. */
sx_status sx_realign_scatter_masked(const sx_plan* plan, const void* src_k, const void* src_v, const void* k_new,
                                    const void* v_new, const uint8_t* mask, void* k_cache, void* v_cache,
                                    void* stream);

/* Eq. sparseq-attn and Eq. sparseq-score with the cross-head sum of Section 3.2:
 *   scores[off_r + j] = sum_h sum_{i in P_r, i >= j} softmax_j(scale * q[i,h] . K[j, h/(Hq/Hkv)])
 * over the probe rows P_r = I_nr U S_tail of request r, reading keys from k_cache (whatever the
 * cache holds: re-aligned cached keys and the fresh keys written so far).  Probabilities and
 * sums are float32 per tile and float64 across tiles; the order of every sum is fixed, so the
 * result is deterministic.  Positions after the last probe get 0.  Uses plan scratch.
 * lse_in: NULL (two passes over the keys: the softmax denominators of the probe rows, then the
 *   column sums), or a DEVICE float32 array [sum T][Hq] of natural-log sums
 *   log sum_{j <= i} exp(scale * q[i,h] . K[j]) over the keys k_cache holds -- exactly what
 *   sx_full_attn writes to its lse output when the selecting layer is the last full layer of a
 *   hybrid stack (Section 3.4), with k_cache holding that layer's keys.  Then the denominators
 *   are taken from it (one pass); only the probe rows are read. */
sx_status sx_sparseq_score(const sx_plan* plan, const void* q, const void* k_cache, const float* lse_in,
                           float* scores, void* stream);

/* sx_sparseq_score in one-pass mode (lse_in required) that allocates nothing and uses no plan scratch:
 * for callers that cannot allocate device memory or should not touch the plan's scratch -- code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same kernels, same fixed
 * summation order, so the scores are bit-identical to sx_sparseq_score's.  Its scratch (the per-KV-head
 * column sums and the gathered probe columns) lives in a 32 MiB array inside the library that each
 * device holds from the first call on that device until the process ends; a plan needing more
 * (8 Hkv sum T + 2 (n_probes + 64) Hq d + 4 (n_probes + 64) Hq bytes, each part rounded up to 256;
 * bfloat16 plans, float32 plans only the first part) returns SX_EUNSUPPORTED.  Every call on a
 * device shares that array: calls that overlap in time on one device (different streams, threads or
 * processes without ordering) race and give wrong scores.  No host synchronisation. */
sx_status sx_sparseq_score_static(const sx_plan* plan, const void* q, const void* k_cache, const float* lse_in,
                                  float* scores, void* stream);

/* Eq. topk, Section 3.3 and Algorithm 1 steps 14-17, per request: S_key = the k_r reused
 * positions (every position with SX_TOPK_ALL_POSITIONS) with the largest score (k_r as in
 * sx_plan_budget; ties go to the lower index),
 * R = sorted(I_nr U S_key U S_ov U S_tail) written in the row-list layout.  Selection compares
 * the float32 scores exactly.  ratio outside [0, 1] -> SX_EINVAL. */
sx_status sx_topk_select(const sx_plan* plan, const float* scores, double ratio, int32_t* rows,
                         int32_t* n_rows, void* stream);

/* Algorithm 1 step 21: for every listed row i of request r and every query head h,
 *   out[off_r + n, h] = sum_{j <= i} softmax_j(scale * q[off_r + i, h] . K[j]) V[j]
 * with K/V read from the paged cache of request r.  bfloat16 runs on matrix cores with float32
 * accumulation and bfloat16 probabilities; float32 runs on vector ALUs.  max_rows as in
 * sx_kv_scatter: the rows n >= min(n_rows[r], max_rows) are neither computed nor written, so the
 * attention covers exactly the rows whose K/V sx_kv_scatter writes for the same list.  Uses the
 * plan's work-queue counters (bfloat16), so calls sharing a plan must be stream-ordered; takes its
 * row tiles in the order sx_rows_mask planned for the same row list, if any. */
sx_status sx_sparse_attn(const sx_plan* plan, const void* q, const int32_t* rows, const int32_t* n_rows,
                         int32_t max_rows, const void* k_cache, const void* v_cache, void* out,
                         void* stream);

/* Plain causal attention over dense fresh tensors (the hybrid layers below the threshold,
 * Section 3.4).  cu_seqlens is a DEVICE int32 array [n_requests + 1] of token offsets
 * (cu_seqlens[0] = 0); max_seqlen (host) must be >= every request length.  lse, when not NULL,
 * receives [sum T][Hq] float32 natural-log sums log(sum_j exp(scale * q.k_j)).  bfloat16 calls
 * run a persistent grid whose work-queue counters sit in the library (64 slots per device,
 * handed out in turn): at most 64 calls may be in flight on one device at a time.  A call made
 * while its stream is being captured into a graph uses no counters (one workgroup per row tile). */
sx_status sx_full_attn(const sx_layer_desc* desc, const void* q, const void* k, const void* v,
                       const int32_t* cu_seqlens, int32_t n_requests, int32_t max_seqlen, void* out,
                       float* lse, void* stream);

/* ------------------------------------------------------------------------------------------
 * Row-sparse layer body (Algorithm 1 steps 19 and 22): the projections, normalisations and the
 * feed-forward module evaluated only on the rows of R, as the paper does after the boundary
 * layer.  bfloat16 plans only (SX_EUNSUPPORTED otherwise); float32 arithmetic inside, bfloat16
 * results rounded to nearest even.
 *
 * Rows: for request r, rows[off_r + n] for n < min(n_rows[r], max_rows) (the row-list layout of
 * sx_topk_select; max_rows is at most the longest request and should be >= every n_rows[r], as for
 * sx_kv_scatter).  An operand row is addressed
 *   by slot  (`*_by_token` = 0): row off_r + n of a [sum T][...] array -- compact per request,
 *            the layout of sx_sparse_attn's output;
 *   by token (`*_by_token` = 1): row off_r + rows[off_r + n] -- the request's token rows, the
 *            layout of fresh q/k/v and of hidden states.
 * Every tensor is caller-owned DEVICE memory; rows not listed are neither read nor written.
 * ------------------------------------------------------------------------------------------ */

/* y[row] = x[row] . w^T (+ residual[row]): x [..][k], w [n][k] (the weight of a linear layer,
 * k contiguous), y and residual [..][n]; residual (nullable) is addressed like y and may be y
 * itself (in-place residual add).  k a multiple of 64, n a multiple of 256.  Matrix cores,
 * float32 accumulation. */
sx_status sx_gemm_rows(const sx_plan* plan, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                       const void* x, int32_t x_by_token, const void* w, int32_t k, int32_t n,
                       const void* residual, void* y, int32_t y_by_token, void* stream);

/* The same product for a weight made of stacked parts, each written to its own output: w is
 * [sum part_n][k] (part i = rows sum_{j<i} part_n[j] .. of w, e.g. the query, key and value
 * projections stacked), and columns of part i land in y_parts[i], [..][part_n[i]], addressed by
 * y_by_token like sx_gemm_rows' y.  part_n (host array of n_parts, 1 <= n_parts <= 4): positive
 * multiples of 256; y_parts: host array of DEVICE pointers.  No residual.  One launch for all the
 * parts, so narrow parts share the machine. */
sx_status sx_gemm_rows_split(const sx_plan* plan, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                             const void* x, int32_t x_by_token, const void* w, int32_t k, int32_t n_parts,
                             const int32_t* part_n, void* const* y_parts, int32_t y_by_token, void* stream);

/* RMSNorm: y[row] = x[row] / sqrt(mean_j x[row][j]^2 + eps) * gamma, rows of h elements
 * (h a multiple of 8), gamma [h]; the sum of squares is float32 in a fixed order. */
sx_status sx_rmsnorm_rows(const sx_plan* plan, const int32_t* rows, const int32_t* n_rows, int32_t max_rows,
                          const void* x, int32_t x_by_token, const void* gamma, float eps, int32_t h, void* y,
                          int32_t y_by_token, void* stream);

/* RoPE of fresh query and key rows, in place, at each listed token's position in the new
 * sequence (new_pos of its segment + offset): q [sum T][Hq][d], k [sum T][Hkv][d], addressed by
 * token.  Pairs and frequencies as in sx_rope_realign (angle and cos/sin in float64, rounded to
 * float32; rotation in float32 without contraction). */
sx_status sx_rope_rows(const sx_plan* plan, const int32_t* rows, const int32_t* n_rows, int32_t max_rows, void* q,
                       void* k, void* stream);

/* SwiGLU activation, by slot: y[row][j] = silu(g) * u with g = gate_up[row][j],
 * u = gate_up[row][f + j], silu(g) = g / (1 + e^-g); gate_up [sum T][2f], y [sum T][f]
 * (f a multiple of 8). */
sx_status sx_silu_mul_rows(const sx_plan* plan, const int32_t* n_rows, int32_t max_rows, const void* gate_up,
                           int32_t f, void* y, void* stream);

/* Text of the last non-OK status returned to this thread ("" if none). */
const char* sx_last_error(void);

/* Library version string. */
const char* sx_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SX_H */
