/*
 * lethe.h -- C ABI of the MI355X (gfx950) Lethe hot path.
 *
 * Lethe (arXiv 2511.06029) prunes the KV cache of a decoding LLM along two
 * axes: per layer, a budget derived from the layer's attention sparsity
 * ("Spatial KV Cache Pruning via Layerwise Sparsity Estimation", Eq. 1-2), and
 * over time, by Recency-Aware Selective Retention (RASR, Eq. 5) which keeps a
 * recent window plus the tokens with the highest decayed attention score.
 *
 * This library implements one decode step (append, grouped-query attention,
 * Eq. 5 score update) and the three calls of a prune round (layer sparsity and
 * budgets, RASR selection, in-place compaction) as HIP kernels.
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every pointer argument and every pointer inside lethe_cache is DEVICE
 *    memory owned by the caller, except `cache` itself, which is a host
 *    struct read during the call only.  The library allocates nothing; its
 *    only device memory of its own is that static scratch array.
 *  - Calls enqueue work on `stream` and return without synchronising the
 *    host.  The returned status covers host-checkable errors only; when it is
 *    not LETHE_OK nothing was enqueued.
 *  - Conditions found on the device are OR-ed into *cache->dev_status
 *    (LETHE_DEV_* bits below); the affected sequence or segment is left
 *    unmodified.  The caller reads the word at its own sync points.
 *  - Calls keep no global mutable state (the one exception is the static
 *    scratch of lethe_decode_attn_score_noalloc, shared by its calls on one
 *    device): concurrent calls on different caches and workspaces are safe.
 *    Calls that share a cache or a workspace must be ordered on one stream.
 *  - Each cache carries a decode state (lethe_cache::state) of
 *    lethe_state_bytes(cache) bytes that the caller allocates and zero-fills
 *    once, before the first call; the calls keep it consistent afterwards.  It
 *    holds the one decode step whose score update is still pending (see
 *    lethe_decode_attn_score).  Whoever changes len, scores or the layout of
 *    a cache other than through these calls first calls lethe_score_flush
 *    (or zero-fills the state again, dropping a pending step).
 *
 * Cache layout (ragged, one layout for K, V and scores)
 * ----------------------------------------------------
 *  Rows are head_dim elements of `dtype`.  Layer l owns rows
 *  [l * rows_per_layer, (l + 1) * rows_per_layer).  The segment of
 *  (layer l, sequence b, KV head h) starts at row
 *      l * rows_per_layer + seq_base[b] + h * cap[b]
 *  and holds cap[b] rows, of which the first len[l * num_seqs + b] are live
 *  (the same count for every KV head of (l, b)).  Live rows are in token
 *  order, oldest first.  score has the same row geometry with one fp32 per
 *  row.  The caller guarantees seq_base[b] + num_kv_heads * cap[b] <=
 *  rows_per_layer; kernels re-check it and flag LETHE_DEV_BAD_LAYOUT.
 */
#ifndef LETHE_H
#define LETHE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LETHE_OK = 0,
  LETHE_ERR_INVALID = -1,     /* bad argument (null pointer, out-of-range value) */
  LETHE_ERR_UNSUPPORTED = -2, /* valid but not built: head_dim, group size, batch */
  LETHE_ERR_WORKSPACE = -3,   /* ws_bytes below lethe_workspace_bytes(...)         */
  LETHE_ERR_HIP = -4          /* the HIP runtime rejected a launch                 */
} lethe_status;

typedef enum { LETHE_BF16 = 0, LETHE_F32 = 1 } lethe_dtype;

/* Bits OR-ed into *dev_status by the kernels. */
#define LETHE_DEV_APPEND_OVERFLOW 1 /* append with len == cap: sequence skipped      */
#define LETHE_DEV_INFEASIBLE 2      /* protected rows exceed the global budget        */
#define LETHE_DEV_BAD_LAYOUT 4      /* len < 0, len > cap or segment past the layer   */
#define LETHE_DEV_HEAD_MISMATCH 8   /* compaction kept different counts across heads  */
#define LETHE_DEV_WAIT_TIMEOUT 16   /* a bounded wait between blocks gave up: the call's
                                       results are unspecified (never expected)      */

typedef struct {
  void* k;                  /* dtype [num_layers][rows_per_layer][head_dim]            */
  void* v;                  /* dtype [num_layers][rows_per_layer][head_dim]            */
  float* score;             /* fp32  [num_layers][rows_per_layer]                      */
  int32_t* len;             /* int32 [num_layers][num_seqs] live rows                  */
  const int64_t* seq_base;  /* int64 [num_seqs] first row of sequence b in a layer     */
  const int32_t* cap;       /* int32 [num_seqs] rows per (layer, sequence, KV head)    */
  int64_t rows_per_layer;
  int32_t num_layers;
  int32_t num_seqs;         /* 1 .. 1024                                               */
  int32_t num_q_heads;
  int32_t num_kv_heads;     /* num_q_heads / num_kv_heads in 1 .. 8                    */
  int32_t head_dim;         /* 64 or 128                                               */
  lethe_dtype dtype;        /* storage of k, v and of the q / k_new / v_new inputs     */
  int32_t* dev_status;      /* int32 [1], LETHE_DEV_* bits                             */
  void* state;              /* lethe_state_bytes(cache) bytes, zero-filled before use  */
} lethe_cache;

/* Operations, for lethe_workspace_bytes. */
#define LETHE_OP_DECODE 0
#define LETHE_OP_SPARSITY 1
#define LETHE_OP_SELECT 2
#define LETHE_OP_COMPACT 3
#define LETHE_OP_DECODE_FINAL 4
#define LETHE_OP_COMPACT_PLAN 5

/*
 * Bytes of device workspace `op` needs for this cache (0 when none).  No
 * workspace needs initialising; its contents are scratch between calls.
 * Returns 0 for an invalid cache description or op (the device pointers,
 * cache->state included, are not looked at).
 */
size_t lethe_workspace_bytes(const lethe_cache* cache, int op);

/*
 * Bytes of the decode state of this cache: two query sets of
 * num_layers * num_seqs * num_q_heads * head_dim elements of dtype, 8 bytes
 * per (layer, sequence, query head), and a few words per (layer, sequence).
 * Independent of rows_per_layer.  Returns 0 for an invalid cache description
 * (the device pointers, cache->state included, are not looked at).
 */
size_t lethe_state_bytes(const lethe_cache* cache);

/*
 * One decode step of layer `layer` for every sequence (the decoding loop of
 * the paper's System Overview; importance update of Eq. 5 in the RASR
 * section, summed over the query heads of each KV group and read per token).
 *
 *  1. Append (when k_new != NULL): for every sequence b and KV head h, row
 *     n = len[layer][b] of the segment receives k_new[b][h][:] and
 *     v_new[b][h][:], and its score starts at 0; len becomes n + 1.  If
 *     n == cap[b] the whole sequence is skipped: LETHE_DEV_APPEND_OVERFLOW is
 *     set, its cache rows, scores and len are untouched and its out rows are
 *     filled with quiet NaN.
 *  2. Attention: query head i = h * G + g (G = num_q_heads / num_kv_heads)
 *     reads KV head h (the repeat-interleave of Eq. 3, never materialised):
 *        x_j = softmax_scale * q[b][i][:] . K[j][:],  p = softmax_j(x),
 *        out[b][i][:] = sum_j p_j V[j][:]
 *     over all live rows j (after the append).  A sequence with no live rows
 *     gets out = 0.
 *  3. Score: s_j <- gamma * s_j + sum_{g < G} p_{hG+g, j} for every live row.
 *     This update is applied one call late.  It needs the step's final
 *     softmax maximum and sum, known only when the whole segment has been
 *     read, so the call keeps q, the scale and the per-head statistics in
 *     cache->state, and the next decode call on the same layer recomputes
 *     the step's logits from the K rows it reads anyway and applies it.  lethe_score_flush, and the
 *     start of lethe_layer_sparsity, lethe_rasr_select and lethe_kv_compact,
 *     apply a pending step at once.  So after a decode call `score` of that
 *     layer lacks the call's own step until one of those runs; out and len
 *     are final when the call's work completes.
 *
 *  q       dtype [num_seqs][num_q_heads][head_dim]
 *  k_new   dtype [num_seqs][num_kv_heads][head_dim], or NULL (no append)
 *  v_new   dtype [num_seqs][num_kv_heads][head_dim], NULL iff k_new is NULL
 *  gamma   decay in (0, 1]; 1 is plain accumulated attention
 *  softmax_scale  > 0, or <= 0 for 1/sqrt(head_dim)
 *  out     fp32 [num_seqs][num_q_heads][head_dim]
 *  ws      at least lethe_workspace_bytes(cache, LETHE_OP_DECODE) bytes.
 * A sequence skipped for overflow or a bad layout keeps its pending step.
 * Work split: each segment is cut into chunks of about the same number of
 * rows, one block each, so that sequences of very different lengths finish
 * together.  The split follows tiling hints, the layer's lengths as the
 * decode state last recorded them (lethe_score_flush, the prune calls, which
 * flush first, lethe_kv_compact, lethe_kv_compact_layers and
 * lethe_kv_compact_plan record them; a zero-filled state has
 * none, and the split is then the same for every segment).  The hints only
 * shape the split, never the result: a length changed since they were
 * recorded is still attended in full.  A segment's blocks take their 32-row
 * steps after the first from a shared counter, so that blocks the memory
 * system serves faster take more; the summation order then varies, and
 * repeated calls on identical inputs can differ in the last bits of out and
 * score.  With the environment variable LETHE_DECODE_DETERMINISTIC set to a
 * non-zero value every block's steps are fixed and repeated calls are
 * bit-identical (about 3% slower on the Llama-8B batch-128 workload, 5% on
 * the Qwen-7B batch-16 one).  By default a call splits its hinted rows into
 * chunks of about 14 steps, at least min(512, N) and at most N chunks, N
 * being one per 1024 rows of capacity (512 to 4096); LETHE_DECODE_BLOCKS
 * fixes the number of chunks instead, LETHE_DECODE_STEPS_PER_CHUNK and
 * LETHE_DECODE_MIN_CHUNKS change the two defaults.
 * Accumulation is fp32; results match the exact result to about 1e-5
 * relative.  Errors: LETHE_ERR_INVALID (null pointer, layer out of range,
 * gamma outside (0, 1] or NaN, NaN scale), LETHE_ERR_UNSUPPORTED,
 * LETHE_ERR_WORKSPACE, LETHE_ERR_HIP.
 */
lethe_status lethe_decode_attn_score(const lethe_cache* cache, int32_t layer, const void* q,
                                     const void* k_new, const void* v_new, float gamma,
                                     float softmax_scale, float* out, void* ws, size_t ws_bytes,
                                     hipStream_t stream);

/*
 * The same decode step (Eq. 5 update included), settled within the call:
 * items 1-3 of lethe_decode_attn_score, except that the call's own score
 * update is applied before its work ends in stream order, so afterwards
 * `score` of the layer is current and no step of it is pending.  Meant for
 * the last step before a prune round, which then finds nothing to apply and
 * reads no K row for it.  The step's logits (8 floats per row of the layer)
 * pass through ws, and a second kernel applies them; the scores equal, bit
 * for bit, those that lethe_decode_attn_score followed by lethe_score_flush
 * gives.
 *  ws  at least lethe_workspace_bytes(cache, LETHE_OP_DECODE_FINAL) bytes:
 *      the LETHE_OP_DECODE bytes plus about 32 bytes per row of a layer.
 * Arguments, layouts, skipped sequences (which keep their pending step) and
 * errors as for lethe_decode_attn_score.
 */
lethe_status lethe_decode_attn_score_final(const lethe_cache* cache, int32_t layer, const void* q,
                                           const void* k_new, const void* v_new, float gamma,
                                           float softmax_scale, float* out, void* ws, size_t ws_bytes,
                                           hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the decode
 * step of lethe_decode_attn_score, items 1-3 with the same arguments, layouts,
 * deferred score update and errors, but without a workspace argument.  The
 * chunk partials go to a static device array of the library, 32 MiB on every
 * device the library runs on, held until the process ends; nothing is
 * allocated, by the library or through any other library.  The caller still
 * owns the cache, its decode state, q, k_new, v_new and out.
 *
 * Every call on one device shares that device's array and leaves its
 * partials there; each call writes every partial it reads, so no call sees an
 * earlier call's contents.  Calls that overlap on one device (on different
 * streams, or from different host threads without ordering) race on the
 * array: order them on one stream.  The first call on a device looks up the
 * array's address there (one HIP runtime query).
 *
 * Limit: one partial of 4 * (G * (head_dim + 2)) bytes, rounded up to 128,
 * per (sequence, KV head) must fit the 32 MiB, i.e. num_seqs * num_kv_heads
 * * that size <= 33554432 (all caches of up to 1024 sequences with 8 KV
 * heads and G <= 4, or 4 KV heads and G <= 8, qualify).  Larger caches get
 * LETHE_ERR_UNSUPPORTED before anything is enqueued.  Within the limit the
 * call may split segments into fewer chunks than lethe_decode_attn_score.
 */
lethe_status lethe_decode_attn_score_noalloc(const lethe_cache* cache, int32_t layer, const void* q,
                                             const void* k_new, const void* v_new, float gamma,
                                             float softmax_scale, float* out, hipStream_t stream);

/*
 * Causal prefill attention that seeds the importance scores, for one layer.
 * Eq. 2 collapses attention over heads and query positions into one
 * importance vector; here the sum runs over the query heads of each KV group
 * (as in lethe_decode_attn_score) and over the call's queries.
 *
 * Sequence b comes with q_len[b] queries, for the q_len[b] newest of its
 * n = len[layer][b] cached rows (the prompt, or one chunk of it, whose K and
 * V the caller has already written into the cache).  Query i sits at position
 * p = n - q_len[b] + i and attends rows 0 .. p.  For query head j = h G + g:
 *     x = softmax_scale * q[row][j][:] . K[0..p][:],  P = softmax(x),
 *     out[row][j][:] = sum_r P_r V[r][:]           (row = q_start[b] + i)
 * and for every row r < n of every KV head h:
 *     s_r <- s_r + sum_{g < G} sum_i P_{hG+g, i, r}
 * No decay between the queries of one call; later decode steps decay the
 * seeded scores as Eq. 5 says.  Chunked prefill (several calls covering
 * consecutive chunks) gives the same outputs and scores as one call.
 *
 *  q        bf16 [q_rows][num_q_heads][head_dim]; out fp32, same layout.
 *  q_start  int64 [num_seqs], q_len int32 [num_seqs] (device): the rows of
 *           sequence b are q_start[b] .. q_start[b] + q_len[b] - 1.
 *  max_q_len, max_kv_len  host upper bounds of q_len[b] and len[layer][b]
 *           (they size the grid).
 *  ws       lethe_prefill_workspace_bytes(cache, q_rows) bytes (per query
 *           row and head: the softmax max and 1 / sum between the passes).
 * A sequence whose sizes do not fit (q_len > len, a bound exceeded, rows
 * outside [0, q_rows), a bad layout) sets LETHE_DEV_BAD_LAYOUT and is left
 * untouched.  Applies a pending decode step first.  bf16 caches only
 * (LETHE_ERR_UNSUPPORTED otherwise).  Accumulation fp32, P kept to fp32
 * accuracy in the P V product.  Errors: LETHE_ERR_INVALID, LETHE_ERR_UNSUPPORTED,
 * LETHE_ERR_WORKSPACE, LETHE_ERR_HIP.
 */
lethe_status lethe_prefill_attn_score(const lethe_cache* cache, int32_t layer, const void* q,
                                      const int64_t* q_start, const int32_t* q_len, int64_t q_rows,
                                      int32_t max_q_len, int32_t max_kv_len, float softmax_scale,
                                      float* out, void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes lethe_prefill_attn_score needs for q_rows query rows. */
size_t lethe_prefill_workspace_bytes(const lethe_cache* cache, int64_t q_rows);

/*
 * Layer sparsity and budgets for every sequence (start of a prune round).
 *
 *  Applies a pending decode step first (as lethe_score_flush).
 *
 *  Sparsity (Eq. 1 applied to Eq. 2's head-summed importance): for every
 *  (b, l), a_j = sum_h s_{l,b,h,j} over the live rows and
 *      S = (sqrt(n) - |a|_1 / |a|_2) / (sqrt(n) - 1), clamped to [0, 1],
 *  with S = 0 when n <= 1 or a == 0.  Accumulated in fp64, stored as fp32.
 *  When sparsity_in != NULL, S is taken from it instead (fp32 [num_seqs][L]).
 *
 *  Budgets: the paper gives layers budgets from their redundancy but no
 *  formula; this library splits the global budget of sequence b,
 *  global_budget[b], over its layers by density weights
 *      w_l = 1 + floor((1 - S_l) * 2^24)   (fp32 arithmetic, S clamped, NaN -> 0)
 *  with floors f_l = min(n_l, recent + sink) and caps n_l, proportional
 *  integer shares and largest remainders (ties to the lower layer), capped
 *  layers fixed and the rest re-split until no cap binds.  Then
 *  sum_l budget = global_budget exactly and f_l <= budget <= n_l.  If
 *  sum n_l <= global_budget every budget is n_l; if sum f_l > global_budget,
 *  LETHE_DEV_INFEASIBLE is set and every budget is n_l.
 *
 *  global_budget int64 [num_seqs]; sparsity_out fp32 [num_seqs][num_layers];
 *  budget_out int32 [num_seqs][num_layers]; recent, sink >= 0.
 *  Needs num_layers <= 256.  ws: lethe_workspace_bytes(cache, LETHE_OP_SPARSITY)
 *  (may be 0 bytes / NULL).
 */
lethe_status lethe_layer_sparsity(const lethe_cache* cache, const int64_t* global_budget,
                                  int32_t recent, int32_t sink, const float* sparsity_in,
                                  float* sparsity_out, int32_t* budget_out, void* ws,
                                  size_t ws_bytes, hipStream_t stream);

/*
 * RASR retention (RASR section; sink and recent sets of Algorithm 1): for every
 * segment (l, b, h) with n live rows and budget k = max(budget[b][l], 0):
 *   k >= n: keep every row.  Otherwise r = min(recent, k), s = min(sink, k - r),
 *   keep rows [0, s) and [n - r, n), and among rows [s, n - r) the first
 *   k - r - s in the order (score descending, row ascending), where +0 and
 *   -0 tie and NaN ranks after every number.  Exactly min(n, k) rows are kept.
 *
 *  budget int32 [num_seqs][num_layers]; keep uint8 [num_layers][rows_per_layer]
 *  (same geometry as score) receives 1 (keep) or 0 (evict) for live rows;
 *  other bytes are not written.  ws: may be NULL (0 bytes).  Applies a
 *  pending decode step first (as lethe_score_flush).
 */
lethe_status lethe_rasr_select(const lethe_cache* cache, const int32_t* budget, int32_t recent,
                               int32_t sink, uint8_t* keep, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * RASR retention with one kept set per (layer, sequence), shared by all its KV
 * heads: Eq. 2 collapses attention over every head into a single importance
 * vector per layer, and the GQA note that follows it (Eq. 3) makes that
 * vector head-invariant.  The rank key of row j is the head-summed score
 *     a_j = (...((s_{h=0,j} + s_{1,j}) + s_{2,j}) + ...) + s_{H_KV-1,j}
 * in fp32 (ascending heads, rounded after each addition); the keep rule is
 * that of lethe_rasr_select applied to a with k = max(budget[b][l], 0), and
 * the same mask is written into the keep rows of every KV head, so
 * lethe_kv_compact then moves the same token positions in every head.
 * Arguments, workspace and errors as lethe_rasr_select.
 */
lethe_status lethe_rasr_select_shared(const lethe_cache* cache, const int32_t* budget,
                                      int32_t recent, int32_t sink, uint8_t* keep, void* ws,
                                      size_t ws_bytes, hipStream_t stream);

/* breakpoint[] values of lethe_segmented_shrink that are not cut points. */
#define LETHE_SHRINK_NO_BREAKPOINT (-1)
#define LETHE_SHRINK_NOT_TRIGGERED (-2)

/*
 * Algorithm 1 (Segmented Attention-Based Token Shrinking) with the size
 * trigger of the System Overview, for every (layer l, sequence b), on the
 * head-summed score a of lethe_rasr_select_shared (one kept set shared by the
 * KV heads).  With n = len[l][b] and L = max(evict_threshold[l][b], 0):
 *
 *  0. n <= L: not triggered; every row is kept, the threshold becomes L,
 *     breakpoint = LETHE_SHRINK_NOT_TRIGGERED.
 *  1. Rank the n rows by (a descending, row ascending), +0 = -0, NaN last;
 *     v[r] is the value at rank r.
 *  2. Cut points c_d = floor(n * d / segments), d = 1 .. segments - 1.
 *  3. The breakpoint is the first c_d whose ratio v[0] / v[c_d] reaches tau,
 *     evaluated exactly as tau * v[c_d] <= v[0] in fp64 (the printed "<= tau"
 *     is read as ">= tau": the prose asks for the cut where attention drops
 *     sharply, and the ratio never falls along the ranking).  A ratio with
 *     v[0] <= 0, v[0] NaN or v[c_d] NaN is undefined and never qualifies.
 *  4. With a breakpoint c: keep rows [0, sink), the c best-ranked rows and
 *     rows [n - recent, n) (windows clipped to [0, n)); the threshold becomes
 *     max(L, c + recent).  Without one pruning is delayed: every row is kept
 *     and the threshold becomes 2 L.  Thresholds saturate at 2^31 - 1.
 *
 *  segments >= 1 (1 gives no cut points); tau > 1 and finite; recent, sink >= 0.
 *  evict_threshold int32 [num_layers][num_seqs], read and updated in place.
 *  breakpoint int32 [num_layers][num_seqs] or NULL: the breakpoint c, or one
 *  of the two codes above.  keep uint8 [num_layers][rows_per_layer] as for
 *  lethe_rasr_select; lethe_kv_compact then drops the evicted rows.
 *  ws may be NULL.  Applies a pending decode step first.  Errors:
 *  LETHE_ERR_INVALID, LETHE_ERR_UNSUPPORTED, LETHE_ERR_HIP.
 */
lethe_status lethe_segmented_shrink(const lethe_cache* cache, int32_t segments, float tau,
                                    int32_t recent, int32_t sink, int32_t* evict_threshold,
                                    int32_t* breakpoint, uint8_t* keep, void* ws, size_t ws_bytes,
                                    hipStream_t stream);

/*
 * In-place, order-preserving compaction (pruned tokens leave the cache, as
 * the paper's System Overview and its pruning illustration describe): in
 * every segment the live rows with keep != 0 move, in order, to the front; K,
 * V and score rows move together and bit-exactly; len becomes the number
 * kept.  If the KV heads of one (l, b) keep different counts, len becomes
 * the smallest and LETHE_DEV_HEAD_MISMATCH is set.  Rows at or after the new
 * len are unspecified.  keep: uint8 [num_layers][rows_per_layer].
 *  ws: lethe_workspace_bytes(cache, LETHE_OP_COMPACT) bytes.  Applies a
 *  pending decode step first (as lethe_score_flush), so the scores that move
 *  are current.  The rows move in 256-row tiles through a work queue in ws
 *  whose counters live in the decode state, so compactions of one cache must
 *  be ordered on one stream.  Blocks wait for one another only within a
 *  bounded number of polls: LETHE_DEV_WAIT_TIMEOUT reports one that gave up
 *  (not expected; the environment variables LETHE_COMPACT_TEST_WAIT=1 and
 *  LETHE_COMPACT_SPIN_LIMIT force it, for tests), and LETHE_COMPACT_BLOCKS
 *  overrides the 512 blocks of the moving launch.  All three are read once
 *  per process.
 */
lethe_status lethe_kv_compact(const lethe_cache* cache, const uint8_t* keep, void* ws,
                              size_t ws_bytes, hipStream_t stream);

/*
 * lethe_kv_compact restricted to layers layer_begin .. layer_begin +
 * layer_count - 1 (the same result for those layers; nothing of the other
 * layers is read or written, their rows of `keep` included).  A pending
 * decode step of those layers is applied first.  Calls on one cache share the
 * workspace and the queue counters in the decode state, so they must be
 * ordered on one stream; a decode call of a layer outside the range may run
 * concurrently on another stream, which lets a prune round compact layer l
 * while the next decode step works on the layers before it (the decode call
 * of layer l waits for its compaction).  layer_count 0 does nothing.  Errors:
 * those of lethe_kv_compact, and LETHE_ERR_INVALID for a range outside
 * 0 .. num_layers - 1.
 */
lethe_status lethe_kv_compact_layers(const lethe_cache* cache, int32_t layer_begin, int32_t layer_count,
                                     const uint8_t* keep, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Compaction carried out by the next decode step (the same result as
 * lethe_kv_compact, with the moves riding on the reads that decode step does
 * anyway, so the rows that move are read once instead of twice).
 *
 * lethe_kv_compact_plan records, for every segment (l, b, h) with n live rows
 * and the keep mask `keep` (uint8 [num_layers][rows_per_layer], as for
 * lethe_kv_compact), the rows kept and, per 32-row step, the rows kept before
 * it and the step's keep mask, into `plan` (lethe_workspace_bytes(cache,
 * LETHE_OP_COMPACT_PLAN) bytes: 16 bytes per segment, and 12 per 32-row step
 * of capacity plus one step per segment, for the step's kept-before count,
 * mask and read flag).  It changes nothing in the cache; the decode state's tiling
 * hints take the kept counts.  If the KV heads of an (l, b) keep different
 * counts, LETHE_DEV_HEAD_MISMATCH is set and that sequence's plan is invalid;
 * a bad layout sets LETHE_DEV_BAD_LAYOUT likewise.
 *
 * lethe_decode_attn_score_compact(..., plan, plan_bytes, ws, ws_bytes, ...)
 * is then, for one layer, the compaction of that layer by the plan followed
 * by the decode step of lethe_decode_attn_score (same arguments, ws of
 * LETHE_OP_DECODE size): the kept rows move in order to the front of their
 * segment (K, V and score bit for bit, a pending score update applied to the
 * rows kept), the new row is appended after them, the attention and the score
 * update run over the kept rows and the new one, and len becomes the rows
 * kept plus the appended one.  Rows past the new len are unspecified.  A
 * sequence whose len differs from the one the plan was made for, or whose
 * plan is invalid, is skipped as a bad layout (LETHE_DEV_BAD_LAYOUT, out =
 * NaN, nothing of it changes).  Call it once per layer with the plan made
 * after the layer's last change; between the plan and the last of those
 * calls only these calls may touch the plan (they set its step flags).
 *
 * The work split is lethe_decode_attn_score's: the wavefronts of a segment
 * take its 32-row steps in increasing order.  From the first step holding
 * an evicted row on, a wavefront marks its step read as soon as the step's
 * loads have landed, and before storing the step's kept rows at their new
 * places (at or before their old ones) waits for the steps those places lie
 * in.  Those steps were taken earlier and are marked without waiting for
 * anything, so every wait ends; each is still bounded (2^20 polls per
 * wavefront, fewer if the environment variable LETHE_COMPACT_SPIN_LIMIT,
 * read at each call, says so), and one that gives up sets
 * LETHE_DEV_WAIT_TIMEOUT.  bf16
 * caches only (LETHE_ERR_UNSUPPORTED otherwise); step indices must fit int32
 * (num_layers * (rows_per_layer / 32 + num_seqs * num_kv_heads) < 2^31) and
 * num_kv_heads <= 64.  Errors: those of lethe_decode_attn_score, and
 * LETHE_ERR_WORKSPACE for a plan buffer below the plan size.
 */
lethe_status lethe_kv_compact_plan(const lethe_cache* cache, const uint8_t* keep, void* plan, size_t plan_bytes,
                                   hipStream_t stream);
lethe_status lethe_decode_attn_score_compact(const lethe_cache* cache, int32_t layer, const void* q,
                                             const void* k_new, const void* v_new, float gamma,
                                             float softmax_scale, float* out, void* plan, size_t plan_bytes,
                                             void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Apply the pending decode step of every (layer, sequence) to its scores
 * (item 3 of lethe_decode_attn_score, Eq. 5): afterwards `score` is current
 * and no step is pending.  Needs no workspace.  Errors: LETHE_ERR_INVALID,
 * LETHE_ERR_UNSUPPORTED, LETHE_ERR_HIP.
 */
lethe_status lethe_score_flush(const lethe_cache* cache, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* lethe_status_string(lethe_status status);

#ifdef __cplusplus
}
#endif

#endif /* LETHE_H */
