/*
 * headkv.h -- C ABI of the head-aware compressed-KV decode path for AMD
 * Instinct MI355X (gfx950).
 *
 * The library keeps, per layer, a KV cache whose retained length differs per
 * (batch row, head), and runs four operations of HeadKV (arXiv 2605.20600) on
 * it with hand-written HIP kernels:
 *
 *   headkv_score_heads       head grouping (Sec. 4, Step 2)
 *   headkv_assign_budgets    per-head budgets (Sec. 5.1, Implementation Details)
 *                            and the one-time move into per-head segments
 *   headkv_append_and_evict  cache append (Sec. 3, KV Cache) and the periodic
 *                            update (Sec. 4, Step 3 and Efficient Cache Update):
 *                            sliding window for local heads (Eq. 3), Stratified
 *                            Token Eviction for global heads (Eqs. 4-6)
 *   headkv_decode_attn       single-query attention, Eq. (1), over the
 *                            conditional prefix and the retained tokens
 *
 * Conventions shared by every entry point:
 *   - Status: every call returns HEADKV_OK (0) or a negative error code and
 *     never aborts; headkv_last_error() returns a message for the calling
 *     thread.  Arguments and the call order are validated before any HIP call.
 *   - Memory: the caller allocates every device buffer (sizes from headkv_plan
 *     and headkv_assign_budgets) and keeps it alive while the handle uses it.
 *     The library calls no hipMalloc.  Device buffers must be 256-byte aligned.
 *   - Streams: `stream` is a hipStream_t (NULL = the default stream).  Calls
 *     are asynchronous on it, except headkv_assign_budgets, which waits for the
 *     stream once to read the budgets back.
 *   - Layouts: bf16 values are passed as uint16_t bit patterns.  Per-step
 *     vectors are [batch][heads][head_dim] row-major; per-head arrays are
 *     [batch][heads].
 *   - Threads: a handle is not thread-safe; use one handle per stream.
 *   - Call order per layer: headkv_prefill once, then for every visual step t
 *     (t = 0, 1, ... consecutively): headkv_append_and_evict(t); at the
 *     grouping step t_g = group_threshold - 1 also headkv_score_heads and
 *     headkv_assign_budgets; then headkv_decode_attn.  Calls out of this order
 *     return HEADKV_ERR_STATE.
 */
#ifndef HEADKV_H
#define HEADKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t headkv_status;

#define HEADKV_OK 0
#define HEADKV_ERR_INVALID_ARG (-1) /* bad pointer, size, value or alignment */
#define HEADKV_ERR_CAPACITY (-2)    /* a caller buffer is too small */
#define HEADKV_ERR_STATE (-3)       /* call out of the documented order */
#define HEADKV_ERR_HIP (-4)         /* a HIP runtime call or launch failed */
#define HEADKV_ERR_UNSUPPORTED (-5) /* a shape this library does not handle */

/* Budget modes (Sec. 5.1, Implementation Details: global heads keep rho*N
 * tokens, local heads a small set of neighbouring tokens). */
#define HEADKV_BUDGET_PAPER 0    /* local: recent_len, global: floor(rho*N) */
#define HEADKV_BUDGET_OVERRIDE 1 /* caller budgets per head, 1..N */
#define HEADKV_BUDGET_TOTAL 2    /* layer keeps floor(rho*N)*heads in total:
                                    local heads recent_len, global heads an
                                    equal share in whole rows, >= recent_len */

/* Attention strategies for heads of unequal length, the three of Sec. 5.1
 * (Implementation Details) and Sec. 5.3 (Efficiency Analysis).  All give the
 * same outputs (up to fp32 summation order) and the same retained sets. */
#define HEADKV_ATTN_VARLEN 0  /* each head attends over its own length */
#define HEADKV_ATTN_PADDED 1  /* after grouping every head's segment has the
                                 layer's largest capacity, and every head reads
                                 the layer's longest length with the rows past
                                 its own length masked (Appendix, padding-based
                                 strategy) */
#define HEADKV_ATTN_GROUPED 2 /* one attention launch per head group (global
                                 heads, then local heads), written into one
                                 output */

/* Eviction scores of global heads. */
#define HEADKV_SCORE_MEAN_LOGIT 0 /* Eq. (6): mean raw logit of the past-P queries */
#define HEADKV_SCORE_ATTN_SUM 1   /* variant (multi-query attention aggregation):
                                     each past-P query's attention weight on the
                                     token over the cache it attended (prefix +
                                     retained tokens up to its step), summed
                                     over the queries; keeps the last P queries
                                     of every head in the metadata buffer */

/* Limits of this library. */
#define HEADKV_MAX_VISUAL 16384  /* num_visual */
#define HEADKV_MAX_PREFIX 2048   /* prefix_len */
#define HEADKV_MAX_CAPACITY 4608 /* visual tokens one head can hold */

typedef struct headkv_config {
    int32_t batch;           /* B >= 1 */
    int32_t num_layers;      /* >= 1 */
    int32_t num_heads;       /* H >= 1; key/value heads = query heads */
    int32_t head_dim;        /* d: 64 or 128 */
    int32_t prefix_len;      /* C: conditional tokens, never evicted (Eq. 2) */
    int32_t row_len;         /* R: tokens per image row, row-end token included */
    int32_t num_visual;      /* N: visual tokens of one image */
    int32_t recent_len;      /* w: recent window (Eq. 2), two rows in the paper */
    int32_t local_window;    /* W_loc: a head is local iff n* < W_loc */
    int32_t period;          /* P: update every P steps (Efficient Cache Update) */
    int32_t group_threshold; /* thr in 1..N: heads are grouped when thr visual
                                tokens are cached, i.e. at step thr - 1 */
    int32_t budget_mode;     /* HEADKV_BUDGET_* */
    int32_t rho_num, rho_den;/* rho = rho_num / rho_den in (0, 1] */
    int32_t rs_num, rs_den;  /* r_s = rs_num / rs_den in [0, 1] (Eq. 5) */
    int32_t attn_strategy;   /* HEADKV_ATTN_*; HEADKV_ATTN_VARLEN by default */
    int32_t score_mode;      /* HEADKV_SCORE_*: how global heads score the
                                history for eviction */
    int32_t cfg_pairs;       /* 1: batch rows 2i and 2i+1 are the conditional and
                                unconditional sequences of one classifier-free-
                                guidance pair, and both take the head labels of
                                row 2i (batch must be even); 0: every row is
                                grouped on its own */
    double tau;              /* grouping mass threshold in (0, 1], 0.9 */
} headkv_config;

typedef struct headkv_ctx* headkv_t;

/* Sizes of the caller-owned device buffers.
 *   dense_kv_bytes: per layer, the cache before grouping (every head holds
 *                   its prefix and up to group_threshold visual tokens);
 *   meta_bytes:     per layer, segment table, lengths, labels, budgets,
 *                   the last `period` queries of every head (the window an
 *                   update scores against), the attention dispatch order, the
 *                   attention chunk table;
 *   workspace_bytes: one buffer shared by all layers: the merge words of the
 *                   attention of layers with fewer heads than compute units,
 *                   which cut each head into chunks of at most one pass
 *                   and merge them in the same kernel.  The library zeroes it before
 *                   its first use and every launch leaves it zero; callers
 *                   must not write it while a handle uses it. */
headkv_status headkv_plan(const headkv_config* cfg, size_t* dense_kv_bytes,
                          size_t* meta_bytes, size_t* workspace_bytes);

/* Creates a host handle.  dense_kv, meta: host arrays of num_layers device
 * pointers; workspace: one device pointer, or NULL for a handle whose callers
 * cannot allocate: a call whose attention would need the workspace (a layer
 * with fewer batch x heads than compute units) then returns HEADKV_ERR_STATE,
 * and headkv_decode_attn_noalloc runs that attention instead.  No device
 * work is done. */
headkv_status headkv_create(const headkv_config* cfg, void* const* dense_kv,
                            void* const* meta, void* workspace, headkv_t* out);

void headkv_destroy(headkv_t h);

/* Step 1, cache prefilling (Sec. 4): stores the conditional keys and values
 * k_c, v_c ([B][H][C][d] bf16, device; NULL allowed when C = 0) as the first
 * C cache entries of every head of `layer`, and resets the layer's state. */
headkv_status headkv_prefill(headkv_t h, int32_t layer, const uint16_t* k_c,
                             const uint16_t* v_c, void* stream);

/* Step 1 with its attention: headkv_prefill, and the causal self-attention of
 * the C conditional tokens, out_c[b][h][i] = softmax(q_i K_c^T / sqrt(d) over
 * keys 0..i) V_c (Eq. 1 over the prefix, token by token).  q_c, k_c, v_c:
 * [B][H][C][d] bf16; out_c: [B][H][C][d] fp32; all device, 16-byte aligned.
 * Needs C >= 1.  bf16 storage, fp32 accumulation (the attention weights enter
 * the weighted sum of V in bf16, on the matrix cores). */
headkv_status headkv_prefill_attn(headkv_t h, int32_t layer, const uint16_t* q_c,
                                  const uint16_t* k_c, const uint16_t* v_c, float* out_c,
                                  void* stream);

/* Cache append K <- [K, k_t], V <- [V, v_t] (Sec. 3, KV Cache) for visual
 * step `step` of `layer`; q, k, v: [B][H][d] bf16, device.  q_t joins the
 * head's window of the past-P queries (Eq. 6).  When the layer is grouped and
 * (step - t_g) is a positive multiple of P, the periodic update follows
 * (Eqs. 2-6): each local head keeps its newest `budget` visual tokens; each
 * global head keeps its recent window and evicts from its history the
 * lowest-scored tokens of the long-range and near-range parts, M/2 each.
 * q, k and v must be 16-byte aligned (HEADKV_ERR_INVALID_ARG otherwise).
 * Steps must be consecutive from 0.  A step past t_g before grouping is
 * HEADKV_ERR_STATE. */
headkv_status headkv_append_and_evict(headkv_t h, int32_t layer, int32_t step,
                                      const uint16_t* q, const uint16_t* k,
                                      const uint16_t* v, void* stream);

/* Head grouping (Sec. 4, Step 2), at step t_g after its append: for each
 * (b, h) the current query q ([B][H][d] bf16, device) attends over the whole
 * key cache (prefix and visual tokens 0..t_g) in fp64; the attention mass is
 * accumulated backward from the newest token; n* is the smallest count whose
 * mass reaches tau, and the head is local iff n* < local_window.
 * Writes n_star ([B][H] int32, device) and is_local ([B][H] uint8, device,
 * 1 = local).  q must be 16-byte aligned. */
headkv_status headkv_score_heads(headkv_t h, int32_t layer, const uint16_t* q,
                                 int32_t* n_star, uint8_t* is_local, void* stream);

/* Budgets (Sec. 5.1) and the move into per-head segments, at step t_g after
 * score_heads.  is_local: [B][H] uint8 labels (device; usually the array
 * score_heads wrote; all zero gives the uniform-budget LineAR layout; with
 * cfg_pairs, row 2i+1 takes the labels of row 2i).
 * budget_override: [B][H] int32 (device) for HEADKV_BUDGET_OVERRIDE, else
 * NULL.  budgets: [B][H] int32 output (device), visual tokens per head, the
 * recent window included and the prefix not counted.
 * Each head then needs prefix_len + min(budget + period, N) slots (with
 * HEADKV_ATTN_PADDED, the largest of these for every head of the layer); the
 * total, with alignment, is written to *ragged_bytes_needed.  Both calls of the
 * two-call pattern first run the budget kernel, which writes `budgets` and the
 * layer's device copy of the labels and budgets, and wait for `stream` to read
 * the budgets back.  If ragged_kv is NULL or ragged_bytes is smaller, the call
 * then returns HEADKV_ERR_CAPACITY after setting *ragged_bytes_needed: the
 * layer stays in its dense layout, nothing else has changed, and a second call
 * with a large enough buffer (the same labels give the same budgets) completes
 * the grouping.  Otherwise the first update runs (Eqs. 2-6), the retained
 * tokens are copied into ragged_kv (device, 256-byte aligned, caller-owned from
 * now on), and the dense buffer of this layer is no longer used.  If a HIP
 * call fails after the budgets were read back (HEADKV_ERR_HIP), the layer's
 * metadata may be half-way to the new layout: every later call on the layer
 * returns HEADKV_ERR_STATE until headkv_prefill runs again. */
headkv_status headkv_assign_budgets(headkv_t h, int32_t layer, const uint8_t* is_local,
                                    const int32_t* budget_override, int32_t* budgets,
                                    void* ragged_kv, size_t ragged_bytes,
                                    size_t* ragged_bytes_needed, void* stream);

/* Decode attention, Eq. (1), of the current step for every (b, h) of
 * `layer`: o = softmax(q K^T / sqrt(d)) V over the prefix and the head's
 * retained visual tokens (the current token included).  q: [B][H][d] bf16,
 * out: [B][H][d] fp32, both device and 16-byte aligned.  bf16 storage, fp32
 * accumulation. */
headkv_status headkv_decode_attn(headkv_t h, int32_t layer, const uint16_t* q,
                                 float* out, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * attention of headkv_decode_attn, same arguments and results, with no
 * workspace.  A layer with fewer (batch x heads) than compute units splits
 * each head into chunks whose partial results headkv_decode_attn keeps in the
 * handle's workspace; this call keeps them in a static device array of
 * 4 MiB that the library holds on each GPU it runs on until the process ends
 * (HEADKV_ERR_CAPACITY if a layer's chunks need more: entries x head_dim x
 * 8 bytes).  It calls no hipMalloc, hipFree or allocating routine.  Every
 * call on one GPU shares that GPU's array (the current device's), so calls
 * that overlap on one GPU, on any streams or handles, race; calls ordered on
 * one stream do not. */
headkv_status headkv_decode_attn_noalloc(headkv_t h, int32_t layer, const uint16_t* q,
                                         float* out, void* stream);

/* Decode attention of layers [layer_begin, layer_end) in one launch, with the
 * results of headkv_decode_attn on each.  q, out: host arrays (indexed by
 * layer - layer_begin) of device pointers as for headkv_decode_attn.  For
 * callers that hold several layers' queries at once; a decoder whose next
 * layer needs this one's output calls headkv_decode_attn per layer.  At most
 * 64 layers; needs at least 256 (batch x heads) and HEADKV_ATTN_VARLEN
 * (HEADKV_ERR_UNSUPPORTED otherwise). */
headkv_status headkv_decode_attn_layers(headkv_t h, int32_t layer_begin, int32_t layer_end,
                                        const uint16_t* const* q, float* const* out,
                                        void* stream);

/* One whole decode step of `layer` in the fewest launches: the append of
 * headkv_append_and_evict (with its periodic update when due) followed by the
 * attention of headkv_decode_attn, with identical results.  Without an update
 * the append is fused into the attention kernel; with one, the append, the
 * update and the attention run in one launch when the layer's attention takes
 * one block per head with Eq. (6) scores, else in two.  Arguments as for those
 * two calls.  The grouping step t_g needs the separate calls
 * (HEADKV_ERR_STATE). */
headkv_status headkv_decode_step(headkv_t h, int32_t layer, int32_t step, const uint16_t* q,
                                 const uint16_t* k, const uint16_t* v, float* out,
                                 void* stream);

/* ---- Driver and measurement (not needed by a model, which calls the
 * per-layer entry points between its own kernels). ---- */

/* Runs headkv_decode_step for steps [step_begin, step_end) of every layer,
 * step by step and layer by layer, from one host call.  q, k, v: host arrays
 * of num_layers device pointers, each to [steps][B][H][d] bf16 with
 * step_stride elements between consecutive steps (a multiple of 8, so that
 * every step's rows stay 16-byte aligned); out: host array of
 * num_layers device pointers to [B][H][d] fp32, overwritten every step.
 * timing_every > 0: every step t with t % timing_every == 0 whose attention is
 * one kernel launch is timed with the kernel's own start/end timestamps (see
 * headkv_timing_reserve / headkv_timing_collect).  The range must not contain
 * the grouping step (HEADKV_ERR_STATE); stops at the first failing call. */
headkv_status headkv_run_steps(headkv_t h, int32_t step_begin, int32_t step_end,
                               const uint16_t* const* q, const uint16_t* const* k,
                               const uint16_t* const* v, int64_t step_stride,
                               float* const* out, int32_t timing_every, void* stream);

/* Creates events for `launches` timed launches (host call).  While reserved
 * events are left, every headkv_prefill_attn launch is timed as well. */
headkv_status headkv_timing_reserve(headkv_t h, int64_t launches);

/* Kinds of timed launches. */
#define HEADKV_TIMED_ATTN_APPEND 0 /* fused append + attention over the
                                      compressed cache (after grouping) */
#define HEADKV_TIMED_ATTN 1        /* attention after an update */
#define HEADKV_TIMED_UPDATE 2      /* append + periodic update */
#define HEADKV_TIMED_PREFILL 3     /* prefix store + causal prefix attention */
#define HEADKV_TIMED_ATTN_APPEND_DENSE 4 /* fused append + attention before
                                            grouping (full cache) */
#define HEADKV_TIMED_UPDATE_ATTN 5 /* append + periodic update + attention in
                                      one launch (one block per head of
                                      256 threads) */
#define HEADKV_TIMED_KINDS 6

/* Waits for the timed launches since the last collect and returns, per kind
 * (arrays of HEADKV_TIMED_KINDS), the sum of their kernel durations (ms), their
 * number and the sum of their algorithmic HBM bytes, plus the number of
 * launches that found no free event.  Algorithmic bytes: K/V of every attended
 * token, q and the output for attention; the appended row, its position and
 * the query-sum update for the append; positions, the history keys of
 * evicting global heads and at most M moved rows for the update; q, k, v of
 * the prefix read, its k, v stored and the fp32 output written for the
 * prefill. */
headkv_status headkv_timing_collect(headkv_t h, double* kernel_ms, int64_t* launches,
                                    double* alg_bytes, int64_t* dropped);

/* Parity export: mask[b][h][p] = 1 iff visual position p is retained
 * ([B][H][N] uint8, device) and count[b][h] = number retained ([B][H] int32,
 * device). */
headkv_status headkv_export_retained(headkv_t h, int32_t layer, uint8_t* mask,
                                     int32_t* count, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* headkv_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
