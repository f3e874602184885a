/*
 * CPU oracle for head-aware KV-cache compression (HeadKV, arXiv 2605.20600).
 *
 * TEST INFRASTRUCTURE ONLY.  Plain, slow fp64 scalar loops that state what the
 * compressed decode path computes, step by step, in the paper's order.  Only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark may call it;
 * the product library never links it and shares no code, header or table with
 * it.  Inputs are bf16 values converted exactly to double by the caller.
 *
 * Functions and the passages they follow:
 *   orc_attention      Eq. (1): o = softmax(q K^T / sqrt(d)) V, one query.
 *   orc_group_head     Sec. 4 Step 2 (head grouping): softmax of the current
 *                      query over the key cache, attention mass accumulated
 *                      backward from the newest token until tau is reached;
 *                      n* = the minimum count; local iff n* < local window.
 *   orc_budgets        Sec. 5.1 Implementation Details: global heads keep
 *                      floor(rho*N) visual tokens, local heads a small window
 *                      (two image rows); plus the caller-override and the
 *                      layer-total variants.
 *   orc_update         Eqs. (2)-(6): cache = [conditional | history | recent];
 *                      local heads drop the history (Eq. 3, sliding window);
 *                      global heads apply Stratified Token Eviction (Eqs. 4-6):
 *                      the history is split at floor(T*r_s) into long-range
 *                      (older) and near-range parts, each token is scored by
 *                      the mean raw logit of the past-P queries, and M/2 lowest
 *                      scores are evicted from each part.  A variant scores a
 *                      token by the attention weights those queries gave it.
 *   orc_run_head       One head through a whole generation: append every step,
 *                      update every P steps from the grouping step on (Sec. 4,
 *                      Efficient Cache Update), attend over prefix + retained.
 *
 * Error behaviour: functions returning int return 0 on success and a negative
 * value on invalid arguments; nothing aborts.
 */
#ifndef HEADKV_ORACLE_H
#define HEADKV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Eq. (1).  q: [d]; K, V: [L][d] row-major; out: [d].  L >= 1. */
int orc_attention(const double* q, const double* K, const double* V, int L, int d,
                  double* out);

/* Sec. 4 Step 2.  q: [d]; K: [L][d] in cache order (prefix, then visual tokens
 * oldest to newest; the newest is the current token).  Writes n* (1..L), the
 * label (1 = local), S(W_loc-1) = attention mass of the W_loc-1 newest tokens,
 * and the distance of the n* decision from tau:
 * min(tau - S(n*-1), S(n*) - tau). */
int orc_group_head(const double* q, const double* K, int L, int d, double tau,
                   int local_window, int32_t* n_star, int32_t* is_local,
                   double* mass_window, double* margin);

/* Budget modes. */
#define ORC_BUDGET_PAPER 0
#define ORC_BUDGET_OVERRIDE 1
#define ORC_BUDGET_TOTAL 2

/* Budgets of the H heads of one (input, layer).  labels: [H] (1 = local);
 * override: [H] or NULL; out: [H] visual-token budgets (recent window included,
 * the conditional prefix not counted). */
int orc_budgets(int mode, int H, const int32_t* labels, const int32_t* override_b,
                int N, int row_len, int recent_len, int rho_num, int rho_den,
                int32_t* out);

/* Scores of the global-head update (Eq. 6 and a variant). */
#define ORC_SCORE_MEAN_LOGIT 0 /* Eq. (6): mean raw logit of the past-P queries */
#define ORC_SCORE_ATTN_SUM 1   /* variant: each past-P query's attention weight
                                  on the token, over the cache that query
                                  attended (prefix + retained tokens up to its
                                  step), summed over the queries in step order */

/* One periodic update of one head.  ret: [*n_ret] retained visual positions in
 * ascending order, rewritten in place; Kvis: [N][d] visual keys by position;
 * qsum: [d] sum of the past-P queries, added in step order starting from 0.
 * u: index of this update (0 at the grouping step) -- an odd M puts its extra
 * eviction in the long-range part when u is odd, in the near-range part when
 * u is even.  Writes the number evicted and the smallest score gap between an
 * evicted and a kept token of the same part (+inf when no comparison arose). */
int orc_update(int32_t* ret, int32_t* n_ret, const double* Kvis, int d,
               const double* qsum, int budget, int is_local, int recent_len,
               int rs_num, int rs_den, int u, int32_t* n_evicted, double* min_gap);

/* The same with a score mode.  For ORC_SCORE_ATTN_SUM: Qwin [n_win][d] are the
 * queries of steps first_step .. first_step + n_win - 1 (the last of them the
 * current step) and Kc [C][d] the conditional keys; qsum is not used. */
int orc_update_ex(int32_t* ret, int32_t* n_ret, const double* Kvis, int d,
                  const double* qsum, int budget, int is_local, int recent_len,
                  int rs_num, int rs_den, int u, int score_mode, const double* Qwin,
                  int n_win, int first_step, const double* Kc, int C, int32_t* n_evicted,
                  double* min_gap);

/* A whole generation of one head.
 *   q, k, v: [N][d] visual tokens by step; kc, vc: [C][d] conditional tokens.
 *   t_g: grouping step (updates at t_g, t_g+P, ...); is_local, budget: the
 *   head's label and budget from steps t_g on.
 *   out: [N][d] attention output of every step, or NULL.
 *   snap_steps: [n_snap] steps after whose attention the retained set is
 *   recorded into snap_mask [n_snap][N] (1 = retained), or NULL.
 *   stats: [4] = {updates, tokens evicted, min score gap, unused}.
 *   score_mode: ORC_SCORE_* of the global-head updates. */
int orc_run_head(const double* q, const double* k, const double* v,
                 const double* kc, const double* vc, int C, int N, int d,
                 int t_g, int P, int is_local, int budget, int recent_len,
                 int rs_num, int rs_den, double* out, const int32_t* snap_steps,
                 int n_snap, uint8_t* snap_mask, double* stats, int score_mode);

#ifdef __cplusplus
}
#endif
#endif
