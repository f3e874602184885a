/*
 * CPU oracle for head-aware KV-cache compression -- TEST INFRASTRUCTURE ONLY.
 * See headkv_oracle.h for the contract and the passages each function follows.
 *
 * Built with -O2 -ffp-contract=off: every product and every sum is a separately
 * rounded IEEE fp64 operation, evaluated in the index order written below.
 */
#include "headkv_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* q . k summed over dims 0..d-1 in order. */
static double dot(const double* a, const double* b, int d) {
    double s = 0.0;
    for (int i = 0; i < d; ++i) s += a[i] * b[i];
    return s;
}

/* Eq. (1) over a cache given as row pointers. */
static void attention_rows(const double* q, const double* const* Krow,
                           const double* const* Vrow, int L, int d, double* out,
                           double* s /* scratch [L] */) {
    const double sd = sqrt((double)d);
    double m = -INFINITY;
    for (int j = 0; j < L; ++j) {
        s[j] = dot(q, Krow[j], d) / sd;
        if (s[j] > m) m = s[j];
    }
    double Z = 0.0;
    for (int j = 0; j < L; ++j) {
        s[j] = exp(s[j] - m);
        Z += s[j];
    }
    for (int i = 0; i < d; ++i) out[i] = 0.0;
    for (int j = 0; j < L; ++j) {
        const double a = s[j] / Z;
        for (int i = 0; i < d; ++i) out[i] += a * Vrow[j][i];
    }
}

int orc_attention(const double* q, const double* K, const double* V, int L, int d,
                  double* out) {
    if (!q || !K || !V || !out || L < 1 || d < 1) return -1;
    const double** kr = malloc(sizeof(double*) * (size_t)L);
    const double** vr = malloc(sizeof(double*) * (size_t)L);
    double* s = malloc(sizeof(double) * (size_t)L);
    if (!kr || !vr || !s) { free(kr); free(vr); free(s); return -2; }
    for (int j = 0; j < L; ++j) { kr[j] = K + (size_t)j * d; vr[j] = V + (size_t)j * d; }
    attention_rows(q, kr, vr, L, d, out, s);
    free(kr); free(vr); free(s);
    return 0;
}

int orc_group_head(const double* q, const double* K, int L, int d, double tau,
                   int local_window, int32_t* n_star, int32_t* is_local,
                   double* mass_window, double* margin) {
    if (!q || !K || L < 1 || d < 1 || !(tau > 0.0 && tau <= 1.0) || local_window < 1)
        return -1;
    double* a = malloc(sizeof(double) * (size_t)L);
    if (!a) return -2;
    /* attention weights of the current query over the whole key cache */
    const double sd = sqrt((double)d);
    double m = -INFINITY;
    for (int j = 0; j < L; ++j) {
        a[j] = dot(q, K + (size_t)j * d, d) / sd;
        if (a[j] > m) m = a[j];
    }
    double Z = 0.0;
    for (int j = 0; j < L; ++j) {
        a[j] = exp(a[j] - m);
        Z += a[j];
    }
    for (int j = 0; j < L; ++j) a[j] = a[j] / Z;
    /* accumulate backward from the current (newest) token */
    double S = 0.0, S_prev = 0.0, S_win = 0.0;
    int ns = -1;
    double mg = INFINITY;
    for (int n = 1; n <= L; ++n) {
        S_prev = S;
        S += a[L - n];
        if (n == local_window - 1) S_win = S;
        if (ns < 0 && S >= tau) {
            ns = n;
            const double lo = tau - S_prev, hi = S - tau;
            mg = lo < hi ? lo : hi;
        }
    }
    if (local_window - 1 > L) S_win = S;
    if (ns < 0) {               /* rounding left the total just below tau */
        ns = L;
        mg = tau - S;
    }
    free(a);
    if (n_star) *n_star = ns;
    if (is_local) *is_local = ns < local_window ? 1 : 0;
    if (mass_window) *mass_window = S_win;
    if (margin) *margin = mg;
    return 0;
}

int orc_budgets(int mode, int H, const int32_t* labels, const int32_t* override_b,
                int N, int row_len, int recent_len, int rho_num, int rho_den,
                int32_t* out) {
    if (H < 1 || !labels || !out || N < 1 || row_len < 1 || recent_len < 1) return -1;
    if (mode == ORC_BUDGET_OVERRIDE) {
        if (!override_b) return -1;
        for (int h = 0; h < H; ++h) {
            if (override_b[h] < 1 || override_b[h] > N) return -1;
            out[h] = override_b[h];
        }
        return 0;
    }
    if (rho_num < 1 || rho_den < 1 || rho_num > rho_den) return -1;
    const long long rhoN = (long long)N * rho_num / rho_den;   /* floor(rho * N) */
    const int b_local = recent_len < N ? recent_len : N;
    if (mode == ORC_BUDGET_PAPER) {
        int b_global = (int)(rhoN < 1 ? 1 : rhoN);
        for (int h = 0; h < H; ++h) out[h] = labels[h] ? b_local : b_global;
        return 0;
    }
    if (mode == ORC_BUDGET_TOTAL) {
        /* the layer's total visual budget floor(rho*N)*H is kept; local heads
         * take the window, global heads share the rest equally, in whole rows */
        int n_local = 0;
        for (int h = 0; h < H; ++h) n_local += labels[h] ? 1 : 0;
        const int n_global = H - n_local;
        long long rest = rhoN * H - (long long)n_local * b_local;
        long long per = n_global > 0 && rest > 0 ? rest / n_global : 0;
        long long b_global = per / row_len * row_len;
        if (b_global < b_local) b_global = b_local;
        if (b_global > N) b_global = N;
        for (int h = 0; h < H; ++h) out[h] = labels[h] ? b_local : (int32_t)b_global;
        return 0;
    }
    return -1;
}

/* candidates of one part with their scores, ordered by (score, position) */
typedef struct { double s; int32_t pos; } cand_t;

static int cand_cmp(const void* x, const void* y) {
    const cand_t* a = (const cand_t*)x;
    const cand_t* b = (const cand_t*)y;
    if (a->s < b->s) return -1;
    if (a->s > b->s) return 1;
    return (a->pos > b->pos) - (a->pos < b->pos);
}

static int int_cmp(const void* x, const void* y) {
    const int32_t a = *(const int32_t*)x, b = *(const int32_t*)y;
    return (a > b) - (a < b);
}

/* Attention weight of each history token (positions ret[0..T-1]) summed over
 * the window queries: query p (step first_step + p) attends over the cache it
 * saw at its step -- the prefix, then the retained visual tokens with position
 * <= its step, in position order -- with weights exp(l - max) / Z, Z summed in
 * that cache order; the weights are added to the scores query by query. */
static int window_attention_scores(const int32_t* ret, int n, int T, const double* Kvis,
                                   int d, const double* Qwin, int n_win, int first_step,
                                   const double* Kc, int C, double* score) {
    const double sd = sqrt((double)d);
    double* e = malloc(sizeof(double) * (size_t)(C + n));
    if (!e) return -2;
    for (int j = 0; j < T; ++j) score[j] = 0.0;
    for (int p = 0; p < n_win; ++p) {
        const double* qp = Qwin + (size_t)p * d;
        const int step = first_step + p;
        int nv = 0;  /* visible visual tokens: positions <= step (ret is sorted) */
        while (nv < n && ret[nv] <= step) ++nv;
        double m = -INFINITY;
        for (int j = 0; j < C + nv; ++j) {
            const double* kr = j < C ? Kc + (size_t)j * d : Kvis + (size_t)ret[j - C] * d;
            e[j] = dot(qp, kr, d) / sd;
            if (e[j] > m) m = e[j];
        }
        double Z = 0.0;
        for (int j = 0; j < C + nv; ++j) {
            e[j] = exp(e[j] - m);
            Z += e[j];
        }
        for (int j = 0; j < T && j < nv; ++j) score[j] += e[C + j] / Z;
    }
    free(e);
    return 0;
}

int orc_update(int32_t* ret, int32_t* n_ret, const double* Kvis, int d,
               const double* qsum, int budget, int is_local, int recent_len,
               int rs_num, int rs_den, int u, int32_t* n_evicted, double* min_gap) {
    return orc_update_ex(ret, n_ret, Kvis, d, qsum, budget, is_local, recent_len, rs_num,
                         rs_den, u, ORC_SCORE_MEAN_LOGIT, NULL, 0, 0, NULL, 0, n_evicted,
                         min_gap);
}

int orc_update_ex(int32_t* ret, int32_t* n_ret, const double* Kvis, int d,
                  const double* qsum, int budget, int is_local, int recent_len,
                  int rs_num, int rs_den, int u, int score_mode, const double* Qwin,
                  int n_win, int first_step, const double* Kc, int C, int32_t* n_evicted,
                  double* min_gap) {
    if (!ret || !n_ret || !Kvis || d < 1 || budget < 1 || recent_len < 1) return -1;
    if (score_mode != ORC_SCORE_MEAN_LOGIT && score_mode != ORC_SCORE_ATTN_SUM) return -1;
    if (!is_local && (rs_den < 1 || rs_num < 0 || rs_num > rs_den)) return -1;
    if (!is_local && score_mode == ORC_SCORE_MEAN_LOGIT && !qsum) return -1;
    if (!is_local && score_mode == ORC_SCORE_ATTN_SUM &&
        (!Qwin || n_win < 1 || first_step < 0 || C < 0 || (C > 0 && !Kc)))
        return -1;
    const int n = *n_ret;
    const int w_eff = recent_len < budget ? recent_len : budget;
    double gap = INFINITY;
    int evicted = 0;
    /* Eq. (2): history = retained tokens older than the recent window */
    const int T = n > w_eff ? n - w_eff : 0;
    const int keep = budget - w_eff;
    const int M = T > keep ? T - keep : 0;
    if (M > 0) {
        uint8_t* gone = calloc((size_t)T, 1);
        if (!gone) return -2;
        if (is_local) {
            /* Eq. (3): sliding window -- the oldest tokens leave */
            for (int j = 0; j < M; ++j) gone[j] = 1;
        } else {
            /* Eq. (5): long-range part = oldest floor(T*r_s) history tokens */
            const int n_long = (int)((long long)T * rs_num / rs_den);
            const int n_near = T - n_long;
            int m_long = (M + (u & 1)) >> 1;
            int m_near = M - m_long;
            if (m_long > n_long) { m_near += m_long - n_long; m_long = n_long; }
            if (m_near > n_near) { m_long += m_near - n_near; m_near = n_near; }
            /* Eq. (6): score = mean over the past-P queries of the raw logit;
             * 1/(P sqrt(d)) is a positive constant, so the order is that of
             * qsum . k.  The variant sums those queries' attention weights. */
            cand_t* c = malloc(sizeof(cand_t) * (size_t)T);
            double* ws = score_mode == ORC_SCORE_ATTN_SUM ? malloc(sizeof(double) * (size_t)T) : NULL;
            if (!c || (score_mode == ORC_SCORE_ATTN_SUM && !ws)) {
                free(c); free(ws); free(gone);
                return -2;
            }
            if (ws && window_attention_scores(ret, n, T, Kvis, d, Qwin, n_win, first_step, Kc, C,
                                              ws)) {
                free(c); free(ws); free(gone);
                return -2;
            }
            for (int j = 0; j < T; ++j) {
                c[j].pos = ret[j];
                c[j].s = ws ? ws[j] : dot(qsum, Kvis + (size_t)ret[j] * d, d);
            }
            free(ws);
            const int lo[2] = {0, n_long}, cnt[2] = {n_long, n_near}, mm[2] = {m_long, m_near};
            for (int part = 0; part < 2; ++part) {
                if (mm[part] == 0) continue;
                cand_t* cp = c + lo[part];
                qsort(cp, (size_t)cnt[part], sizeof(cand_t), cand_cmp);
                if (mm[part] < cnt[part]) {
                    const double g = cp[mm[part]].s - cp[mm[part] - 1].s;
                    if (g < gap) gap = g;
                }
                for (int j = 0; j < mm[part]; ++j) {
                    /* position -> index in the history (history is sorted) */
                    int32_t* hit = bsearch(&cp[j].pos, ret, (size_t)T, sizeof(int32_t), int_cmp);
                    gone[hit - ret] = 1;
                }
            }
            free(c);
        }
        int o = 0;
        for (int j = 0; j < n; ++j) {
            if (j < T && gone[j]) { ++evicted; continue; }
            ret[o++] = ret[j];
        }
        *n_ret = o;
        free(gone);
    }
    if (n_evicted) *n_evicted = evicted;
    if (min_gap) *min_gap = gap;
    return 0;
}

int orc_run_head(const double* q, const double* k, const double* v,
                 const double* kc, const double* vc, int C, int N, int d,
                 int t_g, int P, int is_local, int budget, int recent_len,
                 int rs_num, int rs_den, double* out, const int32_t* snap_steps,
                 int n_snap, uint8_t* snap_mask, double* stats, int score_mode) {
    if (!q || !k || !v || C < 0 || (C > 0 && (!kc || !vc)) || N < 1 || d < 1 ||
        t_g < 0 || P < 1 || budget < 1 || recent_len < 1 || n_snap < 0 ||
        (n_snap > 0 && (!snap_steps || !snap_mask)))
        return -1;
    int32_t* ret = malloc(sizeof(int32_t) * (size_t)N);
    const double** kr = malloc(sizeof(double*) * (size_t)(C + N));
    const double** vr = malloc(sizeof(double*) * (size_t)(C + N));
    double* s = malloc(sizeof(double) * (size_t)(C + N));
    double* qsum = malloc(sizeof(double) * (size_t)d);
    if (!ret || !kr || !vr || !s || !qsum) {
        free(ret); free(kr); free(vr); free(s); free(qsum);
        return -2;
    }
    int32_t n_ret = 0;
    int updates = 0, evicted_total = 0;
    double gap_min = INFINITY;
    for (int j = 0; j < C; ++j) { kr[j] = kc + (size_t)j * d; vr[j] = vc + (size_t)j * d; }
    for (int t = 0; t < N; ++t) {
        ret[n_ret++] = t;                       /* K <- [K, k_t], V <- [V, v_t] */
        if (t >= t_g && (t - t_g) % P == 0) {   /* buffer of P tokens is full */
            const int u = (t - t_g) / P;
            const int p0 = t - P + 1 > 0 ? t - P + 1 : 0;
            for (int i = 0; i < d; ++i) qsum[i] = 0.0;
            for (int p = p0; p <= t; ++p)
                for (int i = 0; i < d; ++i) qsum[i] += q[(size_t)p * d + i];
            int32_t ev = 0;
            double g = INFINITY;
            int rc = orc_update_ex(ret, &n_ret, k, d, qsum, budget, is_local, recent_len,
                                   rs_num, rs_den, u, score_mode, q + (size_t)p0 * d, t - p0 + 1,
                                   p0, kc, C, &ev, &g);
            if (rc) { free(ret); free(kr); free(vr); free(s); free(qsum); return rc; }
            ++updates;
            evicted_total += ev;
            if (g < gap_min) gap_min = g;
        }
        if (out) {
            for (int j = 0; j < n_ret; ++j) {
                kr[C + j] = k + (size_t)ret[j] * d;
                vr[C + j] = v + (size_t)ret[j] * d;
            }
            attention_rows(q + (size_t)t * d, kr, vr, C + n_ret, d, out + (size_t)t * d, s);
        }
        for (int i = 0; i < n_snap; ++i) {
            if (snap_steps[i] != t) continue;
            uint8_t* mrow = snap_mask + (size_t)i * N;
            memset(mrow, 0, (size_t)N);
            for (int j = 0; j < n_ret; ++j) mrow[ret[j]] = 1;
        }
    }
    if (stats) {
        stats[0] = updates;
        stats[1] = evicted_total;
        stats[2] = gap_min;
        stats[3] = 0.0;
    }
    free(ret); free(kr); free(vr); free(s); free(qsum);
    return 0;
}
