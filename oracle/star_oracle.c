/*
 * CPU oracle for the STAR decode-rescheduling hot path (arXiv 2510.13668).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, deliberately naive
 * restatement of what the hot path computes, used to check the HIP library.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  It shares no code, header, table or helper with the HIP
 * path.
 *
 * Arithmetic: fp64 for the predictor (operands are widened exactly from the
 * fp32 / bf16 input bits), int64 for every load and score.  Loops follow the
 * definitions directly: a triple loop for each matrix product, per-decode-step
 * summation for the load curves, a direct maximum over all buckets for each
 * migration candidate, and a full sort for the ranking.
 *
 * Symbols:
 *   N(r)     current tokens of request r  (cur_len; Section 5.2, problem
 *            formulation)
 *   N^(r)    predicted remaining length   (rem_len; same passage)
 *   B_i      requests on instance i       (inst_of)
 *   N^_i(B_{i,t}) predicted token load of instance i at future step t
 *            (Eq. 4); request r holds N(r)+t tokens while t < N^(r).
 */
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "star_oracle.h"

/* ---------------------------------------------------------------------- */
/* input widening                                                          */
/* ---------------------------------------------------------------------- */
static double widen(const void* base, int64_t idx, int dtype) {
    if (dtype == STAR_ORACLE_F32) return (double)((const float*)base)[idx];
    uint32_t bits = (uint32_t)((const uint16_t*)base)[idx] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* phi of Eq. 2 (ReLU) or the erf form of GELU: x * Phi(x). */
static double activation(double x, int act) {
    if (act == STAR_ORACLE_RELU) return x > 0.0 ? x : 0.0;
    return 0.5 * x * (1.0 + erf(x / sqrt(2.0)));
}

/* ---------------------------------------------------------------------- */
/* (a) predictor: Eq. 1 realised as a distribution over length bins         */
/* ---------------------------------------------------------------------- */
int star_oracle_predict(int64_t B, int64_t d, int64_t m, int64_t nb, int dtype, int act,
                        const void* hidden, const void* w1, const float* b1,
                        const void* w2, const float* b2, const float* bin_values,
                        double ema_alpha, int ema_init, double* ema_state,
                        int64_t len_max, double* expected, int32_t* rem_len,
                        double* z1_out, double* z2_out) {
    if (B < 0 || d < 1 || m < 1 || nb < 1 || len_max < 1) return -1;
    if (ema_alpha < 0.0 || ema_alpha > 1.0) return -1;
    if (ema_alpha > 0.0 && ema_state == NULL) return -1;

    /* widen the weights once: exact fp32/bf16 -> fp64 */
    double* W1 = (double*)malloc(sizeof(double) * (size_t)(m * d));
    double* W2 = (double*)malloc(sizeof(double) * (size_t)(nb * m));
    if (!W1 || !W2) { free(W1); free(W2); return -1; }
    for (int64_t e = 0; e < m * d; ++e) W1[e] = widen(w1, e, dtype);
    for (int64_t e = 0; e < nb * m; ++e) W2[e] = widen(w2, e, dtype);

    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < B; ++r) {
        double* h = (double*)malloc(sizeof(double) * (size_t)d);
        double* a1 = (double*)malloc(sizeof(double) * (size_t)m);
        double* z2 = (double*)malloc(sizeof(double) * (size_t)nb);
        for (int64_t k = 0; k < d; ++k) h[k] = widen(hidden, r * d + k, dtype);

        /* hidden layer: a1 = phi(W1 h + b1)  (Eq. 2, first factor) */
        for (int64_t u = 0; u < m; ++u) {
            double acc = 0.0;
            for (int64_t k = 0; k < d; ++k) acc += h[k] * W1[u * d + k];
            if (b1) acc += (double)b1[u];
            if (z1_out) z1_out[r * m + u] = acc;
            a1[u] = activation(acc, act);
        }
        /* bin logits: z2 = W2 a1 + b2 */
        for (int64_t j = 0; j < nb; ++j) {
            double acc = 0.0;
            for (int64_t u = 0; u < m; ++u) acc += a1[u] * W2[j * m + u];
            if (b2) acc += (double)b2[j];
            z2[j] = acc;
            if (z2_out) z2_out[r * nb + j] = acc;
        }
        /* p = softmax(z2); E = sum_j p_j v_j  (mean of p_theta(Y|S)) */
        double zmax = z2[0];
        for (int64_t j = 1; j < nb; ++j) if (z2[j] > zmax) zmax = z2[j];
        double den = 0.0, num = 0.0;
        for (int64_t j = 0; j < nb; ++j) {
            double e = exp(z2[j] - zmax);
            den += e;
            num += e * (double)bin_values[j];
        }
        double E = num / den;
        expected[r] = E;

        /* continuous prediction, smoothed across steps */
        double y = E;
        if (ema_alpha > 0.0) {
            y = ema_init ? E : ema_alpha * E + (1.0 - ema_alpha) * ema_state[r];
            ema_state[r] = y;
        }
        if (rem_len) {
            double q = nearbyint(y);             /* ties to even (default mode) */
            if (q < 1.0) q = 1.0;
            if (q > (double)len_max) q = (double)len_max;
            rem_len[r] = (int32_t)q;
        }
        free(h);
        free(a1);
        free(z2);
    }
    free(W1);
    free(W2);
    return 0;
}

/* ---------------------------------------------------------------------- */
/* request validity (shared rule for (b) and (c))                          */
/* ---------------------------------------------------------------------- */
static int request_flags(int64_t r, int64_t n, const int32_t* cur, const int32_t* rem,
                         const int32_t* inst) {
    int f = 0;
    if (inst[r] < 0 || (int64_t)inst[r] >= n) f |= STAR_ORACLE_BAD_INST;
    if (cur[r] < 1) f |= STAR_ORACLE_BAD_CUR;
    if (rem[r] < 1) f |= STAR_ORACLE_BAD_REM;
    return f;
}

/* ---------------------------------------------------------------------- */
/* (f3) the paper's regression head: a 4-layer ReLU MLP with scalar output */
/* ---------------------------------------------------------------------- */
/* y^ = w4 . phi(W3 phi(W2 phi(W1 h + b1) + b2) + b3) + b4 (Section 4.2,
 * Eq. 2, biases optional), phi = ReLU; then the same EMA and integerisation
 * as the binned head.  Only the rows listed in `rows` (or all when rows is
 * NULL) are computed; outputs are indexed like the rows list.  scale_out
 * (or NULL) receives sum_j |w4_j a3_j| + |b4| per row, the magnitude the
 * result's rounding error is relative to. */
int star_oracle_predict_mlp4(int64_t B, int64_t d, int64_t m1, int64_t m2, int64_t m3,
                             int dtype, const void* hidden, const void* w1, const float* b1,
                             const void* w2, const float* b2, const void* w3, const float* b3,
                             const float* w4, double b4, const int64_t* rows, int64_t n_rows,
                             double ema_alpha, int ema_init, double* ema_state, int64_t len_max,
                             double* expected, int32_t* rem_len, double* scale_out) {
    if (B < 0 || d < 1 || m1 < 1 || m2 < 1 || m3 < 1 || len_max < 1) return -1;
    const int64_t R = rows ? n_rows : B;
    int bad = 0;
    #pragma omp parallel for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t q = 0; q < R; ++q) {
        const int64_t b = rows ? rows[q] : q;
        if (b < 0 || b >= B) { bad = 1; continue; }
        double* a1 = (double*)malloc(sizeof(double) * (size_t)m1);
        double* a2 = (double*)malloc(sizeof(double) * (size_t)m2);
        double* a3 = (double*)malloc(sizeof(double) * (size_t)m3);
        for (int64_t j = 0; j < m1; ++j) {
            double z = b1 ? (double)b1[j] : 0.0;
            for (int64_t k = 0; k < d; ++k)
                z += widen(hidden, b * d + k, dtype) * widen(w1, j * d + k, dtype);
            a1[j] = activation(z, STAR_ORACLE_RELU);
        }
        for (int64_t j = 0; j < m2; ++j) {
            double z = b2 ? (double)b2[j] : 0.0;
            for (int64_t k = 0; k < m1; ++k) z += a1[k] * widen(w2, j * m1 + k, dtype);
            a2[j] = activation(z, STAR_ORACLE_RELU);
        }
        double y = b4, scale = fabs(b4);
        for (int64_t j = 0; j < m3; ++j) {
            double z = b3 ? (double)b3[j] : 0.0;
            for (int64_t k = 0; k < m2; ++k) z += a2[k] * widen(w3, j * m2 + k, dtype);
            a3[j] = activation(z, STAR_ORACLE_RELU);
            y += (double)w4[j] * a3[j];
            scale += fabs((double)w4[j] * a3[j]);
        }
        expected[q] = y;
        if (scale_out) scale_out[q] = scale;
        double yv = y;
        if (ema_alpha > 0.0) {
            yv = ema_init ? y : ema_alpha * y + (1.0 - ema_alpha) * ema_state[q];
            ema_state[q] = yv;
        }
        if (rem_len) {
            double r = nearbyint(yv);
            if (!(r >= 1.0)) r = 1.0;
            if (r > (double)len_max) r = (double)len_max;
            rem_len[q] = (int32_t)r;
        }
        free(a1);
        free(a2);
        free(a3);
    }
    return bad ? -1 : 0;
}

/* ---------------------------------------------------------------------- */
/* (b) predicted per-instance load curve, by per-step summation            */
/* ---------------------------------------------------------------------- */
int star_oracle_project_load(int64_t N, int64_t n, int64_t b, int64_t K,
                             const int32_t* cur, const int32_t* rem, const int32_t* inst,
                             int64_t* load, int32_t* flags_out) {
    if (N < 0 || n < 1 || b < 1 || K < 1) return -1;
    const int64_t H = b * K;
    int flags = 0;
    for (int64_t r = 0; r < N; ++r) flags |= request_flags(r, n, cur, rem, inst);
    if (flags_out) *flags_out = flags;

    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < n; ++i) {
        int64_t* step = (int64_t*)calloc((size_t)H, sizeof(int64_t));
        for (int64_t r = 0; r < N; ++r) {
            if (request_flags(r, n, cur, rem, inst) || inst[r] != i) continue;
            for (int64_t t = 0; t < H && t < (int64_t)rem[r]; ++t)
                step[t] += (int64_t)cur[r] + t;          /* N(r) + t tokens at step t */
        }
        for (int64_t k = 0; k < K; ++k) {
            int64_t s = 0;
            for (int64_t t = k * b; t < (k + 1) * b; ++t) s += step[t];
            load[i * K + k] = s;
        }
        free(step);
    }
    return 0;
}

/* ---------------------------------------------------------------------- */
/* (c1) every request -> instance candidate, scored by the projected peak   */
/* ---------------------------------------------------------------------- */
int star_oracle_score(int64_t N, int64_t n, int64_t b, int64_t K,
                      const int32_t* cur, const int32_t* rem, const int32_t* inst,
                      const int64_t* load, int64_t* scores) {
    if (N < 0 || n < 1 || b < 1 || K < 1) return -1;
    const int64_t H = b * K;

    #pragma omp parallel for schedule(dynamic, 16)
    for (int64_t r = 0; r < N; ++r) {
        if (request_flags(r, n, cur, rem, inst)) {
            for (int64_t t = 0; t < n; ++t) scores[r * n + t] = -1;
            continue;
        }
        /* r's own bucketed occupancy curve, one decode step at a time */
        int64_t* own = (int64_t*)calloc((size_t)K, sizeof(int64_t));
        for (int64_t t = 0; t < H && t < (int64_t)rem[r]; ++t)
            own[t / b] += (int64_t)cur[r] + t;
        for (int64_t t = 0; t < n; ++t) {
            const int64_t* L = load + t * K;
            int64_t best = INT64_MIN;
            for (int64_t k = 0; k < K; ++k) {
                /* staying put: r is already counted in its own instance's curve */
                int64_t v = (t == inst[r]) ? L[k] : L[k] + own[k];
                if (v > best) best = v;
            }
            scores[r * n + t] = best;
        }
        free(own);
    }
    return 0;
}

/* ---------------------------------------------------------------------- */
/* (c2) ranking: total order on (score, request, target), ascending         */
/* ---------------------------------------------------------------------- */
typedef struct { int64_t s; int64_t r; int64_t t; } triple;

static int cmp_triple(const void* a, const void* b) {
    const triple* x = (const triple*)a;
    const triple* y = (const triple*)b;
    if (x->s != y->s) return x->s < y->s ? -1 : 1;
    if (x->r != y->r) return x->r < y->r ? -1 : 1;
    if (x->t != y->t) return x->t < y->t ? -1 : 1;
    return 0;
}

int star_oracle_rank(int64_t N, int64_t n, const int32_t* cur, const int32_t* rem,
                     const int32_t* inst, const int64_t* scores, int64_t top_k,
                     int32_t* best_target, int64_t* best_score,
                     int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score) {
    if (N < 0 || n < 1 || top_k < 0) return -1;
    int64_t cap = N * (n - 1);
    triple* all = (triple*)malloc(sizeof(triple) * (size_t)(cap > 0 ? cap : 1));
    int64_t cnt = 0;
    for (int64_t r = 0; r < N; ++r) {
        if (request_flags(r, n, cur, rem, inst)) continue;
        for (int64_t t = 0; t < n; ++t) {
            if (t == inst[r]) continue;           /* staying is not a migration */
            all[cnt].s = scores[r * n + t];
            all[cnt].r = r;
            all[cnt].t = t;
            ++cnt;
        }
    }
    qsort(all, (size_t)cnt, sizeof(triple), cmp_triple);

    if (best_target || best_score) {
        for (int64_t r = 0; r < N; ++r) {
            if (best_target) best_target[r] = -1;
            if (best_score) best_score[r] = -1;
        }
        /* sorted order visits each request's smallest key first */
        for (int64_t e = cnt - 1; e >= 0; --e) {
            if (best_target) best_target[all[e].r] = (int32_t)all[e].t;
            if (best_score) best_score[all[e].r] = all[e].s;
        }
    }
    for (int64_t q = 0; q < top_k; ++q) {
        int have = q < cnt;
        if (topk_req) topk_req[q] = have ? (int32_t)all[q].r : -1;
        if (topk_tgt) topk_tgt[q] = have ? (int32_t)all[q].t : -1;
        if (topk_score) topk_score[q] = have ? all[q].s : -1;
    }
    free(all);
    return 0;
}

/* ---------------------------------------------------------------------- */
/* (f1) time-weighted variance change of each migration                    */
/* ---------------------------------------------------------------------- */
/* Section 5.2 states the objective as the variance of the instances' token
 * loads now plus a beta-weighted sum of the variances of their predicted
 * loads at future steps (Eq. 3-4).  Over bucketed curves this is
 *     Phi = sum_k beta_k Var_i(L_i[k]),   Var = population variance over i.
 * n^2 Var_k = n sum_i L_i[k]^2 - (sum_i L_i[k])^2 is an integer, so
 * n^2 Phi is an integer; a migration's change of n^2 Phi is always a
 * multiple of 2n, and the oracle reports gain = change / (2n), i.e.
 * (n/2) times the change of Phi (negative = the variance falls).
 *
 * Arithmetic: 128-bit two's complement.  Sums, differences and products are
 * taken modulo 2^128 (unsigned __int128) and read back as signed, which is
 * exact whenever the final value lies in (-2^127, 2^127); the function
 * refuses inputs whose bound (from the actual curves) exceeds 2^125. */
typedef unsigned __int128 u128;
typedef __int128 s128;

/* n^2 Var of one bucket over the n instance values v[0..n) */
static u128 n2_var(const int64_t* v, int64_t n) {
    u128 sum = 0, sq = 0;
    for (int64_t i = 0; i < n; ++i) {
        sum += (u128)(s128)v[i];
        sq += (u128)((s128)v[i] * (s128)v[i]);
    }
    return (u128)n * sq - sum * sum;
}

/* r's own bucketed curve, one decode step at a time (as in the scores) */
static void own_curve(int64_t b, int64_t K, int32_t cur, int32_t rem, int64_t* own) {
    const int64_t H = b * K;
    for (int64_t k = 0; k < K; ++k) own[k] = 0;
    for (int64_t t = 0; t < H && t < (int64_t)rem; ++t) own[t / b] += (int64_t)cur + t;
}

/* |change of n^2 Phi| <= 2n beta_max sum_k R_k (R_k + 2 max|L|) for any r;
 * returns 0 when every candidate of this round stays below 2^125. */
static int variance_in_range(int64_t N, int64_t n, int64_t b, int64_t K, const int32_t* cur,
                             const int32_t* rem, const int32_t* inst, const int64_t* load,
                             const uint16_t* beta) {
    long double lmax = 0, bmax = 0;
    for (int64_t e = 0; e < n * K; ++e) {
        long double a = fabsl((long double)load[e]);
        if (a > lmax) lmax = a;
    }
    for (int64_t k = 0; k < K; ++k)
        if ((long double)beta[k] > bmax) bmax = (long double)beta[k];
    int64_t* own = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    long double worst = 0;
    for (int64_t r = 0; r < N; ++r) {
        if (request_flags(r, n, cur, rem, inst)) continue;
        own_curve(b, K, cur[r], rem[r], own);
        long double acc = 0;
        for (int64_t k = 0; k < K; ++k)
            acc += (long double)own[k] * ((long double)own[k] + 2.0L * lmax);
        if (acc > worst) worst = acc;
    }
    free(own);
    return 2.0L * (long double)n * bmax * worst < ldexpl(1.0L, 125) ? 0 : -1;
}

/* change of n^2 Phi when r (on s, own curve `own`) moves to t: the full
 * weighted variance of the moved curves minus that of the current ones */
static s128 phi_change(int64_t n, int64_t K, const int64_t* load, const uint16_t* beta,
                       int64_t s, int64_t t, const int64_t* own, int64_t* before,
                       int64_t* after) {
    u128 total = 0;
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t i = 0; i < n; ++i) {
            before[i] = load[i * K + k];
            after[i] = load[i * K + k];
        }
        after[s] -= own[k];
        after[t] += own[k];
        total += (u128)beta[k] * (n2_var(after, n) - n2_var(before, n));
    }
    return (s128)total;
}

int star_oracle_score_variance(int64_t N, int64_t n, int64_t b, int64_t K,
                               const int32_t* cur, const int32_t* rem, const int32_t* inst,
                               const int64_t* load, const uint16_t* beta, int64_t* gain) {
    if (N < 0 || n < 1 || b < 1 || K < 1) return -1;
    if (variance_in_range(N, n, b, K, cur, rem, inst, load, beta)) return -2;
    int bad = 0;

    #pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
    for (int64_t r = 0; r < N; ++r) {
        int64_t* own = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
        int64_t* before = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
        int64_t* after = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
        const int valid = request_flags(r, n, cur, rem, inst) == 0;
        if (valid) own_curve(b, K, cur[r], rem[r], own);
        for (int64_t t = 0; t < n; ++t) {
            s128 g = 0;                           /* staying put changes nothing */
            if (valid && t != inst[r]) {
                s128 d = phi_change(n, K, load, beta, inst[r], t, own, before, after);
                if (d % (2 * n) != 0) bad = 1;    /* impossible for consistent curves */
                g = d / (2 * n);
            }
            gain[2 * (r * n + t)] = (int64_t)(uint64_t)(u128)g;
            gain[2 * (r * n + t) + 1] = (int64_t)(g >> 64);
        }
        free(own);
        free(before);
        free(after);
    }
    return bad ? -3 : 0;
}

/* ---------------------------------------------------------------------- */
/* (f1) best target per request and the best feasible migration            */
/* ---------------------------------------------------------------------- */
typedef struct { s128 g; int64_t r; int64_t t; } vtriple;

static int cmp_vtriple(const void* a, const void* b) {
    const vtriple* x = (const vtriple*)a;
    const vtriple* y = (const vtriple*)b;
    if (x->g != y->g) return x->g < y->g ? -1 : 1;
    if (x->r != y->r) return x->r < y->r ? -1 : 1;
    if (x->t != y->t) return x->t < y->t ? -1 : 1;
    return 0;
}

static s128 read_gain(const int64_t* gain, int64_t e) {
    return (s128)(((u128)(uint64_t)gain[2 * e + 1] << 64) | (u128)(uint64_t)gain[2 * e]);
}

static void write_gain(int64_t* out, s128 g) {
    out[0] = (int64_t)(uint64_t)(u128)g;
    out[1] = (int64_t)(g >> 64);
}

int star_oracle_select_variance(int64_t N, int64_t n, const int32_t* cur, const int32_t* rem,
                                const int32_t* inst, const int64_t* gain,
                                int32_t* best_target, int64_t* best_gain, int32_t* move,
                                int64_t* move_gain) {
    if (N < 0 || n < 1) return -1;
    int64_t cap = N * (n - 1);
    vtriple* all = (vtriple*)malloc(sizeof(vtriple) * (size_t)(cap > 0 ? cap : 1));
    int64_t cnt = 0;
    for (int64_t r = 0; r < N; ++r) {
        if (request_flags(r, n, cur, rem, inst)) continue;
        for (int64_t t = 0; t < n; ++t) {
            if (t == inst[r]) continue;
            all[cnt].g = read_gain(gain, r * n + t);
            all[cnt].r = r;
            all[cnt].t = t;
            ++cnt;
        }
    }
    qsort(all, (size_t)cnt, sizeof(vtriple), cmp_vtriple);
    for (int64_t r = 0; r < N; ++r) {
        if (best_target) best_target[r] = -1;
        if (best_gain) write_gain(best_gain + 2 * r, 0);
    }
    for (int64_t e = cnt - 1; e >= 0; --e) {
        if (best_target) best_target[all[e].r] = (int32_t)all[e].t;
        if (best_gain) write_gain(best_gain + 2 * all[e].r, all[e].g);
    }
    /* the best feasible migration: largest reduction, taken only if it
     * reduces the objective at all (the running maximum starts at zero) */
    if (move) {
        const int take = cnt > 0 && all[0].g < 0;
        move[0] = take ? (int32_t)all[0].r : -1;
        move[1] = take ? inst[all[0].r] : -1;
        move[2] = take ? (int32_t)all[0].t : -1;
        if (move_gain) write_gain(move_gain, take ? all[0].g : 0);
    }
    free(all);
    return 0;
}

/* ---------------------------------------------------------------------- */
/* (f2) Algorithm 1 end to end, one migration per pass, repeated           */
/* ---------------------------------------------------------------------- */
/* Each pass is one scheduler interval with no decode progress in between:
 *   classification: w_i = sum_k beta_k L_i[k]; mean w = (1/n) sum_i w_i;
 *     O = {i : w_i > (1 + theta) mean w};
 *     U = {i : N_i(B_i) < (1 + theta) mean w} (u_mode 0, as printed), or
 *         {i : w_i < (1 - theta) mean w}      (u_mode 1);
 *     theta = theta_num / theta_den, all comparisons cross-multiplied;
 *   enumeration: (r, s, t) with s in O, t in U, t != s, r on s valid,
 *     rem_r > min_rem, and N_t(B_t) + rem_r (mem_mode 0, as printed) or
 *     N_t(B_t) + cur_r + rem_r (mem_mode 1) <= mem_cap;
 *   selection: the candidate with the smallest (gain, r, t) among gain < 0;
 *   execution: inst_of[r] = t, and every curve is projected again from
 *     scratch by per-step summation.
 * Stops after max_moves passes, when O is empty, or when no candidate
 * lowers the objective. */
int star_oracle_plan(int64_t N, int64_t n, int64_t b, int64_t K, const int32_t* cur,
                     const int32_t* rem, int32_t* inst, int64_t* load, const uint16_t* beta,
                     int64_t theta_num, int64_t theta_den, int u_mode, int64_t min_rem,
                     int64_t mem_cap, int mem_mode, int64_t max_moves, int32_t* moves,
                     int64_t* move_gains, int64_t* n_moves) {
    if (N < 0 || n < 1 || b < 1 || K < 1 || theta_num < 0 || theta_den < 1 || max_moves < 0)
        return -1;
    if (u_mode != 0 && u_mode != 1) return -1;
    if (mem_mode != 0 && mem_mode != 1) return -1;
    int32_t flags = 0;
    if (star_oracle_project_load(N, n, b, K, cur, rem, inst, load, &flags)) return -1;
    int64_t* own = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    int64_t* before = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
    int64_t* after = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
    s128* w = (s128*)malloc(sizeof(s128) * (size_t)n);
    int64_t* now = (int64_t*)malloc(sizeof(int64_t) * (size_t)n);
    char* over = (char*)malloc((size_t)n);
    char* under = (char*)malloc((size_t)n);
    int rc = 0;
    int64_t done = 0;
    while (done < max_moves) {
        if (variance_in_range(N, n, b, K, cur, rem, inst, load, beta)) { rc = -2; break; }
        /* phase 1: classification */
        s128 wsum = 0;
        for (int64_t i = 0; i < n; ++i) {
            w[i] = 0;
            for (int64_t k = 0; k < K; ++k) w[i] += (s128)beta[k] * (s128)load[i * K + k];
            wsum += w[i];
            now[i] = 0;
        }
        for (int64_t r = 0; r < N; ++r)
            if (!request_flags(r, n, cur, rem, inst)) now[inst[r]] += cur[r];
        int any_over = 0;
        for (int64_t i = 0; i < n; ++i) {
            /* x > (1 + theta) mean  <=>  n den x > (den + num) sum */
            over[i] = (s128)n * theta_den * w[i] > (s128)(theta_den + theta_num) * wsum;
            if (u_mode == 0)
                under[i] = (s128)n * theta_den * now[i] < (s128)(theta_den + theta_num) * wsum;
            else
                under[i] = (s128)n * theta_den * w[i] < (s128)(theta_den - theta_num) * wsum;
            any_over |= over[i];
        }
        if (!any_over) break;
        /* phases 2-3: enumerate the filtered candidates, keep the best */
        int have = 0;
        s128 bg = 0;
        int64_t br = -1, bt = -1;
        for (int64_t r = 0; r < N; ++r) {
            if (request_flags(r, n, cur, rem, inst)) continue;
            const int64_t s = inst[r];
            if (!over[s] || (int64_t)rem[r] <= min_rem) continue;
            own_curve(b, K, cur[r], rem[r], own);
            for (int64_t t = 0; t < n; ++t) {
                if (t == s || !under[t]) continue;
                const int64_t need = now[t] + rem[r] + (mem_mode ? (int64_t)cur[r] : 0);
                if (need > mem_cap) continue;
                s128 d = phi_change(n, K, load, beta, s, t, own, before, after);
                if (d % (2 * n) != 0) { rc = -3; break; }
                s128 g = d / (2 * n);
                /* candidates arrive in (r, t) order: strict < keeps the first */
                if (g < 0 && (!have || g < bg)) { have = 1; bg = g; br = r; bt = t; }
            }
            if (rc) break;
        }
        if (rc || !have) break;
        moves[3 * done] = (int32_t)br;
        moves[3 * done + 1] = inst[br];
        moves[3 * done + 2] = (int32_t)bt;
        write_gain(move_gains + 2 * done, bg);
        inst[br] = (int32_t)bt;
        ++done;
        star_oracle_project_load(N, n, b, K, cur, rem, inst, load, &flags);
    }
    *n_moves = done;
    free(own); free(before); free(after); free(w); free(now); free(over); free(under);
    return rc;
}

int star_oracle_abi_version(void) { return 1; }

/* Threads an OpenMP parallel region of the oracle uses (1 without OpenMP). */
int star_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads later parallel regions use (n >= 1); a timing control only, the
 * results do not depend on it. */
void star_oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
