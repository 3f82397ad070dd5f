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

int star_oracle_abi_version(void) { return 1; }

/* Threads an OpenMP parallel region of the oracle uses (1 without OpenMP). */
int star_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
