/*
 * CPU oracle for the STAR decode-rescheduling hot path: declarations.
 *
 * TEST INFRASTRUCTURE ONLY (see star_oracle.c).  This header belongs to the
 * oracle alone; the HIP library neither includes nor mirrors it.
 *
 * All pointers are host memory.  Matrices are row-major.  Functions return 0
 * on success and -1 on a malformed argument.
 */
#ifndef STAR_ORACLE_H
#define STAR_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { STAR_ORACLE_F32 = 0, STAR_ORACLE_BF16 = 1 };          /* input element type */
enum { STAR_ORACLE_RELU = 0, STAR_ORACLE_GELU = 1 };         /* hidden activation  */
enum { STAR_ORACLE_BAD_INST = 1, STAR_ORACLE_BAD_CUR = 2, STAR_ORACLE_BAD_REM = 4 };

/* Predictor head (Section 4.2, Eq. 1-2; length bins of Section 6.5).
 * hidden [B,d], w1 [m,d], w2 [nb,m] in `dtype` (bf16 as uint16 bits);
 * b1 [m], b2 [nb] fp32 or NULL; bin_values [nb] fp32.
 * expected [B] <- E = sum_j softmax(z2)_j v_j.
 * ema_alpha in [0,1]; 0 disables smoothing.  With smoothing, ema_state [B]
 * (fp64, caller-owned) is set to E when ema_init, else to a E + (1-a) state.
 * rem_len [B] (or NULL) <- clamp(round-half-even(smoothed E), 1, len_max).
 * z1_out [B,m] / z2_out [B,nb] (or NULL) receive the pre-activation and the
 * bin logits for inspection. */
int star_oracle_predict(int64_t B, int64_t d, int64_t m, int64_t nb, int dtype, int act,
                        const void* hidden, const void* w1, const float* b1,
                        const void* w2, const float* b2, const float* bin_values,
                        double ema_alpha, int ema_init, double* ema_state,
                        int64_t len_max, double* expected, int32_t* rem_len,
                        double* z1_out, double* z2_out);

/* The paper's regression head (Section 4.2, Eq. 2): a 4-layer ReLU MLP
 * d -> m1 -> m2 -> m3 -> 1 with optional biases b1..b3 (fp32 or NULL) and
 * output weights w4 [m3] fp32, scalar bias b4; W1 [m1,d], W2 [m2,m1],
 * W3 [m3,m2] in `dtype`.  Computes the rows listed in `rows` (n_rows of
 * them; NULL = all B rows); expected [q] <- y^ of rows[q]; EMA and
 * integerisation as star_oracle_predict (ema_state indexed like the rows
 * list); scale_out [q] (or NULL) <- sum_j |w4_j a3_j| + |b4|. */
int star_oracle_predict_mlp4(int64_t B, int64_t d, int64_t m1, int64_t m2, int64_t m3,
                             int dtype, const void* hidden, const void* w1, const float* b1,
                             const void* w2, const float* b2, const void* w3, const float* b3,
                             const float* w4, double b4, const int64_t* rows, int64_t n_rows,
                             double ema_alpha, int ema_init, double* ema_state, int64_t len_max,
                             double* expected, int32_t* rem_len, double* scale_out);

/* Load curves (Section 5.2, Eq. 4 and the worker-side summary of the
 * complexity analysis).  load [n,K]: load[i,k] = sum over decode steps
 * t in [k b, (k+1) b) of sum_{r in B_i, t < rem_r} (cur_r + t).
 * Requests with inst_of outside [0,n), cur_len < 1 or rem_len < 1 are
 * skipped; the OR of their STAR_ORACLE_BAD_* flags goes to *flags_out. */
int star_oracle_project_load(int64_t N, int64_t n, int64_t b, int64_t K,
                             const int32_t* cur_len, const int32_t* rem_len,
                             const int32_t* inst_of, int64_t* load, int32_t* flags_out);

/* Candidate scores [N,n] (Algorithm 1, best-feasible selection, with the
 * projected peak as the figure of merit): for t != inst(r), the maximum over
 * buckets of load[t] plus r's own bucketed curve; for t == inst(r), the
 * maximum of load[t].  Skipped requests get a row of -1. */
int star_oracle_score(int64_t N, int64_t n, int64_t b, int64_t K,
                      const int32_t* cur_len, const int32_t* rem_len, const int32_t* inst_of,
                      const int64_t* load, int64_t* scores);

/* Ranking of all migrations (t != inst(r)) by (score, r, t) ascending.
 * best_target[r] / best_score[r]: the smallest key of request r, or -1.
 * topk_*[q], q < top_k: the q-th smallest key, or -1 past the end.
 * Any output pointer may be NULL. */
int star_oracle_rank(int64_t N, int64_t n, const int32_t* cur_len, const int32_t* rem_len,
                     const int32_t* inst_of, const int64_t* scores, int64_t top_k,
                     int32_t* best_target, int64_t* best_score,
                     int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score);

/* Time-weighted variance change of every migration (Section 5.2, Eq. 3-4;
 * Algorithm 1's best-feasible selection with prediction).  beta [K] are the
 * bucket weights (16-bit fixed point; only their ratios matter).  For r on
 * s and t != s, gain[r,t] = (change of n^2 Phi) / (2n) when r's curve moves
 * from s to t, Phi = sum_k beta_k Var_i(load[i,k]); 0 for t == s and for
 * skipped requests.  gain is [N*n] 128-bit two's complement values stored as
 * (low, high) int64 pairs.  Returns -2 when the values could leave the
 * exactly representable range, -3 if a change is not a multiple of 2n. */
int star_oracle_score_variance(int64_t N, int64_t n, int64_t b, int64_t K,
                               const int32_t* cur_len, const int32_t* rem_len,
                               const int32_t* inst_of, const int64_t* load,
                               const uint16_t* beta, int64_t* gain);

/* Selection over those gains by (gain, r, t) ascending, t != inst(r):
 * best_target[r] / best_gain[r] (pairs): r's smallest key, or -1 / 0;
 * move[3] = (r, s, t) of the smallest key overall if its gain is negative,
 * else (-1, -1, -1), with its gain in move_gain[2] (0 when none). */
int star_oracle_select_variance(int64_t N, int64_t n, const int32_t* cur_len,
                                const int32_t* rem_len, const int32_t* inst_of,
                                const int64_t* gain, int32_t* best_target, int64_t* best_gain,
                                int32_t* move, int64_t* move_gain);

/* Algorithm 1 end to end, repeated: classification with threshold
 * theta = theta_num / theta_den, candidate filters (rem_len > min_rem;
 * memory check against mem_cap), best-feasible selection on the variance
 * gain, and execution, up to max_moves times.  inst_of is updated in place;
 * load [n,K] receives the final curves.  moves [3*max_moves] get (r, s, t)
 * per executed migration, move_gains [2*max_moves] their gains, *n_moves the
 * count.  u_mode 0: U = {current load < (1+theta) mean w} as printed;
 * 1: U = {w_i < (1-theta) mean w}.  mem_mode 0: N_t + rem_r <= mem_cap as
 * printed; 1: N_t + cur_r + rem_r <= mem_cap. */
int star_oracle_plan(int64_t N, int64_t n, int64_t b, int64_t K, const int32_t* cur_len,
                     const int32_t* rem_len, int32_t* inst_of, int64_t* load,
                     const uint16_t* beta, int64_t theta_num, int64_t theta_den, int u_mode,
                     int64_t min_rem, int64_t mem_cap, int mem_mode, int64_t max_moves,
                     int32_t* moves, int64_t* move_gains, int64_t* n_moves);

int star_oracle_abi_version(void);
int star_oracle_threads(void);
void star_oracle_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
