/*
 * libstar -- MI355X (gfx950) hot path of STAR's decode-phase rescheduler
 * (arXiv 2510.13668): remaining-length prediction, load projection and
 * migration-candidate scoring for one rescheduling round.
 *
 * Vocabulary (Section 5.2, problem formulation):
 *   instances I = {0..n_inst-1}; request r sits on instance inst_of[r]
 *   (its batch B_i); N(r) = cur_len[r] is its current token count;
 *   N^(r) = rem_len[r] its predicted remaining generation length; the load of
 *   instance i at future decode step t is N^_i(B_{i,t}) = sum over r in B_i
 *   with t < N^(r) of (N(r) + t)  (Eq. 4's per-step term).
 *
 * Conventions shared by every entry point
 *   - Every array pointer is DEVICE memory owned by the caller; parameter
 *     structs and status outputs are host memory.  The library never
 *     allocates or frees device memory.
 *   - Calls validate their scalar arguments synchronously (returning a
 *     negative star_status before anything is launched), then enqueue
 *     kernels on `stream` (a hipStream_t; NULL = the null stream) and
 *     return.  Results are valid once the stream has reached that point.
 *   - `ws` is a caller-owned device workspace of at least the size reported
 *     by the matching *_workspace_size() call, 256-byte aligned, zeroed once
 *     before first use (star_workspace_init).  Its first STAR_WS_HEADER_BYTES
 *     bytes are the library's state between calls (a sticky device-error
 *     word; counters and a histogram that every call leaves at zero); the
 *     rest is scratch that any call may overwrite, so one workspace can
 *     serve every entry point.  Calls sharing a workspace must be ordered
 *     (same stream, or synchronised); concurrent calls need distinct
 *     workspaces.
 *   - Array CONTENTS that break a documented precondition (instance index
 *     out of range, cur_len < 1, rem_len < 1) are detected on the device:
 *     the offending request is left out of every curve, score and ranking,
 *     and a STAR_DEV_* bit is OR-ed into the workspace's error word, read
 *     back by star_read_device_error.
 *   - No call prints, aborts or throws.
 */
#ifndef STAR_H
#define STAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define STAR_ABI_VERSION 2
#define STAR_WS_HEADER_BYTES 8192
#define STAR_MAX_TOP_K 1024

typedef enum {
    STAR_OK = 0,
    STAR_ERR_INVALID_ARG = -1,   /* null pointer, non-positive size, bad enum */
    STAR_ERR_UNSUPPORTED = -2,   /* shape or alignment outside what the kernels handle */
    STAR_ERR_OVERFLOW = -3,      /* sizes whose int64 loads could overflow */
    STAR_ERR_WORKSPACE = -4,     /* workspace null, misaligned or too small */
    STAR_ERR_HIP = -5,           /* a HIP runtime call or kernel launch failed */
    STAR_ERR_DEVICE_INPUT = -6,  /* star_read_device_error: array contents broke a precondition
                                    (the device error word was non-zero) */
    STAR_ERR_SCRATCH_LIMIT = -7  /* star_predict_noalloc: the call needs more scratch than
                                    STAR_NOALLOC_SCRATCH_BYTES */
} star_status;

/* bits of the device-error word */
enum { STAR_DEV_BAD_INST = 1, STAR_DEV_BAD_CUR = 2, STAR_DEV_BAD_REM = 4 };

typedef enum { STAR_F32 = 0, STAR_BF16 = 1 } star_dtype;
typedef enum { STAR_ACT_RELU = 0, STAR_ACT_GELU_ERF = 1 } star_act;

/* ------------------------------------------------------------------------
 * (a) Remaining-length predictor head.
 *
 * Section 4.2 feeds the last-layer, last-token hidden state h (size d) of
 * each running request to a small MLP (Eq. 2) to estimate the distribution
 * p(Y | S) of the remaining length Y (Eq. 1).  Here the head is
 *     a1 = act(W1 h + b1)                 W1: [m, d]
 *     z  = W2 a1 + b2                     W2: [nb, m]   (one logit per bin)
 *     p  = softmax(z);  E = sum_j p_j v_j (mean of p over length bins v_j,
 *                                          the binned targets of Section 6.5)
 * and, for continuous prediction (Section 4.3), an exponential moving
 * average across calls: y = alpha E + (1 - alpha) y_prev.
 * Finally rem_len = clamp(round_half_even(y), 1, len_max), the N^(r) that
 * (b) and (c) consume.
 *
 * Precision: bf16 or fp32 operands (dtype applies to hidden, w1 and w2);
 * fp32 accumulation; a1 enters the second product as a bf16 hi/lo pair
 * (bf16 path) or fp32; fp32 softmax and EMA.  STAR_ACT_GELU_ERF is
 * x Phi(x) with Phi from the Abramowitz & Stegun 7.1.26 approximation of
 * erfc (within 1.5e-7 max(1, |x|) of the exact GELU in fp32).
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t n_req;      /* B >= 0 rows of hidden */
    int32_t d_model;    /* d >= 1; multiple of 8 (bf16) or 4 (fp32) */
    int32_t d_hidden;   /* m in [1, 2048]; multiple of 8 (bf16) or 4 (fp32) */
    int32_t n_bins;     /* nb in [1, 256] */
    int32_t dtype;      /* star_dtype of hidden, w1, w2 */
    int32_t act;        /* star_act */
    float   ema_alpha;  /* 0 disables smoothing; else in (0, 1] */
    int32_t ema_init;   /* 1: y := E this call (first step); 0: blend with ema_state */
    int32_t len_max;    /* >= 1, upper clamp of rem_len */
} star_predict_params;

size_t star_predict_workspace_size(const star_predict_params* p);

/* hidden [B, d], w1 [m, d], w2 [nb, m]: row-major, 16-byte aligned.
 * b1 [m]: fp32, 16-byte aligned, or NULL (zero).  b2 [nb]: fp32 or NULL.
 * bin_values [nb]: fp32.
 * ema_state [B]: fp32 in/out, required iff ema_alpha > 0.
 * expected_len [B]: fp32 out, the unsmoothed E.
 * rem_len [B]: int32 out, or NULL. */
star_status star_predict(const star_predict_params* p, const void* hidden, const void* w1,
                         const float* b1, const void* w2, const float* b2,
                         const float* bin_values, float* ema_state, float* expected_len,
                         int32_t* rem_len, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (a) across consecutive batches: the same results as star_predict, with
 * one batch's head and the next batch's first-layer product in one launch.
 * Section 4.3 re-predicts at every decode step, and the first layer of step
 * i + 1 needs only that step's hidden states, not step i's outputs.
 *
 * star_predict splits into a product (hidden -> the split-K partials in the
 * workspace) and a head (partials -> E, EMA, rem_len).  A call does:
 *   - ws_prev != NULL: the head of the batch whose product an earlier call
 *     left in ws_prev, writing expected_len, ema_state and rem_len;
 *   - hidden_next != NULL: the product of hidden_next into ws_next.
 * At least one of the two.  A sequence over batches h_0, h_1, ... with
 * workspaces alternating between two buffers A and B:
 *     (h_0 -> A), (A -> out_0, h_1 -> B), (B -> out_1, h_2 -> A), ...,
 *     (last -> out_last)
 * gives out_i equal to star_predict on h_i with the EMA carried across the
 * calls in order: bit for bit where star_predict runs the same two kernels
 * (products with a K-split).  Products of one K-slice, which star_predict
 * runs as one fused kernel that rounds the second product's sums in another
 * order, run here as the product and the head; their results meet the same
 * 2e-2 contract.  Every call's w1, b1, w2, b2, bin_values and params (p)
 * must be the same, except p->ema_init, which applies to the head the call
 * runs.
 *
 * Arguments as for star_predict.  w1 may be NULL when hidden_next is NULL;
 * w2, bin_values, expected_len, ema_state and rem_len may be NULL when
 * ws_prev is NULL.  ws_next and ws_prev: each
 * star_predict_overlap_workspace_size(p) bytes (ws_bytes; the same as
 * star_predict_workspace_size(p) except for one-slice products), 256-byte
 * aligned, not overlapping; ws_prev keeps the product of the call that
 * filled it until its head has run.
 * Errors: STAR_ERR_INVALID_ARG when both sides are NULL or the workspaces
 * overlap; otherwise as star_predict.
 * One launch where the product takes 64 x 64 tiles (bf16) and the head is
 * the 4-row one, else the head and the product as two launches on `stream`.
 * ---------------------------------------------------------------------- */
size_t star_predict_overlap_workspace_size(const star_predict_params* p);
star_status star_predict_overlap(const star_predict_params* p, const void* hidden_next,
                                 void* ws_next, const void* ws_prev, const void* w1,
                                 const float* b1, const void* w2, const float* b2,
                                 const float* bin_values, float* ema_state, float* expected_len,
                                 int32_t* rem_len, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (a) without allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, results and kernels as star_predict, minus
 * the workspace: the scratch (split-K partials or logit shares, and the
 * fused kernel's counters) is a fixed array of STAR_NOALLOC_SCRATCH_BYTES in
 * device memory, one per GPU, held until the process ends.  The call
 * allocates and frees nothing; its first call on a GPU looks up the array's
 * device address and clears its counters (one small kernel on `stream`).
 * Calls on one GPU share that array, so they must not overlap (same stream,
 * or synchronised); overlapping calls race.  Sizes whose scratch exceeds the
 * array return STAR_ERR_SCRATCH_LIMIT before anything is launched (batches of
 * 512 to 4096 rows at d = 4096-5120, m = 512 fit; 32768 rows at m = 1024 do
 * not).
 * ---------------------------------------------------------------------- */
#define STAR_NOALLOC_SCRATCH_BYTES (32 << 20)

star_status star_predict_noalloc(const star_predict_params* p, const void* hidden,
                                 const void* w1, const float* b1, const void* w2,
                                 const float* b2, const float* bin_values, float* ema_state,
                                 float* expected_len, int32_t* rem_len, void* stream);

/* ------------------------------------------------------------------------
 * (f3) The paper's regression head.
 *
 * Section 4.2 (Eq. 2) predicts the remaining length directly with a 4-layer
 * MLP on the same last-layer, last-token hidden state h:
 *     y^ = w4 . relu(W3 relu(W2 relu(W1 h + b1) + b2) + b3) + b4
 * W1 [m1, d], W2 [m2, m1], W3 [m3, m2] (dtype of hidden), w4 [m3] fp32;
 * b1 [m1], b2 [m2], b3 [m3] fp32 or NULL (Eq. 2 has none); b4 in the params.
 * The paper's sizes: d = 3584, m1 = 2048, m2 = 512, m3 = 64 (8.4 M weights).
 * expected_len [B] <- y^; the EMA and rem_len follow as in (a).
 * Precision: bf16 (or fp32) operands, fp32 accumulation; the first layer's
 * output is rounded to the operand type before the second product; the
 * second layer's output enters the third as a bf16 hi/lo pair (bf16) or
 * fp32; fp32 for the rest.
 * Workspace: split-K partials of the first two layers and the first layer's
 * output.  Limits: d, m1, m2 multiples of 8 (bf16) or 4 (fp32); m2 <= 2048;
 * m3 <= 256.
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t n_req;      /* B >= 0 */
    int32_t d_model;    /* d >= 1 */
    int32_t m1, m2, m3; /* hidden widths */
    int32_t dtype;      /* star_dtype of hidden, w1, w2, w3 */
    float   ema_alpha;  /* 0 disables smoothing; else in (0, 1] */
    int32_t ema_init;
    int32_t len_max;    /* >= 1 */
    float   b4;         /* output bias */
} star_mlp4_params;

size_t star_predict_mlp4_workspace_size(const star_mlp4_params* p);

star_status star_predict_mlp4(const star_mlp4_params* p, const void* hidden, const void* w1,
                              const float* b1, const void* w2, const float* b2, const void* w3,
                              const float* b3, const float* w4, float* ema_state,
                              float* expected_len, int32_t* rem_len, void* ws, size_t ws_bytes,
                              void* stream);

/* ------------------------------------------------------------------------
 * (b) Per-instance predicted load curves.
 *
 * Worker-side future-load simulation of Section 5.2's complexity analysis,
 * over a horizon of H = bucket * n_buckets decode steps grouped in buckets
 * of `bucket` steps:
 *     load[i, k] = sum_{t = k*bucket}^{(k+1)*bucket - 1}
 *                  sum_{r in B_i, t < rem_len[r]} (cur_len[r] + t)
 * (int64 token-steps; with bucket = 1, load[i, 0] = N_i(B_i)).
 * cur_len, rem_len, inst_of: int32 [n_req], any order.
 * load: int64 [n_inst, n_buckets], fully overwritten.
 * ---------------------------------------------------------------------- */
typedef struct {
    int32_t n_req;      /* N >= 0 */
    int32_t n_inst;     /* n >= 1 */
    int32_t bucket;     /* b >= 1 */
    int32_t n_buckets;  /* K >= 1; b * K <= 2^30 */
} star_load_params;

/* The header, plus, for long request streams (n_req >= 8192, n_buckets <=
 * 1024, n_inst <= 960), per-instance histograms of each request slice that
 * the last workgroup of the instance sums; the request arrays are then read
 * in 16-byte groups when all three are 16-byte aligned (other alignments
 * take a kernel that needs no more than the header). */
size_t star_project_load_workspace_size(const star_load_params* p);

star_status star_project_load(const star_load_params* p, const int32_t* cur_len,
                              const int32_t* rem_len, const int32_t* inst_of, int64_t* load,
                              void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (c) Migration candidates scored by projected peak load, and ranked.
 *
 * Algorithm 1 (candidate enumeration and best-feasible selection) applied
 * to every request -> instance pair.  For request r on s = inst_of[r]:
 *     scores[r, t] = max_k (load[t, k] + R_r[k])   for t != s,
 *     scores[r, s] = max_k load[s, k]              (staying: r is already in it),
 * where R_r is r's own bucketed curve as defined in (b).  `load` must be
 * the curves of these same requests (normally star_project_load's output).
 * Migrations (t != s) are ranked by the key (score, r, t) ascending:
 *     best_target[r] / best_score[r]: r's smallest key, or -1 / -1 when r
 *         has none (n_inst == 1 or r invalid);
 *     topk_*[q], q < top_k: the q-th smallest key overall, -1 past the end.
 * Outputs: scores int64 [n_req, n_inst] or NULL; best_target int32 [n_req]
 * or NULL; best_score int64 [n_req] or NULL; topk_req/topk_tgt int32 and
 * topk_score int64 [top_k], all three non-NULL iff top_k > 0.
 * ---------------------------------------------------------------------- */
typedef struct {
    star_load_params load;  /* same meaning as for star_project_load */
    int32_t top_k;          /* 0 .. STAR_MAX_TOP_K */
} star_score_params;

size_t star_score_workspace_size(const star_score_params* p);

star_status star_score_migrations(const star_score_params* p, const int32_t* cur_len,
                                  const int32_t* rem_len, const int32_t* inst_of,
                                  const int64_t* load, int64_t* scores, int32_t* best_target,
                                  int64_t* best_score, int32_t* topk_req, int32_t* topk_tgt,
                                  int64_t* topk_score, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (b) + (c) in one call: the load projection of the requests followed by
 * the scoring and ranking of their migrations (Section 5.2, Eq. 4;
 * Algorithm 1), with the same arguments and results as star_project_load
 * then star_score_migrations on that load, except that `load` (int64
 * [n_inst, n_buckets], fully overwritten) is an output here and the two
 * share one workspace of star_project_and_score_workspace_size() bytes.
 * Rounds whose curves fit on-chip (and with at most 8192 requests) skip
 * the projection kernel: every scoring workgroup builds the curves itself
 * and one of them writes `load`; other sizes run the projection first, and
 * where it takes request slices (see star_project_load_workspace_size) and
 * the curves do not fit on-chip, it also writes the scoring's bucket-major
 * curve terms, so no separate preparation pass runs.
 * ---------------------------------------------------------------------- */
size_t star_project_and_score_workspace_size(const star_score_params* p);

star_status star_project_and_score(const star_score_params* p, const int32_t* cur_len,
                                   const int32_t* rem_len, const int32_t* inst_of, int64_t* load,
                                   int64_t* scores, int32_t* best_target, int64_t* best_score,
                                   int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score,
                                   void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (f1) Migration candidates scored by the change of the time-weighted load
 * variance.
 *
 * Section 5.2 sets the migration objective to the variance of the
 * instances' token loads now plus a beta-weighted sum of the variances of
 * their predicted loads at later steps (Eq. 3-4); Algorithm 1's best-feasible
 * selection executes the candidate that reduces it most, if any does.  Over
 * the bucketed curves of (b), Phi = sum_k beta_k Var_i(load[i, k]) (population
 * variance over instances; bucket 0 holds the current step, so the paper's
 * separate current-variance term is beta_0's share).  Moving request r
 * (own curve R_r as in (c)) from s = inst_of[r] to t changes Phi by 2G/n with
 *     gain[r, t] = G = sum_k beta_k R_r[k] (R_r[k] + load[t, k] - load[s, k]),
 * reported exactly as a 128-bit integer; gain[r, s] = 0, and rows of invalid
 * requests are 0.  Negative = the variance falls.
 *   beta: uint16 [n_buckets] device array, the weights in fixed point (only
 *         their ratios matter; 0 ignores a bucket).
 *   best_target[r] / best_gain[r]: r's smallest key (gain, t) over t != s,
 *         or -1 / 0 when r has none; the target may raise the variance.
 *   best_move: ONE device star_move: the smallest key (gain, r, t) with
 *         gain < 0 over all migrations, src = inst_of[req]; or
 *         req = src = tgt = -1, gain 0 when no migration lowers Phi.
 * Any of gain, best_target, best_gain, best_move may be NULL.
 * STAR_ERR_OVERFLOW also when some gain could reach 2^126 in magnitude
 * (bounded from n_req, bucket, n_buckets and the worst int32 cur_len).
 * ---------------------------------------------------------------------- */
typedef struct {
    uint64_t lo;   /* two's complement: value = hi * 2^64 + lo */
    int64_t hi;
} star_i128;

typedef struct {
    int32_t req, src, tgt;
    int32_t reserved;
    star_i128 gain;
} star_move;

size_t star_score_variance_workspace_size(const star_load_params* p);

star_status star_score_variance(const star_load_params* p, const int32_t* cur_len,
                                const int32_t* rem_len, const int32_t* inst_of,
                                const int64_t* load, const uint16_t* beta, star_i128* gain,
                                int32_t* best_target, star_i128* best_gain,
                                star_move* best_move, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * (f2) Algorithm 1 end to end, repeated: a migration plan.
 *
 * One pass is one scheduler interval of Algorithm 1 with the variance gain
 * of (f1) as the figure of merit and no decode progress in between:
 *   classification: w_i = sum_k beta_k load[i, k]; mean w = (1/n) sum_i w_i;
 *     O = {i : w_i > (1 + theta) mean w};
 *     U = {i : N_i < (1 + theta) mean w}    (u_rule 0, as printed), or
 *         {i : w_i < (1 - theta) mean w}    (u_rule 1),
 *     N_i = sum of cur_len over the valid requests on i (current load);
 *   enumeration: (r, s, t) with s = inst_of[r] in O, t in U, t != s,
 *     rem_len[r] > min_rem (the remaining-length-versus-migration-cost
 *     filter), and N_t + rem_len[r] <= mem_cap (mem_rule 0, as printed) or
 *     N_t + cur_len[r] + rem_len[r] <= mem_cap (mem_rule 1);
 *   selection: the smallest key (gain, r, t) with gain < 0;
 *   execution: inst_of[r] = t and r's curve moves from load[s] to load[t].
 * Passes repeat until max_moves migrations are made, O is empty, or no
 * candidate lowers the objective.  theta = theta_num / theta_den; all
 * comparisons are exact (cross-multiplied, 128-bit).
 *   inst_of: int32 [n_req] device, IN/OUT (the placement after the plan).
 *   load: int64 [n_inst, n_buckets] device, IN/OUT: on entry the curves of
 *         exactly these requests (star_project_load), on exit the curves
 *         after the plan.
 *   beta: uint16 [n_buckets] device (as in star_score_variance).
 *   moves: star_move [max_moves] device; moves[q] = q-th migration
 *         (req, src, tgt, gain) in execution order.  n_moves: int32 [1]
 *         device, the number made.
 * Cost: one classification-and-scoring pass over all N x n candidates and
 * one small update per allowed move (2 launches each; once the plan stops,
 * the remaining launches exit at once).
 * ---------------------------------------------------------------------- */
#define STAR_MAX_MOVES 4096

typedef struct {
    star_load_params load;
    int32_t max_moves;          /* 0 .. STAR_MAX_MOVES */
    int32_t theta_num;          /* 0 .. 2^20 */
    int32_t theta_den;          /* 1 .. 2^20 */
    int32_t u_rule;             /* 0 or 1, see above */
    int32_t mem_rule;           /* 0 or 1, see above */
    int32_t min_rem;            /* candidates need rem_len > min_rem */
    int64_t mem_cap;            /* >= 0, tokens */
} star_plan_params;

size_t star_plan_workspace_size(const star_plan_params* p);

star_status star_plan_migrations(const star_plan_params* p, const int32_t* cur_len,
                                 const int32_t* rem_len, int32_t* inst_of, int64_t* load,
                                 const uint16_t* beta, star_move* moves, int32_t* n_moves,
                                 void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Housekeeping.
 * ---------------------------------------------------------------------- */
/* Zero the whole workspace on `stream` (a fill kernel, no memset node).
 * Call once after allocating a workspace; the error word then stays
 * consistent across calls. */
star_status star_workspace_init(void* ws, size_t ws_bytes, void* stream);

/* Synchronise `stream`, return the workspace's device-error word (OR of
 * STAR_DEV_* bits since the last read) in *code, and clear it.  Returns
 * STAR_ERR_DEVICE_INPUT when that word was non-zero (*code names the
 * broken preconditions), STAR_OK when it was zero. */
star_status star_read_device_error(void* ws, void* stream, int32_t* code);

const char* star_status_string(star_status s);
int32_t star_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* STAR_H */
