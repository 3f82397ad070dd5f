// Internal launch interfaces between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "star.h"

namespace star {

struct GemmPlan {
    int tiles_m = 0, tiles_n = 0, ktiles = 0, splits = 1;
    enum { kSmall = 0, kBig = 1, kWide = 2, kHuge = 3, kMid = 4 };
    int shape = kBig;     // 64 x 64 tiles on 4 waves; 128 x 128 on 8; 128 x 128 on 4;
                          // 256 x 256 on 8; 128 x 64 on 8
};
GemmPlan plan_gemm(int M, int N, int K, int elem);

struct PredictPlan {
    GemmPlan gemm;
    int tiles_m = 0, tiles_n = 0, ktiles = 0, splits = 1;
    size_t partial_bytes = 0;   // fp32 split-K partials [splits, B, m]
    size_t head_lds = 0;        // dynamic LDS of the head kernel
    int head_rows = 4;          // rows per head workgroup
    bool head_tiled = false;    // the K-chunked head (large bf16 batches), 64 rows per workgroup
    bool fused = false;         // one kernel: product (one K-slice) and head
    size_t lpart_bytes = 0;     // fused: logit shares [tiles_m][tiles_n][BM * nb32] fp32
};
// allow: 1 = the fused kernel where it applies, 0 = never (the two-kernel path)
PredictPlan plan_predict(const star_predict_params& p, bool tiled_ok = true, bool fused_ok = true);
// The head of a batch whose partials are `partials_prev` and the product of
// the next batch into `partials_next`, in one launch where the plan allows,
// else as two launches (two-kernel plans, plan_predict(p, true, false);
// hipErrorInvalidValue for a fused plan).  Either side may be null.
hipError_t launch_predict_overlap(const star_predict_params& p, const PredictPlan& pl,
                                  const void* hidden_next, float* partials_next,
                                  const float* partials_prev, const void* w1, const float* b1,
                                  const void* w2, const float* b2, const float* bins,
                                  float* ema_state, float* expected, int32_t* rem_len,
                                  hipStream_t stream);
hipError_t launch_predict(const star_predict_params& p, const PredictPlan& pl, const void* hidden,
                          const void* w1, const float* b1, const void* w2, const float* b2,
                          const float* bins, float* ema_state, float* expected, int32_t* rem_len,
                          char* scratch, uint32_t* tickets, hipStream_t stream);

struct Mlp4Plan {
    GemmPlan g1;          // layer 1
    PredictPlan head;     // layer 2 (its split-K partials) and the last two layers
    size_t p1_off = 0, a1_off = 0, p2_off = 0, total = 0;
};
Mlp4Plan plan_mlp4(const star_mlp4_params& p);
hipError_t launch_mlp4(const star_mlp4_params& p, const Mlp4Plan& pl, const void* hidden,
                       const void* w1, const float* b1, const void* w2, const float* b2,
                       const void* w3, const float* b3, const float* w4, float* ema_state,
                       float* expected, int32_t* rem_len, char* ws, hipStream_t stream);

struct LoadPlan {
    int chunk = 0;       // buckets per workgroup
    int n_chunks = 0;
    bool split = false;  // request slices per instance, met by a last arriver (16-byte
                         // aligned request arrays; otherwise the chunked kernel)
    int slices = 0, slice_len = 0, kp = 0;
    size_t part_bytes = 0;  // the slices' histograms, after the workspace header
};
LoadPlan plan_load(const star_load_params& p);

// Planes of every instance's curve terms, for scoring from them; entry
// (k, t), k = 0..K, at k sk + t st (bucket-major: sk = n, st = 1;
// instance-major: sk = 1, st = K + 1):
//     tpm(k, t) = PM_t[k] = max_{j < k} (L_t[j] + b^2 j)   (-inf at k = 0)
//     tl(k, t)  = L_t[k], -inf at k = K
//     tsm(k, t) = SM_t[min(k + 1, K)], SM_t[k] = max_{j >= k} L_t[j], SM_t[K] = -inf
//     peak[t]   = SM_t[0]
struct CurvePlanes {
    int64_t* tpm = nullptr;
    int64_t* tl = nullptr;
    int64_t* tsm = nullptr;
    int64_t* peak = nullptr;
    int64_t sk = 0, st = 0;
};

// ws: the workspace (its header); part: part_bytes for the split projection's
// histograms.  With planes set, the split projection writes them as well and
// sets *planes_written.
hipError_t launch_project_load(const star_load_params& p, const LoadPlan& pl,
                               const int32_t* cur, const int32_t* rem, const int32_t* inst,
                               int64_t* load, char* ws, char* part, const CurvePlanes* planes,
                               bool* planes_written, hipStream_t stream);

struct ScorePlan {
    bool fused = false;   // PM/SM built in LDS by the scoring kernel
    bool one = false;     // one 1024-thread workgroup projects, scores and ranks everything
                          // (up to 1024 requests on up to 8 instances)
    bool small = false;   // one workgroup scores and ranks everything
    bool rank2 = false;   // fused scoring that code-sorts its keys, then one ranking workgroup
    bool project_in = false; // rank2: the scoring workgroups project the curves themselves
                             // (star_project_and_score only)
    size_t ghist_off = 0, base_off = 0, keys_s_off = 0, keys_i_off = 0, offs_off = 0;
    int rpb = 0;          // requests per scoring workgroup
    int cand = 0;         // candidates per scoring workgroup (rpb * n)
    int groups = 0;       // scoring workgroups
    bool topk_direct = false;  // top-k over all migrations (else over the k best requests' ones)
    int topk_rj = 8;           // direct top-k: keys per thread in registers (8 or 16)
    bool topk_reg1 = false;    // pruned top-k: best keys fit registers
    int topk_rj2 = 0;          // pruned top-k: the k requests' migrations per thread in
                               // registers (8 or 16), 0: streamed
    bool topk_pruned = false;  // pruned top-k: the scoring kernel writes the key-code base
    bool topk_hist = false;    // pruned top-k, best keys beyond registers: the top-k counts
                               // their codes and gathers those up to the k-th
    size_t bcode_off = 0, gs_off = 0, gi_off = 0;  // topk_hist: best-key codes, gathered keys
    size_t tpm_off = 0, tl_off = 0, tsm_off = 0, peak_off = 0;  // curve planes (not fused)
    bool by_bucket = false;  // the planes bucket-major (else instance-major)
    int lg = 0;           // planar scoring: 2^lg lanes per request
    size_t scores_off = 0, bscore_off = 0, btarget_off = 0, total = 0;
    size_t lds = 0;       // dynamic LDS of the scoring kernel (or of the small path's one)
};
ScorePlan plan_score(const star_score_params& p, bool project = false);
// The planes of the non-fused path, inside ws.
CurvePlanes score_planes(const star_score_params& p, const ScorePlan& pl, char* ws);
// planes_ready: the projection has already written the planes.
hipError_t launch_score(const star_score_params& p, const ScorePlan& pl, const int32_t* cur,
                        const int32_t* rem, const int32_t* inst, const int64_t* load,
                        int64_t* scores, int32_t* best_target, int64_t* best_score,
                        int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score, char* ws,
                        int32_t* err_word, hipStream_t stream, int64_t* load_out = nullptr,
                        bool planes_ready = false);

struct VarPlan {
    int lg = 0;           // lanes per request = 2^lg (<= 16)
    int blocks = 0;       // scoring workgroups
    bool ticketed = false;  // best move found inside the scoring kernel
    size_t qt_off = 0, lt_off = 0, bs_off = 0, part_off = 0, total = 0;
};
VarPlan plan_variance(const star_load_params& p);
hipError_t launch_variance(const star_load_params& p, const VarPlan& pl, const int32_t* cur,
                           const int32_t* rem, const int32_t* inst, const int64_t* load,
                           const uint16_t* beta, star_i128* gain, int32_t* best_target,
                           star_i128* best_gain, star_move* move, char* ws, int32_t* err,
                           hipStream_t stream);

struct PlanPlan {
    VarPlan v;
    size_t now_off = 0, total = 0;
};
PlanPlan plan_plan(const star_plan_params& p);
hipError_t launch_plan(const star_plan_params& p, const PlanPlan& pl, const int32_t* cur,
                       const int32_t* rem, int32_t* inst, int64_t* load, const uint16_t* beta,
                       star_move* moves, int32_t* n_moves, char* ws, int32_t* err,
                       hipStream_t stream);

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream);

}  // namespace star
