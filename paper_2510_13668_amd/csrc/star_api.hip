// C-ABI of libstar: argument validation, workspace layout and launches.
// Every check that can be made from scalars happens here, synchronously,
// before anything is enqueued; see include/star.h for the contract.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "star_common.hpp"
#include "star_internal.hpp"

#define STAR_API extern "C" __attribute__((visibility("default")))

namespace star {

__global__ void fill_zero_kernel(uint32_t* p, size_t words) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < words;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream) {
    const size_t words = bytes / 4;
    if (words == 0) return hipSuccess;
    size_t blocks = (words + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                       (uint32_t*)p, words);
    return hipGetLastError();
}

static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

static star_status check_ws(const void* ws, size_t ws_bytes, size_t need) {
    if (!ws || !aligned(ws, 256) || ws_bytes < need) return STAR_ERR_WORKSPACE;
    return STAR_OK;
}

static star_status check_load_params(const star_load_params* p) {
    if (!p) return STAR_ERR_INVALID_ARG;
    if (p->n_req < 0 || p->n_inst < 1 || p->bucket < 1 || p->n_buckets < 1)
        return STAR_ERR_INVALID_ARG;
    const int64_t H = (int64_t)p->bucket * p->n_buckets;
    if (H > ((int64_t)1 << 30)) return STAR_ERR_UNSUPPORTED;
    // Every load, score and intermediate is at most (N + 1) b (c_max + H) + b H
    // with c_max < 2^31; keep that below 2^62.
    const __int128 bound = (__int128)(p->n_req + 1) * p->bucket * (((__int128)1 << 31) + H) +
                           (__int128)p->bucket * H;
    if (bound >= ((__int128)1 << 62)) return STAR_ERR_OVERFLOW;
    return STAR_OK;
}

static star_status check_predict_params(const star_predict_params* p) {
    if (!p) return STAR_ERR_INVALID_ARG;
    if (p->n_req < 0 || p->d_model < 1 || p->d_hidden < 1 || p->n_bins < 1 || p->len_max < 1)
        return STAR_ERR_INVALID_ARG;
    if (p->dtype != STAR_F32 && p->dtype != STAR_BF16) return STAR_ERR_INVALID_ARG;
    if (p->act != STAR_ACT_RELU && p->act != STAR_ACT_GELU_ERF) return STAR_ERR_INVALID_ARG;
    if (!(p->ema_alpha >= 0.0f && p->ema_alpha <= 1.0f)) return STAR_ERR_INVALID_ARG;
    if (p->ema_init != 0 && p->ema_init != 1) return STAR_ERR_INVALID_ARG;
    const int vec = p->dtype == STAR_BF16 ? 8 : 4;      // elements per 16-byte load
    if (p->d_model % vec || p->d_hidden % vec) return STAR_ERR_UNSUPPORTED;
    if (p->d_hidden > 2048 || p->n_bins > 256) return STAR_ERR_UNSUPPORTED;
    return STAR_OK;
}

}  // namespace star

using namespace star;

STAR_API int32_t star_abi_version(void) { return STAR_ABI_VERSION; }

STAR_API const char* star_status_string(star_status s) {
    switch (s) {
        case STAR_OK: return "STAR_OK";
        case STAR_ERR_INVALID_ARG: return "STAR_ERR_INVALID_ARG: null pointer, bad size or bad enum";
        case STAR_ERR_UNSUPPORTED: return "STAR_ERR_UNSUPPORTED: shape or alignment not handled";
        case STAR_ERR_OVERFLOW: return "STAR_ERR_OVERFLOW: int64 loads could overflow at these sizes";
        case STAR_ERR_WORKSPACE: return "STAR_ERR_WORKSPACE: workspace null, misaligned or too small";
        case STAR_ERR_HIP: return "STAR_ERR_HIP: HIP runtime or launch failure";
        case STAR_ERR_DEVICE_INPUT:
            return "STAR_ERR_DEVICE_INPUT: array contents broke a precondition (device error word set)";
        case STAR_ERR_SCRATCH_LIMIT:
            return "STAR_ERR_SCRATCH_LIMIT: the call needs more than the built-in scratch of the "
                   "allocation-free entry point (STAR_NOALLOC_SCRATCH_BYTES)";
    }
    return "unknown star_status";
}

// ---------------------------------------------------------------------------
// predictor
// ---------------------------------------------------------------------------
STAR_API size_t star_predict_workspace_size(const star_predict_params* p) {
    if (check_predict_params(p) != STAR_OK) return 0;
    return STAR_WS_HEADER_BYTES + align_up(plan_predict(*p).partial_bytes, 256);
}

STAR_API star_status star_predict(const star_predict_params* p, const void* hidden,
                                  const void* w1, const float* b1, const void* w2,
                                  const float* b2, const float* bin_values, float* ema_state,
                                  float* expected_len, int32_t* rem_len, void* ws,
                                  size_t ws_bytes, void* stream) {
    star_status st = check_predict_params(p);
    if (st != STAR_OK) return st;
    if (p->n_req > 0) {
        if (!hidden || !w1 || !w2 || !bin_values || !expected_len) return STAR_ERR_INVALID_ARG;
        if (p->ema_alpha > 0.0f && !ema_state) return STAR_ERR_INVALID_ARG;
        if (!aligned(hidden, 16) || !aligned(w1, 16) || !aligned(w2, 16) || !aligned(b1, 16))
            return STAR_ERR_UNSUPPORTED;
    }
    const PredictPlan pl = plan_predict(*p);
    st = check_ws(ws, ws_bytes, STAR_WS_HEADER_BYTES + align_up(pl.partial_bytes, 256));
    if (st != STAR_OK) return st;
    char* scratch = (char*)ws + STAR_WS_HEADER_BYTES;
    uint32_t* tickets = (uint32_t*)((char*)ws + kHdrTickets);
    hipError_t e = launch_predict(*p, pl, hidden, w1, b1, w2, b2, bin_values, ema_state,
                                  expected_len, rem_len, scratch, tickets, (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// star_predict_overlap runs the two-kernel plan (product, then head) for
// every shape: one-slice products, which star_predict runs as one fused
// kernel, keep their fp32 partial plane in the workspace here.
STAR_API size_t star_predict_overlap_workspace_size(const star_predict_params* p) {
    if (check_predict_params(p) != STAR_OK) return 0;
    return STAR_WS_HEADER_BYTES + align_up(plan_predict(*p, true, false).partial_bytes, 256);
}

STAR_API star_status star_predict_overlap(const star_predict_params* p, const void* hidden_next,
                                          void* ws_next, const void* ws_prev, const void* w1,
                                          const float* b1, const void* w2, const float* b2,
                                          const float* bin_values, float* ema_state,
                                          float* expected_len, int32_t* rem_len, size_t ws_bytes,
                                          void* stream) {
    star_status st = check_predict_params(p);
    if (st != STAR_OK) return st;
    if (!hidden_next && !ws_prev) return STAR_ERR_INVALID_ARG;
    const PredictPlan pl = plan_predict(*p, true, false);
    const size_t need = STAR_WS_HEADER_BYTES + align_up(pl.partial_bytes, 256);
    if (hidden_next) {
        if (p->n_req > 0 && !w1) return STAR_ERR_INVALID_ARG;
        if (p->n_req > 0 && (!aligned(hidden_next, 16) || !aligned(w1, 16)))
            return STAR_ERR_UNSUPPORTED;
        st = check_ws(ws_next, ws_bytes, need);
        if (st != STAR_OK) return st;
    }
    if (ws_prev) {
        if (p->n_req > 0) {
            if (!w2 || !bin_values || !expected_len) return STAR_ERR_INVALID_ARG;
            if (p->ema_alpha > 0.0f && !ema_state) return STAR_ERR_INVALID_ARG;
            if (!aligned(w2, 16) || !aligned(b1, 16)) return STAR_ERR_UNSUPPORTED;
        }
        st = check_ws(ws_prev, ws_bytes, need);
        if (st != STAR_OK) return st;
    }
    if (hidden_next && ws_prev) {             // the two workspaces must not overlap
        const char* a = (const char*)ws_next;
        const char* b = (const char*)ws_prev;
        if (a < b + need && b < a + need) return STAR_ERR_INVALID_ARG;
    }
    float* next = hidden_next ? (float*)((char*)ws_next + STAR_WS_HEADER_BYTES) : nullptr;
    const float* prev = ws_prev ? (const float*)((const char*)ws_prev + STAR_WS_HEADER_BYTES)
                                : nullptr;
    hipError_t e = launch_predict_overlap(*p, pl, hidden_next, next, prev, w1, b1, w2, b2,
                                          bin_values, ema_state, expected_len, rem_len,
                                          (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// predictor without allocation: the scratch is a fixed array in device
// memory, one copy per GPU (each GPU that runs it holds the array until the
// process ends).  Its device address is looked up once per device, with that
// device current; host code never uses the array's own name as a device
// address.  Calls on one GPU share the array: they must not overlap.
// ---------------------------------------------------------------------------
__device__ __attribute__((aligned(256))) char scratch[STAR_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<char*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// The device address of `scratch` on the current device, or nullptr on a
// HIP error.  The first call on a device also clears the header (the fused
// predictor's counters start at zero; every call leaves them at zero).
char* noalloc_scratch(hipStream_t stream) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    char* p = g_scratch[dev].load(std::memory_order_acquire);
    if (p) return p;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_relaxed);
    if (p) return p;
    void* addr = nullptr;
    if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return nullptr;
    if (launch_fill_zero(addr, STAR_WS_HEADER_BYTES, stream) != hipSuccess) return nullptr;
    p = (char*)addr;
    g_scratch[dev].store(p, std::memory_order_release);
    return p;
}
}  // namespace

STAR_API star_status star_predict_noalloc(const star_predict_params* p, const void* hidden,
                                          const void* w1, const float* b1, const void* w2,
                                          const float* b2, const float* bin_values,
                                          float* ema_state, float* expected_len,
                                          int32_t* rem_len, void* stream) {
    star_status st = check_predict_params(p);
    if (st != STAR_OK) return st;
    if (p->n_req > 0) {
        if (!hidden || !w1 || !w2 || !bin_values || !expected_len) return STAR_ERR_INVALID_ARG;
        if (p->ema_alpha > 0.0f && !ema_state) return STAR_ERR_INVALID_ARG;
        if (!aligned(hidden, 16) || !aligned(w1, 16) || !aligned(w2, 16) || !aligned(b1, 16))
            return STAR_ERR_UNSUPPORTED;
    }
    const PredictPlan pl = plan_predict(*p);
    if (STAR_WS_HEADER_BYTES + align_up(pl.partial_bytes, 256) > (size_t)STAR_NOALLOC_SCRATCH_BYTES)
        return STAR_ERR_SCRATCH_LIMIT;
    char* ws = noalloc_scratch((hipStream_t)stream);
    if (!ws) return STAR_ERR_HIP;
    hipError_t e = launch_predict(*p, pl, hidden, w1, b1, w2, b2, bin_values, ema_state,
                                  expected_len, rem_len, ws + STAR_WS_HEADER_BYTES,
                                  (uint32_t*)(ws + kHdrTickets), (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// regression head
// ---------------------------------------------------------------------------
static star_status check_mlp4_params(const star_mlp4_params* p) {
    if (!p) return STAR_ERR_INVALID_ARG;
    if (p->n_req < 0 || p->d_model < 1 || p->m1 < 1 || p->m2 < 1 || p->m3 < 1 || p->len_max < 1)
        return STAR_ERR_INVALID_ARG;
    if (p->dtype != STAR_F32 && p->dtype != STAR_BF16) return STAR_ERR_INVALID_ARG;
    if (!(p->ema_alpha >= 0.0f && p->ema_alpha <= 1.0f)) return STAR_ERR_INVALID_ARG;
    if (p->ema_init != 0 && p->ema_init != 1) return STAR_ERR_INVALID_ARG;
    if (!(p->b4 == p->b4) || p->b4 > 3.0e38f || p->b4 < -3.0e38f) return STAR_ERR_INVALID_ARG;
    const int vec = p->dtype == STAR_BF16 ? 8 : 4;
    if (p->d_model % vec || p->m1 % vec || p->m2 % vec) return STAR_ERR_UNSUPPORTED;
    if (p->m2 > 2048 || p->m3 > 256) return STAR_ERR_UNSUPPORTED;
    return STAR_OK;
}

STAR_API size_t star_predict_mlp4_workspace_size(const star_mlp4_params* p) {
    if (check_mlp4_params(p) != STAR_OK) return 0;
    return STAR_WS_HEADER_BYTES + plan_mlp4(*p).total;
}

STAR_API star_status star_predict_mlp4(const star_mlp4_params* p, const void* hidden,
                                       const void* w1, const float* b1, const void* w2,
                                       const float* b2, const void* w3, const float* b3,
                                       const float* w4, float* ema_state, float* expected_len,
                                       int32_t* rem_len, void* ws, size_t ws_bytes,
                                       void* stream) {
    star_status st = check_mlp4_params(p);
    if (st != STAR_OK) return st;
    if (p->n_req > 0) {
        if (!hidden || !w1 || !w2 || !w3 || !w4 || !expected_len) return STAR_ERR_INVALID_ARG;
        if (p->ema_alpha > 0.0f && !ema_state) return STAR_ERR_INVALID_ARG;
        if (!aligned(hidden, 16) || !aligned(w1, 16) || !aligned(w2, 16) || !aligned(w3, 16) ||
            !aligned(b1, 16))
            return STAR_ERR_UNSUPPORTED;
    }
    const Mlp4Plan pl = plan_mlp4(*p);
    st = check_ws(ws, ws_bytes, STAR_WS_HEADER_BYTES + pl.total);
    if (st != STAR_OK) return st;
    hipError_t e = launch_mlp4(*p, pl, hidden, w1, b1, w2, b2, w3, b3, w4, ema_state,
                               expected_len, rem_len, (char*)ws + STAR_WS_HEADER_BYTES,
                               (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// load projection
// ---------------------------------------------------------------------------
STAR_API size_t star_project_load_workspace_size(const star_load_params* p) {
    if (check_load_params(p) != STAR_OK) return 0;
    return STAR_WS_HEADER_BYTES + plan_load(*p).part_bytes;
}

STAR_API star_status star_project_load(const star_load_params* p, const int32_t* cur_len,
                                       const int32_t* rem_len, const int32_t* inst_of,
                                       int64_t* load, void* ws, size_t ws_bytes, void* stream) {
    star_status st = check_load_params(p);
    if (st != STAR_OK) return st;
    if (!load) return STAR_ERR_INVALID_ARG;
    if (p->n_req > 0 && (!cur_len || !rem_len || !inst_of)) return STAR_ERR_INVALID_ARG;
    const LoadPlan pl = plan_load(*p);
    st = check_ws(ws, ws_bytes, STAR_WS_HEADER_BYTES + pl.part_bytes);
    if (st != STAR_OK) return st;
    hipError_t e = launch_project_load(*p, pl, cur_len, rem_len, inst_of, load, (char*)ws,
                                       (char*)ws + STAR_WS_HEADER_BYTES, nullptr, nullptr,
                                       (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// scoring and ranking
// ---------------------------------------------------------------------------
static star_status check_score_params(const star_score_params* p) {
    if (!p) return STAR_ERR_INVALID_ARG;
    star_status st = check_load_params(&p->load);
    if (st != STAR_OK) return st;
    if (p->top_k < 0 || p->top_k > STAR_MAX_TOP_K) return STAR_ERR_INVALID_ARG;
    if (p->load.n_inst > 4096) return STAR_ERR_UNSUPPORTED;
    if ((int64_t)p->load.n_req * p->load.n_inst >= ((int64_t)1 << 31)) return STAR_ERR_UNSUPPORTED;
    return STAR_OK;
}

STAR_API size_t star_score_workspace_size(const star_score_params* p) {
    if (check_score_params(p) != STAR_OK) return 0;
    return plan_score(*p).total;
}

STAR_API star_status star_score_migrations(const star_score_params* p, const int32_t* cur_len,
                                           const int32_t* rem_len, const int32_t* inst_of,
                                           const int64_t* load, int64_t* scores,
                                           int32_t* best_target, int64_t* best_score,
                                           int32_t* topk_req, int32_t* topk_tgt,
                                           int64_t* topk_score, void* ws, size_t ws_bytes,
                                           void* stream) {
    star_status st = check_score_params(p);
    if (st != STAR_OK) return st;
    if (!load) return STAR_ERR_INVALID_ARG;
    if (p->load.n_req > 0 && (!cur_len || !rem_len || !inst_of)) return STAR_ERR_INVALID_ARG;
    const bool any_topk = topk_req || topk_tgt || topk_score;
    const bool all_topk = topk_req && topk_tgt && topk_score;
    if (p->top_k > 0 ? !all_topk : any_topk) return STAR_ERR_INVALID_ARG;
    const ScorePlan pl = plan_score(*p);
    st = check_ws(ws, ws_bytes, pl.total);
    if (st != STAR_OK) return st;
    int32_t* err = (int32_t*)((char*)ws + kHdrErrorWord);
    hipError_t e = launch_score(*p, pl, cur_len, rem_len, inst_of, load, scores, best_target,
                                best_score, topk_req, topk_tgt, topk_score, (char*)ws, err,
                                (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// The split projection's histograms follow the scoring's scratch (its last
// workgroups write the scoring's curve planes while others still read them).
static size_t project_and_score_part(const ScorePlan& pl) { return align_up(pl.total, 256); }
static size_t project_and_score_bytes(const star_score_params& p, const ScorePlan& pl) {
    if (pl.project_in) return pl.total;
    return project_and_score_part(pl) + plan_load(p.load).part_bytes;
}

STAR_API size_t star_project_and_score_workspace_size(const star_score_params* p) {
    if (check_score_params(p) != STAR_OK) return 0;
    return project_and_score_bytes(*p, plan_score(*p, true));
}

STAR_API star_status star_project_and_score(const star_score_params* p, const int32_t* cur_len,
                                            const int32_t* rem_len, const int32_t* inst_of,
                                            int64_t* load, int64_t* scores, int32_t* best_target,
                                            int64_t* best_score, int32_t* topk_req,
                                            int32_t* topk_tgt, int64_t* topk_score, void* ws,
                                            size_t ws_bytes, void* stream) {
    star_status st = check_score_params(p);
    if (st != STAR_OK) return st;
    if (!load) return STAR_ERR_INVALID_ARG;
    if (p->load.n_req > 0 && (!cur_len || !rem_len || !inst_of)) return STAR_ERR_INVALID_ARG;
    const bool any_topk = topk_req || topk_tgt || topk_score;
    const bool all_topk = topk_req && topk_tgt && topk_score;
    if (p->top_k > 0 ? !all_topk : any_topk) return STAR_ERR_INVALID_ARG;
    const ScorePlan pl = plan_score(*p, true);
    st = check_ws(ws, ws_bytes, project_and_score_bytes(*p, pl));
    if (st != STAR_OK) return st;
    int32_t* err = (int32_t*)((char*)ws + kHdrErrorWord);
    hipError_t e = hipSuccess;
    bool planes_ready = false;
    if (!pl.project_in) {
        const CurvePlanes cp = score_planes(*p, pl, (char*)ws);
        e = launch_project_load(p->load, plan_load(p->load), cur_len, rem_len, inst_of, load,
                                (char*)ws, (char*)ws + project_and_score_part(pl),
                                cp.tpm ? &cp : nullptr, &planes_ready, (hipStream_t)stream);
    }
    if (e == hipSuccess)
        e = launch_score(*p, pl, cur_len, rem_len, inst_of, load, scores, best_target, best_score,
                         topk_req, topk_tgt, topk_score, (char*)ws, err, (hipStream_t)stream,
                         pl.project_in ? load : nullptr, planes_ready);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// time-weighted variance gains
// ---------------------------------------------------------------------------
static star_status check_variance_params(const star_load_params* p) {
    star_status st = check_load_params(p);
    if (st != STAR_OK) return st;
    if ((int64_t)p->n_req * p->n_inst >= ((int64_t)1 << 31)) return STAR_ERR_UNSUPPORTED;
    // |G| <= beta_max * sum_k R_k * (R_max + L_max), with R_k summing to at
    // most H (c_max + H), R_max = b (c_max + H), L_max = N R_max, c_max < 2^31.
    const long double cH = 2147483648.0L + (long double)p->bucket * p->n_buckets;
    const long double H = (long double)p->bucket * p->n_buckets;
    const long double rmax = (long double)p->bucket * cH;
    const long double bound = 65535.0L * H * cH * ((long double)p->n_req + 1.0L) * rmax;
    if (!(bound < ldexpl(1.0L, 126))) return STAR_ERR_OVERFLOW;
    return STAR_OK;
}

STAR_API size_t star_score_variance_workspace_size(const star_load_params* p) {
    if (check_variance_params(p) != STAR_OK) return 0;
    return plan_variance(*p).total;
}

STAR_API star_status star_score_variance(const star_load_params* p, const int32_t* cur_len,
                                         const int32_t* rem_len, const int32_t* inst_of,
                                         const int64_t* load, const uint16_t* beta,
                                         star_i128* gain, int32_t* best_target,
                                         star_i128* best_gain, star_move* best_move, void* ws,
                                         size_t ws_bytes, void* stream) {
    star_status st = check_variance_params(p);
    if (st != STAR_OK) return st;
    if (!load || !beta) return STAR_ERR_INVALID_ARG;
    if (p->n_req > 0 && (!cur_len || !rem_len || !inst_of)) return STAR_ERR_INVALID_ARG;
    if (!aligned(gain, 16) || !aligned(best_gain, 16) || !aligned(best_move, 16))
        return STAR_ERR_UNSUPPORTED;
    const VarPlan pl = plan_variance(*p);
    st = check_ws(ws, ws_bytes, pl.total);
    if (st != STAR_OK) return st;
    int32_t* err = (int32_t*)((char*)ws + kHdrErrorWord);
    hipError_t e = launch_variance(*p, pl, cur_len, rem_len, inst_of, load, beta, gain,
                                   best_target, best_gain, best_move, (char*)ws, err,
                                   (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// migration plans
// ---------------------------------------------------------------------------
static star_status check_plan_params(const star_plan_params* p) {
    if (!p) return STAR_ERR_INVALID_ARG;
    star_status st = check_variance_params(&p->load);
    if (st != STAR_OK) return st;
    if (p->max_moves < 0 || p->max_moves > STAR_MAX_MOVES) return STAR_ERR_INVALID_ARG;
    if (p->theta_num < 0 || p->theta_num > (1 << 20) || p->theta_den < 1 ||
        p->theta_den > (1 << 20))
        return STAR_ERR_INVALID_ARG;
    if ((p->u_rule != 0 && p->u_rule != 1) || (p->mem_rule != 0 && p->mem_rule != 1))
        return STAR_ERR_INVALID_ARG;
    if (p->mem_cap < 0) return STAR_ERR_INVALID_ARG;
    if (p->load.n_inst > 1024) return STAR_ERR_UNSUPPORTED;
    // n (theta_den + theta_num) w_i with w_i <= 65535 * sum of every load
    const long double H = (long double)p->load.bucket * p->load.n_buckets;
    const long double w = 65535.0L * ((long double)p->load.n_req + 1.0L) * H *
                          (2147483648.0L + H);
    const long double bound = (long double)p->load.n_inst * (2.0L * 1048576.0L) * w;
    if (!(bound < ldexpl(1.0L, 126))) return STAR_ERR_OVERFLOW;
    return STAR_OK;
}

STAR_API size_t star_plan_workspace_size(const star_plan_params* p) {
    if (check_plan_params(p) != STAR_OK) return 0;
    return plan_plan(*p).total;
}

STAR_API star_status star_plan_migrations(const star_plan_params* p, const int32_t* cur_len,
                                          const int32_t* rem_len, int32_t* inst_of,
                                          int64_t* load, const uint16_t* beta, star_move* moves,
                                          int32_t* n_moves, void* ws, size_t ws_bytes,
                                          void* stream) {
    star_status st = check_plan_params(p);
    if (st != STAR_OK) return st;
    if (!load || !beta || !n_moves) return STAR_ERR_INVALID_ARG;
    if (p->max_moves > 0 && !moves) return STAR_ERR_INVALID_ARG;
    if (p->load.n_req > 0 && (!cur_len || !rem_len || !inst_of)) return STAR_ERR_INVALID_ARG;
    if (!aligned(moves, 16)) return STAR_ERR_UNSUPPORTED;
    const PlanPlan pl = plan_plan(*p);
    st = check_ws(ws, ws_bytes, pl.total);
    if (st != STAR_OK) return st;
    int32_t* err = (int32_t*)((char*)ws + kHdrErrorWord);
    hipError_t e = launch_plan(*p, pl, cur_len, rem_len, inst_of, load, beta, moves, n_moves,
                               (char*)ws, err, (hipStream_t)stream);
    return e == hipSuccess ? STAR_OK : STAR_ERR_HIP;
}

// ---------------------------------------------------------------------------
// housekeeping
// ---------------------------------------------------------------------------
STAR_API star_status star_workspace_init(void* ws, size_t ws_bytes, void* stream) {
    star_status st = check_ws(ws, ws_bytes, STAR_WS_HEADER_BYTES);
    if (st != STAR_OK) return st;
    return launch_fill_zero(ws, ws_bytes, (hipStream_t)stream) == hipSuccess
               ? STAR_OK
               : STAR_ERR_HIP;
}

STAR_API star_status star_read_device_error(void* ws, void* stream, int32_t* code) {
    if (!code) return STAR_ERR_INVALID_ARG;
    if (!ws || !aligned(ws, 256)) return STAR_ERR_WORKSPACE;
    hipStream_t s = (hipStream_t)stream;
    if (hipStreamSynchronize(s) != hipSuccess) return STAR_ERR_HIP;
    int32_t v = 0;
    if (hipMemcpy(&v, (char*)ws + kHdrErrorWord, sizeof v, hipMemcpyDeviceToHost) != hipSuccess)
        return STAR_ERR_HIP;
    if (launch_fill_zero((char*)ws + kHdrErrorWord, 4, s) != hipSuccess) return STAR_ERR_HIP;
    if (hipStreamSynchronize(s) != hipSuccess) return STAR_ERR_HIP;
    *code = v;
    return v ? STAR_ERR_DEVICE_INPUT : STAR_OK;
}
