// (f1) Time-weighted variance change of every migration, on gfx950.
//
// Section 5.2 takes as the migration objective the variance of the
// instances' token loads now plus a beta-weighted sum of the variances of
// their predicted loads at later steps (Eq. 3-4).  Over bucketed curves that
// is Phi = sum_k beta_k Var_i(L_i[k]).  Moving request r (own curve R) from s
// to t keeps every bucket's mean, and changes bucket k's population variance
// by (2/n) R_k (R_k + L_t[k] - L_s[k]).  The library reports
//     G(r, t) = sum_k beta_k R_k (R_k + L_t[k] - L_s[k])   (= (n/2) dPhi),
// exactly, in 128-bit two's complement.  Sums, differences and products are
// taken modulo 2^128, which gives the exact value whenever |G| < 2^127; the
// host rejects sizes for which that could fail.
//
// With R_k = alpha + b^2 k below the request's end bucket k_e, p at k_e
// (the load model of Section 5.2), and the prefix sums
//     B0[k] = sum_{j<k} beta_j,   B1[k] = sum_{j<k} beta_j j,
//     B2[k] = sum_{j<k} beta_j j^2,
//     QA_i[k] = sum_{j<k} beta_j L_i[j],   QB_i[k] = sum_{j<k} beta_j j L_i[j],
// all read at k = k_e,
//     G = alpha^2 B0 + 2 alpha b^2 B1 + b^4 B2 + alpha (QA_t - QA_s)
//         + b^2 (QB_t - QB_s) + beta_{k_e} p (p + L_t[k_e] - L_s[k_e]),
// where the last term is present only when k_e < K.  The target enters
// through three gathers, so a candidate costs O(1) instead of the O(H)
// incremental update of the complexity analysis.
//
// Algorithm 1's best-feasible selection keeps the migration with the largest
// reduction, and only if it reduces the objective at all.  That is the
// smallest key (G, r n + t) with G < 0.
//
// Kernels:
//  * var_prep_kernel: one workgroup per instance row (QA, QB) plus one for
//    the weight sums (B0, B1, B2); a chunked block scan in LDS.
//  * var_score_kernel: each wave takes requests in groups of 64 / P lanes,
//    P = the power of two >= n (capped at 64; larger n loops over targets).
//    A lane scores one candidate, writes its gain, and the group's best
//    target comes from a butterfly of lane shuffles.  Negative best keys are
//    reduced per workgroup; the last workgroup to finish (atomic ticket)
//    reduces the workgroups' partials and writes the best feasible move.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

typedef unsigned __int128 u128;
typedef __int128 s128;

constexpr int VP_THREADS = 256;
constexpr int VS_THREADS = 256;
constexpr int VS_WAVES = VS_THREADS / kWave;
constexpr int VS_MAX_BLOCKS = 1024;

constexpr size_t kHdrVarTicket = 64;   // workspace header: finished-workgroup ticket

__device__ inline u128 wide(int64_t v) { return (u128)(s128)v; }

// ---------------------------------------------------------------------------
// prefix tables
// ---------------------------------------------------------------------------
// Row i < n: QA_i[k], QB_i[k] for k = 0..K.  Row n: B0[k], B1[k], B2[k].
// Thread j of the workgroup owns the buckets [j*per, (j+1)*per); its sums
// are scanned across the workgroup in LDS (inclusive Hillis-Steele; the
// exclusive prefix is the inclusive one minus the thread's own sum, which
// modular arithmetic allows), then each thread writes its run.
__global__ __launch_bounds__(VP_THREADS) void var_prep_kernel(const int64_t* __restrict__ load,
                                                              const uint16_t* __restrict__ beta,
                                                              int n, int K, u128* __restrict__ qa,
                                                              u128* __restrict__ qb,
                                                              u128* __restrict__ bs,
                                                              uint32_t* __restrict__ ticket) {
    __shared__ u128 sx[3][VP_THREADS];
    const int row = blockIdx.x, tid = threadIdx.x;
    const int K1 = K + 1;
    const bool wrow = row == n;
    const int per = (K + VP_THREADS - 1) / VP_THREADS;
    const int j0 = min(tid * per, K), j1 = min(j0 + per, K);
    const int64_t* L = load + (size_t)(wrow ? 0 : row) * K;

    if (row == 0 && tid == 0) *ticket = 0u;   // the scoring kernel runs after this one

    u128 x0 = 0, x1 = 0, x2 = 0;
    for (int j = j0; j < j1; ++j) {
        const u128 w = beta[j], uj = (u128)j;
        if (wrow) {
            x0 += w;
            x1 += w * uj;
            x2 += w * uj * uj;
        } else {
            const u128 wl = w * wide(L[j]);
            x0 += wl;
            x1 += wl * uj;
        }
    }
    sx[0][tid] = x0;
    sx[1][tid] = x1;
    sx[2][tid] = x2;
    __syncthreads();
    for (int o = 1; o < VP_THREADS; o <<= 1) {
        u128 y0 = 0, y1 = 0, y2 = 0;
        if (tid >= o) {
            y0 = sx[0][tid - o];
            y1 = sx[1][tid - o];
            y2 = sx[2][tid - o];
        }
        __syncthreads();
        sx[0][tid] += y0;
        sx[1][tid] += y1;
        sx[2][tid] += y2;
        __syncthreads();
    }
    u128 p0 = sx[0][tid] - x0, p1 = sx[1][tid] - x1, p2 = sx[2][tid] - x2;
    u128* o0 = wrow ? bs : qa + (size_t)row * K1;
    u128* o1 = wrow ? bs + K1 : qb + (size_t)row * K1;
    u128* o2 = bs + 2 * (size_t)K1;
    for (int j = j0; j < j1; ++j) {
        o0[j] = p0;
        o1[j] = p1;
        if (wrow) o2[j] = p2;
        const u128 w = beta[j], uj = (u128)j;
        if (wrow) {
            p0 += w;
            p1 += w * uj;
            p2 += w * uj * uj;
        } else {
            const u128 wl = w * wide(L[j]);
            p0 += wl;
            p1 += wl * uj;
        }
    }
    if (tid == VP_THREADS - 1) {
        o0[K] = sx[0][tid];
        o1[K] = sx[1][tid];
        if (wrow) o2[K] = sx[2][tid];
    }
}

// ---------------------------------------------------------------------------
// keys (gain, r n + t), ascending
// ---------------------------------------------------------------------------
struct VKey {
    s128 g;
    uint32_t idx;
};
constexpr uint32_t kNoIdx = 0xFFFFFFFFu;
__device__ inline VKey no_key() { return VKey{(s128)(~(u128)0 >> 1), kNoIdx}; }
__device__ inline bool vless(const VKey& a, const VKey& b) {
    return a.g < b.g || (a.g == b.g && a.idx < b.idx);
}
__device__ inline VKey vmin(const VKey& a, const VKey& b) { return vless(b, a) ? b : a; }

__device__ inline VKey shfl_xor_key(const VKey& k, int m) {
    const u128 u = (u128)k.g;
    const uint32_t w0 = (uint32_t)__shfl_xor((int)(uint32_t)u, m, kWave);
    const uint32_t w1 = (uint32_t)__shfl_xor((int)(uint32_t)(u >> 32), m, kWave);
    const uint32_t w2 = (uint32_t)__shfl_xor((int)(uint32_t)(u >> 64), m, kWave);
    const uint32_t w3 = (uint32_t)__shfl_xor((int)(uint32_t)(u >> 96), m, kWave);
    VKey o;
    o.g = (s128)(((u128)w3 << 96) | ((u128)w2 << 64) | ((u128)w1 << 32) | (u128)w0);
    o.idx = (uint32_t)__shfl_xor((int)k.idx, m, kWave);
    return o;
}

// min over lanes whose indexes differ only in the bits of [lo, hi)
__device__ inline VKey butterfly_min(VKey k, int lo, int hi) {
    for (int m = lo; m < hi; m <<= 1) k = vmin(k, shfl_xor_key(k, m));
    return k;
}

// A workgroup's partial, written and read with device-scope atomics so the
// last workgroup sees every other XCD's value.
struct VPart {
    uint64_t w[3];   // gain low, gain high, index
    uint64_t pad;
};
__device__ inline void store_part(VPart* p, const VKey& k) {
    const u128 u = (u128)k.g;
    __hip_atomic_store(&p->w[0], (uint64_t)u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->w[1], (uint64_t)(u >> 64), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&p->w[2], (uint64_t)k.idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline VKey load_part(VPart* p) {
    const uint64_t lo = __hip_atomic_load(&p->w[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t hi = __hip_atomic_load(&p->w[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint64_t ix = __hip_atomic_load(&p->w[2], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return VKey{(s128)(((u128)hi << 64) | (u128)lo), (uint32_t)ix};
}

struct VarArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* load;
    const uint16_t* beta;
    const u128* qa;
    const u128* qb;
    const u128* bs;
    u128* gain;              // [N, n] or null
    int32_t* best_target;    // [N] or null
    u128* best_gain;         // [N] or null
    star_move* move;         // one, or null
    VPart* part;             // [gridDim.x] when move != null
    uint32_t* ticket;
    int32_t* err;
    int N, n, b, K;
    int lpr_log2;            // lanes per request = 1 << lpr_log2 (<= 64)
    int groups;              // request groups of 64 >> lpr_log2 requests
    int64_t H;
};

__global__ __launch_bounds__(VS_THREADS) void var_score_kernel(VarArgs a) {
    __shared__ VKey wbest[VS_WAVES];
    __shared__ bool last;
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    const int lpr = 1 << a.lpr_log2, rpw = kWave >> a.lpr_log2;
    const int sub = lane >> a.lpr_log2, tl = lane & (lpr - 1);
    const int n = a.n, K = a.K, K1 = K + 1;
    const u128 bb = (u128)a.b * (u128)a.b;
    VKey feas = no_key();   // this lane's view of the wave's best negative key

    for (int grp = blockIdx.x * VS_WAVES + wid; grp < a.groups; grp += gridDim.x * VS_WAVES) {
        const int r = grp * rpw + sub;
        const bool live = r < a.N;
        ReqTerms q{};
        if (live) q = request_terms(a.inst[r], a.cur[r], a.rem[r], n, a.b, a.H);
        const bool valid = live && q.bad == 0;
        if (live && tl == 0) report_error(a.err, q.bad);

        // the request's part of G, independent of the target
        u128 base = 0, bp = 0, al = 0;
        const int ke = q.ke;
        const bool part = valid && ke < K;
        if (valid) {
            al = wide(q.alpha);
            const u128 b0 = a.bs[ke], b1 = a.bs[K1 + ke], b2 = a.bs[2 * K1 + ke];
            const size_t so = (size_t)q.s * K1 + ke;
            base = al * al * b0 + (u128)2 * al * bb * b1 + bb * bb * b2 - al * a.qa[so] -
                   bb * a.qb[so];
            if (part) {
                bp = (u128)a.beta[ke] * wide(q.p);
                base += bp * (wide(q.p) - wide(a.load[(size_t)q.s * K + ke]));
            }
        }
        VKey best = no_key();
        for (int t = tl; t < n; t += lpr) {
            if (!live) break;
            u128 g = 0;
            if (valid && t != q.s) {
                const size_t to = (size_t)t * K1 + ke;
                g = base + al * a.qa[to] + bb * a.qb[to];
                if (part) g += bp * wide(a.load[(size_t)t * K + ke]);
                best = vmin(best, VKey{(s128)g, (uint32_t)r * (uint32_t)n + (uint32_t)t});
            }
            if (a.gain) a.gain[(size_t)r * n + t] = g;
        }
        best = butterfly_min(best, 1, lpr);
        if (live && tl == 0) {
            const bool has = best.idx != kNoIdx;
            if (a.best_target)
                a.best_target[r] = has ? (int32_t)(best.idx - (uint32_t)r * (uint32_t)n) : -1;
            if (a.best_gain) a.best_gain[r] = has ? (u128)best.g : (u128)0;
        }
        if (best.g < 0) feas = vmin(feas, best);
    }
    if (!a.move) return;

    // best negative key of the workgroup, then of the grid
    feas = butterfly_min(feas, 1, kWave);
    if (lane == 0) wbest[wid] = feas;
    __syncthreads();
    if (threadIdx.x == 0) {
        VKey k = wbest[0];
        for (int w = 1; w < VS_WAVES; ++w) k = vmin(k, wbest[w]);
        store_part(&a.part[blockIdx.x], k);
        __threadfence();
        const uint32_t done = atomicAdd(a.ticket, 1u);
        last = done == gridDim.x - 1;
    }
    __syncthreads();
    if (!last) return;
    __threadfence();
    VKey k = no_key();
    for (int g = threadIdx.x; g < (int)gridDim.x; g += VS_THREADS) k = vmin(k, load_part(&a.part[g]));
    k = butterfly_min(k, 1, kWave);
    if (lane == 0) wbest[wid] = k;
    __syncthreads();
    if (threadIdx.x == 0) {
        VKey m = wbest[0];
        for (int w = 1; w < VS_WAVES; ++w) m = vmin(m, wbest[w]);
        star_move mv;
        if (m.idx != kNoIdx) {
            const int r = (int)(m.idx / (uint32_t)n);
            mv.req = r;
            mv.src = a.inst[r];
            mv.tgt = (int)(m.idx - (uint32_t)r * (uint32_t)n);
            mv.gain.lo = (uint64_t)(u128)m.g;
            mv.gain.hi = (int64_t)(m.g >> 64);
        } else {
            mv.req = mv.src = mv.tgt = -1;
            mv.gain.lo = 0;
            mv.gain.hi = 0;
        }
        mv.reserved = 0;
        *a.move = mv;
        *a.ticket = 0u;
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
VarPlan plan_variance(const star_load_params& p) {
    VarPlan pl;
    const int n = p.n_inst, N = p.n_req;
    const size_t K1 = (size_t)p.n_buckets + 1;
    int lg = 0;
    while ((1 << lg) < n && lg < 6) ++lg;
    pl.lpr_log2 = lg;
    const int rpw = kWave >> lg;
    pl.groups = (int)ceil_div(N, rpw);
    const int64_t blocks = ceil_div(pl.groups, VS_WAVES);
    pl.blocks = (int)(blocks < 1 ? 1 : blocks > VS_MAX_BLOCKS ? VS_MAX_BLOCKS : blocks);
    size_t off = STAR_WS_HEADER_BYTES;
    pl.qa_off = off;
    off += align_up((size_t)n * K1 * sizeof(u128), 256);
    pl.qb_off = off;
    off += align_up((size_t)n * K1 * sizeof(u128), 256);
    pl.bs_off = off;
    off += align_up(3 * K1 * sizeof(u128), 256);
    pl.part_off = off;
    off += align_up((size_t)pl.blocks * sizeof(VPart), 256);
    pl.total = off;
    return pl;
}

hipError_t launch_variance(const star_load_params& p, const VarPlan& pl, const int32_t* cur,
                           const int32_t* rem, const int32_t* inst, const int64_t* load,
                           const uint16_t* beta, star_i128* gain, int32_t* best_target,
                           star_i128* best_gain, star_move* move, char* ws, int32_t* err,
                           hipStream_t stream) {
    static_assert(sizeof(star_i128) == sizeof(u128), "star_i128 is one 128-bit integer");
    const int n = p.n_inst, K = p.n_buckets;
    u128* qa = (u128*)(ws + pl.qa_off);
    u128* qb = (u128*)(ws + pl.qb_off);
    u128* bs = (u128*)(ws + pl.bs_off);
    uint32_t* ticket = (uint32_t*)(ws + kHdrVarTicket);
    hipLaunchKernelGGL(var_prep_kernel, dim3(n + 1), dim3(VP_THREADS), 0, stream, load, beta, n,
                       K, qa, qb, bs, ticket);
    VarArgs a;
    a.cur = cur;
    a.rem = rem;
    a.inst = inst;
    a.load = load;
    a.beta = beta;
    a.qa = qa;
    a.qb = qb;
    a.bs = bs;
    a.gain = (u128*)gain;
    a.best_target = best_target;
    a.best_gain = (u128*)best_gain;
    a.move = move;
    a.part = (VPart*)(ws + pl.part_off);
    a.ticket = ticket;
    a.err = err;
    a.N = p.n_req;
    a.n = n;
    a.b = p.bucket;
    a.K = K;
    a.lpr_log2 = pl.lpr_log2;
    a.groups = pl.groups;
    a.H = (int64_t)p.bucket * K;
    hipLaunchKernelGGL(var_score_kernel, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
    return hipGetLastError();
}

}  // namespace star
