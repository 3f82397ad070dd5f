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
//  * var_prep_kernel: one workgroup per instance (QA, QB) plus one for the
//    weight sums (B0, B1, B2); a chunked block scan in LDS.  The
//    per-instance tables are stored bucket-major, [k][t] (and a bucket-major
//    copy of the curves), so that the lanes scoring one request's targets
//    read one contiguous run.
//  * var_score_kernel: up to 16 lanes per request; a lane walks every 16th
//    target (reads and writes stay contiguous across the request's lanes)
//    and keeps its best key in registers, and a short DPP scan combines the
//    lanes.  Negative best keys are reduced per workgroup.  In small grids the last workgroup to finish
//    (atomic ticket) reduces the workgroups' partials and writes the best
//    feasible move; larger grids leave that to var_final_kernel.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

typedef unsigned __int128 u128;
typedef __int128 s128;

constexpr int VP_THREADS = 256;
constexpr int VS_THREADS = 256;
constexpr int VS_WAVES = VS_THREADS / kWave;

// Grids up to this many workgroups find the best move in the scoring kernel
// (the last workgroup to finish reduces the partials); larger ones hand the
// partials to a one-workgroup kernel, because every workgroup's release
// fence would write back its XCD's L2, full of freshly written gains.
constexpr int VS_TICKET_BLOCKS = 64;
constexpr int VS_MAX_LG = 4;             // at most 16 lanes per request
constexpr int PLAN_MAX_INST = 1024;      // instances a plan classifies in LDS
constexpr int PA_THREADS = 256;          // the plan's update workgroup
constexpr int PLAN_MAX_BLOCKS = 1 << 20; // scoring workgroups of a plan pass (one tile each)


__device__ inline u128 wide(int64_t v) { return (u128)(s128)v; }

// a * x modulo 2^128 for a 128-bit a and a non-negative 64-bit x: one full
// 64 x 64 product and one low half
__device__ inline u128 mul_u64(u128 a, uint64_t x) {
    return (u128)(uint64_t)a * x + ((u128)((uint64_t)(a >> 64) * x) << 64);
}
// a * x modulo 2^128 for a signed 64-bit x (x sign-extended to 128 bits)
__device__ inline u128 mul_s64(u128 a, int64_t x) {
    u128 r = mul_u64(a, (uint64_t)x);
    if (x < 0) r -= a << 64;
    return r;
}

// one bucket-major table entry: QA_t[k], QB_t[k]
struct QEntry {
    u128 qa, qb;
};

// ---------------------------------------------------------------------------
// prefix tables
// ---------------------------------------------------------------------------
// Row i < n: QA_i[k], QB_i[k] for k = 0..K.  Row n: B0[k], B1[k], B2[k].
// Thread j of the workgroup owns the buckets [j*per, (j+1)*per); its sums
// are scanned across the workgroup in LDS (inclusive Hillis-Steele; the
// exclusive prefix is the inclusive one minus the thread's own sum, which
// modular arithmetic allows), then each thread writes its run.  Up to
// VP_REG buckets per thread stay in registers between the two passes, so
// that no load waits behind the table stores (loads and stores share one
// counter on gfx9).
constexpr int VP_REG = 8;

__device__ inline void prep_load(const uint16_t* beta, const int64_t* L, bool wrow, int c0,
                                 int last, uint32_t* wv, int64_t* lv) {
#pragma unroll
    for (int i = 0; i < VP_REG; ++i) {
        const int j = c0 + i < last ? c0 + i : last;   // clamped: no branch per slot
        wv[i] = beta[j];
        lv[i] = wrow ? 0 : L[j];
    }
}

// The tables of one row, computed by the whole workgroup (sx: LDS of
// 3 x VP_THREADS entries).  L is the instance's curve (row < n) or unused
// (the weights' row, wrow).  A thread reads back only buckets it owns, so
// a caller may have just written them itself.
__device__ void prep_row(const int64_t* __restrict__ L, const uint16_t* __restrict__ beta, int n,
                         int K, int row, bool wrow, QEntry* __restrict__ qt,
                         int64_t* __restrict__ lt, u128* __restrict__ bs, u128 (*sx)[VP_THREADS]) {
    const int tid = threadIdx.x;
    const int K1 = K + 1;
    const int per = (K + VP_THREADS - 1) / VP_THREADS;
    const int j0 = min(tid * per, K), j1 = min(j0 + per, K);
    __syncthreads();   // sx may still be read by a previous row

    uint32_t wv[VP_REG];
    int64_t lv[VP_REG];
    u128 x0 = 0, x1 = 0, x2 = 0;
    for (int c0 = j0; c0 < j1; c0 += VP_REG) {
        prep_load(beta, L, wrow, c0, j1 - 1, wv, lv);
#pragma unroll
        for (int i = 0; i < VP_REG; ++i) {
            const bool in = c0 + i < j1;
            const u128 w = in ? (u128)wv[i] : (u128)0, uj = (u128)(c0 + i);
            if (wrow) {
                x0 += w;
                x1 += w * uj;
                x2 += w * uj * uj;
            } else {
                const u128 wl = mul_s64(w, lv[i]);
                x0 += wl;
                x1 += wl * uj;
            }
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
    for (int c0 = j0; c0 < j1; c0 += VP_REG) {
        if (per > VP_REG) prep_load(beta, L, wrow, c0, j1 - 1, wv, lv);
#pragma unroll
        for (int i = 0; i < VP_REG; ++i) {
            const int j = c0 + i;
            if (j >= j1) break;
            const u128 w = wv[i], uj = (u128)j;
            if (wrow) {
                bs[j] = p0;
                bs[K1 + j] = p1;
                bs[2 * (size_t)K1 + j] = p2;
                p0 += w;
                p1 += w * uj;
                p2 += w * uj * uj;
            } else {
                qt[(size_t)j * n + row] = QEntry{p0, p1};
                lt[(size_t)j * n + row] = lv[i];
                const u128 wl = mul_s64(w, lv[i]);
                p0 += wl;
                p1 += wl * uj;
            }
        }
    }
    if (tid == VP_THREADS - 1) {
        if (wrow) {
            bs[K] = sx[0][tid];
            bs[K1 + K] = sx[1][tid];
            bs[2 * (size_t)K1 + K] = sx[2][tid];
        } else {
            qt[(size_t)K * n + row] = QEntry{sx[0][tid], sx[1][tid]};
        }
    }
}

__global__ __launch_bounds__(VP_THREADS) void var_prep_kernel(const int64_t* __restrict__ load,
                                                              const uint16_t* __restrict__ beta,
                                                              int n, int K,
                                                              QEntry* __restrict__ qt,
                                                              int64_t* __restrict__ lt,
                                                              u128* __restrict__ bs,
                                                              uint32_t* __restrict__ ticket) {
    __shared__ u128 sx[3][VP_THREADS];
    const int row = blockIdx.x;
    if (row == 0 && threadIdx.x == 0) *ticket = 0u;   // the scoring kernel runs after this one
    prep_row(load + (size_t)(row == n ? 0 : row) * K, beta, n, K, row, row == n, qt, lt, bs, sx);
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

// DPP move of a whole key; a lane whose source lies outside its row, or in
// a row that kRowMask leaves out, receives the no-key sentinel
template <int kCtrl, int kRowMask>
__device__ inline VKey dpp_key(const VKey& k) {
    const u128 u = (u128)k.g;
    const u128 inf = ~(u128)0 >> 1;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
        w[i] = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(inf >> (32 * i)),
                                                    (int)(uint32_t)(u >> (32 * i)), kCtrl,
                                                    kRowMask, 0xF, false);
    VKey o;
    o.g = (s128)(((u128)w[3] << 96) | ((u128)w[2] << 64) | ((u128)w[1] << 32) | (u128)w[0]);
    o.idx = (uint32_t)__builtin_amdgcn_update_dpp((int)kNoIdx, (int)k.idx, kCtrl, kRowMask, 0xF,
                                                  false);
    return o;
}

// Minimum over each aligned group of 2^lg lanes (lg <= 6), valid in the
// group's last lane: an inclusive min-scan by DPP row shifts, where a lane
// ignores a source in the previous group (tl = lane index in its group),
// then the row broadcasts for groups of 32 and 64 lanes.  Every lane of the
// wave must be active.
__device__ inline VKey group_min(VKey k, int lg, int tl) {
    VKey o;
    if (lg >= 1) {
        o = dpp_key<kDppRowShr1, 0xF>(k);
        if (tl >= 1 && vless(o, k)) k = o;
    }
    if (lg >= 2) {
        o = dpp_key<kDppRowShr2, 0xF>(k);
        if (tl >= 2 && vless(o, k)) k = o;
    }
    if (lg >= 3) {
        o = dpp_key<kDppRowShr4, 0xF>(k);
        if (tl >= 4 && vless(o, k)) k = o;
    }
    if (lg >= 4) {
        o = dpp_key<kDppRowShr8, 0xF>(k);
        if (tl >= 8 && vless(o, k)) k = o;
    }
    if (lg >= 5) {
        o = dpp_key<kDppRowBcast15, 0xA>(k);
        if (vless(o, k)) k = o;
    }
    if (lg >= 6) {
        o = dpp_key<kDppRowBcast31, 0xC>(k);
        if (vless(o, k)) k = o;
    }
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

// One workgroup: the smallest of `parts` partial keys, written as the move
// (or the no-move record when none is negative).
// One workgroup: the smallest of `parts` partial keys, returned to every
// thread.
template <bool kAtomic, int kThreads = VS_THREADS>
__device__ VKey reduce_keys(VPart* part, int parts, VKey* wbest) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    constexpr int kBatch = 8;   // partials in flight per thread
    VKey k = no_key();
    for (int g0 = tid; g0 < parts; g0 += kThreads * kBatch) {
        VKey p[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int g = g0 + i * kThreads;
            VPart* src = &part[g < parts ? g : parts - 1];
            if (kAtomic) {
                p[i] = load_part(src);
            } else {
                const VPart v = *src;
                p[i] = VKey{(s128)(((u128)v.w[1] << 64) | (u128)v.w[0]), (uint32_t)v.w[2]};
            }
        }
#pragma unroll
        for (int i = 0; i < kBatch; ++i) k = vmin(k, p[i]);   // repeats are harmless
    }
    k = group_min(k, 6, lane);
    if (lane == kWave - 1) wbest[wid] = k;
    __syncthreads();
    VKey m = wbest[0];
    for (int w = 1; w < kThreads / kWave; ++w) m = vmin(m, wbest[w]);
    __syncthreads();
    return m;
}

// The move record of key m (or the no-move record).
__device__ inline star_move move_of(const VKey& m, const int32_t* inst, int n) {
    star_move mv;
    if (m.idx != kNoIdx) {
        const int r = (int)(m.idx / (uint32_t)n);
        mv.req = r;
        mv.src = inst[r];
        mv.tgt = (int)(m.idx - (uint32_t)r * (uint32_t)n);
        mv.gain.lo = (uint64_t)(u128)m.g;
        mv.gain.hi = (int64_t)(m.g >> 64);
    } else {
        mv.req = mv.src = mv.tgt = -1;
        mv.gain.lo = 0;
        mv.gain.hi = 0;
    }
    mv.reserved = 0;
    return mv;
}

template <bool kAtomic>
__device__ void reduce_parts(VPart* part, int parts, const int32_t* inst, int n, star_move* move,
                             VKey* wbest) {
    const VKey m = reduce_keys<kAtomic>(part, parts, wbest);
    if (threadIdx.x == 0) *move = move_of(m, inst, n);
}

// A request's target-independent part of G, staged in LDS.
struct ReqStash {
    u128 base, bp;
    uint64_t al;
    int32_t ke;
    int32_t s;        // source instance; -2: no candidates (invalid request, or a
                      // source Algorithm 1 does not move from); -1: past the end
    int64_t need;     // memory the request takes on a target (plans)
};

struct VarArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const uint16_t* beta;
    const QEntry* qt;        // [K + 1][n]
    const int64_t* lt;       // [K][n]
    const u128* bs;          // [3][K + 1]
    u128* gain;              // [N, n] or null
    int32_t* best_target;    // [N] or null
    u128* best_gain;         // [N] or null
    star_move* move;         // one, or null
    VPart* part;             // [gridDim.x] when move != null
    uint32_t* ticket;
    int32_t* err;
    int N, n, b, K;
    int ticketed;            // 1: the last workgroup reduces the partials
    int tiles;               // request tiles (workgroups loop over them in plans)
    int64_t H;
    // plans (Algorithm 1's classification and candidate filters)
    const int64_t* now;      // [n] current loads N_i
    const int32_t* done;     // nonzero: the plan has stopped
    int theta_num, theta_den, u_rule, mem_rule, min_rem;
    int64_t mem_cap;
};

constexpr int VS_M = 4;      // targets per lane per chunk

// (g, t) keys of one request: smaller gain, then smaller target
__device__ inline bool gt_less(s128 ga, int ta, s128 gb, int tb) {
    return ga < gb || (ga == gb && (uint32_t)ta < (uint32_t)tb);
}

// One DPP step of the per-request reduction: the key of lane - S (row
// shift) replaces this lane's if smaller; lanes whose source lies in the
// previous request's group (or row) keep theirs.
template <int kCtrl, int S>
__device__ inline void dpp_step(s128& g, int& t, int tl) {
    const u128 u = (u128)g;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int x = (int)(uint32_t)(u >> (32 * i));
        w[i] = (uint32_t)__builtin_amdgcn_update_dpp(x, x, kCtrl, 0xF, 0xF, false);
    }
    const int to = __builtin_amdgcn_update_dpp(t, t, kCtrl, 0xF, 0xF, false);
    const s128 go =
        (s128)(((u128)w[3] << 96) | ((u128)w[2] << 64) | ((u128)w[1] << 32) | (u128)w[0]);
    if (tl >= S && gt_less(go, to, g, t)) {
        g = go;
        t = to;
    }
}

// A workgroup takes VS_WAVES * 64 / P requests (P = 2^LG <= 16 lanes per
// request).  Phase A: thread j stages request j's target-independent terms
// in LDS (coalesced reads, one gather of the weight sums and of its
// source's entry).  Phase B: each wave takes 64 / P requests at once; lane
// l of a request's group walks the targets l, l + P, ... in chunks of
// VS_M, loading a chunk's table entries (contiguous across the group)
// before storing its gains and keeping its best key in registers; then an
// LG-step DPP row-shift scan leaves the request's best key in the group's
// last lane.  One pass per wave: on gfx9 loads and stores share one
// counter, so a second pass's loads would wait for the first pass's stores.
//
// Plans (kPlan): Algorithm 1's classification runs first in every
// workgroup.  w_i = QA_i[K] comes straight from the tables; O = {w_i > (1 +
// theta) mean w}; U by the chosen rule; for each target the memory room
// C_mem - N_t (or -1 outside U).  Only requests on an instance of O with
// rem_len > min_rem are staged as sources, a candidate must fit the room,
// and only the workgroup's best negative key is written.
template <int LG, bool kPlan>
__global__ __launch_bounds__(VS_THREADS) void var_score_kernel(VarArgs a) {
    constexpr int P = 1 << LG, RPW = kWave / P, TILE = VS_WAVES * RPW;
    constexpr int NM = kPlan ? PLAN_MAX_INST : 1;
    __shared__ ReqStash st[TILE];
    __shared__ VKey wbest[VS_WAVES];
    __shared__ bool last;
    __shared__ uint8_t over_m[NM];
    __shared__ int64_t room_m[NM];
    __shared__ u128 wred[kPlan ? VS_THREADS : 1];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int sub = lane >> LG, tl = lane & (P - 1);
    const int n = a.n, K = a.K, K1 = K + 1;
    const uint64_t bb = (uint64_t)a.b * (uint64_t)a.b;
    const QEntry* __restrict__ qt = a.qt;
    const int64_t* __restrict__ lt = a.lt;
    u128* __restrict__ gain = a.gain;

    if (kPlan) {
        if (*a.done) return;
        // classification: sum of w, then O and the targets' room
        u128 acc = 0;
        for (int i = tid; i < n; i += VS_THREADS) acc += qt[(size_t)K * n + i].qa;
        wred[tid] = acc;
        __syncthreads();
        for (int o = VS_THREADS / 2; o > 0; o >>= 1) {
            if (tid < o) wred[tid] += wred[tid + o];
            __syncthreads();
        }
        const s128 wsum = (s128)wred[0];
        const s128 den = a.theta_den, num = a.theta_num;
        const s128 hi = (den + num) * wsum, lo = (den - num) * wsum;   // n den (1 +- theta) mean w
        for (int i = tid; i < n; i += VS_THREADS) {
            const s128 nw = (s128)n * den * (s128)qt[(size_t)K * n + i].qa;
            const int64_t now = a.now[i];
            over_m[i] = nw > hi;
            const bool under = a.u_rule == 0 ? (s128)n * den * (s128)now < hi : nw < lo;
            room_m[i] = under ? a.mem_cap - now : -1;
        }
        __syncthreads();
    }

    VKey feas = no_key();   // best key of this lane's requests that lowers the objective
    for (int tile = blockIdx.x; tile < a.tiles; tile += gridDim.x) {
        const int r0 = tile * TILE;
        __syncthreads();   // the previous tile's stash has been read
        if (tid < TILE) {
            const int r = r0 + tid;
            ReqStash e;
            e.base = 0;
            e.bp = 0;
            e.al = 0;
            e.ke = 0;
            e.s = -1;
            e.need = 0;
            if (r < a.N) {
                const ReqTerms q = request_terms(a.inst[r], a.cur[r], a.rem[r], n, a.b, a.H);
                if (!kPlan) report_error(a.err, q.bad);
                bool src_ok = !q.bad;
                if (kPlan && src_ok) {
                    src_ok = over_m[q.s] && a.rem[r] > a.min_rem;
                    e.need = a.rem[r] + (a.mem_rule ? a.cur[r] : 0);
                }
                e.s = src_ok ? q.s : -2;
                if (src_ok) {
                    // alpha, b^2 and p are non-negative and below 2^62
                    const uint64_t al = (uint64_t)q.alpha;
                    const int ke = q.ke;
                    const u128 b0 = a.bs[ke], b1 = a.bs[K1 + ke], b2 = a.bs[2 * K1 + ke];
                    const QEntry qs = qt[(size_t)ke * n + q.s];
                    u128 base = mul_u64(mul_u64(b0, al), al) + mul_u64(mul_u64(b1, al), 2 * bb) +
                                mul_u64(mul_u64(b2, bb), bb) - mul_u64(qs.qa, al) -
                                mul_u64(qs.qb, bb);
                    u128 bp = 0;
                    if (ke < K) {
                        bp = (u128)a.beta[ke] * (u128)(uint64_t)q.p;
                        base += mul_s64(bp, q.p - lt[(size_t)ke * n + q.s]);
                    }
                    e.base = base;
                    e.bp = bp;
                    e.al = al;
                    e.ke = ke;
                }
            }
            st[tid] = e;
        }
        __syncthreads();

        const int j = wid * RPW + sub;
        const int r = r0 + j;
        const u128 base = st[j].base, bp = st[j].bp;
        const uint64_t al = st[j].al;
        const int ke = st[j].ke, src = st[j].s;
        const int64_t need = st[j].need;
        const bool live = src != -1, valid = src >= 0;
        const size_t row = valid ? (size_t)ke * n : 0;   // others read entry 0, unused
        s128 bg = ~(u128)0 >> 1;
        int bt = -1;
        for (int c0 = 0; c0 < n; c0 += P * VS_M) {
            QEntry qe[VS_M];
            int64_t le[VS_M];
#pragma unroll
            for (int i = 0; i < VS_M; ++i) {
                const int t = c0 + tl + P * i;
                const size_t o = row + (t < n ? t : 0);
                qe[i] = qt[o];
                le[i] = lt[o];
            }
#pragma unroll
            for (int i = 0; i < VS_M; ++i) {
                const int t = c0 + tl + P * i;
                u128 g = 0;
                if (valid) {   // whole waves without a source skip the arithmetic
                    g = base + mul_u64(qe[i].qa, al) + mul_u64(qe[i].qb, bb);
                    if (ke < K) g += mul_s64(bp, le[i]);
                }
                bool mig = valid && t < n && t != src;
                if (kPlan) mig = mig && need <= room_m[t < n ? t : 0];
                if (!mig) g = 0;
                if (mig && (s128)g < bg) {   // targets ascend within a lane
                    bg = (s128)g;
                    bt = t;
                }
                if (!kPlan && gain && live && t < n) gain[(size_t)r * n + t] = g;
            }
        }
        if (LG >= 1) dpp_step<kDppRowShr1, 1>(bg, bt, tl);
        if (LG >= 2) dpp_step<kDppRowShr2, 2>(bg, bt, tl);
        if (LG >= 3) dpp_step<kDppRowShr4, 4>(bg, bt, tl);
        if (LG >= 4) dpp_step<kDppRowShr8, 8>(bg, bt, tl);

        if (live && tl == P - 1) {
            if (!kPlan && a.best_target) a.best_target[r] = bt;
            if (!kPlan && a.best_gain) a.best_gain[r] = bt >= 0 ? (u128)bg : (u128)0;
            if (bt >= 0 && bg < 0)
                feas = vmin(feas, VKey{bg, (uint32_t)r * (uint32_t)n + (uint32_t)bt});
        }
    }
    if (!kPlan && !a.move) return;

    // best negative key of the workgroup, then (small grids) of the grid
    feas = group_min(feas, 6, lane);
    if (lane == kWave - 1) wbest[wid] = feas;
    __syncthreads();
    if (tid == 0) {
        VKey k = wbest[0];
        for (int w = 1; w < VS_WAVES; ++w) k = vmin(k, wbest[w]);
        store_part(&a.part[blockIdx.x], k);
        if (!kPlan && a.ticketed) {
            // small grids only: this release fence writes back the XCD's L2
            __threadfence();
            last = atomicAdd(a.ticket, 1u) == gridDim.x - 1;
        }
    }
    if (kPlan || !a.ticketed) return;
    __syncthreads();
    if (!last) return;
    __threadfence();
    reduce_parts<true>(a.part, gridDim.x, a.inst, n, a.move, wbest);
    if (tid == 0) *a.ticket = 0u;
}

// The best feasible move from the scoring workgroups' partials (large grids,
// after the scoring kernel has finished).
__global__ __launch_bounds__(VS_THREADS) void var_final_kernel(VPart* part, int parts,
                                                               const int32_t* inst, int n,
                                                               star_move* move) {
    __shared__ VKey wbest[VS_WAVES];
    reduce_parts<false>(part, parts, inst, n, move, wbest);
}

// ---------------------------------------------------------------------------
// (f2) Algorithm 1 end to end: one migration per pass, repeated
// ---------------------------------------------------------------------------
struct PlanArgs {
    const int32_t* cur;
    const int32_t* rem;
    int32_t* inst;           // updated in place
    int64_t* load;           // [n, K], updated in place
    const uint16_t* beta;
    QEntry* qt;
    int64_t* lt;
    u128* bs;
    VPart* part;
    int parts;
    int64_t* now;            // [n] current loads N_i
    int32_t* done;
    int32_t* count;
    int32_t* n_moves;        // caller's move count
    star_move* moves;        // caller's [max_moves]
    int32_t* err;
    int N, n, b, K;
    int64_t H;
};

// The plan's state: current loads (accumulated by plan_prep_kernel), stop
// flag and move counts.
__global__ void plan_zero_kernel(int64_t* now, int n, int32_t* done, int32_t* count,
                                 int32_t* n_moves) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) now[i] = 0;
    if (threadIdx.x == 0) {
        *done = 0;
        *count = 0;
        *n_moves = 0;
    }
}

constexpr int PLAN_REQ_CHUNK = 4096;     // requests per current-load workgroup

// Workgroups 0..n: the tables of every row (as var_prep_kernel).  The
// others: each sums cur_len per instance over a chunk of valid requests in
// LDS and adds the sums to N_i (int64 atomics: exact, any order), and
// reports invalid requests.
__global__ __launch_bounds__(VP_THREADS) void plan_prep_kernel(PlanArgs a) {
    __shared__ u128 sx[3][VP_THREADS];
    __shared__ unsigned long long hist[PLAN_MAX_INST];
    const int row = blockIdx.x, tid = threadIdx.x, n = a.n;
    if (row <= n) {
        prep_row(a.load + (size_t)(row == n ? 0 : row) * a.K, a.beta, n, a.K, row, row == n,
                 a.qt, a.lt, a.bs, sx);
        return;
    }
    for (int i = tid; i < n; i += VP_THREADS) hist[i] = 0;
    __syncthreads();
    const int r0 = (row - n - 1) * PLAN_REQ_CHUNK;
    const int r1 = min(a.N, r0 + PLAN_REQ_CHUNK);
    int32_t bad = 0;
    for (int r = r0 + tid; r < r1; r += VP_THREADS) {
        const int s = a.inst[r], c = a.cur[r], l = a.rem[r];
        int32_t f = 0;
        if (s < 0 || s >= n) f |= STAR_DEV_BAD_INST;
        if (c < 1) f |= STAR_DEV_BAD_CUR;
        if (l < 1) f |= STAR_DEV_BAD_REM;
        if (!f) atomicAdd(&hist[s], (unsigned long long)c);
        bad |= f;
    }
    report_error(a.err, bad);
    __syncthreads();
    for (int i = tid; i < n; i += VP_THREADS)
        if (hist[i]) atomicAdd((unsigned long long*)&a.now[i], hist[i]);
}

// One workgroup after each scoring pass: the best feasible key of the
// pass; none stops the plan.  Otherwise the move is recorded and executed:
// inst_of[r] = t, N_s and N_t adjusted, r's own curve R taken from row s
// and added to row t of the curves.  The tables change by closed forms, so
// no scan is needed: with F_A(k) = sum_{j<k} beta_j R_j and
// F_B(k) = sum_{j<k} beta_j j R_j,
//     F_A(k) = alpha B0[k] + b^2 B1[k],  F_B(k) = alpha B1[k] + b^2 B2[k]
// for k <= k_e, and for k > k_e the value at k_e plus beta_{k_e} p (times
// k_e for F_B); QA and QB of row s fall by F, those of row t rise by F.
__global__ __launch_bounds__(PA_THREADS) void plan_apply_kernel(PlanArgs a) {
    __shared__ VKey wbest[PA_THREADS / kWave];
    if (*a.done) return;
    const int tid = threadIdx.x, n = a.n, K = a.K, K1 = K + 1;
    const VKey m = reduce_keys<false, PA_THREADS>(a.part, a.parts, wbest);
    if (m.idx == kNoIdx) {
        if (tid == 0) *a.done = 1;
        return;
    }
    const int r = (int)(m.idx / (uint32_t)n);
    const int t = (int)(m.idx - (uint32_t)r * (uint32_t)n);
    const int s = a.inst[r];
    const int c = a.cur[r];
    __syncthreads();   // every thread has read inst[r] before it changes
    if (tid == 0) {
        const int q = *a.count;
        star_move mv;
        mv.req = r;
        mv.src = s;
        mv.tgt = t;
        mv.reserved = 0;
        mv.gain.lo = (uint64_t)(u128)m.g;
        mv.gain.hi = (int64_t)(m.g >> 64);
        a.moves[q] = mv;
        *a.count = q + 1;
        *a.n_moves = q + 1;
        a.inst[r] = t;
        a.now[s] -= c;
        a.now[t] += c;
    }
    const ReqTerms rq = request_terms(t, c, a.rem[r], n, a.b, a.H);
    const int ke = rq.ke;
    const uint64_t al = (uint64_t)rq.alpha;
    const uint64_t bb = (uint64_t)a.b * (uint64_t)a.b;
    const u128 tail = ke < K ? (u128)a.beta[ke] * (u128)(uint64_t)rq.p : (u128)0;
    for (int k = tid; k <= K; k += PA_THREADS) {
        const int kk = k <= ke ? k : ke;
        u128 fa = mul_u64(a.bs[kk], al) + mul_u64(a.bs[K1 + kk], bb);
        u128 fb = mul_u64(a.bs[K1 + kk], al) + mul_u64(a.bs[2 * (size_t)K1 + kk], bb);
        if (k > ke) {
            fa += tail;
            fb += mul_u64(tail, (uint64_t)ke);
        }
        QEntry* es = &a.qt[(size_t)k * n + s];
        QEntry* et = &a.qt[(size_t)k * n + t];
        const QEntry vs = *es, vt = *et;
        *es = QEntry{vs.qa - fa, vs.qb - fb};
        *et = QEntry{vt.qa + fa, vt.qb + fb};
        if (k < K && k <= ke) {
            const int64_t R = k < ke ? rq.alpha + (int64_t)bb * k : rq.p;
            a.lt[(size_t)k * n + s] -= R;
            a.lt[(size_t)k * n + t] += R;
            a.load[(size_t)s * K + k] -= R;
            a.load[(size_t)t * K + k] += R;
        }
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <bool kPlan>
static void launch_score_lg(int lg, int blocks, const VarArgs& a, hipStream_t stream) {
    switch (lg) {
        case 0:
            hipLaunchKernelGGL((var_score_kernel<0, kPlan>), dim3(blocks), dim3(VS_THREADS), 0,
                               stream, a);
            break;
        case 1:
            hipLaunchKernelGGL((var_score_kernel<1, kPlan>), dim3(blocks), dim3(VS_THREADS), 0,
                               stream, a);
            break;
        case 2:
            hipLaunchKernelGGL((var_score_kernel<2, kPlan>), dim3(blocks), dim3(VS_THREADS), 0,
                               stream, a);
            break;
        case 3:
            hipLaunchKernelGGL((var_score_kernel<3, kPlan>), dim3(blocks), dim3(VS_THREADS), 0,
                               stream, a);
            break;
        default:
            hipLaunchKernelGGL((var_score_kernel<4, kPlan>), dim3(blocks), dim3(VS_THREADS), 0,
                               stream, a);
            break;
    }
}

VarPlan plan_variance(const star_load_params& p) {
    VarPlan pl;
    const int n = p.n_inst, N = p.n_req;
    const size_t K1 = (size_t)p.n_buckets + 1;
    int lg = 0;
    while ((1 << lg) < n && lg < VS_MAX_LG) ++lg;
    pl.lg = lg;
    const int64_t blocks = ceil_div(N, (int64_t)VS_WAVES * (kWave >> lg));
    pl.blocks = (int)(blocks < 1 ? 1 : blocks);
    pl.ticketed = pl.blocks <= VS_TICKET_BLOCKS;
    size_t off = STAR_WS_HEADER_BYTES;
    pl.qt_off = off;
    off += align_up((size_t)n * K1 * sizeof(QEntry), 256);
    pl.lt_off = off;
    off += align_up((size_t)n * K1 * sizeof(int64_t), 256);
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
    QEntry* qt = (QEntry*)(ws + pl.qt_off);
    int64_t* lt = (int64_t*)(ws + pl.lt_off);
    u128* bs = (u128*)(ws + pl.bs_off);
    uint32_t* ticket = (uint32_t*)(ws + kHdrVarTicket);
    hipLaunchKernelGGL(var_prep_kernel, dim3(n + 1), dim3(VP_THREADS), 0, stream, load, beta, n,
                       K, qt, lt, bs, ticket);
    VarArgs a;
    a.cur = cur;
    a.rem = rem;
    a.inst = inst;
    a.beta = beta;
    a.qt = qt;
    a.lt = lt;
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
    a.ticketed = pl.ticketed;
    a.tiles = pl.blocks;
    a.H = (int64_t)p.bucket * K;
    launch_score_lg<false>(pl.lg, pl.blocks, a, stream);
    if (move && !pl.ticketed)
        hipLaunchKernelGGL(var_final_kernel, dim3(1), dim3(VS_THREADS), 0, stream, a.part,
                           pl.blocks, inst, n, move);
    return hipGetLastError();
}

PlanPlan plan_plan(const star_plan_params& p) {
    PlanPlan pl;
    pl.v = plan_variance(p.load);
    size_t off = pl.v.total;
    pl.now_off = off;
    off += align_up((size_t)p.load.n_inst * sizeof(int64_t), 256);
    pl.total = off;
    return pl;
}

hipError_t launch_plan(const star_plan_params& p, const PlanPlan& pl, const int32_t* cur,
                       const int32_t* rem, int32_t* inst, int64_t* load, const uint16_t* beta,
                       star_move* moves, int32_t* n_moves, char* ws, int32_t* err,
                       hipStream_t stream) {
    const int n = p.load.n_inst, K = p.load.n_buckets;
    PlanArgs a;
    a.cur = cur;
    a.rem = rem;
    a.inst = inst;
    a.load = load;
    a.beta = beta;
    a.qt = (QEntry*)(ws + pl.v.qt_off);
    a.lt = (int64_t*)(ws + pl.v.lt_off);
    a.bs = (u128*)(ws + pl.v.bs_off);
    a.part = (VPart*)(ws + pl.v.part_off);
    const int grid = pl.v.blocks < PLAN_MAX_BLOCKS ? pl.v.blocks : PLAN_MAX_BLOCKS;
    a.parts = grid;
    a.now = (int64_t*)(ws + pl.now_off);
    a.done = (int32_t*)(ws + kHdrPlanDone);
    a.count = (int32_t*)(ws + kHdrPlanCount);
    a.n_moves = n_moves;
    a.moves = moves;
    a.err = err;
    a.N = p.load.n_req;
    a.n = n;
    a.b = p.load.bucket;
    a.K = K;
    a.H = (int64_t)p.load.bucket * K;
    hipLaunchKernelGGL(plan_zero_kernel, dim3(1), dim3(256), 0, stream, a.now, n, a.done, a.count,
                       n_moves);
    const int chunks = (int)ceil_div(a.N, PLAN_REQ_CHUNK);
    hipLaunchKernelGGL(plan_prep_kernel, dim3(n + 1 + chunks), dim3(VP_THREADS), 0, stream, a);

    VarArgs v;
    v.cur = cur;
    v.rem = rem;
    v.inst = inst;
    v.beta = beta;
    v.qt = a.qt;
    v.lt = a.lt;
    v.bs = a.bs;
    v.gain = nullptr;
    v.best_target = nullptr;
    v.best_gain = nullptr;
    v.move = nullptr;
    v.part = a.part;
    v.ticket = nullptr;
    v.err = err;
    v.N = a.N;
    v.n = n;
    v.b = a.b;
    v.K = K;
    v.ticketed = 0;
    v.tiles = pl.v.blocks;
    v.H = a.H;
    v.now = a.now;
    v.done = a.done;
    v.theta_num = p.theta_num;
    v.theta_den = p.theta_den;
    v.u_rule = p.u_rule;
    v.mem_rule = p.mem_rule;
    v.min_rem = p.min_rem;
    v.mem_cap = p.mem_cap;
    for (int m = 0; m < p.max_moves; ++m) {
        launch_score_lg<true>(pl.v.lg, grid, v, stream);
        hipLaunchKernelGGL(plan_apply_kernel, dim3(1), dim3(PA_THREADS), 0, stream, a);
    }
    return hipGetLastError();
}

}  // namespace star
