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

constexpr size_t kHdrVarTicket = 64;   // workspace header: finished-workgroup ticket
// Grids up to this many workgroups find the best move in the scoring kernel
// (the last workgroup to finish reduces the partials); larger ones hand the
// partials to a one-workgroup kernel, because every workgroup's release
// fence would write back its XCD's L2, full of freshly written gains.
constexpr int VS_TICKET_BLOCKS = 64;
constexpr int VS_MAX_LG = 4;             // at most 16 lanes per request

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

__global__ __launch_bounds__(VP_THREADS) void var_prep_kernel(const int64_t* __restrict__ load,
                                                              const uint16_t* __restrict__ beta,
                                                              int n, int K,
                                                              QEntry* __restrict__ qt,
                                                              int64_t* __restrict__ lt,
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
template <bool kAtomic>
__device__ void reduce_parts(VPart* part, int parts, const int32_t* inst, int n, star_move* move,
                             VKey* wbest) {
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    VKey k = no_key();
    for (int g = tid; g < parts; g += VS_THREADS) {
        VKey p;
        if (kAtomic) {
            p = load_part(&part[g]);
        } else {
            const VPart v = part[g];
            p = VKey{(s128)(((u128)v.w[1] << 64) | (u128)v.w[0]), (uint32_t)v.w[2]};
        }
        k = vmin(k, p);
    }
    k = group_min(k, 6, lane);
    if (lane == kWave - 1) wbest[wid] = k;
    __syncthreads();
    if (tid == 0) {
        VKey m = wbest[0];
        for (int w = 1; w < VS_WAVES; ++w) m = vmin(m, wbest[w]);
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
        *move = mv;
    }
}

// A request's target-independent part of G, staged in LDS.
struct ReqStash {
    u128 base, bp;
    uint64_t al;
    int32_t ke;
    int32_t s;        // source instance; -2: invalid request, -1: past the end
    int32_t pad[2];
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
    int64_t H;
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
template <int LG>
__global__ __launch_bounds__(VS_THREADS) void var_score_kernel(VarArgs a) {
    constexpr int P = 1 << LG, RPW = kWave / P, TILE = VS_WAVES * RPW;
    __shared__ ReqStash st[TILE];
    __shared__ VKey wbest[VS_WAVES];
    __shared__ bool last;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wid = tid / kWave;
    const int sub = lane >> LG, tl = lane & (P - 1);
    const int n = a.n, K = a.K, K1 = K + 1;
    const uint64_t bb = (uint64_t)a.b * (uint64_t)a.b;
    const int r0 = blockIdx.x * TILE;
    const QEntry* __restrict__ qt = a.qt;
    const int64_t* __restrict__ lt = a.lt;
    u128* __restrict__ gain = a.gain;

    if (tid < TILE) {
        const int r = r0 + tid;
        ReqStash e;
        e.base = 0;
        e.bp = 0;
        e.al = 0;
        e.ke = 0;
        e.s = -1;
        if (r < a.N) {
            const ReqTerms q = request_terms(a.inst[r], a.cur[r], a.rem[r], n, a.b, a.H);
            report_error(a.err, q.bad);
            e.s = q.bad ? -2 : q.s;
            if (!q.bad) {
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
            u128 g = base + mul_u64(qe[i].qa, al) + mul_u64(qe[i].qb, bb);
            if (ke < K) g += mul_s64(bp, le[i]);
            const bool mig = valid && t < n && t != src;
            if (!mig) g = 0;
            if (mig && (s128)g < bg) {   // targets ascend within a lane
                bg = (s128)g;
                bt = t;
            }
            if (gain && live && t < n) gain[(size_t)r * n + t] = g;
        }
    }
    if (LG >= 1) dpp_step<kDppRowShr1, 1>(bg, bt, tl);
    if (LG >= 2) dpp_step<kDppRowShr2, 2>(bg, bt, tl);
    if (LG >= 3) dpp_step<kDppRowShr4, 4>(bg, bt, tl);
    if (LG >= 4) dpp_step<kDppRowShr8, 8>(bg, bt, tl);

    VKey feas = no_key();   // the request's best key if it lowers the objective
    if (live && tl == P - 1) {
        if (a.best_target) a.best_target[r] = bt;
        if (a.best_gain) a.best_gain[r] = bt >= 0 ? (u128)bg : (u128)0;
        if (bt >= 0 && bg < 0) feas = VKey{bg, (uint32_t)r * (uint32_t)n + (uint32_t)bt};
    }
    if (!a.move) return;

    // best negative key of the workgroup, then (small grids) of the grid
    feas = group_min(feas, 6, lane);
    if (lane == kWave - 1) wbest[wid] = feas;
    __syncthreads();
    if (tid == 0) {
        VKey k = wbest[0];
        for (int w = 1; w < VS_WAVES; ++w) k = vmin(k, wbest[w]);
        store_part(&a.part[blockIdx.x], k);
        if (a.ticketed) {
            // small grids only: this release fence writes back the XCD's L2
            __threadfence();
            last = atomicAdd(a.ticket, 1u) == gridDim.x - 1;
        }
    }
    if (!a.ticketed) return;
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
// host side
// ---------------------------------------------------------------------------
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
    a.H = (int64_t)p.bucket * K;
    switch (pl.lg) {
        case 0:
            hipLaunchKernelGGL(var_score_kernel<0>, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
            break;
        case 1:
            hipLaunchKernelGGL(var_score_kernel<1>, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
            break;
        case 2:
            hipLaunchKernelGGL(var_score_kernel<2>, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
            break;
        case 3:
            hipLaunchKernelGGL(var_score_kernel<3>, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL(var_score_kernel<4>, dim3(pl.blocks), dim3(VS_THREADS), 0, stream, a);
            break;
    }
    if (move && !pl.ticketed)
        hipLaunchKernelGGL(var_final_kernel, dim3(1), dim3(VS_THREADS), 0, stream, a.part,
                           pl.blocks, inst, n, move);
    return hipGetLastError();
}

}  // namespace star
