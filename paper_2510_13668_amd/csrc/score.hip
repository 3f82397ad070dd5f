// (c) Migration candidates scored by projected peak load, and ranked, on gfx950.
//
// Algorithm 1 (candidate enumeration, best-feasible selection) over every
// request -> instance pair, with the projected peak of the target's curve
// as the figure of merit.  For r on s with l' = min(l, H), k_e = l' div b,
// mu = l' mod b, alpha_r = b c + b(b-1)/2 and P_r = mu c + mu k_e b +
// mu(mu-1)/2, r's own curve is R_r[k] = alpha_r + b^2 k (k < k_e),
// P_r (k = k_e), 0 (k > k_e).  With, per instance t,
//     PM_t[k] = max_{j<k} (L_t[j] + b^2 j),   SM_t[k] = max_{j>=k} L_t[j],
// the peak of L_t + R_r is
//     max(PM_t[k_e] + alpha_r,  L_t[k_e] + P_r,  SM_t[k_e + 1])
// (terms outside [0, K) dropped): three gathers per candidate instead of a
// K-long scan.  This is the scheduler-side incremental update of the
// complexity analysis in Section 5.2 taken to O(1) per candidate.
//
// Kernel score (many workgroups, each a block of requests against every
// target): PM/SM from LDS when all curves fit there (built per workgroup
// with DPP wavefront scans), else from a separate prep kernel; writes every
// score and each request's best migration (the smallest key
// (score, r*n + t) over t != s; keys are a total order).
//
// Kernel top-k (one workgroup of 1024 threads): the k smallest keys.
// Exact pruning: a migration in the global top-k belongs to one of the k
// requests whose best key is smallest (its key is >= its request's best
// key, and k distinct requests have best keys below the k-th smallest
// migration key otherwise).  So when N(n-1) is large, a block radix select
// over the N best keys first picks those k requests, and only their
// k(n-1) migrations are ranked.  Radix select: 11-bit digits over the key
// (score - min score, then r*n + t), LDS histograms, DPP scans; the winners
// are then ordered by counting ranks.  No sorting network, no cross-
// workgroup synchronisation.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

constexpr int PREP_THREADS = 512;
constexpr int PREP_SEG = 4;
constexpr int SC_THREADS = 256;
constexpr int SC_CAND = 256;                 // target candidates per scoring workgroup
constexpr int SC_FUSED_ENTRIES = 2600;       // n*(K+1) up to which PM/SM live in LDS
constexpr int SC_LBATCH = (SC_FUSED_ENTRIES + SC_THREADS - 1) / SC_THREADS;  // curve reads per thread
constexpr int TK_THREADS = 1024;
constexpr int TK_DIGIT = 11;                 // radix-select digit width
constexpr int TK_BINS = 1 << TK_DIGIT;
constexpr int TK_MAX_KEYS = 16 * TK_THREADS; // migrations the direct top-k holds in registers

constexpr int64_t kInfS = INT64_MAX;
constexpr uint32_t kInfI = 0xFFFFFFFFu;

__device__ inline int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }

__device__ inline bool key_less(int64_t s0, uint32_t i0, int64_t s1, uint32_t i1) {
    return s0 < s1 || (s0 == s1 && i0 < i1);
}

// ---------------------------------------------------------------------------
// prep (large curve sets): PM_t[0..K] (PM_t[0] unused), SM_t[0..K] (SM_t[K] unused)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(PREP_THREADS) void score_prep_kernel(const int64_t* __restrict__ load,
                                                                  int K, int b,
                                                                  int64_t* __restrict__ PM,
                                                                  int64_t* __restrict__ SM) {
    __shared__ int64_t tmp[PREP_THREADS / 64 + 1];
    const int tid = threadIdx.x;
    const int t = blockIdx.x;
    const int64_t* L = load + (int64_t)t * K;
    int64_t* pm = PM + (int64_t)t * (K + 1);
    int64_t* sm = SM + (int64_t)t * (K + 1);
    const int64_t bb = (int64_t)b * b;
    constexpr int CH = PREP_THREADS * PREP_SEG;

    int64_t carry = INT64_MIN;                 // exclusive prefix max of L[j] + b^2 j
    for (int base = 0; base < K; base += CH) {
        const int j0 = base + tid * PREP_SEG;
        int64_t loc = INT64_MIN;
        for (int j = j0; j < j0 + PREP_SEG && j < K; ++j) loc = imax(loc, L[j] + bb * j);
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64<PREP_THREADS>(loc, OpMax(), INT64_MIN, tmp, &tot);
        int64_t run = imax(carry, ex);
        for (int j = j0; j < j0 + PREP_SEG && j < K; ++j) {
            pm[j] = run;
            run = imax(run, L[j] + bb * j);
        }
        carry = imax(carry, tot);
    }
    if (tid == 0) pm[K] = carry;

    carry = INT64_MIN;                         // inclusive suffix max of L[j]
    for (int base = 0; base < K; base += CH) {
        const int p0 = base + tid * PREP_SEG;  // reversed position p <-> j = K-1-p
        int64_t loc = INT64_MIN;
        for (int p = p0; p < p0 + PREP_SEG && p < K; ++p) loc = imax(loc, L[K - 1 - p]);
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64<PREP_THREADS>(loc, OpMax(), INT64_MIN, tmp, &tot);
        int64_t run = imax(carry, ex);
        for (int p = p0; p < p0 + PREP_SEG && p < K; ++p) {
            run = imax(run, L[K - 1 - p]);
            sm[K - 1 - p] = run;
        }
        carry = imax(carry, tot);
    }
    if (tid == 0) sm[K] = INT64_MIN;
}

// ---------------------------------------------------------------------------
// score
// ---------------------------------------------------------------------------
struct ScoreArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* load;
    const int64_t* PM;            // global PM/SM (non-fused path)
    const int64_t* SM;
    int64_t* scores;              // caller's array or workspace copy
    int32_t* best_target;         // caller's array or workspace copy
    int64_t* best_score;
    int32_t* err_word;
    int N, n, b, K, rpb, cand;
};

template <bool kFused>
__global__ __launch_bounds__(SC_THREADS) void score_kernel(ScoreArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int n = a.n, K = a.K, b = a.b;
    const int K1 = K + 1;
    const int cand = a.cand;                       // rpb * n keys in this workgroup
    const int rpb = a.rpb;

    // LDS: [L | PM | SM] (fused), keys, per-request values
    int64_t* lL = (int64_t*)smem;
    int64_t* lPM = lL + (kFused ? n * K1 : 0);
    int64_t* lSM = lPM + (kFused ? n * K1 : 0);
    int64_t* ks = lSM + (kFused ? n * K1 : 0);
    int64_t* r_alpha = ks + cand;
    int64_t* r_p = r_alpha + rpb;
    uint32_t* ki = (uint32_t*)(r_p + rpb);
    int32_t* r_ke = (int32_t*)(ki + cand);
    int32_t* r_s = r_ke + rpb;

    const int row0 = blockIdx.x * rpb;
    const int64_t H = (int64_t)b * K;
    const int64_t bb = (int64_t)b * b;
    const int64_t bb2 = (int64_t)b * (b - 1) / 2;

    // 0) per-request values; curves into LDS.  All reads are issued before
    //    the first is used (clamped indices, unconditional loads).
    int32_t bad = 0;
    int64_t lv[SC_LBATCH];
    const int nK = n * K;
    if constexpr (kFused) {
#pragma unroll
        for (int j = 0; j < SC_LBATCH; ++j) {
            const int e = j * SC_THREADS + tid;
            lv[j] = a.load[e < nK ? e : nK - 1];
        }
    }
    for (int q0 = 0; q0 < rpb; q0 += SC_THREADS * 2) {
        int sv[2], cv[2], rv[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int q = q0 + j * SC_THREADS + tid;
            int r = row0 + q;
            r = r < a.N ? r : a.N - 1;
            sv[j] = a.inst[r];
            cv[j] = a.cur[r];
            rv[j] = a.rem[r];
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int q = q0 + j * SC_THREADS + tid;
            if (q >= rpb) continue;
            const int r = row0 + q;
            int s = -1;
            if (r < a.N) {
                s = sv[j];
                const int cr = cv[j];
                const int lr = rv[j];
                int32_t f = 0;
                if (s < 0 || s >= n) f |= STAR_DEV_BAD_INST;
                if (cr < 1) f |= STAR_DEV_BAD_CUR;
                if (lr < 1) f |= STAR_DEV_BAD_REM;
                bad |= f;
                if (f) {
                    s = -1;
                } else {
                    const int64_t lp = (int64_t)lr < H ? (int64_t)lr : H;
                    const int64_t ke = lp / b;
                    const int64_t mu = lp - ke * b;
                    r_alpha[q] = (int64_t)b * cr + bb2;
                    r_p[q] = mu * cr + mu * ke * b + mu * (mu - 1) / 2;
                    r_ke[q] = (int32_t)ke;
                }
            }
            r_s[q] = s;
        }
    }
    bad = wave_or_i32(bad);
    if (lane == 0) report_error(a.err_word, bad);
    if constexpr (kFused) {
#pragma unroll
        for (int j = 0; j < SC_LBATCH; ++j) {
            const int e = j * SC_THREADS + tid;
            if (e < nK) {
                const int t = e / K, k = e - t * K;
                lL[t * K1 + k] = lv[j];
            }
        }
        __syncthreads();
        // Per instance (one wave each, round robin): every lane reduces a
        // contiguous segment of SEG buckets serially, one DPP wavefront scan
        // combines the 64 segment maxima, and a second serial pass writes.
        // For the suffix maxima lane l takes segment 63 - l, so that a
        // prefix scan over lanes is a suffix scan over buckets.
        const int SEG = (K + 63) >> 6;
        for (int t = wid; t < n; t += SC_THREADS / 64) {
            const int64_t* L = lL + t * K1;
            int64_t* pm = lPM + t * K1;
            int64_t* sm = lSM + t * K1;
            const int f0 = lane * SEG;
            const int f1 = f0 + SEG < K ? f0 + SEG : K;
            const int g0 = (63 - lane) * SEG;
            const int g1 = g0 + SEG < K ? g0 + SEG : K;
            int64_t fwd = INT64_MIN, bwd = INT64_MIN;
            for (int u = 0; u < SEG; ++u) {
                if (f0 + u < f1) fwd = imax(fwd, L[f0 + u] + bb * (f0 + u));
                if (g0 + u < g1) bwd = imax(bwd, L[g0 + u]);
            }
            const int64_t finc = wave_incl_max_i64(fwd);
            const int64_t binc = wave_incl_max_i64(bwd);
            int64_t fex = __shfl_up(finc, 1, 64);
            int64_t bex = __shfl_up(binc, 1, 64);
            if (lane == 0) { fex = INT64_MIN; bex = INT64_MIN; }
            for (int j = f0; j < f1; ++j) {
                pm[j] = fex;
                fex = imax(fex, L[j] + bb * j);
            }
            for (int j = g1 - 1; j >= g0; --j) {
                bex = imax(bex, L[j]);
                sm[j] = bex;
            }
            if (lane == 63) pm[K] = finc;
            if (lane == 0) sm[K] = INT64_MIN;
        }
    }
    __syncthreads();
    const int64_t* gL = kFused ? lL : a.load;
    const int64_t* gPM = kFused ? lPM : a.PM;
    const int64_t* gSM = kFused ? lSM : a.SM;
    const int Ls = kFused ? K1 : K;              // row stride of the curve array

    // 1) candidates -> scores and keys (self-candidates and invalid requests
    //    get the +inf key)
    for (int e = tid; e < cand; e += SC_THREADS) {
        int64_t key_s = kInfS;
        uint32_t key_i = kInfI;
        const int q = e / n, t = e - q * n;
        const int r = row0 + q;
        if (r < a.N) {
            const int s = r_s[q];
            int64_t sc = -1;
            if (s >= 0) {
                const int64_t* sm = gSM + (int64_t)t * K1;
                if (t == s) {
                    sc = sm[0];
                } else {
                    const int ke = r_ke[q];
                    sc = INT64_MIN;
                    if (ke >= 1) sc = imax(sc, gPM[(int64_t)t * K1 + ke] + r_alpha[q]);
                    if (ke < K) sc = imax(sc, gL[(int64_t)t * Ls + ke] + r_p[q]);
                    if (ke + 1 < K) sc = imax(sc, sm[ke + 1]);
                    key_s = sc;
                    key_i = (uint32_t)((int64_t)r * n + t);
                }
            }
            if (a.scores) a.scores[(int64_t)r * n + t] = sc;
        }
        ks[e] = key_s;
        ki[e] = key_i;
    }
    __syncthreads();

    // 2) best migration per request: smallest (score, t) over t != s
    for (int q = tid; q < rpb; q += SC_THREADS) {
        const int r = row0 + q;
        if (r >= a.N) continue;
        int64_t bs = kInfS;
        uint32_t bi = kInfI;
        for (int t = 0; t < n; ++t) {
            const int e = q * n + t;
            if (key_less(ks[e], ki[e], bs, bi)) { bs = ks[e]; bi = ki[e]; }
        }
        const bool none = bi == kInfI;
        if (a.best_target) a.best_target[r] = none ? -1 : (int32_t)(bi - (uint32_t)((int64_t)r * n));
        if (a.best_score) a.best_score[r] = none ? -1 : bs;
    }
}

// ---------------------------------------------------------------------------
// top-k: block-wide helpers (1024 threads)
// ---------------------------------------------------------------------------
struct TkShared {
    int hist[TK_BINS];
    int wsum[TK_THREADS / 64];
    int64_t red64[TK_THREADS / 64];
    int64_t bcast[4];
};

// Sum of one int over the block; every thread gets the total.
__device__ inline int block_sum_i32(int v, TkShared& sh) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_incl_add_i32(v);
    if (lane == 63) sh.wsum[wid] = v;
    __syncthreads();
    int t = 0;
#pragma unroll
    for (int w = 0; w < TK_THREADS / 64; ++w) t += sh.wsum[w];
    __syncthreads();
    return t;
}

// Exclusive prefix of one int over the block (thread order); *total = sum.
__device__ inline int block_excl_i32(int v, TkShared& sh, int* total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int inc = wave_incl_add_i32(v);
    if (lane == 63) sh.wsum[wid] = inc;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < TK_THREADS / 64; ++w) {
        const int x = sh.wsum[w];
        before += w < wid ? x : 0;
        all += x;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

// Min (kMin) or max of one int64 over the block; every thread gets it.
template <bool kMin>
__device__ inline int64_t block_minmax_i64(int64_t v, TkShared& sh) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const int64_t u = __shfl_xor(v, o, 64);
        v = kMin ? (u < v ? u : v) : (u > v ? u : v);
    }
    if (lane == 0) sh.red64[wid] = v;
    __syncthreads();
    int64_t r = sh.red64[0];
#pragma unroll
    for (int w = 1; w < TK_THREADS / 64; ++w) {
        const int64_t x = sh.red64[w];
        r = kMin ? (x < r ? x : r) : (x > r ? x : r);
    }
    __syncthreads();
    return r;
}

// Key sources for block_select.  A source visits this thread's keys
// (s, i), s >= 0, calling f(s, i); s == kInfS marks "no key".
template <int RJ>
struct RegKeys {                  // keys held in registers
    int64_t s[RJ];
    uint32_t i[RJ];
    template <class F>
    __device__ inline void visit(F&& f) const {
#pragma unroll
        for (int j = 0; j < RJ; ++j) f(s[j], i[j]);
    }
};

constexpr int TK_SBATCH = 8;      // global reads per thread in flight in a streaming visit

struct BestKeys {                 // (best score, r) of every request with a migration
    const int64_t* best_score;
    const int32_t* best_target;
    int N;
    template <class F>
    __device__ inline void visit(F&& f) const {
        for (int r0 = 0; r0 < N; r0 += TK_THREADS * TK_SBATCH) {
            int64_t bs[TK_SBATCH];
            int32_t bt[TK_SBATCH];
#pragma unroll
            for (int u = 0; u < TK_SBATCH; ++u) {
                const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
                const int rc = r < N ? r : N - 1;
                bs[u] = best_score[rc];
                bt[u] = best_target[rc];
            }
#pragma unroll
            for (int u = 0; u < TK_SBATCH; ++u) {
                const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
                const bool ok = r < N && bt[u] >= 0;
                f(ok ? bs[u] : kInfS, ok ? (uint32_t)r : kInfI);
            }
        }
    }
};

struct PrunedKeys {               // every migration of the requests rk[0..nr)
    const int64_t* scores;
    const int32_t* rk;            // LDS: request ids
    const int32_t* rk_inst;       // LDS: their instances
    int nr, n;
    template <class F>
    __device__ inline void visit(F&& f) const {
        const int M = nr * (n - 1);
        for (int e0 = 0; e0 < M; e0 += TK_THREADS * TK_SBATCH) {
            int64_t sv[TK_SBATCH];
            uint32_t iv[TK_SBATCH];
#pragma unroll
            for (int u = 0; u < TK_SBATCH; ++u) {
                const int e = e0 + u * TK_THREADS + (int)threadIdx.x;
                const int ec = e < M ? e : M - 1;
                const int q = ec / (n - 1), v = ec - q * (n - 1);
                const int r = rk[q];
                const int t = v < rk_inst[q] ? v : v + 1;     // skip staying put
                iv[u] = (uint32_t)((int64_t)r * n + t);
                sv[u] = scores[(int64_t)r * n + t];
            }
#pragma unroll
            for (int u = 0; u < TK_SBATCH; ++u) {
                const int e = e0 + u * TK_THREADS + (int)threadIdx.x;
                f(e < M ? sv[u] : kInfS, e < M ? iv[u] : kInfI);
            }
        }
    }
};

// Returns the upper bound U = (us, ui) such that exactly min(k, #keys)
// keys of the source are <= U.
template <class Src>
__device__ void block_select(const Src& src, int k, TkShared& sh, int64_t* us, uint32_t* ui) {
    int mine = 0;
    int64_t lo = kInfS, hi = -1;
    src.visit([&](int64_t s, uint32_t) {
        if (s != kInfS) {
            ++mine;
            lo = s < lo ? s : lo;
            hi = s > hi ? s : hi;
        }
    });
    const int total = block_sum_i32(mine, sh);
    if (total <= k) {                              // every key is a winner
        *us = kInfS - 1;
        *ui = kInfI;
        return;
    }
    const int64_t smin = block_minmax_i64<true>(lo, sh);
    const int64_t smax = block_minmax_i64<false>(hi, sh);
    const uint64_t range = (uint64_t)(smax - smin);
    int sbits = 0;
    while (sbits < 64 && (range >> sbits) != 0) ++sbits;

    // digits over the (sbits + 32)-bit value (d << 32) | i, d = s - smin
    uint64_t pd = 0, md = 0;                       // chosen prefix / mask on d
    uint32_t pi = 0, mi = 0;                       // chosen prefix / mask on i
    int kk = k;
    bool done = false;
    for (int pos = sbits + 32; pos > 0 && !done; pos -= TK_DIGIT) {
        const int lowbit = pos > TK_DIGIT ? pos - TK_DIGIT : 0;     // digit bits [lowbit, pos)
        const int width = pos - lowbit;
        for (int b = threadIdx.x; b < TK_BINS; b += TK_THREADS) sh.hist[b] = 0;
        __syncthreads();
        src.visit([&](int64_t s, uint32_t i) {
            if (s == kInfS) return;
            const uint64_t d = (uint64_t)(s - smin);
            if ((d & md) != pd || (i & mi) != pi) return;
            uint32_t dig;
            if (lowbit >= 32) dig = (uint32_t)(d >> (lowbit - 32));
            else if (pos <= 32) dig = i >> lowbit;
            else dig = (uint32_t)((d << (32 - lowbit)) | (i >> lowbit));
            dig &= (1u << width) - 1;
            atomicAdd(&sh.hist[dig], 1);
        });
        __syncthreads();
        // find the bin holding the kk-th key: each thread owns PER bins
        constexpr int PER = TK_BINS / TK_THREADS;
        int c[PER], own = 0;
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            c[u] = sh.hist[threadIdx.x * PER + u];
            own += c[u];
        }
        int tot;
        int before = block_excl_i32(own, sh, &tot);
#pragma unroll
        for (int u = 0; u < PER; ++u) {
            if (before < kk && kk <= before + c[u]) {
                sh.bcast[0] = threadIdx.x * PER + u;
                sh.bcast[1] = kk - before;
                sh.bcast[2] = c[u];
            }
            before += c[u];
        }
        __syncthreads();
        const uint32_t bin = (uint32_t)sh.bcast[0];
        kk = (int)sh.bcast[1];
        const int cnt = (int)sh.bcast[2];
        __syncthreads();
        for (int bit = lowbit; bit < pos; ++bit) {  // extend the prefix by this digit
            const uint32_t v = (bin >> (bit - lowbit)) & 1u;
            if (bit >= 32) {
                md |= 1ull << (bit - 32);
                pd |= (uint64_t)v << (bit - 32);
            } else {
                mi |= 1u << bit;
                pi |= v << bit;
            }
        }
        done = cnt == kk;                          // the whole bin is needed
    }
    // U: the prefix with every unchosen bit set (within the sbits bits every
    // d has); no overflow since smin + 2^sbits <= 2 smax + 1 < 2^63
    uint64_t du = pd | ~md;
    du &= sbits >= 64 ? ~0ull : ((1ull << sbits) - 1);
    *us = smin + (int64_t)du;
    *ui = pi | ~mi;
}

// Writes the source's keys <= U to (os, oi) in thread order; returns their
// count (every thread gets it).
template <class Src>
__device__ int block_gather(const Src& src, int64_t us, uint32_t ui, TkShared& sh, int64_t* os,
                            uint32_t* oi, int cap) {
    int mine = 0;
    src.visit([&](int64_t s, uint32_t i) {
        if (s != kInfS && !key_less(us, ui, s, i)) ++mine;
    });
    int total;
    int at = block_excl_i32(mine, sh, &total);
    src.visit([&](int64_t s, uint32_t i) {
        if (s != kInfS && !key_less(us, ui, s, i)) {
            if (at < cap) {
                os[at] = s;
                oi[at] = i;
            }
            ++at;
        }
    });
    __syncthreads();
    return total < cap ? total : cap;
}

// ---------------------------------------------------------------------------
// top-k kernel
// ---------------------------------------------------------------------------
struct TopkArgs {
    const int32_t* inst;
    const int64_t* scores;        // [N, n] (caller's array or workspace copy)
    const int32_t* best_target;   // [N]
    const int64_t* best_score;    // [N]
    int32_t* topk_req;
    int32_t* topk_tgt;
    int64_t* topk_score;
    int N, n, top_k;
};

__device__ inline void rank_and_write(const TopkArgs& a, const int64_t* ws_s, const uint32_t* ws_i,
                                      int nw) {
    for (int w = threadIdx.x; w < nw; w += TK_THREADS) {
        const int64_t xs = ws_s[w];
        const uint32_t xi = ws_i[w];
        int rank = 0;
        for (int j = 0; j < nw; ++j) rank += key_less(ws_s[j], ws_i[j], xs, xi) ? 1 : 0;
        a.topk_req[rank] = (int32_t)(xi / (uint32_t)a.n);
        a.topk_tgt[rank] = (int32_t)(xi % (uint32_t)a.n);
        a.topk_score[rank] = xs;
    }
    for (int q = nw + threadIdx.x; q < a.top_k; q += TK_THREADS) {
        a.topk_req[q] = -1;
        a.topk_tgt[q] = -1;
        a.topk_score[q] = -1;
    }
}

// Every migration of every request held in registers (N n <= RJ * 1024).
template <int RJ>
__global__ __launch_bounds__(TK_THREADS) void topk_direct_kernel(TopkArgs a) {
    __shared__ TkShared sh;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    const int tid = threadIdx.x;
    const int n = a.n, M = a.N * a.n;
    RegKeys<RJ> keys;
    {
        int64_t sv[RJ];
        int32_t iv[RJ], bv[RJ];
#pragma unroll
        for (int j = 0; j < RJ; ++j) {
            const int e = j * TK_THREADS + tid;
            const int ec = e < M ? e : M - 1;
            sv[j] = a.scores[ec];
            iv[j] = a.inst[ec / n];
            bv[j] = a.best_target[ec / n];
        }
#pragma unroll
        for (int j = 0; j < RJ; ++j) {
            const int e = j * TK_THREADS + tid;
            const bool ok = e < M && bv[j] >= 0 && (e % n) != iv[j];
            keys.s[j] = ok ? sv[j] : kInfS;
            keys.i[j] = ok ? (uint32_t)e : kInfI;
        }
    }
    int64_t us;
    uint32_t ui;
    block_select(keys, a.top_k, sh, &us, &ui);
    const int nw = block_gather(keys, us, ui, sh, ws_s, ws_i, STAR_MAX_TOP_K);
    rank_and_write(a, ws_s, ws_i, nw);
}

// First the k requests with the smallest best keys, then the k smallest of
// their migrations (both streamed from global memory).
__global__ __launch_bounds__(TK_THREADS) void topk_pruned_kernel(TopkArgs a) {
    __shared__ TkShared sh;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    __shared__ int32_t rk[STAR_MAX_TOP_K];
    __shared__ int32_t rk_inst[STAR_MAX_TOP_K];
    BestKeys bk{a.best_score, a.best_target, a.N};
    int64_t us;
    uint32_t ui;
    block_select(bk, a.top_k, sh, &us, &ui);
    const int nr = block_gather(bk, us, ui, sh, ws_s, ws_i, STAR_MAX_TOP_K);
    for (int q = threadIdx.x; q < nr; q += TK_THREADS) {
        const int r = (int)ws_i[q];
        rk[q] = r;
        rk_inst[q] = a.inst[r];
    }
    __syncthreads();
    PrunedKeys pk{a.scores, rk, rk_inst, nr, a.n};
    block_select(pk, a.top_k, sh, &us, &ui);
    const int nw = block_gather(pk, us, ui, sh, ws_s, ws_i, STAR_MAX_TOP_K);
    rank_and_write(a, ws_s, ws_i, nw);
}

__global__ void fill_i32_kernel(int32_t* p, int count, int32_t v) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < count; i += gridDim.x * 256) p[i] = v;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
ScorePlan plan_score(const star_score_params& p) {
    ScorePlan pl;
    const int n = p.load.n_inst;
    const int N = p.load.n_req;
    const int K1 = p.load.n_buckets + 1;
    pl.fused = (int64_t)n * K1 <= SC_FUSED_ENTRIES;
    pl.rpb = SC_CAND / n > 1 ? SC_CAND / n : 1;
    if (N > 0 && pl.rpb > N) pl.rpb = N;
    pl.cand = pl.rpb * n;
    pl.groups = N > 0 ? (int)ceil_div(N, pl.rpb) : 0;
    // top-k: select over all migrations when they fit one workgroup's
    // registers, else over the k requests with the smallest best keys first
    const int64_t migr = (int64_t)N * n;
    pl.topk_direct = migr <= TK_MAX_KEYS;
    int rj = 1;
    while ((int64_t)rj * TK_THREADS < migr && rj < TK_MAX_KEYS / TK_THREADS) rj *= 2;
    pl.topk_rj = rj;
    pl.topk_ok = true;

    size_t off = STAR_WS_HEADER_BYTES;
    pl.pm_off = off;
    if (!pl.fused) off = align_up(off + (size_t)n * K1 * 8, 256);
    pl.sm_off = off;
    if (!pl.fused) off = align_up(off + (size_t)n * K1 * 8, 256);
    pl.scores_off = off;                          // used when the caller passes no scores
    off = align_up(off + (size_t)N * n * 8, 256);
    pl.bscore_off = off;
    off = align_up(off + (size_t)N * 8, 256);
    pl.btarget_off = off;
    off = align_up(off + (size_t)N * 4, 256);
    pl.total = off;
    pl.lds = (pl.fused ? (size_t)3 * n * K1 * 8 : 0) + (size_t)pl.cand * 12 + (size_t)pl.rpb * 24;
    return pl;
}

template <bool kFused>
static hipError_t launch_score_kernel(const ScorePlan& pl, const ScoreArgs& a, hipStream_t stream) {
    if (pl.lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)score_kernel<kFused>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(score_kernel<kFused>, dim3(pl.groups), dim3(SC_THREADS), pl.lds, stream, a);
    return hipGetLastError();
}

static hipError_t fill_i32(int32_t* p, int count, int32_t v, hipStream_t stream) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3((count + 255) / 256), dim3(256), 0, stream, p, count, v);
    return hipGetLastError();
}

template <int RJ>
static hipError_t launch_topk_rj(const TopkArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL(topk_direct_kernel<RJ>, dim3(1), dim3(TK_THREADS), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_score(const star_score_params& p, const ScorePlan& pl, const int32_t* cur,
                        const int32_t* rem, const int32_t* inst, const int64_t* load,
                        int64_t* scores, int32_t* best_target, int64_t* best_score,
                        int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score, char* ws,
                        int32_t* err_word, hipStream_t stream) {
    const star_load_params& lp = p.load;
    if (lp.n_req == 0) {
        if (p.top_k > 0) {                       // no candidates: top-k is all -1
            hipError_t e = fill_i32(topk_req, p.top_k, -1, stream);
            if (e == hipSuccess) e = fill_i32(topk_tgt, p.top_k, -1, stream);
            if (e == hipSuccess) e = fill_i32((int32_t*)topk_score, 2 * p.top_k, -1, stream);
            return e;
        }
        return hipSuccess;
    }
    const bool need_all = p.top_k > 0;           // the top-k kernel reads scores and best moves
    ScoreArgs a = {};
    a.cur = cur; a.rem = rem; a.inst = inst; a.load = load;
    a.PM = (const int64_t*)(ws + pl.pm_off);
    a.SM = (const int64_t*)(ws + pl.sm_off);
    a.scores = scores ? scores : (need_all ? (int64_t*)(ws + pl.scores_off) : nullptr);
    a.best_target = best_target ? best_target : (need_all ? (int32_t*)(ws + pl.btarget_off) : nullptr);
    a.best_score = best_score ? best_score : (need_all ? (int64_t*)(ws + pl.bscore_off) : nullptr);
    a.err_word = err_word;
    a.N = lp.n_req; a.n = lp.n_inst; a.b = lp.bucket; a.K = lp.n_buckets;
    a.rpb = pl.rpb; a.cand = pl.cand;
    hipError_t e;
    if (pl.fused) {
        e = launch_score_kernel<true>(pl, a, stream);
    } else {
        hipLaunchKernelGGL(score_prep_kernel, dim3(lp.n_inst), dim3(PREP_THREADS), 0, stream, load,
                           lp.n_buckets, lp.bucket, (int64_t*)(ws + pl.pm_off),
                           (int64_t*)(ws + pl.sm_off));
        e = hipGetLastError();
        if (e == hipSuccess) e = launch_score_kernel<false>(pl, a, stream);
    }
    if (e != hipSuccess || p.top_k == 0) return e;
    if (lp.n_inst == 1) {                        // nowhere to migrate to
        e = fill_i32(topk_req, p.top_k, -1, stream);
        if (e == hipSuccess) e = fill_i32(topk_tgt, p.top_k, -1, stream);
        if (e == hipSuccess) e = fill_i32((int32_t*)topk_score, 2 * p.top_k, -1, stream);
        return e;
    }

    TopkArgs t = {};
    t.inst = inst;
    t.scores = a.scores;
    t.best_target = a.best_target;
    t.best_score = a.best_score;
    t.topk_req = topk_req; t.topk_tgt = topk_tgt; t.topk_score = topk_score;
    t.N = lp.n_req; t.n = lp.n_inst; t.top_k = p.top_k;
    if (!pl.topk_direct) {
        hipLaunchKernelGGL(topk_pruned_kernel, dim3(1), dim3(TK_THREADS), 0, stream, t);
        return hipGetLastError();
    }
    switch (pl.topk_rj) {
        case 1: return launch_topk_rj<1>(t, stream);
        case 2: return launch_topk_rj<2>(t, stream);
        case 4: return launch_topk_rj<4>(t, stream);
        case 8: return launch_topk_rj<8>(t, stream);
        case 16: return launch_topk_rj<16>(t, stream);
    }
    return hipErrorInvalidValue;
}

}  // namespace star
