// (c) Migration candidates scored by projected peak load, and ranked, on gfx950.
//
// Algorithm 1 (candidate enumeration, best-feasible selection) over every
// request -> instance pair, with the projected peak of the target's curve
// as the figure of merit.  For r on s with l' = min(l, H), k_e = l' div b,
// mu = l' mod b, alpha_r = b c + b(b-1)/2 and P_r = mu c + mu k_e b +
// mu(mu-1)/2, r's own curve is R_r[k] = alpha_r + b^2 k (k < k_e),
// P_r (k = k_e), 0 (k > k_e).  With, per instance t,
//     PM_t[k] = max_{j<k} (L_t[j] + b^2 j),   SM_t[k] = max_{j>=k} L_t[j],
// (PM_t[0] = SM_t[K] = -inf) the peak of L_t + R_r is
//     max(PM_t[k_e] + alpha_r,  L_t[k_e] + P_r,  SM_t[min(k_e + 1, K)])
// (the middle term only for k_e < K): three gathers per candidate instead
// of a K-long scan.  This is the scheduler-side incremental update of the
// complexity analysis in Section 5.2 taken to O(1) per candidate.
//
// Migrations (t != s) are ranked by the key (score, r*n + t), a total order.
// The k smallest are found by a block radix select: 12-bit digits of the
// key packed as ((score - min score) << ibits) | (r*n + t), LDS
// histograms, DPP scans, stopping as soon as the bin that holds the k-th key
// is needed whole; the <= k winners are then put in order by a bucket sort
// on their top 12 bits (LDS counts, offsets, scatter, and a rank count only
// among equal buckets).
//
// Three paths:
//  * small rounds (N <= 1024, N n <= 8192, curves fit LDS): ONE workgroup of
//    512 threads loads the curves, builds PM/SM, scores every candidate with
//    the keys in registers, takes each request's best move with LDS atomics
//    and runs the selection.  No intermediate array goes through HBM.
//  * otherwise many workgroups score blocks of requests (PM/SM built in LDS
//    per workgroup, or by a prep kernel for large curve sets), writing
//    scores and best moves; then one 1024-thread workgroup selects, over all
//    migrations when they fit its registers, else with exact pruning: a
//    migration in the global top-k belongs to one of the k requests whose
//    best key is smallest (its key is >= its request's best key, and k
//    distinct requests have best keys below the k-th smallest migration key
//    otherwise), so the k requests are selected first and only their k(n-1)
//    migrations are ranked.  When there are more requests than best keys fit
//    its registers, the top-k counts the best keys' codes (a monotone summary
//    of the score) in an LDS histogram and gathers only the best keys up to
//    the code that holds the k-th.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

constexpr int PREP_THREADS = 512;
constexpr int PREP_SEG = 4;
constexpr int SC_THREADS = 256;
constexpr int SC_CAND = 256;                 // target candidates per scoring workgroup
// Separate scoring workgroups (score_kernel) take more requests each while
// SC_MIN_GROUPS of them remain, up to SC_CAND_MAX candidates: the per-group
// work (request terms, curve base) is then shared by more candidates
// (measured at 32768 requests x 64 instances: 8192 -> 2048 groups, the call
// 80.2 -> 73.5 us; at 256 groups, making them longer was slower).
constexpr int SC_CAND_MAX = 1024;
constexpr int SC_MIN_GROUPS = 2048;
constexpr int SC_FUSED_ENTRIES = 2600;       // n*(K+1) up to which PM/SM live in LDS
constexpr int SC_LBATCH = (SC_FUSED_ENTRIES + SC_THREADS - 1) / SC_THREADS;  // curve reads per thread
constexpr int SC_PBATCH = 4;                 // requests per thread in flight (in-kernel projection)
constexpr int SC_PROJECT_MAX_REQ = 8192;     // requests up to which every group projects for itself

constexpr int SEL_DIGIT = 12;                // radix-select digit width
constexpr int SEL_BINS = 1 << SEL_DIGIT;
constexpr int SEL_SBATCH = 8;                // reads per thread in flight when streaming keys

constexpr int TK_THREADS = 1024;             // top-k workgroup of the multi-workgroup path
constexpr int TK_RJ = 16;                    // migration keys per thread held in registers there
constexpr int TK_REG_KEYS = TK_RJ * TK_THREADS;
constexpr int TK_RJ1 = 8;                    // best keys per thread in registers (pruned, stage 1)
constexpr int TK_REG_BEST = TK_RJ1 * TK_THREADS;

constexpr int SS_THREADS = 512;              // the one workgroup of the small path
constexpr int SS_RJ = 16;                    // candidates per thread
constexpr int SS_MAX_REQ = 1024;
constexpr int SS_LBATCH = (SC_FUSED_ENTRIES + SS_THREADS - 1) / SS_THREADS;
constexpr int SS_RBATCH = SS_MAX_REQ / SS_THREADS;

constexpr int RK_CODES = 1024;               // key codes (monotone in score - base)
constexpr int RK_MAX_GROUPS = 1024;          // scoring workgroups the ranking kernel can take
constexpr int RK_BCAP = 4096;                // boundary-code keys gathered into LDS

constexpr int64_t kInfS = INT64_MAX;
constexpr uint32_t kInfI = 0xFFFFFFFFu;

__device__ inline int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }
__device__ inline int64_t imin64(int64_t a, int64_t b) { return a < b ? a : b; }

__device__ inline bool key_less(int64_t s0, uint32_t i0, int64_t s1, uint32_t i1) {
    return s0 < s1 || (s0 == s1 && i0 < i1);
}

__device__ inline int bit_length(uint64_t x) { return x ? 64 - __clzll((long long)x) : 0; }

// A key's code is a monotone 10-bit summary of d = score - base (base: the
// smallest target peak, which no migration score is below): the position of
// d's leading one and the four bits after it.  Keys with a smaller code are
// smaller keys, so the k smallest keys are all keys whose code is below some
// c*, plus the smallest few of those with code c*.
__device__ inline uint32_t key_code(uint64_t d) {
    const int e = bit_length(d);                         // 0..63
    if (e <= 4) return (uint32_t)d;
    return ((uint32_t)(e - 4) << 4) | (uint32_t)((d >> (e - 5)) & 15);   // < 960
}
constexpr uint16_t kNoCode = 0xFFFF;                     // a request without a migration

// q = x / d for d >= 1 with m = floor((2^32 - 1) / d) + 1 (m = 0 encodes
// d = 1): the multiply-high estimate is exact or one too large (x + d < 2^32).
__device__ inline uint32_t fast_div(uint32_t x, uint32_t d, uint32_t m) {
    if (m == 0) return x;
    const uint32_t q = __umulhi(x, m);
    return q * d > x ? q - 1 : q;
}
static uint32_t div_magic(uint32_t d) { return d == 1 ? 0u : (uint32_t)(0xFFFFFFFFull / d) + 1u; }

// Value of lane l - 1 (lane 0 gets `ident`): DPP wave_shr:1.
__device__ inline int64_t wave_shr1_i64(int64_t v, int64_t ident) {
    constexpr int kWaveShr1 = 0x138;
    const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)ident, (int)(uint32_t)v, kWaveShr1,
                                               0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(ident >> 32), (int)(v >> 32), kWaveShr1, 0xF,
                                               0xF, false);
    return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Inclusive prefix max over the 32 lanes of each half wave (lane order):
// DPP row shifts, then row 1 / row 3 take lane 15 of row 0 / row 2.
__device__ inline int64_t half_incl_max_i64(int64_t v) {
    v = dpp_max_step_i64<kDppRowShr1, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr2, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr4, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr8, 0xF>(v);
    v = dpp_max_step_i64<kDppRowBcast15, 0xA>(v);
    return v;
}

// PM/SM of every instance from curves in LDS with row stride K+1 (entry K
// of each row is padding).  Each instance is taken by a group of 32 lanes
// (half a wave; kT/32 instances at a time); lane l owns a run of S (odd,
// >= ceil(K/32)) consecutive buckets: a max over its run, one DPP scan across
// the 32 runs, then a pass that writes.  Runs are read PMSM_BATCH entries at
// a time so that their LDS reads are in flight together.  For SM the runs
// are numbered from the end of the curve.
constexpr int PMSM_BATCH = 8;
template <int kT>
__device__ inline void build_pm_sm(const int64_t* lL, int64_t* lPM, int64_t* lSM, int n, int K,
                                   int64_t bb) {
    const int l = threadIdx.x & 31;
    const int K1 = K + 1;
    // run length: at least ceil(K/32), and odd, so that the 32 lanes' runs
    // start on different LDS banks (an even stride of 2^j buckets would put
    // them on a few banks only)
    const int S = ((K + 31) >> 5) | 1;
    for (int t0 = 0; t0 < n; t0 += kT / 32) {
        const int t = t0 + (int)(threadIdx.x >> 5);
        // waves whose two instances are both past n sit out (no barrier
        // inside: the DPP moves stay within the wave)
        if (t0 + 2 * (int)(threadIdx.x >> 6) >= n) continue;
        const bool live = t < n;
        const int tc = live ? t : 0;
        const int64_t* L = lL + tc * K1;
        int64_t* pm = lPM + tc * K1;
        int64_t* sm = lSM + tc * K1;
        const int j0 = l * S;
        const int j1 = j0 + S < K ? j0 + S : K;      // run [j0, j1) (empty past the end)
        // PM: exclusive prefix max of L[j] + b^2 j
        int64_t run = INT64_MIN;
        for (int jb = j0; jb < j1; jb += PMSM_BATCH) {
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb + u;
                x[u] = L[j < j1 ? j : j0];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u)
                if (jb + u < j1) run = imax(run, x[u] + bb * (jb + u));
        }
        const int64_t pinc = half_incl_max_i64(run);
        const int64_t pex = wave_shr1_i64(pinc, INT64_MIN);
        run = l == 0 ? INT64_MIN : pex;
        for (int jb = j0; jb < j1; jb += PMSM_BATCH) {
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb + u;
                x[u] = L[j < j1 ? j : j0];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb + u;
                if (j < j1) {
                    if (live) pm[j] = run;
                    run = imax(run, x[u] + bb * j);
                }
            }
        }
        if (live && l == 31) pm[K] = pinc;
        // SM: inclusive suffix max of L[j]; lane l takes j = K-1-j0 down to K-j1
        const int q0 = K - 1 - j0, q1 = K - j1;      // run [q1, q0], walked downwards
        run = INT64_MIN;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb - u;
                x[u] = L[j >= q1 ? j : q0];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u)
                if (jb - u >= q1) run = imax(run, x[u]);
        }
        const int64_t sinc = half_incl_max_i64(run);
        const int64_t sex = wave_shr1_i64(sinc, INT64_MIN);
        run = l == 0 ? INT64_MIN : sex;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb - u;
                x[u] = L[j >= q1 ? j : q0];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int j = jb - u;
                if (j >= q1) {
                    run = imax(run, x[u]);
                    if (live) sm[j] = run;
                }
            }
        }
        if (live && l == 0) sm[K] = INT64_MIN;
    }
}

// Inclusive prefix sum over the 32 lanes of each half wave (lane order),
// DPP as in half_incl_max_i64; lanes without a source add 0.
template <int kCtrl, int kRowMask>
__device__ inline int64_t dpp_add_step_i64(int64_t v) {
    const int lo = dpp_i32<kCtrl, kRowMask>((int)(uint32_t)v, 0);
    const int hi = dpp_i32<kCtrl, kRowMask>((int)(v >> 32), 0);
    return v + (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
__device__ inline int64_t half_incl_add_i64(int64_t v) {
    v = dpp_add_step_i64<kDppRowShr1, 0xF>(v);
    v = dpp_add_step_i64<kDppRowShr2, 0xF>(v);
    v = dpp_add_step_i64<kDppRowShr4, 0xF>(v);
    v = dpp_add_step_i64<kDppRowShr8, 0xF>(v);
    v = dpp_add_step_i64<kDppRowBcast15, 0xA>(v);
    return v;
}

// Exclusive maximum over the lanes above this one in its half wave (lanes
// l+1..31 of the same 32), -inf for lane 31: shuffles down.
__device__ inline int64_t half_excl_max_above_i64(int64_t v) {
    const int l = threadIdx.x & 31;
    int64_t inc = v;
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
        const uint32_t lo = (uint32_t)__shfl_down((int)(uint32_t)inc, o, 32);
        const uint32_t hi = (uint32_t)__shfl_down((int)(inc >> 32), o, 32);
        const int64_t u = (int64_t)(((uint64_t)hi << 32) | lo);
        inc = l + o < 32 ? imax(inc, u) : inc;
    }
    const uint32_t lo = (uint32_t)__shfl_down((int)(uint32_t)inc, 1, 32);
    const uint32_t hi = (uint32_t)__shfl_down((int)(inc >> 32), 1, 32);
    const int64_t ex = (int64_t)(((uint64_t)hi << 32) | lo);
    return l == 31 ? INT64_MIN : ex;
}

// Section 5.2's curves of every instance from its requests, with their PM
// and SM, in LDS (rows of stride K+1).  In: hA / hN hold alpha_r and the
// request count by k_e (1..K), hP the partial-bucket terms by k_e (0..K-1).
// With S_A(k), S_n(k) the sums of hA, hN over k_e > k, the curve is
// L[k] = S_A(k) + b^2 k S_n(k) + hP[k], written over hP.  Each instance is
// taken by half a wave; lane l owns a run of S (odd) buckets counted from
// the end (lane 0 the top ones), and makes three passes over it:
//   1) run sums of hA, hN; exclusive suffix sums across lanes (DPP);
//   2) L over the run, written, with the run's max of L and of L[j] + b^2 j;
//   3) SM = suffix max (lanes above in bucket order come first: the same
//      DPP direction), PM = exclusive prefix max of L[j] + b^2 j (the lanes
//      holding lower buckets: shuffles down), both written from the run.
// PM_t[K] is the maximum over every bucket; SM_t[K] and L_t[K] are -inf.
template <int kT>
__device__ inline void build_curves_pm_sm(const int64_t* hA, const int64_t* hN, int64_t* hPL,
                                          int64_t* lPM, int64_t* lSM, int n, int K, int64_t bb) {
    const int l = threadIdx.x & 31;
    const int K1 = K + 1;
    const int S = ((K + 31) >> 5) | 1;
    for (int t0 = 0; t0 < n; t0 += kT / 32) {
        const int t = t0 + (int)(threadIdx.x >> 5);
        // waves whose two instances are both past n sit out (no barrier
        // inside: the DPP moves stay within the wave)
        if (t0 + 2 * (int)(threadIdx.x >> 6) >= n) continue;
        const bool live = t < n;
        const int tc = live ? t : 0;
        const int64_t* A = hA + tc * K1;
        const int64_t* C = hN + tc * K1;
        int64_t* L = hPL + tc * K1;
        const int j0 = l * S;
        const int j1 = j0 + S < K ? j0 + S : K;
        const int q0 = K - 1 - j0, q1 = K - j1;      // buckets [q1, q0]
        // 1) run sums
        int64_t sa = 0, sn = 0;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t xa[PMSM_BATCH], xn[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                xa[u] = A[q + 1];
                xn[u] = C[q + 1];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u)
                if (jb - u >= q1) {
                    sa += xa[u];
                    sn += xn[u];
                }
        }
        // every lane runs the lane shifts (a DPP move inside one arm of a
        // branch would read disabled lanes)
        const int64_t ia = half_incl_add_i64(sa), in = half_incl_add_i64(sn);
        const int64_t ea = wave_shr1_i64(ia, 0), en = wave_shr1_i64(in, 0);
        int64_t ra = l == 0 ? 0 : ea;
        int64_t rn = l == 0 ? 0 : en;
        // 2) L over the run (downwards) and the run's maxima
        int64_t smax = INT64_MIN, pmax = INT64_MIN;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t xa[PMSM_BATCH], xn[PMSM_BATCH], xp[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                xa[u] = A[q + 1];
                xn[u] = C[q + 1];
                xp[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u;
                if (q >= q1) {
                    ra += xa[u];
                    rn += xn[u];
                    const int64_t v = ra + bb * q * rn + xp[u];
                    if (live) L[q] = v;
                    smax = imax(smax, v);
                    pmax = imax(pmax, v + bb * q);
                }
            }
        }
        // 3) SM: suffix max, lanes below l hold the higher buckets (same
        //    direction as the sums); PM: prefix max over lower buckets =
        //    lanes above l
        const int64_t si = half_incl_max_i64(smax);
        const int64_t se = wave_shr1_i64(si, INT64_MIN);
        int64_t srun = l == 0 ? INT64_MIN : se;
        int64_t prun = half_excl_max_above_i64(pmax);
        const int64_t ptot = imax(prun, pmax);       // lane 0: max over every bucket
        // the run's L values are this lane's own writes: no barrier needed
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {         // SM downwards
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                x[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u;
                if (q >= q1) {
                    srun = imax(srun, x[u]);
                    if (live) lSM[tc * K1 + q] = srun;
                }
            }
        }
        for (int jb = q1; jb <= q0; jb += PMSM_BATCH) {         // PM upwards, exclusive
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb + u <= q0 ? jb + u : q1;
                x[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb + u;
                if (q <= q0) {
                    if (live) lPM[tc * K1 + q] = prun;
                    prun = imax(prun, x[u] + bb * q);
                }
            }
        }
        if (live && l == 0) {
            L[K] = INT64_MIN;
            lSM[tc * K1 + K] = INT64_MIN;
            lPM[tc * K1 + K] = ptot;
        }
    }
}

// Exclusive maximum over the lanes above this one (lanes l+1..63), -inf for
// lane 63: the wave reversed by an LDS permute, a DPP prefix maximum, and
// the result gathered back by a second permute.
__device__ inline int64_t perm_i64(int64_t x, int src_lane) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_ds_bpermute(src_lane * 4, (int)(uint32_t)x);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_ds_bpermute(src_lane * 4, (int)(x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ inline int64_t wave_excl_max_above_i64(int64_t v) {
    const int l = threadIdx.x & 63;
    const int64_t inc = wave_incl_max_i64(perm_i64(v, 63 - l));   // lane l: max of v[63-l..63]
    const int64_t x = perm_i64(inc, l < 63 ? 62 - l : 0);
    return l < 63 ? x : INT64_MIN;
}

// build_curves_pm_sm with a whole wave per instance (runs of S = ceil(K/64),
// made odd, buckets per lane): half the serial depth, and every wave of a
// larger workgroup takes an instance.
template <int kT>
__device__ inline void build_curves_pm_sm_w(const int64_t* hA, const int64_t* hN, int64_t* hPL,
                                            int64_t* lPM, int64_t* lSM, int n, int K,
                                            int64_t bb) {
    const int l = threadIdx.x & 63;
    const int K1 = K + 1;
    const int S = ((K + 63) >> 6) | 1;
    for (int t = (int)(threadIdx.x >> 6); t < n; t += kT / 64) {   // wave-uniform
        const int64_t* A = hA + t * K1;
        const int64_t* C = hN + t * K1;
        int64_t* L = hPL + t * K1;
        const int j0 = l * S;
        const int j1 = j0 + S < K ? j0 + S : K;
        const int q0 = K - 1 - j0, q1 = K - j1;      // buckets [q1, q0] (none when j0 >= K)
        // 1) run sums
        int64_t sa = 0, sn = 0;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t xa[PMSM_BATCH], xn[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                xa[u] = A[q + 1];
                xn[u] = C[q + 1];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u)
                if (jb - u >= q1) {
                    sa += xa[u];
                    sn += xn[u];
                }
        }
        int64_t ra = wave_shr1_i64(wave_incl_add_i64(sa), 0);   // sums over the lanes below
        int64_t rn = wave_shr1_i64(wave_incl_add_i64(sn), 0);
        // 2) L over the run (downwards) and the run's maxima
        int64_t smax = INT64_MIN, pmax = INT64_MIN;
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {
            int64_t xa[PMSM_BATCH], xn[PMSM_BATCH], xp[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                xa[u] = A[q + 1];
                xn[u] = C[q + 1];
                xp[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u;
                if (q >= q1) {
                    ra += xa[u];
                    rn += xn[u];
                    const int64_t v = ra + bb * q * rn + xp[u];
                    L[q] = v;
                    smax = imax(smax, v);
                    pmax = imax(pmax, v + bb * q);
                }
            }
        }
        // 3) SM from the lanes below (higher buckets), PM from the lanes above
        int64_t srun = wave_shr1_i64(wave_incl_max_i64(smax), INT64_MIN);
        int64_t prun = wave_excl_max_above_i64(pmax);
        const int64_t ptot = imax(prun, pmax);       // lane 0: max over every bucket
        for (int jb = q0; jb >= q1; jb -= PMSM_BATCH) {         // SM downwards
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u >= q1 ? jb - u : q0;
                x[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb - u;
                if (q >= q1) {
                    srun = imax(srun, x[u]);
                    lSM[t * K1 + q] = srun;
                }
            }
        }
        for (int jb = q1; jb <= q0; jb += PMSM_BATCH) {         // PM upwards, exclusive
            int64_t x[PMSM_BATCH];
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb + u <= q0 ? jb + u : q1;
                x[u] = L[q];
            }
#pragma unroll
            for (int u = 0; u < PMSM_BATCH; ++u) {
                const int q = jb + u;
                if (q <= q0) {
                    lPM[t * K1 + q] = prun;
                    prun = imax(prun, x[u] + bb * q);
                }
            }
        }
        if (l == 0) {
            L[K] = INT64_MIN;
            lSM[t * K1 + K] = INT64_MIN;
            lPM[t * K1 + K] = ptot;
        }
    }
}

// The same with a run of at most kS buckets per lane (K <= 64 kS, S odd)
// held in registers: every LDS read of the histograms and partial terms is
// issued at once at the start, and L, SM and PM come from the registers, so
// the lane reads LDS once instead of three times.
constexpr int PMSM_REG_RUN = 5;
template <int kT, int kS>
__device__ inline void build_curves_pm_sm_wr(const int64_t* hA, const int64_t* hN, int64_t* hPL,
                                             int64_t* lPM, int64_t* lSM, int n, int K,
                                             int64_t bb) {
    const int l = threadIdx.x & 63;
    const int K1 = K + 1;
    const int S = ((K + 63) >> 6) | 1;                 // <= kS (the caller checks)
    for (int t = (int)(threadIdx.x >> 6); t < n; t += kT / 64) {   // wave-uniform
        const int64_t* A = hA + t * K1;
        const int64_t* C = hN + t * K1;
        int64_t* L = hPL + t * K1;
        const int j0 = l * S;
        const int q0 = K - 1 - j0;                     // buckets q0, q0 - 1, ... (u < len)
        const int len = j0 < K ? (K - j0 < S ? K - j0 : S) : 0;
        int64_t xa[kS], xn[kS], xv[kS];
#pragma unroll
        for (int u = 0; u < kS; ++u) {
            const int q = u < len ? q0 - u : 0;        // in range: read, then ignored
            xa[u] = A[q + 1];
            xn[u] = C[q + 1];
            xv[u] = L[q];
        }
        int64_t sa = 0, sn = 0;
#pragma unroll
        for (int u = 0; u < kS; ++u)
            if (u < len) {
                sa += xa[u];
                sn += xn[u];
            }
        int64_t ra = wave_shr1_i64(wave_incl_add_i64(sa), 0);   // sums over the lanes below
        int64_t rn = wave_shr1_i64(wave_incl_add_i64(sn), 0);
        int64_t smax = INT64_MIN, pmax = INT64_MIN;
#pragma unroll
        for (int u = 0; u < kS; ++u)
            if (u < len) {
                const int q = q0 - u;
                ra += xa[u];
                rn += xn[u];
                xv[u] = ra + bb * q * rn + xv[u];      // L[q]
                L[q] = xv[u];
                smax = imax(smax, xv[u]);
                pmax = imax(pmax, xv[u] + bb * q);
            }
        int64_t srun = wave_shr1_i64(wave_incl_max_i64(smax), INT64_MIN);
        int64_t prun = wave_excl_max_above_i64(pmax);
        const int64_t ptot = imax(prun, pmax);        // lane 0: max over every bucket
#pragma unroll
        for (int u = 0; u < kS; ++u)                   // SM downwards
            if (u < len) {
                srun = imax(srun, xv[u]);
                lSM[t * K1 + q0 - u] = srun;
            }
#pragma unroll
        for (int u = kS - 1; u >= 0; --u)              // PM upwards, exclusive
            if (u < len) {
                const int q = q0 - u;
                lPM[t * K1 + q] = prun;
                prun = imax(prun, xv[u] + bb * q);
            }
        if (l == 0) {
            L[K] = INT64_MIN;
            lSM[t * K1 + K] = INT64_MIN;
            lPM[t * K1 + K] = ptot;
        }
    }
}


// Minimum of a 64-bit value over aligned groups of g lanes (g a power of
// two, 2..64); every lane of a group gets it.  DPP quad permutes for lane
// distances 1 and 2, row shifts under bank masks for 4 and 8, and
// ds_bpermute-based shuffles above.
template <int kCtrl, int kBankMask>
__device__ inline uint64_t dpp_u64(uint64_t old, uint64_t v) {
    const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)old, (int)(uint32_t)v, kCtrl, 0xF,
                                               kBankMask, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(old >> 32), (int)(v >> 32), kCtrl, 0xF,
                                               kBankMask, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}
__device__ inline uint64_t umin64(uint64_t a, uint64_t b) { return a < b ? a : b; }
__device__ inline uint64_t group_min_u64(uint64_t v, int g) {
    constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E;      // quad_perm [1,0,3,2], [2,3,0,1]
    constexpr int kRowShr4 = 0x114, kRowShl4 = 0x104, kRowShr8 = 0x118, kRowShl8 = 0x108;
    if (g > 1) v = umin64(v, dpp_u64<kQuadXor1, 0xF>(v, v));
    if (g > 2) v = umin64(v, dpp_u64<kQuadXor2, 0xF>(v, v));
    if (g > 4) v = umin64(v, dpp_u64<kRowShl4, 0x5>(dpp_u64<kRowShr4, 0xA>(v, v), v));
    if (g > 8) v = umin64(v, dpp_u64<kRowShl8, 0x3>(dpp_u64<kRowShr8, 0xC>(v, v), v));
    for (int o = 16; o < g; o <<= 1) {
        const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, o, 64);
        const uint32_t hi = (uint32_t)__shfl_xor((int)(v >> 32), o, 64);
        v = umin64(v, ((uint64_t)hi << 32) | lo);
    }
    return v;
}

// Score of moving a request with terms (ke, alpha, p) to t, from PM/SM rows
// of stride K+1 and a curve row L_t whose entry K reads as -inf.
__device__ inline int64_t move_score(const int64_t* pm_t, const int64_t* sm_t, int64_t l_ke, int ke,
                                     int K, int64_t alpha, int64_t p) {
    const int64_t a = pm_t[ke] + alpha;              // PM_t[0] = -inf + alpha: no overflow
    const int64_t m = l_ke + p;
    const int64_t c = sm_t[ke + 1 < K ? ke + 1 : K];
    return imax(imax(a, m), c);
}

// ---------------------------------------------------------------------------
// prep (large curve sets): planes of every instance's PM, L and SM, entry
// (k, t) at k sk + t st (k = 0..K):
//     TPM(k, t) = PM_t[k]                    (PM_t[K] = max over all j)
//     TL(k, t)  = L_t[k], -inf at k = K
//     TSM(k, t) = SM_t[min(k + 1, K)]        (SM_t[K] = -inf)
//     PEAK[t]   = SM_t[0], the instance's peak
// Bucket-major (sk = n, st = 1) puts one request's reads for every target
// at its k_e side by side; instance-major (sk = 1, st = K + 1) makes these
// writes contiguous, for rounds with few requests per bucket.  One workgroup
// per instance.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(PREP_THREADS) void score_prep_kernel(const int64_t* __restrict__ load,
                                                                  int K, int b, int64_t sk,
                                                                  int64_t st,
                                                                  int64_t* __restrict__ TPM,
                                                                  int64_t* __restrict__ TL,
                                                                  int64_t* __restrict__ TSM,
                                                                  int64_t* __restrict__ PEAK) {
    __shared__ int64_t tmp[PREP_THREADS / 64 + 1];
    const int tid = threadIdx.x;
    const int t = blockIdx.x;
    const int64_t* L = load + (int64_t)t * K;
    const int64_t bb = (int64_t)b * b;
    constexpr int CH = PREP_THREADS * PREP_SEG;

    int64_t carry = INT64_MIN;                 // exclusive prefix max of L[j] + b^2 j
    for (int base = 0; base < K; base += CH) {
        const int j0 = base + tid * PREP_SEG;
        int64_t x[PREP_SEG];
        int64_t loc = INT64_MIN;
#pragma unroll
        for (int u = 0; u < PREP_SEG; ++u) {
            const int j = j0 + u;
            x[u] = j < K ? L[j] : 0;
            if (j < K) loc = imax(loc, x[u] + bb * j);
        }
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64<PREP_THREADS>(loc, OpMax(), INT64_MIN, tmp, &tot);
        int64_t run = imax(carry, ex);
#pragma unroll
        for (int u = 0; u < PREP_SEG; ++u) {
            const int j = j0 + u;
            if (j < K) {
                TPM[j * sk + t * st] = run;
                TL[j * sk + t * st] = x[u];
                run = imax(run, x[u] + bb * j);
            }
        }
        carry = imax(carry, tot);
    }
    if (tid == 0) {
        TPM[K * sk + t * st] = carry;
        TL[K * sk + t * st] = INT64_MIN;
        TSM[(K - 1) * sk + t * st] = INT64_MIN;
        TSM[K * sk + t * st] = INT64_MIN;
    }

    carry = INT64_MIN;                         // inclusive suffix max of L[j]
    for (int base = 0; base < K; base += CH) {
        const int p0 = base + tid * PREP_SEG;  // reversed position p <-> j = K-1-p
        int64_t x[PREP_SEG];
        int64_t loc = INT64_MIN;
#pragma unroll
        for (int u = 0; u < PREP_SEG; ++u) {
            const int p = p0 + u;
            x[u] = p < K ? L[K - 1 - p] : INT64_MIN;
            loc = imax(loc, x[u]);
        }
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64<PREP_THREADS>(loc, OpMax(), INT64_MIN, tmp, &tot);
        int64_t run = imax(carry, ex);
#pragma unroll
        for (int u = 0; u < PREP_SEG; ++u) {
            const int p = p0 + u;
            if (p < K) {
                run = imax(run, x[u]);
                const int j = K - 1 - p;       // SM_t[j] = run
                if (j > 0) TSM[(j - 1) * sk + t * st] = run;
                else PEAK[t] = run;
            }
        }
        carry = imax(carry, tot);
    }
}

// ---------------------------------------------------------------------------
// score (multi-workgroup path)
// ---------------------------------------------------------------------------
struct ScoreArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* load;
    int64_t* scores;              // caller's array or workspace copy
    int32_t* best_target;         // caller's array or workspace copy
    int64_t* best_score;
    int32_t* err_word;
    int64_t* load_out;            // curves built by the scoring kernel itself (group 0 writes)
    int64_t* bbase;               // code base for the top-k's best keys (group 0 writes), or null
    uint16_t* bcode;              // [N] code of each request's best key (kNoCode: none), or null
    int N, n, b, K, rpb, cand;
    uint32_t magic_K, magic_n;
};

// Curve sets that fit the LDS: every workgroup builds PM/SM of every
// instance there, then scores its rpb requests against every target.
__global__ __launch_bounds__(SC_THREADS) void score_kernel(ScoreArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int n = a.n, K = a.K, b = a.b;
    const int K1 = K + 1;
    const int cand = a.cand;                       // rpb * n keys in this workgroup
    const int rpb = a.rpb;

    // LDS: [L | PM | SM], keys, per-request values
    int64_t* lL = (int64_t*)smem;
    int64_t* lPM = lL + n * K1;
    int64_t* lSM = lPM + n * K1;
    int64_t* ks = lSM + n * K1;
    int64_t* r_alpha = ks + cand;
    int64_t* r_p = r_alpha + rpb;
    uint32_t* ki = (uint32_t*)(r_p + rpb);
    int32_t* r_ke = (int32_t*)(ki + cand);
    int32_t* r_s = r_ke + rpb;

    const int row0 = blockIdx.x * rpb;
    const int64_t H = (int64_t)b * K;
    const int64_t bb = (int64_t)b * b;

    // 0) per-request values; curves into LDS.  All reads are issued before
    //    the first is used (clamped indices, unconditional loads).
    int32_t bad = 0;
    int64_t lv[SC_LBATCH];
    const int nK = n * K;
#pragma unroll
    for (int j = 0; j < SC_LBATCH; ++j) {
        const int e = j * SC_THREADS + tid;
        lv[j] = a.load[e < nK ? e : nK - 1];
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
            const bool live = row0 + q < a.N;
            const ReqTerms rt = request_terms(sv[j], cv[j], rv[j], n, b, H);
            bad |= live ? rt.bad : 0;
            r_s[q] = live ? rt.s : -1;
            r_ke[q] = rt.ke;
            r_alpha[q] = rt.alpha;
            r_p[q] = rt.p;
        }
    }
    bad = wave_or_i32(bad);
    if (lane == 0) report_error(a.err_word, bad);
#pragma unroll
    for (int j = 0; j < SC_LBATCH; ++j) {
        const int e = j * SC_THREADS + tid;
        if (e < nK) {
            const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
            lL[t * K1 + (e - t * K)] = lv[j];
        }
    }
    for (int t = tid; t < n; t += SC_THREADS) lL[t * K1 + K] = INT64_MIN;
    __syncthreads();
    build_pm_sm<SC_THREADS>(lL, lPM, lSM, n, K, bb);
    __syncthreads();

    // 1) candidates -> scores and keys (self-candidates and invalid requests
    //    get the +inf key)
    for (int e = tid; e < cand; e += SC_THREADS) {
        int64_t key_s = kInfS;
        uint32_t key_i = kInfI;
        const int q = e / n, t = e - q * n;
        const int r = row0 + q;
        if (r < a.N) {
            const int s = r_s[q];
            const int ke = r_ke[q];
            const int64_t l_ke = lL[t * K1 + ke];          // entry K is -inf
            const int64_t* pm_t = lPM + t * K1;
            const int64_t* sm_t = lSM + t * K1;
            const int64_t mv = move_score(pm_t, sm_t, l_ke, ke, K, r_alpha[q], r_p[q]);
            const int64_t sc = s < 0 ? -1 : (t == s ? sm_t[0] : mv);
            if (s >= 0 && t != s) {
                key_s = sc;
                key_i = (uint32_t)((int64_t)r * n + t);
            }
            if (a.scores) a.scores[(int64_t)r * n + t] = sc;
        }
        ks[e] = key_s;
        ki[e] = key_i;
    }
    __syncthreads();

    // the code base of the top-k's best keys: the smallest target peak (no
    // migration scores below it), one read per thread and a block minimum
    int64_t base = INT64_MAX;
    if (a.bbase) {
        __shared__ int64_t wmin[SC_THREADS / 64];
        for (int t = tid; t < n; t += SC_THREADS) {
            const int64_t v = lSM[t * K1];
            base = v < base ? v : base;
        }
        base = -readlane_i64(wave_incl_max_i64(-base), 63);
        if (lane == 0) wmin[tid >> 6] = base;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < SC_THREADS / 64; ++w) base = wmin[w] < base ? wmin[w] : base;
        if (blockIdx.x == 0 && tid == 0) *a.bbase = base;
    }

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
        if (a.bcode) a.bcode[r] = none ? kNoCode : (uint16_t)key_code((uint64_t)(bs - base));
    }
}

// ---------------------------------------------------------------------------
// score from the bucket-major planes (curve sets too large for LDS)
// ---------------------------------------------------------------------------
// One group of G lanes per request, lane l of the group scoring targets
// t = l + G c (c < TPL; G = 16 when n > 16, else the power of two >= n;
// more than 16 TPL targets are taken TPL per lane at a time).  Bucket-major
// planes put every target's PM, L and SM at a request's k_e side by side, so
// a request's reads are a few contiguous lines.  A lane keeps the smallest
// (score, t) of its targets (t ascends, so the first minimum stays), and
// the group minimum is taken with DPP moves inside the 16-lane row.  Each
// group takes REQ consecutive requests, whose reads are issued together.
constexpr int SP_THREADS = 256;
constexpr int SP_ROW = 16;                 // lanes per request when n > 16

struct PlanarArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* tpm;           // planes of PM, L, SM: entry (k, t) at k sk + t st
    const int64_t* tl;
    const int64_t* tsm;
    const int64_t* peak;          // [n]
    int64_t sk, st;
    int64_t* scores;              // [N, n] or null
    int32_t* best_target;         // [N] or null
    int64_t* best_score;          // [N] or null
    int32_t* err_word;
    int64_t* bbase;               // code base of the best keys (workgroup 0 writes), or null
    uint16_t* bcode;              // [N] code of each request's best key, or null
    int N, n, b, K, lg;           // G = 2^lg lanes per request
};

template <int TPL, int REQ>
__global__ __launch_bounds__(SP_THREADS) void score_planar_kernel(PlanarArgs a) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int n = a.n, b = a.b, K = a.K;
    const int G = 1 << a.lg;
    const int gl = lane & (G - 1);
    const int gpw = 64 >> a.lg;                          // groups per wave
    const int wave = blockIdx.x * (SP_THREADS / 64) + (tid >> 6);
    const int64_t H = (int64_t)b * K;
    const int64_t alpha0 = (int64_t)b * (b - 1) / 2;

    int rv[REQ], sv[REQ], cv[REQ], lv[REQ];
#pragma unroll
    for (int j = 0; j < REQ; ++j) {
        rv[j] = (wave * REQ + j) * gpw + (lane >> a.lg);
        const int rc = rv[j] < a.N ? rv[j] : a.N - 1;
        sv[j] = a.inst[rc];
        cv[j] = a.cur[rc];
        lv[j] = a.rem[rc];
    }
    // the code base: the smallest peak (no migration scores below it)
    int64_t base = INT64_MAX;
    if (a.bbase) {
        for (int t = lane; t < n; t += 64) base = imin64(base, a.peak[t]);
        base = -readlane_i64(wave_incl_max_i64(-base), 63);
        if (blockIdx.x == 0 && tid == 0) *a.bbase = base;
    }
    // request terms (Section 5.2's load model, as the projection takes them)
    int32_t bad = 0;
    int ke[REQ], s[REQ];
    int64_t al[REQ], pp[REQ];
#pragma unroll
    for (int j = 0; j < REQ; ++j) {
        int32_t f = 0;
        if (sv[j] < 0 || sv[j] >= n) f |= STAR_DEV_BAD_INST;
        if (cv[j] < 1) f |= STAR_DEV_BAD_CUR;
        if (lv[j] < 1) f |= STAR_DEV_BAD_REM;
        const bool live = rv[j] < a.N;
        bad |= live ? f : 0;
        const uint32_t lp = (uint32_t)((int64_t)lv[j] < H ? (int64_t)lv[j] : H);
        const uint32_t k = lp / (uint32_t)b;
        const int64_t mu = (int64_t)(lp - k * (uint32_t)b);
        const bool ok = f == 0;
        s[j] = ok && live ? sv[j] : -1;
        ke[j] = ok ? (int)k : 0;
        al[j] = (int64_t)b * cv[j] + alpha0;
        pp[j] = mu * cv[j] + mu * (int64_t)k * b + mu * (mu - 1) / 2;
    }
    bad = wave_or_i32(bad);
    if (lane == 0) report_error(a.err_word, bad);

    int64_t bs[REQ];
    int bt[REQ];
#pragma unroll
    for (int j = 0; j < REQ; ++j) {
        bs[j] = kInfS;
        bt[j] = -1;
    }
    for (int t0 = 0; t0 < n; t0 += G * TPL) {
        int tv[TPL];
        int64_t pk[TPL];
        int64_t xm[REQ][TPL], xl[REQ][TPL], xs[REQ][TPL];
#pragma unroll
        for (int c = 0; c < TPL; ++c) {
            tv[c] = t0 + gl + G * c;
            const int tc = tv[c] < n ? tv[c] : n - 1;
            pk[c] = a.peak[tc];
#pragma unroll
            for (int j = 0; j < REQ; ++j) {
                const int64_t idx = ke[j] * a.sk + tc * a.st;
                xm[j][c] = a.tpm[idx];
                xl[j][c] = a.tl[idx];
                xs[j][c] = a.tsm[idx];
            }
        }
#pragma unroll
        for (int j = 0; j < REQ; ++j) {
#pragma unroll
            for (int c = 0; c < TPL; ++c) {
                const int t = tv[c];
                const int64_t mv = imax(imax(xm[j][c] + al[j], xl[j][c] + pp[j]), xs[j][c]);
                const int64_t sc = s[j] < 0 ? -1 : (t == s[j] ? pk[c] : mv);
                const bool tin = t < n;
                if (tin && rv[j] < a.N && a.scores) a.scores[(int64_t)rv[j] * n + t] = sc;
                if (tin && s[j] >= 0 && t != s[j] && sc < bs[j]) {
                    bs[j] = sc;
                    bt[j] = t;
                }
            }
        }
    }
    // best (score, t) of each request over its group
#pragma unroll
    for (int j = 0; j < REQ; ++j) {
        const uint64_t u = bt[j] >= 0 ? (uint64_t)bs[j] ^ 0x8000000000000000ull : ~0ull;
        const uint64_t um = group_min_u64(u, G);
        const uint64_t tt = bt[j] >= 0 && u == um ? (uint64_t)(uint32_t)bt[j] : ~0ull;
        const uint64_t tm = group_min_u64(tt, G);
        if (gl == 0 && rv[j] < a.N) {
            const bool none = um == ~0ull;
            const int64_t best = (int64_t)(um ^ 0x8000000000000000ull);
            if (a.best_target) a.best_target[rv[j]] = none ? -1 : (int32_t)tm;
            if (a.best_score) a.best_score[rv[j]] = none ? -1 : best;
            if (a.bcode) a.bcode[rv[j]] = none ? kNoCode : (uint16_t)key_code((uint64_t)(best - base));
        }
    }
}

// Targets per lane and requests per group of the planar scoring: a dozen
// plane reads in flight per lane (two dozen with four targets per lane,
// where two requests per group halve the waves: at 32768 requests on 64
// instances they then fit the chip at once, 11.4 against 11.9 us with one).
static int planar_tpl(int n) { return n <= SP_ROW ? 1 : n <= 2 * SP_ROW ? 2 : 4; }
static int planar_req(int tpl) { return tpl == 4 ? 2 : 4 / tpl; }

static hipError_t launch_planar(const PlanarArgs& q, int groups, int tpl, hipStream_t stream) {
    switch (tpl) {
    case 1:
        hipLaunchKernelGGL((score_planar_kernel<1, 4>), dim3(groups), dim3(SP_THREADS), 0, stream, q);
        break;
    case 2:
        hipLaunchKernelGGL((score_planar_kernel<2, 2>), dim3(groups), dim3(SP_THREADS), 0, stream, q);
        break;
    default:
        hipLaunchKernelGGL((score_planar_kernel<4, 2>), dim3(groups), dim3(SP_THREADS), 0, stream, q);
        break;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// block-wide helpers for a workgroup of kT threads (full exec mask)
// ---------------------------------------------------------------------------
template <int kT>
struct alignas(16) SelShared {
    static constexpr int W = kT / 64;
    int hist[SEL_BINS];           // digit histogram (int4-accessed); bucket offsets when ordering
    int fill[SEL_BINS];           // bucket fill counters when ordering
    int wcnt[W];
    int64_t wlo[W];
    int64_t whi[W];
    alignas(16) int bcast[4];
};

__device__ inline int wave_total_add_i32(int v) {
    return __builtin_amdgcn_readlane(wave_incl_add_i32(v), 63);
}

// Count, min and max over the block in one LDS round; every thread gets them.
template <int kT>
__device__ inline void block_stats(int cnt, int64_t lo, int64_t hi, SelShared<kT>& sh, int* total,
                                   int64_t* mn, int64_t* mx) {
    constexpr int W = kT / 64;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    cnt = wave_total_add_i32(cnt);
    const int64_t nlo = readlane_i64(wave_incl_max_i64(-lo), 63);
    hi = readlane_i64(wave_incl_max_i64(hi), 63);
    if (lane == 0) {
        sh.wcnt[wid] = cnt;
        sh.wlo[wid] = -nlo;
        sh.whi[wid] = hi;
    }
    __syncthreads();
    const int c = lane < W ? sh.wcnt[lane] : 0;
    const int64_t l = lane < W ? -sh.wlo[lane] : -kInfS;
    const int64_t h = lane < W ? sh.whi[lane] : -1;
    *total = wave_total_add_i32(c);
    *mn = -readlane_i64(wave_incl_max_i64(l), 63);
    *mx = readlane_i64(wave_incl_max_i64(h), 63);
    __syncthreads();
}

// Exclusive prefix of one int over the block (thread order); *total = sum.
template <int kT>
__device__ inline int block_excl_i32(int v, SelShared<kT>& sh, int* total) {
    constexpr int W = kT / 64;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int inc = wave_incl_add_i32(v);
    if (lane == 63) sh.wcnt[wid] = inc;
    __syncthreads();
    const int xs = wave_incl_add_i32(lane < W ? sh.wcnt[lane] : 0);
    const int before = wid > 0 ? __builtin_amdgcn_readlane(xs, wid - 1) : 0;
    *total = __builtin_amdgcn_readlane(xs, W - 1);
    __syncthreads();
    return before + inc - v;
}

// ---------------------------------------------------------------------------
// key sources: visit(f) calls f(s, i) on each of this thread's keys; s ==
// kInfS marks "no key".  Every thread makes the same calls (uniform control).
// ---------------------------------------------------------------------------
template <int RJ>
struct RegKeys {                  // RJ keys in registers (unused slots hold kInfS)
    int64_t s[RJ];
    uint32_t i[RJ];
    template <class F>
    __device__ inline void visit(F&& f) const {
#pragma unroll
        for (int j = 0; j < RJ; ++j) f(s[j], i[j]);
    }
};

struct BestKeys {                 // (best score, r) of every request with a migration
    const int64_t* best_score;
    const int32_t* best_target;
    int N;
    template <class F>
    __device__ inline void visit(F&& f) const {
        for (int r0 = 0; r0 < N; r0 += TK_THREADS * SEL_SBATCH) {
            int64_t bs[SEL_SBATCH];
            int32_t bt[SEL_SBATCH];
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) {
                const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
                const int rc = r < N ? r : N - 1;
                bs[u] = best_score[rc];
                bt[u] = best_target[rc];
            }
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) {
                const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
                const bool ok = r < N && bt[u] >= 0;
                f(ok ? bs[u] : kInfS, ok ? (uint32_t)r : kInfI);
            }
        }
    }
};

struct TopkArgs {
    const int32_t* inst;
    const int64_t* scores;        // [N, n] (caller's array or workspace copy)
    const int32_t* best_target;   // [N]
    const int64_t* best_score;    // [N]
    int32_t* topk_req;
    int32_t* topk_tgt;
    int64_t* topk_score;
    const int64_t* bbase;         // code base of the best keys (the smallest target peak)
    const uint16_t* bcode;        // [N] code of each best key (kNoCode: none), code stage only
    int64_t* gs;                  // [TK_REG_BEST] best keys gathered at or below the k-th code
    uint32_t* gi;
    int N, n, top_k;
    uint32_t magic_n, magic_n1;   // fast_div multipliers for n and n - 1
};

// Migration e of the pruned set: the v-th other instance of request rk[q],
// with (q, v) = divmod(e, n - 1).
__device__ inline void pruned_key(const TopkArgs& a, const int32_t* rk, const int32_t* rk_inst,
                                  uint32_t e, int64_t* s, uint32_t* i) {
    const uint32_t n1 = (uint32_t)a.n - 1;
    const uint32_t q = fast_div(e, n1, a.magic_n1);
    const int v = (int)(e - q * n1);
    const int r = rk[q];
    const int t = v < rk_inst[q] ? v : v + 1;             // skip staying put
    *i = (uint32_t)((int64_t)r * a.n + t);
    *s = a.scores[(int64_t)r * a.n + t];
}

struct PrunedKeys {               // every migration of the requests rk[0..nr), streamed
    const TopkArgs* a;
    const int32_t* rk;            // LDS: request ids
    const int32_t* rk_inst;       // LDS: their instances
    int M;                        // nr * (n - 1)
    template <class F>
    __device__ inline void visit(F&& f) const {
        for (int e0 = 0; e0 < M; e0 += TK_THREADS * SEL_SBATCH) {
            int64_t sv[SEL_SBATCH];
            uint32_t iv[SEL_SBATCH];
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) {
                const int e = e0 + u * TK_THREADS + (int)threadIdx.x;
                pruned_key(*a, rk, rk_inst, (uint32_t)(e < M ? e : M - 1), &sv[u], &iv[u]);
            }
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) {
                const int e = e0 + u * TK_THREADS + (int)threadIdx.x;
                f(e < M ? sv[u] : kInfS, e < M ? iv[u] : kInfI);
            }
        }
    }
};

// Register loaders of the 1024-thread top-k: every slot is loaded (clamped
// index) and masked afterwards, so the reads are issued together.
template <int RJ>
__device__ inline void load_migrations(RegKeys<RJ>& k, const TopkArgs& a) {
    const int M = a.N * a.n;                               // >= 1
    int32_t iv[RJ], bv[RJ];
    uint32_t qv[RJ];
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        const uint32_t ec = (uint32_t)(e < M ? e : M - 1);
        qv[j] = fast_div(ec, (uint32_t)a.n, a.magic_n);
        k.s[j] = a.scores[ec];
        iv[j] = a.inst[qv[j]];
        bv[j] = a.best_target[qv[j]];
    }
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        const bool ok = e < M && bv[j] >= 0 && (int)((uint32_t)e - qv[j] * (uint32_t)a.n) != iv[j];
        k.s[j] = ok ? k.s[j] : kInfS;
        k.i[j] = ok ? (uint32_t)e : kInfI;
    }
}

__device__ inline void load_best(RegKeys<TK_RJ1>& k, const TopkArgs& a) {
    int32_t bt[TK_RJ1];
#pragma unroll
    for (int j = 0; j < TK_RJ1; ++j) {
        const int r = j * TK_THREADS + (int)threadIdx.x;
        const int rc = r < a.N ? r : a.N - 1;              // N >= 1
        k.s[j] = a.best_score[rc];
        bt[j] = a.best_target[rc];
    }
#pragma unroll
    for (int j = 0; j < TK_RJ1; ++j) {
        const int r = j * TK_THREADS + (int)threadIdx.x;
        const bool ok = r < a.N && bt[j] >= 0;
        k.s[j] = ok ? k.s[j] : kInfS;
        k.i[j] = ok ? (uint32_t)r : kInfI;
    }
}

template <int RJ>
__device__ inline void load_pruned(RegKeys<RJ>& k, const TopkArgs& a, const int32_t* rk,
                                   const int32_t* rk_inst, int M) {
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        k.s[j] = kInfS;
        k.i[j] = kInfI;
    }
    if (M == 0) return;                                    // no request has a migration
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        pruned_key(a, rk, rk_inst, (uint32_t)(e < M ? e : M - 1), &k.s[j], &k.i[j]);
    }
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        k.s[j] = e < M ? k.s[j] : kInfS;
        k.i[j] = e < M ? k.i[j] : kInfI;
    }
}

// ---------------------------------------------------------------------------
// radix select
// ---------------------------------------------------------------------------
template <int kT>
__device__ inline void clear_bins(int* h) {
    for (int q = threadIdx.x * 4; q < SEL_BINS; q += kT * 4) *(int4*)&h[q] = make_int4(0, 0, 0, 0);
}

// The bin holding the kk-th key (1-based); updates kk to the rank inside it,
// *cnt = its size.
template <int kT>
__device__ inline uint32_t find_bin(SelShared<kT>& sh, int* kk, int* cnt) {
    constexpr int PER = SEL_BINS / kT;
    static_assert(PER % 4 == 0, "int4 of bins per thread");
    int c[PER], own = 0;
#pragma unroll
    for (int u = 0; u < PER; u += 4) {
        const int4 c4 = *(const int4*)&sh.hist[threadIdx.x * PER + u];
        c[u] = c4.x; c[u + 1] = c4.y; c[u + 2] = c4.z; c[u + 3] = c4.w;
        own += c4.x + c4.y + c4.z + c4.w;
    }
    int tot;
    int before = block_excl_i32<kT>(own, sh, &tot);
    const int want = *kk;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        if (before < want && want <= before + c[u]) {
            sh.bcast[0] = threadIdx.x * PER + u;
            sh.bcast[1] = want - before;
            sh.bcast[2] = c[u];
        }
        before += c[u];
    }
    __syncthreads();
    const int4 b4 = *(const int4*)sh.bcast;
    *kk = b4.y;
    *cnt = b4.z;
    __syncthreads();
    return (uint32_t)b4.x;
}

// Keys packed as v = ((s - smin) << ibits) | i (nbits bits), a 64-bit value
// that orders like (s, i).  Returns the bound U on v.
template <int kT, class Src>
__device__ uint64_t select_packed(const Src& src, int k, int64_t smin, int nbits, int ibits,
                                  SelShared<kT>& sh) {
    uint64_t prefix = 0;                  // v >> pos == prefix for the keys still in play
    int kk = k, pos = nbits;
    while (pos > 0) {
        const int lowbit = pos > SEL_DIGIT ? pos - SEL_DIGIT : 0;
        const uint32_t mask = (1u << (pos - lowbit)) - 1;
        clear_bins<kT>(sh.hist);
        __syncthreads();
        src.visit([&](int64_t s, uint32_t i) {
            if (s == kInfS) return;
            const uint64_t v = ((uint64_t)(s - smin) << ibits) | i;
            if (pos < 64 && (v >> pos) != prefix) return;
            atomicAdd(&sh.hist[(uint32_t)(v >> lowbit) & mask], 1);
        });
        __syncthreads();
        int cnt;
        const uint32_t bin = find_bin<kT>(sh, &kk, &cnt);
        prefix = (prefix << (pos - lowbit)) | bin;
        pos = lowbit;
        if (cnt == kk) break;             // the whole bin is needed
    }
    return (prefix << pos) | ((1ull << pos) - 1);
}

// Wide keys (score range and index need more than 64 bits): digits over the
// (sbits + 32)-bit value (d << 32) | i, d = s - smin.  Returns U as (us, ui).
template <int kT, class Src>
__device__ void select_wide(const Src& src, int k, int64_t smin, int sbits, SelShared<kT>& sh,
                            int64_t* us, uint32_t* ui) {
    uint64_t pd = 0, md = 0;              // chosen prefix / mask on d
    uint32_t pi = 0, mi = 0;              // chosen prefix / mask on i
    int kk = k;
    for (int pos = sbits + 32; pos > 0;) {
        const int lowbit = pos > SEL_DIGIT ? pos - SEL_DIGIT : 0;     // digit bits [lowbit, pos)
        const int width = pos - lowbit;
        clear_bins<kT>(sh.hist);
        __syncthreads();
        src.visit([&](int64_t s, uint32_t i) {
            if (s == kInfS) return;
            const uint64_t d = (uint64_t)(s - smin);
            if ((d & md) != pd || (i & mi) != pi) return;
            uint32_t dig;
            if (lowbit >= 32) dig = (uint32_t)(d >> (lowbit - 32));
            else if (pos <= 32) dig = i >> lowbit;
            else dig = (uint32_t)((d << (32 - lowbit)) | (i >> lowbit));
            atomicAdd(&sh.hist[dig & ((1u << width) - 1)], 1);
        });
        __syncthreads();
        int cnt;
        const uint32_t bin = find_bin<kT>(sh, &kk, &cnt);
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
        pos = lowbit;
        if (cnt == kk) break;
    }
    // U: the prefix with every unchosen bit set, within the sbits bits every
    // d has (smin + 2^sbits - 1 <= 2 smax < 2^63: no overflow)
    uint64_t du = pd | ~md;
    du &= sbits >= 64 ? ~0ull : ((1ull << sbits) - 1);
    *us = smin + (int64_t)du;
    *ui = pi | ~mi;
}

// Given the source's count / min / max, the bound U = (us, ui) such that
// exactly min(k, total) keys are <= U.  ibits: bits of the largest index.
template <int kT, class Src>
__device__ void select_bound(const Src& src, int k, int ibits, int total, int64_t smin,
                             int64_t smax, SelShared<kT>& sh, int64_t* us, uint32_t* ui) {
    if (total <= k) {                     // every key is a winner
        *us = kInfS - 1;
        *ui = kInfI;
        return;
    }
    const int sbits = bit_length((uint64_t)(smax - smin));
    if (sbits + ibits <= 64) {
        const uint64_t U = select_packed<kT>(src, k, smin, sbits + ibits, ibits, sh);
        *us = smin + (int64_t)(U >> ibits);
        *ui = (uint32_t)(U & ((1ull << ibits) - 1));
    } else {
        select_wide<kT>(src, k, smin, sbits, sh, us, ui);
    }
}

template <int kT, class Src>
__device__ void source_stats(const Src& src, SelShared<kT>& sh, int* total, int64_t* smin,
                             int64_t* smax) {
    int mine = 0;
    int64_t lo = kInfS, hi = -1;
    src.visit([&](int64_t s, uint32_t) {
        if (s != kInfS) {
            ++mine;
            lo = s < lo ? s : lo;
            hi = s > hi ? s : hi;
        }
    });
    block_stats<kT>(mine, lo, hi, sh, total, smin, smax);
}

// Writes the source's keys <= U to (os, oi) in thread order; returns their
// count (every thread gets it).
template <int kT, class Src>
__device__ int block_gather(const Src& src, int64_t us, uint32_t ui, SelShared<kT>& sh,
                            int64_t* os, uint32_t* oi, int cap) {
    int mine = 0;
    src.visit([&](int64_t s, uint32_t i) {
        if (s != kInfS && !key_less(us, ui, s, i)) ++mine;
    });
    int total;
    int at = block_excl_i32<kT>(mine, sh, &total);
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

// Puts the nw winners (ws_s, ws_i), all with score in [smin, smax_w], in key
// order and writes them as (i / n, i % n, s); -1 past nw up to top_k.
// Bucket sort on the top SEL_DIGIT bits of the packed key, then a rank
// count among the members of each bucket.
template <int kT>
__device__ void order_and_write(const int64_t* ws_s, const uint32_t* ws_i, int nw, int64_t smin,
                                int64_t smax_w, int ibits, int n, uint32_t magic_n,
                                int32_t* out_r, int32_t* out_t, int64_t* out_s, int top_k,
                                SelShared<kT>& sh, uint64_t* sv) {
    const int tid = threadIdx.x;
    const int sbits = nw > 0 ? bit_length((uint64_t)(smax_w - smin)) : 0;
    const uint64_t imask = (1ull << ibits) - 1;
    if (nw > 0 && sbits + ibits <= 64) {
        // about two buckets per winner (at least one per thread, at most
        // SEL_BINS): the scan below touches only those
        int bb = kT;
        while (bb < 2 * nw && bb < SEL_BINS) bb <<= 1;
        const int bbits = bit_length((uint64_t)(bb - 1));
        const int nbits = sbits + ibits;
        const int shift = nbits > bbits ? nbits - bbits : 0;
        for (int q = tid; q < bb; q += kT) {
            sh.hist[q] = 0;
            sh.fill[q] = 0;
        }
        __syncthreads();
        for (int p = tid; p < nw; p += kT) {
            const uint64_t v = ((uint64_t)(ws_s[p] - smin) << ibits) | ws_i[p];
            atomicAdd(&sh.hist[(uint32_t)(v >> shift)], 1);
        }
        __syncthreads();
        {                                                   // counts -> exclusive offsets
            constexpr int PER = SEL_BINS / kT;
            const int per = bb / kT;                        // 1 .. PER
            int c[PER], own = 0;
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                c[u] = u < per ? sh.hist[tid * per + u] : 0;
                own += c[u];
            }
            int tot;
            int before = block_excl_i32<kT>(own, sh, &tot);
#pragma unroll
            for (int u = 0; u < PER; ++u) {
                if (u < per) sh.hist[tid * per + u] = before;
                before += c[u];
            }
        }
        __syncthreads();
        for (int p = tid; p < nw; p += kT) {
            const uint64_t v = ((uint64_t)(ws_s[p] - smin) << ibits) | ws_i[p];
            const uint32_t bkt = (uint32_t)(v >> shift);
            sv[sh.hist[bkt] + atomicAdd(&sh.fill[bkt], 1)] = v;
        }
        __syncthreads();
        for (int q = tid; q < nw; q += kT) {
            const uint64_t v = sv[q];
            const uint32_t bkt = (uint32_t)(v >> shift);
            const int lo = sh.hist[bkt], cnt = sh.fill[bkt];
            int rank = 0;
            for (int j = lo; j < lo + cnt; ++j) rank += sv[j] < v ? 1 : 0;
            const int pos = lo + rank;
            const uint32_t i = (uint32_t)(v & imask);
            const uint32_t r = fast_div(i, (uint32_t)n, magic_n);
            out_r[pos] = (int32_t)r;
            out_t[pos] = (int32_t)(i - r * (uint32_t)n);
            out_s[pos] = smin + (int64_t)(v >> ibits);
        }
    } else if (nw > 0) {                                    // rank count over all winners
        for (int w = tid; w < nw; w += kT) {
            const int64_t xs = ws_s[w];
            const uint32_t xi = ws_i[w];
            int rank = 0;
            for (int j = 0; j < nw; ++j) rank += key_less(ws_s[j], ws_i[j], xs, xi) ? 1 : 0;
            const uint32_t r = fast_div(xi, (uint32_t)n, magic_n);
            out_r[rank] = (int32_t)r;
            out_t[rank] = (int32_t)(xi - r * (uint32_t)n);
            out_s[rank] = xs;
        }
    }
    for (int q = nw + tid; q < top_k; q += kT) {
        out_r[q] = -1;
        out_t[q] = -1;
        out_s[q] = -1;
    }
}

// Full selection over a source: stats, bound, gather, order, write.
template <int kT, class Src>
__device__ int select_top(const Src& src, int k, int ibits, SelShared<kT>& sh, int64_t* ws_s,
                          uint32_t* ws_i, int64_t* smin_out, int64_t* smax_w_out) {
    int total;
    int64_t smin, smax, us;
    uint32_t ui;
    source_stats<kT>(src, sh, &total, &smin, &smax);
    select_bound<kT>(src, k, ibits, total, smin, smax, sh, &us, &ui);
    *smin_out = smin;
    *smax_w_out = us < smax ? us : smax;
    return block_gather<kT>(src, us, ui, sh, ws_s, ws_i, STAR_MAX_TOP_K);
}

// ---------------------------------------------------------------------------
// top-k kernels of the multi-workgroup path (one workgroup)
// ---------------------------------------------------------------------------
// Every migration held in registers, kRJ per thread (N n <= kRJ TK_THREADS).
template <int kRJ>
__global__ __launch_bounds__(TK_THREADS) void topk_direct_kernel(TopkArgs a) {
    __shared__ SelShared<TK_THREADS> sh;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    __shared__ uint64_t sv[STAR_MAX_TOP_K];
    RegKeys<kRJ> keys;
    load_migrations(keys, a);
    const int ibits = bit_length((uint64_t)(a.N * a.n - 1));
    int64_t smin, smax_w;
    const int nw = select_top<TK_THREADS>(keys, a.top_k, ibits, sh, ws_s, ws_i, &smin, &smax_w);
    order_and_write<TK_THREADS>(ws_s, ws_i, nw, smin, smax_w, ibits, a.n, a.magic_n, a.topk_req,
                                a.topk_tgt, a.topk_score, a.top_k, sh, sv);
}

// Boundary keys of select_by_code, and its counters.
constexpr int TK_BCAP = 2048;
struct CodeLds {
    int64_t bs_s[TK_BCAP];
    uint32_t bs_i[TK_BCAP];
    int na, nb;
};

// The k smallest of a register source's keys, by their codes relative to
// base (no key is below it).  An LDS histogram of the codes gives c*, the
// code that holds the k-th key: every key below c* wins, and the k - na
// smallest of the nb keys of code c* are ranked directly when nb <=
// TK_THREADS, radix-selected from LDS when nb <= TK_BCAP, and otherwise (a
// crowded code) the whole source is radix-selected.  The winners go to
// (ws_s, ws_i) unordered, with their score range; returns their count.
template <int RJ>
__device__ __forceinline__ int select_by_code(const RegKeys<RJ>& keys, int k, int64_t base, int ibits,
                              SelShared<TK_THREADS>& sh, CodeLds& cl, int64_t* ws_s,
                              uint32_t* ws_i, int64_t* smin, int64_t* smax_w) {
    static_assert(RK_CODES == TK_THREADS && RK_CODES <= SEL_BINS, "one code per thread");
    constexpr uint32_t kNone = 0xFFFFFFFFu;
    const int tid = threadIdx.x;
    sh.hist[tid] = 0;
    if (tid == 0) {
        cl.na = 0;
        cl.nb = 0;
    }
    __syncthreads();
    uint32_t code[RJ];
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        code[j] = keys.s[j] != kInfS ? key_code((uint64_t)(keys.s[j] - base)) : kNone;
        if (code[j] != kNone) atomicAdd(&sh.hist[code[j]], 1);
    }
    __syncthreads();
    const int h = sh.hist[tid];
    int total;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &total);
    const int kk = k < total ? k : total;
    if (tid == 0) sh.bcast[0] = RK_CODES;              // every key wins when total <= k
    __syncthreads();
    if (kk < total && before < kk && kk <= before + h) {
        sh.bcast[0] = tid;
        sh.bcast[1] = h;
    }
    __syncthreads();
    const uint32_t cstar = (uint32_t)sh.bcast[0];
    const int nbc = cstar < (uint32_t)RK_CODES ? sh.bcast[1] : 0;
    __syncthreads();
    if (nbc > TK_BCAP) return select_top<TK_THREADS>(keys, k, ibits, sh, ws_s, ws_i, smin, smax_w);
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        if (code[j] < cstar) {                            // fewer than kk <= STAR_MAX_TOP_K
            const int p = atomicAdd(&cl.na, 1);
            ws_s[p] = keys.s[j];
            ws_i[p] = keys.i[j];
        } else if (code[j] == cstar) {                    // nbc <= TK_BCAP of them
            const int p = atomicAdd(&cl.nb, 1);
            cl.bs_s[p] = keys.s[j];
            cl.bs_i[p] = keys.i[j];
        }
    }
    __syncthreads();
    const int na = cl.na, nb = cl.nb;
    const int need = kk - na;                             // 0 <= need <= nb
    int nw = na;
    if (need > 0) {
        if (nb <= TK_THREADS) {
            if (tid < nb) {
                const int64_t xs = cl.bs_s[tid];
                const uint32_t xi = cl.bs_i[tid];
                int rank = 0;
                for (int q = 0; q < nb; ++q) rank += key_less(cl.bs_s[q], cl.bs_i[q], xs, xi) ? 1 : 0;
                if (rank < need) {
                    ws_s[na + rank] = xs;
                    ws_i[na + rank] = xi;
                }
            }
            nw += need;
        } else {
            RegKeys<TK_BCAP / TK_THREADS> bk;
#pragma unroll
            for (int j = 0; j < TK_BCAP / TK_THREADS; ++j) {
                const int p = j * TK_THREADS + tid;
                bk.s[j] = p < nb ? cl.bs_s[p] : kInfS;
                bk.i[j] = p < nb ? cl.bs_i[p] : kInfI;
            }
            int cnt;
            int64_t us, mn, mx;
            uint32_t ui;
            source_stats<TK_THREADS>(bk, sh, &cnt, &mn, &mx);
            select_bound<TK_THREADS>(bk, need, ibits, cnt, mn, mx, sh, &us, &ui);
            nw += block_gather<TK_THREADS>(bk, us, ui, sh, ws_s + na, ws_i + na,
                                           STAR_MAX_TOP_K - na);
        }
    }
    __syncthreads();
    int64_t lo = kInfS, hi = -1;
    for (int p = tid; p < nw; p += TK_THREADS) {
        lo = ws_s[p] < lo ? ws_s[p] : lo;
        hi = ws_s[p] > hi ? ws_s[p] : hi;
    }
    int cntw;
    block_stats<TK_THREADS>(0, lo, hi, sh, &cntw, smin, smax_w);
    return nw;
}

// The k smallest of the g gathered best keys, RJ per thread in registers.
template <int RJ>
__device__ __forceinline__ int select_gathered(const TopkArgs& a, int g, int ib1, SelShared<TK_THREADS>& sh,
                               CodeLds& cl, int64_t base, int64_t* ws_s, uint32_t* ws_i,
                               int64_t* smin, int64_t* smax_w) {
    RegKeys<RJ> keys;
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        const int ec = e < g ? e : 0;
        keys.s[j] = a.gs[ec];
        keys.i[j] = a.gi[ec];
    }
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const int e = j * TK_THREADS + (int)threadIdx.x;
        keys.s[j] = e < g ? keys.s[j] : kInfS;
        keys.i[j] = e < g ? keys.i[j] : kInfI;
    }
    return select_by_code<RJ>(keys, a.top_k, base, ib1, sh, cl, ws_s, ws_i, smin, smax_w);
}

// Best-key code of request r (kNoCode: none), loaded in batches of
// SEL_SBATCH per thread; f(r, code) for each.
template <class F>
__device__ inline void visit_codes(const TopkArgs& a, F&& f) {
    for (int r0 = 0; r0 < a.N; r0 += TK_THREADS * SEL_SBATCH) {
        uint16_t cv[SEL_SBATCH];
#pragma unroll
        for (int u = 0; u < SEL_SBATCH; ++u) {
            const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
            cv[u] = a.bcode[r < a.N ? r : a.N - 1];
        }
#pragma unroll
        for (int u = 0; u < SEL_SBATCH; ++u) {
            const int r = r0 + u * TK_THREADS + (int)threadIdx.x;
            f(r, r < a.N ? cv[u] : kNoCode);
        }
    }
}

// The k smallest best keys by their codes, which the scoring kernel wrote
// (2 bytes per request): one pass counts them in an LDS histogram and finds
// the code c* that holds the k-th key, a second gathers every best key of
// code <= c* (all of the k smallest, and only keys no larger than the rest
// of code c*), and those are selected in registers.  More than TK_REG_BEST
// such keys (a crowded code c*) take the streamed selection over all best
// keys instead.
__device__ __forceinline__ int select_best_by_code(const TopkArgs& a, int ib1, SelShared<TK_THREADS>& sh,
                                   CodeLds& cl, int64_t* ws_s, uint32_t* ws_i, int64_t* smin,
                                   int64_t* smax_w, int* gcount) {
    static_assert(RK_CODES == TK_THREADS && RK_CODES <= SEL_BINS, "one code per thread");
    const int tid = threadIdx.x;
    const int64_t base = *a.bbase;
    sh.hist[tid] = 0;
    __syncthreads();
    visit_codes(a, [&](int, uint16_t c) {
        if (c != kNoCode) atomicAdd(&sh.hist[c], 1);
    });
    __syncthreads();
    const int h = sh.hist[tid];
    int total;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &total);
    const bool all = total <= a.top_k;
    if (all ? tid == RK_CODES - 1 : (before < a.top_k && before + h >= a.top_k)) {
        sh.bcast[0] = tid;                     // c*
        sh.bcast[1] = before + h;              // best keys of code <= c*
    }
    if (tid == 0) *gcount = 0;
    __syncthreads();
    const uint32_t cstar = (uint32_t)sh.bcast[0];
    const int nle = sh.bcast[1];
    __syncthreads();
    if (nle > TK_REG_BEST) {
        BestKeys bk{a.best_score, a.best_target, a.N};
        return select_top<TK_THREADS>(bk, a.top_k, ib1, sh, ws_s, ws_i, smin, smax_w);
    }
    visit_codes(a, [&](int r, uint16_t c) {
        if (c != kNoCode && c <= cstar) {
            const int at = atomicAdd(gcount, 1);
            if (at < TK_REG_BEST) {
                a.gs[at] = a.best_score[r];
                a.gi[at] = (uint32_t)r;
            }
        }
    });
    __syncthreads();                           // the gathered keys are visible to the workgroup
    const int g = *gcount < TK_REG_BEST ? *gcount : TK_REG_BEST;
    return select_gathered<TK_RJ1>(a, g, ib1, sh, cl, base, ws_s, ws_i, smin, smax_w);
}

// Counting sort of the pruned top-k: up to TK_SORT_CAP candidate keys,
// first compacted in thread order (each thread's count, a block prefix, then
// plain LDS writes: no per-key atomic round trips), then placed in slots
// grouped by code (sh.hist holds each code's offset, sh.fill its count) and
// ranked among the keys that share their code.
constexpr int TK_SORT_CAP = TK_THREADS;
constexpr int TK_CODE_V = 4;                            // 16-byte code reads per thread
constexpr int TK_CODE_REG = TK_CODE_V * 8 * TK_THREADS; // best-key codes held in registers
struct SortLds {
    int64_t s[TK_SORT_CAP];       // keys in code order
    uint32_t i[TK_SORT_CAP];
    uint16_t c[TK_SORT_CAP];
    int64_t cs[TK_SORT_CAP];      // the candidates, compacted in thread order
    uint32_t ci[TK_SORT_CAP];
    uint16_t cc[TK_SORT_CAP];
};

// Thread t's key (s, i) of code c goes to the next slot of its code (t < P;
// sh.hist: code offsets, sh.fill: zero); returns its place in key order: the
// code's offset plus the number of keys of the code below it (-1 for t >= P).
__device__ __forceinline__ int sort_place(SelShared<TK_THREADS>& sh, SortLds& sl, int P, int64_t s,
                                          uint32_t i, uint16_t c) {
    const int tid = threadIdx.x;
    if (tid < P) {
        const int slot = sh.hist[c] + atomicAdd(&sh.fill[c], 1);
        sl.s[slot] = s;
        sl.i[slot] = i;
        sl.c[slot] = c;
    }
    __syncthreads();
    if (tid >= P) return -1;
    const int lo = sh.hist[c], hi = lo + sh.fill[c];
    int rank = 0;
    int j = lo;
    for (; j + 4 <= hi; j += 4) {                       // four LDS reads in flight
        int64_t xs[4];
        uint32_t xi[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            xs[u] = sl.s[j + u];
            xi[u] = sl.i[j + u];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) rank += key_less(xs[u], xi[u], s, i) ? 1 : 0;
    }
    for (; j < hi; ++j) rank += key_less(sl.s[j], sl.i[j], s, i) ? 1 : 0;
    return lo + rank;
}

// Code u (0..7) of eight consecutive 2-byte codes read as one 16-byte word.
__device__ __forceinline__ uint16_t code_of(const uint4& v, int u) {
    const uint32_t w = u < 2 ? v.x : u < 4 ? v.y : u < 6 ? v.z : v.w;
    return (uint16_t)((u & 1) ? w >> 16 : w & 0xFFFFu);
}

// Stage 1 with every best-key code in registers (N <= TK_CODE_REG): the code
// histogram gives c*, the code of the k-th smallest best key; every best key
// of code <= c* is compacted and counting-sorted, so (ws_s, ws_i)[0, nr)
// holds the nr = min(k, keys) smallest best keys in key order and *smax_w
// the largest of them.  Returns -1 (with the workgroup synchronised) when
// more than TK_SORT_CAP best keys have codes <= c*.
__device__ __forceinline__ int best_sorted(const TopkArgs& a, SelShared<TK_THREADS>& sh,
                                           SortLds& sl, int64_t* ws_s, uint32_t* ws_i,
                                           int64_t* smax_w) {
    static_assert(RK_CODES == TK_THREADS && TK_SORT_CAP <= TK_THREADS, "one code per thread");
    const int tid = threadIdx.x;
    const uint4* cp = reinterpret_cast<const uint4*>(a.bcode);   // 256-byte aligned, padded
    const int nv = (a.N + 7) >> 3;
    uint4 cv[TK_CODE_V];
#pragma unroll
    for (int j = 0; j < TK_CODE_V; ++j) {
        const int v = j * TK_THREADS + tid;
        cv[j] = cp[v < nv ? v : 0];
    }
    sh.hist[tid] = 0;
    sh.fill[tid] = 0;
    // codes past N read as kNoCode from here on (masked once, in registers)
#pragma unroll
    for (int j = 0; j < TK_CODE_V; ++j) {
        const int v = j * TK_THREADS + tid;
        const int valid = v < nv ? a.N - v * 8 : 0;      // codes of this group below N
        auto pad = [valid](int d) -> uint32_t {      // kNoCode in slots 2d, 2d+1 past N
            return (2 * d >= valid ? 0x0000FFFFu : 0u) | (2 * d + 1 >= valid ? 0xFFFF0000u : 0u);
        };
        cv[j].x |= pad(0);
        cv[j].y |= pad(1);
        cv[j].z |= pad(2);
        cv[j].w |= pad(3);
    }
    __syncthreads();
    auto code = [&](int j, int u) -> uint16_t { return code_of(cv[j], u); };
#pragma unroll
    for (int j = 0; j < TK_CODE_V; ++j)
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const uint16_t c = code(j, u);
            if (c != kNoCode) atomicAdd(&sh.hist[c], 1);
        }
    __syncthreads();
    const int h = sh.hist[tid];
    int total;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &total);
    const bool all = total <= a.top_k;
    if (all ? tid == RK_CODES - 1 : (before < a.top_k && before + h >= a.top_k)) {
        sh.bcast[0] = tid;                                // c*
        sh.bcast[1] = before + h;                         // best keys of code <= c*
    }
    sh.hist[tid] = before;                                // code offsets
    __syncthreads();
    const uint32_t cstar = (uint32_t)sh.bcast[0];
    const int nle = sh.bcast[1];
    if (nle > TK_SORT_CAP) {
        __syncthreads();
        return -1;
    }
    // which of this thread's codes are <= c*, as one bit each; their
    // compacted positions follow a block prefix of the bit counts
    uint32_t sel = 0;
#pragma unroll
    for (int j = 0; j < TK_CODE_V; ++j)
#pragma unroll
        for (int u = 0; u < 8; ++u) sel |= (code(j, u) <= cstar ? 1u : 0u) << (j * 8 + u);
    int tot;
    int pos = block_excl_i32<TK_THREADS>(__builtin_popcount(sel), sh, &tot);
    if (sel) {                                            // few threads have any
#pragma unroll
        for (int j = 0; j < TK_CODE_V; ++j)
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (sel & (1u << (j * 8 + u))) {
                    sl.ci[pos] = (uint32_t)((j * TK_THREADS + tid) * 8 + u);
                    sl.cc[pos] = code(j, u);
                    ++pos;
                }
    }
    __syncthreads();
    int64_t s = 0;
    uint32_t r = 0;
    uint16_t c = 0;
    if (tid < nle) {
        r = sl.ci[tid];
        c = sl.cc[tid];
        s = a.best_score[r];
    }
    const int nr = a.top_k < nle ? a.top_k : nle;
    const int p = sort_place(sh, sl, nle, s, r, c);
    if (p >= 0 && p < nr) {
        ws_s[p] = s;
        ws_i[p] = r;
    }
    __syncthreads();
    *smax_w = nr > 0 ? ws_s[nr - 1] : -1;
    return nr;
}

// The k smallest of a register source's keys (no key below base), in key
// order: the code histogram gives c*, and every key of code <= c* is
// compacted and counting-sorted, so (ws_s, ws_i)[0, nr) holds the nr =
// min(k, keys) smallest and *smax_w the largest of them.  Returns -1 (with
// the workgroup synchronised) when more than TK_SORT_CAP keys have codes
// <= c*.
template <int RJ>
__device__ __forceinline__ int regs_sorted(const RegKeys<RJ>& keys, int k, int64_t base,
                                           SelShared<TK_THREADS>& sh, SortLds& sl,
                                           int64_t* ws_s, uint32_t* ws_i, int64_t* smax_w) {
    constexpr uint16_t kNone = 0xFFFF;
    const int tid = threadIdx.x;
    sh.hist[tid] = 0;
    sh.fill[tid] = 0;
    __syncthreads();
    uint16_t code[RJ];
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        const bool ok = keys.s[j] != kInfS;
        code[j] = ok ? (uint16_t)key_code((uint64_t)(keys.s[j] - base)) : kNone;
        if (ok) atomicAdd(&sh.hist[code[j]], 1);
    }
    __syncthreads();
    const int h = sh.hist[tid];
    int total;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &total);
    const bool all = total <= k;
    if (all ? tid == RK_CODES - 1 : (before < k && before + h >= k)) {
        sh.bcast[0] = tid;                                // c*
        sh.bcast[1] = before + h;                         // keys of code <= c*
    }
    sh.hist[tid] = before;                                // code offsets
    __syncthreads();
    const uint32_t cstar = (uint32_t)sh.bcast[0];
    const int nle = sh.bcast[1];
    if (nle > TK_SORT_CAP) {
        __syncthreads();
        return -1;
    }
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < RJ; ++j) cnt += code[j] <= cstar ? 1 : 0;
    int tot;
    int pos = block_excl_i32<TK_THREADS>(cnt, sh, &tot);
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        if (code[j] <= cstar) {
            sl.cs[pos] = keys.s[j];
            sl.ci[pos] = keys.i[j];
            sl.cc[pos] = code[j];
            ++pos;
        }
    }
    __syncthreads();
    int64_t ks = 0;
    uint32_t ki = 0;
    uint16_t kc = 0;
    if (tid < nle) {
        ks = sl.cs[tid];
        ki = sl.ci[tid];
        kc = sl.cc[tid];
    }
    const int nr = k < nle ? k : nle;
    const int p = sort_place(sh, sl, nle, ks, ki, kc);
    if (p >= 0 && p < nr) {
        ws_s[p] = ks;
        ws_i[p] = ki;
    }
    __syncthreads();
    *smax_w = nr > 0 ? ws_s[nr - 1] : -1;
    return nr;
}

// Stage 2 from registers: the k smallest migrations of the nr requests,
// written in key order.  When nr = k, the k requests' best keys are k
// distinct migrations, so the k-th smallest migration is at most the largest
// of them (smax_w) and only migrations scored at most smax_w can win; when
// nr < k every migration of the nr requests is a candidate.  The candidates
// are compacted and counting-sorted on their codes.  Returns false, with
// nothing written and the workgroup synchronised, when more than
// TK_SORT_CAP are candidates.
template <int RJ>
__device__ __forceinline__ bool pruned_sorted_write(const RegKeys<RJ>& keys, const TopkArgs& a,
                                                    int nr, int64_t smax_w, int64_t base,
                                                    SelShared<TK_THREADS>& sh, SortLds& sl) {
    const int tid = threadIdx.x;
    const int64_t thr = nr == a.top_k ? smax_w : kInfS;
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < RJ; ++j) cnt += keys.s[j] != kInfS && keys.s[j] <= thr ? 1 : 0;
    int P;
    int pos = block_excl_i32<TK_THREADS>(cnt, sh, &P);
    if (P > TK_SORT_CAP) return false;                    // block_excl_i32 ends synchronised
#pragma unroll
    for (int j = 0; j < RJ; ++j) {
        if (keys.s[j] != kInfS && keys.s[j] <= thr) {
            sl.cs[pos] = keys.s[j];
            sl.ci[pos] = keys.i[j];
            ++pos;
        }
    }
    sh.hist[tid] = 0;
    sh.fill[tid] = 0;
    __syncthreads();
    int64_t s = 0;
    uint32_t i = 0;
    uint16_t c = 0;
    if (tid < P) {
        s = sl.cs[tid];
        i = sl.ci[tid];
        c = (uint16_t)key_code((uint64_t)(s - base));
        atomicAdd(&sh.hist[c], 1);
    }
    __syncthreads();
    const int h = sh.hist[tid];
    int tot;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &tot);
    sh.hist[tid] = before;
    __syncthreads();
    const int kk = a.top_k < P ? a.top_k : P;
    const int p = sort_place(sh, sl, P, s, i, c);
    if (p >= 0 && p < kk) {
        const uint32_t r = fast_div(i, (uint32_t)a.n, a.magic_n);
        a.topk_req[p] = (int32_t)r;
        a.topk_tgt[p] = (int32_t)(i - r * (uint32_t)a.n);
        a.topk_score[p] = s;
    }
    for (int q = kk + tid; q < a.top_k; q += TK_THREADS) {
        a.topk_req[q] = -1;
        a.topk_tgt[q] = -1;
        a.topk_score[q] = -1;
    }
    return true;
}

// How the pruned top-k finds the k requests with the smallest best keys: all
// best keys in registers, or those the code histogram leaves.
enum : int { kStage1Reg = 0, kStage1Code = 1 };

// First the k requests with the smallest best keys, then the k smallest of
// their migrations (kRJ2 per thread in registers, or streamed when 0).
template <int kStage1, int kRJ2>
__global__ __launch_bounds__(TK_THREADS) void topk_pruned_kernel(TopkArgs a) {
    __shared__ SelShared<TK_THREADS> sh;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    __shared__ uint64_t sv[STAR_MAX_TOP_K];
    __shared__ int32_t rk[STAR_MAX_TOP_K];
    __shared__ int32_t rk_inst[STAR_MAX_TOP_K];
    __shared__ int gcount;
    __shared__ CodeLds cl;
    __shared__ SortLds sl;
    int nr;
    int64_t smin, smax_w;
    const int64_t base = *a.bbase;
    const int ib1 = bit_length((uint64_t)(a.N - 1));
    if constexpr (kStage1 == kStage1Reg) {
        RegKeys<TK_RJ1> keys;
        load_best(keys, a);
        nr = kRJ2 > 0 ? regs_sorted<TK_RJ1>(keys, a.top_k, base, sh, sl, ws_s, ws_i, &smax_w) : -1;
        if (nr < 0)
            nr = select_by_code<TK_RJ1>(keys, a.top_k, base, ib1, sh, cl, ws_s, ws_i, &smin,
                                        &smax_w);
    } else {
        // (the streamed stage 2 keeps the histogram-and-gather stage 1: the
        // two together exceed the registers of a 1024-thread workgroup)
        nr = kRJ2 > 0 && a.N <= TK_CODE_REG ? best_sorted(a, sh, sl, ws_s, ws_i, &smax_w) : -1;
        if (nr < 0) nr = select_best_by_code(a, ib1, sh, cl, ws_s, ws_i, &smin, &smax_w, &gcount);
    }
    for (int q = threadIdx.x; q < nr; q += TK_THREADS) {
        const int r = (int)ws_i[q];
        rk[q] = r;
        rk_inst[q] = a.inst[r];
    }
    __syncthreads();
    const int M = nr * (a.n - 1);
    const int ib2 = bit_length((uint64_t)((int64_t)a.N * a.n - 1));
    int nw;
    if constexpr (kRJ2 > 0) {
        RegKeys<kRJ2> keys;
        load_pruned(keys, a, rk, rk_inst, M);
        if (pruned_sorted_write<kRJ2>(keys, a, nr, smax_w, base, sh, sl)) return;
        nw = select_by_code<kRJ2>(keys, a.top_k, base, ib2, sh, cl, ws_s, ws_i, &smin, &smax_w);
    } else {
        PrunedKeys pk{&a, rk, rk_inst, M};
        nw = select_top<TK_THREADS>(pk, a.top_k, ib2, sh, ws_s, ws_i, &smin, &smax_w);
    }
    order_and_write<TK_THREADS>(ws_s, ws_i, nw, smin, smax_w, ib2, a.n, a.magic_n, a.topk_req,
                                a.topk_tgt, a.topk_score, a.top_k, sh, sv);
}

// ---------------------------------------------------------------------------
// score + first ranking stage (many workgroups), then one workgroup ranks
// ---------------------------------------------------------------------------
struct RankArgs {
    uint32_t* ghist;              // [RK_CODES] counts over all groups (zero on entry)
    int64_t* base;                // the code base, written by group 0
    int64_t* keys_s;              // [groups, cand] each group's migrations in code order
    uint32_t* keys_i;
    int32_t* offs;                // [groups, RK_CODES + 1] exclusive code offsets per group
};

struct FinalArgs {
    uint32_t* ghist;              // zeroed here after use
    const int32_t* offs;
    const int64_t* keys_s;
    const uint32_t* keys_i;
    int32_t* topk_req;
    int32_t* topk_tgt;
    int64_t* topk_score;
    int groups, cand, n, top_k, ibits;
    uint32_t magic_n;
};

constexpr int RK_THREADS = 256;               // the ranking workgroup

// Keys of code c* of every group, streamed: slot x of the flattened
// [groups, cand] array is one when lo[w] <= j < hi[w] (w, j = divmod(x, cand)).
struct BoundaryKeys {
    const FinalArgs* a;
    const int32_t* lo;            // LDS [groups]
    const int32_t* hi;
    template <class F>
    __device__ inline void visit(F&& f) const {
        const int X = a->groups * a->cand;
        for (int x0 = 0; x0 < X; x0 += RK_THREADS * SEL_SBATCH) {
            int64_t sv[SEL_SBATCH];
            uint32_t iv[SEL_SBATCH];
            bool ok[SEL_SBATCH];
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) {
                const int x = x0 + u * RK_THREADS + (int)threadIdx.x;
                const int xc = x < X ? x : X - 1;
                const int w = xc / a->cand, j = xc - w * a->cand;
                ok[u] = x < X && j >= lo[w] && j < hi[w];
                sv[u] = a->keys_s[xc];
                iv[u] = a->keys_i[xc];
            }
#pragma unroll
            for (int u = 0; u < SEL_SBATCH; ++u) f(ok[u] ? sv[u] : kInfS, ok[u] ? iv[u] : kInfI);
        }
    }
};

// Position p of a concatenation whose part w starts at pre[w] (pre[0] = 0,
// nondecreasing, parts 0..G-1): the part holding p.
__device__ inline int find_part(const int32_t* pre, int G, int p) {
    int lo = 0, hi = G - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= p) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// LDS of the final ranking workgroup.
struct FinalLds {
    SelShared<RK_THREADS> sh;
    int64_t ws_s[STAR_MAX_TOP_K];
    uint32_t ws_i[STAR_MAX_TOP_K];
    uint64_t sv[STAR_MAX_TOP_K];
    int32_t lo_w[RK_MAX_GROUPS], hi_w[RK_MAX_GROUPS];
    int32_t pre_a[RK_MAX_GROUPS], pre_b[RK_MAX_GROUPS];
    int64_t bs_s[RK_BCAP];
    uint32_t bs_i[RK_BCAP];
};

__device__ __forceinline__ void rank_final_body(const FinalArgs& a, FinalLds& F) {
    SelShared<RK_THREADS>& sh = F.sh;
    int64_t* ws_s = F.ws_s;
    uint32_t* ws_i = F.ws_i;
    uint64_t* sv = F.sv;
    int32_t* lo_w = F.lo_w;
    int32_t* hi_w = F.hi_w;
    int32_t* pre_a = F.pre_a;
    int32_t* pre_b = F.pre_b;
    int64_t* bs_s = F.bs_s;
    uint32_t* bs_i = F.bs_i;
    const int tid = threadIdx.x;
    const int G = a.groups;

    // 1) c*: the code holding the k-th smallest key (four codes per thread);
    //    the histogram is zeroed for the next call
    constexpr int CPT = RK_CODES / RK_THREADS;
    int hc[CPT], own = 0;
#pragma unroll
    for (int u = 0; u < CPT; ++u) {
        hc[u] = (int)a.ghist[tid * CPT + u];
        own += hc[u];
    }
#pragma unroll
    for (int u = 0; u < CPT; ++u) a.ghist[tid * CPT + u] = 0;
    int total;
    int ex = block_excl_i32<RK_THREADS>(own, sh, &total);
    const int k = a.top_k < total ? a.top_k : total;
    if (tid == 0) sh.bcast[0] = RK_CODES;             // all keys win when total <= k
    __syncthreads();
    if (k < total) {
#pragma unroll
        for (int u = 0; u < CPT; ++u) {
            if (ex < k && k <= ex + hc[u]) sh.bcast[0] = tid * CPT + u;
            ex += hc[u];
        }
    }
    __syncthreads();
    const int cstar = sh.bcast[0];

    // 2) per group: keys below c* ([0, lo)) and at c* ([lo, hi)); thread
    //    tid owns the groups [tid*GPT, tid*GPT + GPT)
    const int GPT = (G + RK_THREADS - 1) / RK_THREADS;
    int sa = 0, sb = 0;
    for (int u = 0; u < GPT; ++u) {
        const int w = tid * GPT + u;
        if (w < G) {
            const int32_t* o = a.offs + (int64_t)w * (RK_CODES + 1);
            const int l = o[cstar];
            const int h = cstar < RK_CODES ? o[cstar + 1] : l;
            lo_w[w] = l;
            hi_w[w] = h;
            sa += l;
            sb += h - l;
        }
    }
    int na, nb;
    int pa = block_excl_i32<RK_THREADS>(sa, sh, &na);
    int pb = block_excl_i32<RK_THREADS>(sb, sh, &nb);
    for (int u = 0; u < GPT; ++u) {
        const int w = tid * GPT + u;
        if (w < G) {
            pre_a[w] = pa;
            pre_b[w] = pb;
            pa += lo_w[w];
            pb += hi_w[w] - lo_w[w];
        }
    }
    __syncthreads();

    // 3) every key below c* wins (na < k <= STAR_MAX_TOP_K)
    for (int p = tid; p < na; p += RK_THREADS) {
        const int w = find_part(pre_a, G, p);
        const int64_t x = (int64_t)w * a.cand + (p - pre_a[w]);
        ws_s[p] = a.keys_s[x];
        ws_i[p] = a.keys_i[x];
    }

    // 4) the k - na smallest keys of code c*
    const int need = k - na;
    int nw = na;
    if (need > 0 && nb <= RK_BCAP) {
        for (int p = tid; p < nb; p += RK_THREADS) {
            const int w = find_part(pre_b, G, p);
            const int64_t x = (int64_t)w * a.cand + lo_w[w] + (p - pre_b[w]);
            bs_s[p] = a.keys_s[x];
            bs_i[p] = a.keys_i[x];
        }
        __syncthreads();
        if (nb <= RK_THREADS) {
            // few keys: each one's rank among them, directly
            if (tid < nb) {
                const int64_t xs = bs_s[tid];
                const uint32_t xi = bs_i[tid];
                int rank = 0;
                for (int q = 0; q < nb; ++q) rank += key_less(bs_s[q], bs_i[q], xs, xi) ? 1 : 0;
                if (rank < need) {
                    ws_s[na + rank] = xs;
                    ws_i[na + rank] = xi;
                }
            }
            nw += need;
        } else {
            RegKeys<RK_BCAP / RK_THREADS> keys;
#pragma unroll
            for (int j = 0; j < RK_BCAP / RK_THREADS; ++j) {
                const int p = j * RK_THREADS + tid;
                keys.s[j] = p < nb ? bs_s[p] : kInfS;
                keys.i[j] = p < nb ? bs_i[p] : kInfI;
            }
            int cnt;
            int64_t us, smin, smax;
            uint32_t ui;
            source_stats<RK_THREADS>(keys, sh, &cnt, &smin, &smax);
            select_bound<RK_THREADS>(keys, need, a.ibits, cnt, smin, smax, sh, &us, &ui);
            nw += block_gather<RK_THREADS>(keys, us, ui, sh, ws_s + na, ws_i + na,
                                           STAR_MAX_TOP_K - na);
        }
    } else if (need > 0) {
        BoundaryKeys src{&a, lo_w, hi_w};
        int cnt;
        int64_t us, smin, smax;
        uint32_t ui;
        source_stats<RK_THREADS>(src, sh, &cnt, &smin, &smax);
        select_bound<RK_THREADS>(src, need, a.ibits, cnt, smin, smax, sh, &us, &ui);
        nw += block_gather<RK_THREADS>(src, us, ui, sh, ws_s + na, ws_i + na, STAR_MAX_TOP_K - na);
    }
    __syncthreads();

    // 5) order the winners and write them out
    int64_t lo = kInfS, hi = -1;
    for (int p = tid; p < nw; p += RK_THREADS) {
        lo = ws_s[p] < lo ? ws_s[p] : lo;
        hi = ws_s[p] > hi ? ws_s[p] : hi;
    }
    int cntw;
    int64_t wmin, wmax;
    block_stats<RK_THREADS>(0, lo, hi, sh, &cntw, &wmin, &wmax);
    order_and_write<RK_THREADS>(ws_s, ws_i, nw, wmin, wmax, a.ibits, a.n, a.magic_n, a.topk_req,
                                a.topk_tgt, a.topk_score, a.top_k, sh, sv);
}

__global__ __launch_bounds__(RK_THREADS) void rank_final_kernel(FinalArgs a) {
    __shared__ FinalLds F;
    rank_final_body(a, F);
}

// Fused scoring (all curves in LDS) plus each group's migration keys sorted
// by code (a counting sort in LDS), its code offsets and the global code
// histogram.
// kProject: every group builds the curves itself from all N requests (the
//   load projection, redundantly per group: N is small on this path) and
//   group 0 writes them to a.load_out, so no projection kernel runs first.
//   (Measured on MI355X: one launch fewer per round is worth more than the
//   repeated reads of the requests.  Handing the final ranking to the last
//   group to finish was not: its device-scope fences and the ranking's LDS
//   in every group cost more than the ranking kernel's launch.)
template <bool kProject>
__global__ __launch_bounds__(SC_THREADS) void score_rank_kernel(ScoreArgs a, RankArgs rk) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ int lhist[RK_CODES];
    __shared__ int wtot[SC_THREADS / 64];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int n = a.n, K = a.K, b = a.b;
    const int K1 = K + 1;
    const int cand = a.cand;                       // rpb * n <= SC_THREADS: one per thread
    const int rpb = a.rpb;

    int64_t* lL = (int64_t*)smem;
    int64_t* lPM = lL + n * K1;
    int64_t* lSM = lPM + n * K1;
    int64_t* ks = lSM + n * K1;
    int64_t* r_alpha = ks + cand;
    int64_t* r_p = r_alpha + rpb;
    uint32_t* ki = (uint32_t*)(r_p + rpb);
    int32_t* r_ke = (int32_t*)(ki + cand);
    int32_t* r_s = r_ke + rpb;

    const int g = blockIdx.x;
    const int row0 = g * rpb;
    const int64_t H = (int64_t)b * K;
    const int64_t bb = (int64_t)b * b;

    // 0) curves and per-request terms (all reads issued first)
    const int nK = n * K;
    int64_t lv[kProject ? 1 : SC_LBATCH];
    if constexpr (!kProject) {
#pragma unroll
        for (int j = 0; j < SC_LBATCH; ++j) {
            const int e = j * SC_THREADS + tid;
            lv[j] = a.load[e < nK ? e : nK - 1];
        }
    }
    int32_t bad = 0;
    {
        const int q = tid;                           // rpb <= SC_THREADS
        int r = row0 + q;
        r = r < a.N ? r : a.N - 1;
        const int sv = a.inst[r], cv = a.cur[r], rv = a.rem[r];
        if (q < rpb) {
            const bool live = row0 + q < a.N;
            const ReqTerms rt = request_terms(sv, cv, rv, n, b, H);
            bad = live ? rt.bad : 0;
            r_s[q] = live ? rt.s : -1;
            r_ke[q] = rt.ke;
            r_alpha[q] = rt.alpha;
            r_p[q] = rt.p;
        }
    }
    bad = wave_or_i32(bad);
    if (lane == 0) report_error(a.err_word, bad);
    if constexpr (kProject) {
        // histograms by k_e: hA in PM's rows, hN in SM's, hP in L's (the
        // three are contiguous); invalid requests add nothing
        for (int e = tid; e < 3 * n * K1; e += SC_THREADS) lL[e] = 0;
        __syncthreads();
        for (int base = 0; base < a.N; base += SC_THREADS * SC_PBATCH) {
            int sv[SC_PBATCH], cv[SC_PBATCH], rv[SC_PBATCH];
#pragma unroll
            for (int j = 0; j < SC_PBATCH; ++j) {
                const int r = base + j * SC_THREADS + tid;
                const int rc = r < a.N ? r : a.N - 1;
                sv[j] = a.inst[rc];
                cv[j] = a.cur[rc];
                rv[j] = a.rem[rc];
            }
#pragma unroll
            for (int j = 0; j < SC_PBATCH; ++j) {
                if (base + j * SC_THREADS + tid >= a.N) continue;
                const ReqTerms rt = request_terms(sv[j], cv[j], rv[j], n, b, H);
                if (rt.s < 0) continue;
                const int row = rt.s * K1;
                if (rt.ke > 0) {
                    atomicAdd((unsigned long long*)&lPM[row + rt.ke], (unsigned long long)rt.alpha);
                    atomicAdd((unsigned long long*)&lSM[row + rt.ke], 1ull);
                }
                if (rt.p != 0) atomicAdd((unsigned long long*)&lL[row + rt.ke], (unsigned long long)rt.p);
            }
        }
        __syncthreads();
        // the histograms hA / hN sit in PM's / SM's rows: every lane reads
        // them (its own run and one entry of the next) in the first two
        // sweeps, which the whole wave finishes before any lane writes PM
        // or SM in the third; instances use disjoint rows
        build_curves_pm_sm<SC_THREADS>(lPM, lSM, lL, lPM, lSM, n, K, bb);
        __syncthreads();
        if (g == 0)
            for (int e = tid; e < nK; e += SC_THREADS) {
                const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
                a.load_out[e] = lL[t * K1 + (e - t * K)];
            }
    } else {
#pragma unroll
        for (int j = 0; j < SC_LBATCH; ++j) {
            const int e = j * SC_THREADS + tid;
            if (e < nK) {
                const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
                lL[t * K1 + (e - t * K)] = lv[j];
            }
        }
        for (int t = tid; t < n; t += SC_THREADS) lL[t * K1 + K] = INT64_MIN;
    }
    for (int c = tid; c < RK_CODES; c += SC_THREADS) lhist[c] = 0;
    __syncthreads();
    if constexpr (!kProject) {
        build_pm_sm<SC_THREADS>(lL, lPM, lSM, n, K, bb);
        __syncthreads();
    }

    // 1) this thread's candidate e = q n + t
    int64_t base = INT64_MAX;                         // smallest target peak
    for (int t = 0; t < n; ++t) {
        const int64_t v = lSM[t * K1];
        base = v < base ? v : base;
    }
    const int e = tid;
    const uint32_t ec = (uint32_t)(e < cand ? e : cand - 1);
    const int q = (int)fast_div(ec, (uint32_t)n, a.magic_n);
    const int t = (int)ec - q * n;
    const int r = row0 + q;
    const bool live = e < cand && r < a.N;
    const int s = r_s[q], ke = r_ke[q];
    const int64_t* pm_t = lPM + t * K1;
    const int64_t* sm_t = lSM + t * K1;
    const int64_t mv = move_score(pm_t, sm_t, lL[t * K1 + ke], ke, K, r_alpha[q], r_p[q]);
    const int64_t sc = s < 0 ? -1 : (t == s ? sm_t[0] : mv);
    const bool mig = live && s >= 0 && t != s;
    if (live && a.scores) a.scores[(int64_t)r * n + t] = sc;
    if (e < cand) {
        ks[e] = mig ? sc : kInfS;
        ki[e] = mig ? (uint32_t)((int64_t)r * n + t) : kInfI;
    }
    // code and rank of this key among the group's keys of equal code
    const uint32_t code = mig ? key_code((uint64_t)(sc - base)) : 0;
    const int lrank = mig ? atomicAdd(&lhist[code], 1) : 0;
    __syncthreads();

    // 2) best migration per request: smallest (score, t) over t != s
    for (int qq = tid; qq < rpb; qq += SC_THREADS) {
        const int rr = row0 + qq;
        if (rr >= a.N) continue;
        int64_t bs = kInfS;
        uint32_t bi = kInfI;
        for (int tt = 0; tt < n; ++tt) {
            const int ee = qq * n + tt;
            if (key_less(ks[ee], ki[ee], bs, bi)) { bs = ks[ee]; bi = ki[ee]; }
        }
        const bool none = bi == kInfI;
        if (a.best_target) a.best_target[rr] = none ? -1 : (int32_t)(bi - (uint32_t)((int64_t)rr * n));
        if (a.best_score) a.best_score[rr] = none ? -1 : bs;
    }

    // 3) code histogram -> exclusive offsets (4 codes per thread), global counts
    constexpr int PER = RK_CODES / SC_THREADS;
    int c4[PER], own = 0;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        c4[u] = lhist[tid * PER + u];
        own += c4[u];
    }
    const int inc = wave_incl_add_i32(own);
    if (lane == 63) wtot[tid >> 6] = inc;
    __syncthreads();
    int before = inc - own;
    for (int w = 0; w < (tid >> 6); ++w) before += wtot[w];
    int32_t* go = rk.offs + (int64_t)g * (RK_CODES + 1);
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int c = tid * PER + u;
        go[c] = before;
        if (c4[u]) atomicAdd(&rk.ghist[c], (uint32_t)c4[u]);
        lhist[c] = before;                            // now the offset
        before += c4[u];
    }
    if (tid == SC_THREADS - 1) go[RK_CODES] = before;  // this group's migration count
    if (g == 0 && tid == 0) *rk.base = base;
    __syncthreads();
    if (mig) {
        const int64_t at = (int64_t)g * cand + lhist[code] + lrank;
        rk.keys_s[at] = sc;
        rk.keys_i[at] = (uint32_t)((int64_t)r * n + t);
    }
}


// ---------------------------------------------------------------------------
// small rounds: one workgroup scores and ranks
// ---------------------------------------------------------------------------
struct SmallArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* load;
    int64_t* scores;              // [N, n] or NULL
    int32_t* best_target;         // [N] or NULL
    int64_t* best_score;          // [N] or NULL
    int32_t* topk_req;            // [top_k] (top_k > 0)
    int32_t* topk_tgt;
    int64_t* topk_score;
    int32_t* err_word;
    int N, n, b, K, top_k;
    uint32_t magic_n, magic_K;
};

// Dynamic LDS: [L | PM | SM] (n (K+1) int64 each), then per request
// {alpha, p} (2 x int64), best (uint64) and {ke, s} (2 x int32).
constexpr size_t SS_STATIC_LDS = sizeof(SelShared<SS_THREADS>) + STAR_MAX_TOP_K * (8 + 4 + 8);
static size_t small_lds_bytes(int N, int n, int K) {
    const size_t E = ((size_t)n * (K + 1) + 1) & ~(size_t)1;   // even: keeps {alpha, p} 16-B aligned
    return 3 * E * 8 + (size_t)N * (16 + 8 + 8);
}

// One workgroup of 8 waves (two per SIMD): up to 256 VGPRs per lane, so the
// candidate slots' LDS round trips can all be in flight.
__global__ __launch_bounds__(SS_THREADS) __attribute__((amdgpu_waves_per_eu(1, 2)))
void score_small_kernel(SmallArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ SelShared<SS_THREADS> sh;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    __shared__ uint64_t sv[STAR_MAX_TOP_K];
    const int tid = threadIdx.x, lane = tid & 63;
    const int N = a.N, n = a.n, b = a.b, K = a.K, K1 = K + 1, E = (n * K1 + 1) & ~1;
    int64_t* lL = (int64_t*)smem;
    int64_t* lPM = lL + E;
    int64_t* lSM = lPM + E;
    longlong2* r_ap = (longlong2*)(lSM + E);           // {alpha, p}; E * 3 * 8 keeps 16-B alignment
    uint64_t* r_best = (uint64_t*)(r_ap + N);
    int2* r_ks = (int2*)(r_best + N);                   // {ke, s}
    const int64_t H = (int64_t)b * K;
    const int64_t bb = (int64_t)b * b;

    // 0) curves and requests: every read issued before the first is used
    const int nK = n * K;
    int64_t lv[SS_LBATCH];
#pragma unroll
    for (int j = 0; j < SS_LBATCH; ++j) {
        const int e = j * SS_THREADS + tid;
        lv[j] = a.load[e < nK ? e : nK - 1];
    }
    int sv_[SS_RBATCH], cv[SS_RBATCH], rv[SS_RBATCH];
#pragma unroll
    for (int j = 0; j < SS_RBATCH; ++j) {
        const int r = j * SS_THREADS + tid;
        const int rc = r < N ? r : N - 1;
        sv_[j] = a.inst[rc];
        cv[j] = a.cur[rc];
        rv[j] = a.rem[rc];
    }
    int32_t bad = 0;
#pragma unroll
    for (int j = 0; j < SS_RBATCH; ++j) {
        const int r = j * SS_THREADS + tid;
        if (r < N) {
            const ReqTerms rt = request_terms(sv_[j], cv[j], rv[j], n, b, H);
            bad |= rt.bad;
            r_ks[r] = make_int2(rt.ke, rt.s);
            r_ap[r] = make_longlong2(rt.alpha, rt.p);
            r_best[r] = ~0ull;
        }
    }
    bad = wave_or_i32(bad);
    if (lane == 0) report_error(a.err_word, bad);
#pragma unroll
    for (int j = 0; j < SS_LBATCH; ++j) {
        const int e = j * SS_THREADS + tid;
        if (e < nK) {
            const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
            lL[t * K1 + (e - t * K)] = lv[j];
        }
    }
    for (int t = tid; t < n; t += SS_THREADS) lL[t * K1 + K] = INT64_MIN;
    __syncthreads();

    // 1) PM/SM
    build_pm_sm<SS_THREADS>(lL, lPM, lSM, n, K, bb);
    __syncthreads();

    // 2) every candidate e = r n + t: score (written out), migration key in
    //    registers.  All slots are computed (clamped index) and masked.
    //    Slots go eight at a time, their LDS reads issued in two batches
    //    (request terms, then the three curve gathers); stores come after.
    const int M = N * n;
    RegKeys<SS_RJ> keys;
    int64_t scv[SS_RJ];
    constexpr int SB = 8;
#pragma unroll
    for (int h = 0; h < SS_RJ; h += SB) {
        int tt[SB];
        int2 ks[SB];
        longlong2 ap[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int e = (h + u) * SS_THREADS + tid;
            const uint32_t ec = (uint32_t)(e < M ? e : M - 1);
            const int r = (int)fast_div(ec, (uint32_t)n, a.magic_n);
            tt[u] = (int)ec - r * n;
            ks[u] = r_ks[r];
            ap[u] = r_ap[r];
        }
        int64_t g0[SB], g1[SB], g2[SB], g3[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int base = tt[u] * K1, ke = ks[u].x;
            g0[u] = lPM[base + ke];
            g1[u] = lL[base + ke];                                  // entry K is -inf
            g2[u] = lSM[base + (ke + 1 < K ? ke + 1 : K)];
            g3[u] = lSM[base];
        }
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int e = (h + u) * SS_THREADS + tid;
            const int s = ks[u].y, t = tt[u];
            const int64_t mv = imax(imax(g0[u] + ap[u].x, g1[u] + ap[u].y), g2[u]);
            scv[h + u] = s < 0 ? -1 : (t == s ? g3[u] : mv);
            const bool mig = e < M && s >= 0 && t != s;
            keys.s[h + u] = mig ? scv[h + u] : kInfS;
            keys.i[h + u] = mig ? (uint32_t)e : kInfI;
        }
    }
    if (a.scores) {
#pragma unroll
        for (int j = 0; j < SS_RJ; ++j) {
            const int e = j * SS_THREADS + tid;
            if (e < M) a.scores[e] = scv[j];
        }
    }

    // 3) best move per request, as the minimum of ((score - smin) << tbits) | t
    //    when that fits 64 bits: over the request's group of n lanes when n
    //    divides 64 (candidates e = r n + t are consecutive lanes), else by
    //    LDS atomic min; wider keys take the minimum of (score - smin) and then
    //    of t among the moves that reach it.
    int total;
    int64_t smin, smax;
    source_stats<SS_THREADS>(keys, sh, &total, &smin, &smax);
    const int tbits = bit_length((uint64_t)(n - 1));
    const uint64_t tmask = (1ull << tbits) - 1;
    const bool packed = total > 0 && bit_length((uint64_t)(smax - smin)) + tbits <= 64;
    const bool grouped = packed && (64 % n) == 0;
    if (grouped) {
#pragma unroll
        for (int j = 0; j < SS_RJ; ++j) {
            const int e = j * SS_THREADS + tid;
            const uint32_t r = fast_div((uint32_t)e, (uint32_t)n, a.magic_n);
            const uint64_t v = keys.s[j] == kInfS
                                   ? ~0ull
                                   : ((uint64_t)(keys.s[j] - smin) << tbits) | ((uint32_t)e - r * n);
            const uint64_t g = group_min_u64(v, n);
            if (e < M && (lane & (n - 1)) == 0) r_best[r] = g;
        }
    } else if (total > 0) {
        keys.visit([&](int64_t s, uint32_t i) {
            if (s == kInfS) return;
            const uint32_t r = fast_div(i, (uint32_t)n, a.magic_n);
            const uint64_t d = (uint64_t)(s - smin);
            atomicMin((unsigned long long*)&r_best[r],
                      (unsigned long long)(packed ? (d << tbits) | (i - r * (uint32_t)n) : d));
        });
        if (!packed) {
            for (int r = tid; r < N; r += SS_THREADS) r_ks[r].x = -1;  // min target, as unsigned
            __syncthreads();
            keys.visit([&](int64_t s, uint32_t i) {
                if (s == kInfS) return;
                const uint32_t r = fast_div(i, (uint32_t)n, a.magic_n);
                if ((uint64_t)(s - smin) == r_best[r])
                    atomicMin((unsigned int*)&r_ks[r].x, i - r * (uint32_t)n);
            });
        }
    }
    __syncthreads();
    for (int r = tid; r < N; r += SS_THREADS) {
        const uint64_t v = r_best[r];
        const bool none = v == ~0ull;
        const int64_t bs = none ? -1 : smin + (int64_t)(packed ? v >> tbits : v);
        const int32_t bt = none ? -1 : (packed ? (int32_t)(v & tmask) : r_ks[r].x);
        if (a.best_target) a.best_target[r] = bt;
        if (a.best_score) a.best_score[r] = bs;
    }

    // 4) top-k
    if (a.top_k > 0) {
        const int ibits = bit_length((uint64_t)(M - 1));
        int64_t us;
        uint32_t ui;
        select_bound<SS_THREADS>(keys, a.top_k, ibits, total, smin, smax, sh, &us, &ui);
        const int nw = block_gather<SS_THREADS>(keys, us, ui, sh, ws_s, ws_i, STAR_MAX_TOP_K);
        order_and_write<SS_THREADS>(ws_s, ws_i, nw, smin, us < smax ? us : smax, ibits, n,
                                    a.magic_n, a.topk_req, a.topk_tgt, a.topk_score, a.top_k, sh,
                                    sv);
    }
}

// ---------------------------------------------------------------------------
// one workgroup scores and ranks a whole round (up to 1024 requests on up to
// 8 instances, curves in LDS)
// ---------------------------------------------------------------------------
// Thread r takes request r: it adds its terms to the LDS histograms by k_e
// (or the curves are read), the curves and PM/SM are built in LDS, and the
// thread scores its request against every target, keeping the migration
// keys in registers.  The top-k takes the code histogram of those keys and
// c*, the code of the k-th smallest; every key of code <= c* is compacted
// and counting-sorted, so the k smallest come out in key order (more than
// TK_SORT_CAP keys up to c* take the radix selection instead).  One kernel,
// no global round trip between scoring and ranking.
constexpr int SO_THREADS = TK_THREADS;
constexpr int SO_MAX_N = 8;                  // instances (keys per thread)
constexpr int SO_LB = (SC_FUSED_ENTRIES + SO_THREADS - 1) / SO_THREADS;  // curve reads per thread
constexpr size_t SO_STATIC_LDS =
    sizeof(SelShared<TK_THREADS>) + sizeof(SortLds) + STAR_MAX_TOP_K * (8 + 4 + 8);

struct OneArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    const int64_t* load;          // the curves, when not projecting
    int64_t* load_out;            // the curves built here, when projecting
    int64_t* scores;              // [N, n] or NULL
    int32_t* best_target;         // [N] or NULL
    int64_t* best_score;          // [N] or NULL
    int32_t* topk_req;            // [top_k] (top_k > 0)
    int32_t* topk_tgt;
    int64_t* topk_score;
    int32_t* err_word;
    int N, n, b, K, top_k, ibits;
    uint32_t magic_n, magic_K;
};

template <bool kProject>
__global__ __launch_bounds__(SO_THREADS) void score_one_kernel(OneArgs a) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ SelShared<TK_THREADS> sh;
    __shared__ SortLds sl;
    __shared__ int64_t ws_s[STAR_MAX_TOP_K];
    __shared__ uint32_t ws_i[STAR_MAX_TOP_K];
    __shared__ uint64_t sv[STAR_MAX_TOP_K];
    static_assert(RK_CODES == SO_THREADS, "one code per thread");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int N = a.N, n = a.n, K = a.K, b = a.b;
    const int K1 = K + 1, nK = n * K;
    const int64_t H = (int64_t)b * K;
    const int64_t bb = (int64_t)b * b;
    int64_t* lL = (int64_t*)smem;
    int64_t* lPM = lL + n * K1;
    int64_t* lSM = lPM + n * K1;

    // the top-k's code histogram and fill counters (one code per thread)
    sh.hist[tid] = 0;
    sh.fill[tid] = 0;
    // 0) this thread's request (and the curves when given); reads first
    const int r = tid;
    const bool live = r < N;
    const int rc = live ? r : N - 1;
    const int sr = a.inst[rc], cr = a.cur[rc], lr = a.rem[rc];
    int64_t lv[kProject ? 1 : SO_LB];
    if constexpr (!kProject) {
#pragma unroll
        for (int j = 0; j < SO_LB; ++j) {
            const int e = j * SO_THREADS + tid;
            lv[j] = a.load[e < nK ? e : nK - 1];
        }
    } else {
        for (int e = tid; e < 3 * n * K1; e += SO_THREADS) lL[e] = 0;
    }
    int32_t f = 0;
    if (sr < 0 || sr >= n) f |= STAR_DEV_BAD_INST;
    if (cr < 1) f |= STAR_DEV_BAD_CUR;
    if (lr < 1) f |= STAR_DEV_BAD_REM;
    const bool ok = live && f == 0;
    const uint32_t lp = (uint32_t)((int64_t)lr < H ? (int64_t)lr : H);
    const uint32_t kq = lp / (uint32_t)b;
    const int64_t mu = (int64_t)(lp - kq * (uint32_t)b);
    const int s = ok ? sr : -1;
    const int ke = ok ? (int)kq : 0;
    const int64_t alpha = (int64_t)b * cr + (int64_t)b * (b - 1) / 2;
    const int64_t pr = mu * cr + mu * (int64_t)kq * b + mu * (mu - 1) / 2;
    const int32_t bad = wave_or_i32(live ? f : 0);
    if (lane == 0) report_error(a.err_word, bad);
    __syncthreads();

    // 1) curves, PM, SM in LDS
    if constexpr (kProject) {
        // histograms by k_e: alpha in PM's rows, counts in SM's, partial
        // buckets in L's (build_curves_pm_sm reads them there)
        if (ok) {
            const int row = s * K1;
            if (ke > 0) {
                atomicAdd((unsigned long long*)&lPM[row + ke], (unsigned long long)alpha);
                atomicAdd((unsigned long long*)&lSM[row + ke], 1ull);
            }
            if (pr != 0) atomicAdd((unsigned long long*)&lL[row + ke], (unsigned long long)pr);
        }
        __syncthreads();
        if (K <= 64 * PMSM_REG_RUN)
            build_curves_pm_sm_wr<SO_THREADS, PMSM_REG_RUN>(lPM, lSM, lL, lPM, lSM, n, K, bb);
        else
            build_curves_pm_sm_w<SO_THREADS>(lPM, lSM, lL, lPM, lSM, n, K, bb);
        __syncthreads();
    } else {
#pragma unroll
        for (int j = 0; j < SO_LB; ++j) {
            const int e = j * SO_THREADS + tid;
            if (e < nK) {
                const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
                lL[t * K1 + (e - t * K)] = lv[j];
            }
        }
        for (int t = tid; t < n; t += SO_THREADS) lL[t * K1 + K] = INT64_MIN;
        __syncthreads();
        build_pm_sm<SO_THREADS>(lL, lPM, lSM, n, K, bb);
        __syncthreads();
    }

    // 2) scores of request r against every target; its best migration
    int64_t base = INT64_MAX;                     // smallest target peak
    for (int t = 0; t < n; ++t) base = imin64(base, lSM[t * K1]);
    // and the key code of each migration, counted in the top-k's histogram
    constexpr uint16_t kNone = 0xFFFF;
    int64_t sc[SO_MAX_N];
    uint16_t code[SO_MAX_N];
    int64_t bs = kInfS;
    int bt = -1;
#pragma unroll
    for (int t = 0; t < SO_MAX_N; ++t) {
        sc[t] = -1;
        code[t] = kNone;
        if (t < n) {
            const int64_t* pm_t = lPM + t * K1;
            const int64_t* sm_t = lSM + t * K1;
            const int64_t mv = move_score(pm_t, sm_t, lL[t * K1 + ke], ke, K, alpha, pr);
            sc[t] = s < 0 ? -1 : (t == s ? sm_t[0] : mv);
            const bool mig = s >= 0 && t != s;
            if (mig && sc[t] < bs) {              // t ascends: the first minimum stays
                bs = sc[t];
                bt = t;
            }
            if (mig && a.top_k > 0) {
                code[t] = (uint16_t)key_code((uint64_t)(sc[t] - base));
                atomicAdd(&sh.hist[code[t]], 1);
            }
        }
    }
    // the round's global writes, issued last.  Barriers do not wait for
    // stores here, but issuing these right after the scoring, under the
    // ranking's phases, measured slower (12.1-12.2 against 11.8 us a call)
    auto write_round = [&]() {
        if (live && a.scores) {
            int64_t* out = a.scores + (int64_t)r * n;
            if ((n & 1) == 0) {                   // 16-byte aligned pairs
#pragma unroll
                for (int t = 0; t < SO_MAX_N; t += 2)
                    if (t < n) *(longlong2*)(out + t) = make_longlong2(sc[t], sc[t + 1]);
            } else {
#pragma unroll
                for (int t = 0; t < SO_MAX_N; ++t)
                    if (t < n) out[t] = sc[t];
            }
        }
        if (live && a.best_target) a.best_target[r] = bt;
        if (live && a.best_score) a.best_score[r] = bt < 0 ? -1 : bs;
        if constexpr (kProject)
            for (int e = tid; e < nK; e += SO_THREADS) {
                const int t = (int)fast_div((uint32_t)e, (uint32_t)K, a.magic_K);
                a.load_out[e] = lL[t * K1 + (e - t * K)];
            }
    };
    if (a.top_k == 0) {
        write_round();
        return;
    }

    // 3) top-k over the migration keys (sc[t], r n + t), t != s
    __syncthreads();
    const int h = sh.hist[tid];
    int total;
    const int before = block_excl_i32<TK_THREADS>(h, sh, &total);
    const bool all = total <= a.top_k;
    if (all ? tid == RK_CODES - 1 : (before < a.top_k && before + h >= a.top_k)) {
        sh.bcast[0] = tid;                        // c*
        sh.bcast[1] = before + h;                 // keys of code <= c*
    }
    sh.hist[tid] = before;                        // code offsets
    __syncthreads();
    const uint32_t cstar = (uint32_t)sh.bcast[0];
    const int nle = sh.bcast[1];
    if (nle <= TK_SORT_CAP) {
        int cnt = 0;
#pragma unroll
        for (int t = 0; t < SO_MAX_N; ++t) cnt += code[t] <= cstar ? 1 : 0;
        int tot;
        int pos = block_excl_i32<TK_THREADS>(cnt, sh, &tot);
#pragma unroll
        for (int t = 0; t < SO_MAX_N; ++t) {
            if (code[t] <= cstar) {
                sl.cs[pos] = sc[t];
                sl.ci[pos] = (uint32_t)(r * n + t);
                sl.cc[pos] = code[t];
                ++pos;
            }
        }
        __syncthreads();
        int64_t ks = 0;
        uint32_t ki = 0;
        uint16_t kc = 0;
        if (tid < nle) {
            ks = sl.cs[tid];
            ki = sl.ci[tid];
            kc = sl.cc[tid];
        }
        const int kk = a.top_k < total ? a.top_k : total;
        const int p = sort_place(sh, sl, nle, ks, ki, kc);
        if (p >= 0 && p < kk) {
            const uint32_t rr = fast_div(ki, (uint32_t)n, a.magic_n);
            a.topk_req[p] = (int32_t)rr;
            a.topk_tgt[p] = (int32_t)(ki - rr * (uint32_t)n);
            a.topk_score[p] = ks;
        }
        for (int q = kk + tid; q < a.top_k; q += SO_THREADS) {
            a.topk_req[q] = -1;
            a.topk_tgt[q] = -1;
            a.topk_score[q] = -1;
        }
        write_round();
        return;
    }
    // a crowded code c*: radix selection over the registers
    RegKeys<SO_MAX_N> keys;
#pragma unroll
    for (int t = 0; t < SO_MAX_N; ++t) {
        const bool mig = code[t] != kNone;
        keys.s[t] = mig ? sc[t] : kInfS;
        keys.i[t] = mig ? (uint32_t)(r * n + t) : kInfI;
    }
    int64_t smin, smax_w;
    const int nw = select_top<TK_THREADS>(keys, a.top_k, a.ibits, sh, ws_s, ws_i, &smin, &smax_w);
    order_and_write<TK_THREADS>(ws_s, ws_i, nw, smin, smax_w, a.ibits, n, a.magic_n, a.topk_req,
                                a.topk_tgt, a.topk_score, a.top_k, sh, sv);
    write_round();
}

__global__ void fill_i32_kernel(int32_t* p, int count, int32_t v) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < count; i += gridDim.x * 256) p[i] = v;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
ScorePlan plan_score(const star_score_params& p, bool project) {
    ScorePlan pl;
    const int n = p.load.n_inst;
    const int N = p.load.n_req;
    const int K1 = p.load.n_buckets + 1;
    pl.fused = (int64_t)n * K1 <= SC_FUSED_ENTRIES;
    pl.small = pl.fused && N <= SS_MAX_REQ && (int64_t)N * n <= (int64_t)SS_RJ * SS_THREADS;
    pl.rpb = SC_CAND / n > 1 ? SC_CAND / n : 1;
    if (N > 0 && pl.rpb > N) pl.rpb = N;
    pl.cand = pl.rpb * n;
    pl.groups = N > 0 ? (int)ceil_div(N, pl.rpb) : 0;
    // top-k: select over all migrations when they fit one workgroup's
    // registers, else over the k requests with the smallest best keys first
    // register slots per thread: 8 when that holds every key, else 16
    const int64_t nmig = (int64_t)N * n, npr = (int64_t)p.top_k * (n - 1);
    pl.topk_direct = nmig <= TK_REG_KEYS;
    pl.topk_rj = nmig <= 8 * TK_THREADS ? 8 : TK_RJ;
    pl.topk_reg1 = N <= TK_REG_BEST;
    pl.topk_rj2 = npr <= 8 * TK_THREADS ? 8 : npr <= TK_REG_KEYS ? TK_RJ : 0;

    size_t off = STAR_WS_HEADER_BYTES;
    // fused scoring with the two-stage ranking: the scoring workgroups sort
    // their keys by code, one workgroup ranks
    // a whole round in one workgroup: up to 1024 requests on up to 8 instances
    pl.one = pl.fused && N > 0 && N <= SO_THREADS && n <= SO_MAX_N;
    if (pl.one) {
        pl.small = false;
        pl.project_in = project;
        pl.total = off;
        pl.lds = (size_t)3 * n * K1 * 8;
        return pl;
    }
    pl.rank2 = pl.fused && p.top_k > 0 && pl.groups <= RK_MAX_GROUPS && pl.cand <= SC_THREADS;
    if (pl.rank2) {
        pl.small = false;
        pl.project_in = project && N > 0 && N <= SC_PROJECT_MAX_REQ;
        static_assert(RK_CODES == 1024, "the header's histogram has 1024 codes");
        pl.ghist_off = kHdrScoreHist;             // in the header: zero between calls
        pl.base_off = off;
        off = align_up(off + 8, 256);
        pl.keys_s_off = off;
        off = align_up(off + (size_t)pl.groups * pl.cand * 8, 256);
        pl.keys_i_off = off;
        off = align_up(off + (size_t)pl.groups * pl.cand * 4, 256);
        pl.offs_off = off;
        off = align_up(off + (size_t)pl.groups * (RK_CODES + 1) * 4, 256);
        pl.total = off;
        pl.lds = (size_t)3 * n * K1 * 8 + (size_t)pl.cand * 12 + (size_t)pl.rpb * 24;
        return pl;
    }
    if (pl.small) {
        pl.total = off;
        pl.lds = small_lds_bytes(N, n, p.load.n_buckets);
        return pl;
    }
    while (N > 0 && pl.cand * 2 <= SC_CAND_MAX && ceil_div(N, pl.rpb * 2) >= SC_MIN_GROUPS) {
        pl.rpb *= 2;
        pl.cand = pl.rpb * n;
        pl.groups = (int)ceil_div(N, pl.rpb);
    }
    if (!pl.fused) {                              // planes and peaks
        // bucket-major when requests outnumber buckets (the scoring gathers
        // dominate), else instance-major (the preparation's writes do)
        pl.by_bucket = N >= p.load.n_buckets;
        const size_t plane = align_up((size_t)n * K1 * 8, 256);
        pl.tpm_off = off;
        pl.tl_off = off + plane;
        pl.tsm_off = off + 2 * plane;
        pl.peak_off = off + 3 * plane;
        off = align_up(pl.peak_off + (size_t)n * 8, 256);
        pl.lg = 0;
        while ((1 << pl.lg) < n && (1 << pl.lg) < SP_ROW) ++pl.lg;
        const int tpl = planar_tpl(n);
        const int per_wg = (SP_THREADS / 64) * planar_req(tpl) * (64 >> pl.lg);
        pl.groups = N > 0 ? (int)ceil_div(N, per_wg) : 0;
    }
    pl.scores_off = off;                          // used when the caller passes no scores
    off = align_up(off + (size_t)N * n * 8, 256);
    pl.bscore_off = off;
    off = align_up(off + (size_t)N * 8, 256);
    pl.btarget_off = off;
    off = align_up(off + (size_t)N * 4, 256);
    pl.topk_pruned = p.top_k > 0 && n > 1 && !pl.topk_direct;
    pl.topk_hist = pl.topk_pruned && !pl.topk_reg1;
    if (pl.topk_pruned) {
        pl.base_off = off;
        off = align_up(off + 8, 256);
    }
    if (pl.topk_hist) {
        pl.bcode_off = off;
        off = align_up(off + (size_t)N * 2, 256);
        pl.gs_off = off;
        off = align_up(off + (size_t)TK_REG_BEST * 8, 256);
        pl.gi_off = off;
        off = align_up(off + (size_t)TK_REG_BEST * 4, 256);
    }
    pl.total = off;
    pl.lds = pl.fused ? (size_t)3 * n * K1 * 8 + (size_t)pl.cand * 12 + (size_t)pl.rpb * 24 : 0;
    return pl;
}

// Dynamic LDS beyond the default needs the kernel's limit raised (static +
// dynamic stays within the 160 KB of a gfx950 CU).
static hipError_t set_lds(const void* fn, size_t lds, size_t static_lds) {
    if (lds + static_lds <= 64 * 1024) return hipSuccess;
    return hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

static hipError_t launch_score_kernel(const ScorePlan& pl, const ScoreArgs& a, hipStream_t stream) {
    hipError_t e = set_lds((const void*)score_kernel, pl.lds, 64);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_kernel, dim3(pl.groups), dim3(SC_THREADS), pl.lds, stream, a);
    return hipGetLastError();
}

static hipError_t fill_i32(int32_t* p, int count, int32_t v, hipStream_t stream) {
    hipLaunchKernelGGL(fill_i32_kernel, dim3((count + 255) / 256), dim3(256), 0, stream, p, count, v);
    return hipGetLastError();
}

template <int S1, int RJ2>
static hipError_t launch_topk_pruned1(const TopkArgs& a, hipStream_t stream) {
    hipLaunchKernelGGL((topk_pruned_kernel<S1, RJ2>), dim3(1), dim3(TK_THREADS), 0, stream, a);
    return hipGetLastError();
}

template <int S1>
static hipError_t launch_topk_pruned(const TopkArgs& a, int rj2, hipStream_t stream) {
    return rj2 == 8 ? launch_topk_pruned1<S1, 8>(a, stream)
         : rj2 == TK_RJ ? launch_topk_pruned1<S1, TK_RJ>(a, stream)
                        : launch_topk_pruned1<S1, 0>(a, stream);
}

CurvePlanes score_planes(const star_score_params& p, const ScorePlan& pl, char* ws) {
    CurvePlanes c;
    if (pl.fused) return c;
    c.tpm = (int64_t*)(ws + pl.tpm_off);
    c.tl = (int64_t*)(ws + pl.tl_off);
    c.tsm = (int64_t*)(ws + pl.tsm_off);
    c.peak = (int64_t*)(ws + pl.peak_off);
    c.sk = pl.by_bucket ? p.load.n_inst : 1;
    c.st = pl.by_bucket ? 1 : p.load.n_buckets + 1;
    return c;
}

hipError_t launch_score(const star_score_params& p, const ScorePlan& pl, const int32_t* cur,
                        const int32_t* rem, const int32_t* inst, const int64_t* load,
                        int64_t* scores, int32_t* best_target, int64_t* best_score,
                        int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score, char* ws,
                        int32_t* err_word, hipStream_t stream, int64_t* load_out,
                        bool planes_ready) {
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
    if (pl.one) {
        OneArgs o = {};
        o.cur = cur; o.rem = rem; o.inst = inst; o.load = load; o.load_out = load_out;
        o.scores = scores; o.best_target = best_target; o.best_score = best_score;
        o.topk_req = topk_req; o.topk_tgt = topk_tgt; o.topk_score = topk_score;
        o.err_word = err_word;
        o.N = lp.n_req; o.n = lp.n_inst; o.b = lp.bucket; o.K = lp.n_buckets; o.top_k = p.top_k;
        o.ibits = 0;
        for (int64_t x = (int64_t)lp.n_req * lp.n_inst - 1; x > 0; x >>= 1) ++o.ibits;
        o.magic_n = div_magic((uint32_t)lp.n_inst);
        o.magic_K = div_magic((uint32_t)lp.n_buckets);
        const void* kern = load_out ? (const void*)score_one_kernel<true>
                                    : (const void*)score_one_kernel<false>;
        hipError_t e = set_lds(kern, pl.lds, SO_STATIC_LDS);
        if (e != hipSuccess) return e;
        if (load_out)
            hipLaunchKernelGGL(score_one_kernel<true>, dim3(1), dim3(SO_THREADS), pl.lds, stream, o);
        else
            hipLaunchKernelGGL(score_one_kernel<false>, dim3(1), dim3(SO_THREADS), pl.lds, stream, o);
        return hipGetLastError();
    }
    if (pl.rank2) {
        ScoreArgs a = {};
        a.cur = cur; a.rem = rem; a.inst = inst; a.load = load;
        a.scores = scores; a.best_target = best_target; a.best_score = best_score;
        a.err_word = err_word;
        a.N = lp.n_req; a.n = lp.n_inst; a.b = lp.bucket; a.K = lp.n_buckets;
        a.rpb = pl.rpb; a.cand = pl.cand;
        a.magic_K = div_magic((uint32_t)lp.n_buckets);
        a.magic_n = div_magic((uint32_t)lp.n_inst);
        RankArgs rk;
        rk.ghist = (uint32_t*)(ws + pl.ghist_off);
        rk.base = (int64_t*)(ws + pl.base_off);
        rk.keys_s = (int64_t*)(ws + pl.keys_s_off);
        rk.keys_i = (uint32_t*)(ws + pl.keys_i_off);
        rk.offs = (int32_t*)(ws + pl.offs_off);
        a.load_out = load_out;
        using Kern = void (*)(ScoreArgs, RankArgs);
        const Kern kern = pl.project_in ? score_rank_kernel<true> : score_rank_kernel<false>;
        hipError_t e = set_lds((const void*)kern, pl.lds, RK_CODES * 4 + 64);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(kern, dim3(pl.groups), dim3(SC_THREADS), pl.lds, stream, a, rk);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        FinalArgs f = {};
        f.ghist = rk.ghist;
        f.offs = rk.offs;
        f.keys_s = rk.keys_s;
        f.keys_i = rk.keys_i;
        f.topk_req = topk_req; f.topk_tgt = topk_tgt; f.topk_score = topk_score;
        f.groups = pl.groups; f.cand = pl.cand; f.n = lp.n_inst; f.top_k = p.top_k;
        f.ibits = 0;
        for (int64_t x = (int64_t)lp.n_req * lp.n_inst - 1; x > 0; x >>= 1) ++f.ibits;
        f.magic_n = div_magic((uint32_t)lp.n_inst);
        hipLaunchKernelGGL(rank_final_kernel, dim3(1), dim3(RK_THREADS), 0, stream, f);
        return hipGetLastError();
    }
    if (pl.small) {
        SmallArgs s = {};
        s.cur = cur; s.rem = rem; s.inst = inst; s.load = load;
        s.scores = scores; s.best_target = best_target; s.best_score = best_score;
        s.topk_req = topk_req; s.topk_tgt = topk_tgt; s.topk_score = topk_score;
        s.err_word = err_word;
        s.N = lp.n_req; s.n = lp.n_inst; s.b = lp.bucket; s.K = lp.n_buckets; s.top_k = p.top_k;
        s.magic_n = div_magic((uint32_t)lp.n_inst);
        s.magic_K = div_magic((uint32_t)lp.n_buckets);
        hipError_t e = set_lds((const void*)score_small_kernel, pl.lds, SS_STATIC_LDS);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(score_small_kernel, dim3(1), dim3(SS_THREADS), pl.lds, stream, s);
        return hipGetLastError();
    }
    const bool need_all = p.top_k > 0;           // the top-k kernel reads scores and best moves
    ScoreArgs a = {};
    a.cur = cur; a.rem = rem; a.inst = inst; a.load = load;
    a.scores = scores ? scores : (need_all ? (int64_t*)(ws + pl.scores_off) : nullptr);
    a.best_target = best_target ? best_target : (need_all ? (int32_t*)(ws + pl.btarget_off) : nullptr);
    a.best_score = best_score ? best_score : (need_all ? (int64_t*)(ws + pl.bscore_off) : nullptr);
    a.err_word = err_word;
    a.N = lp.n_req; a.n = lp.n_inst; a.b = lp.bucket; a.K = lp.n_buckets;
    a.rpb = pl.rpb; a.cand = pl.cand;
    a.magic_K = div_magic((uint32_t)lp.n_buckets);
    a.magic_n = div_magic((uint32_t)lp.n_inst);
    if (pl.topk_pruned) a.bbase = (int64_t*)(ws + pl.base_off);
    if (pl.topk_hist) a.bcode = (uint16_t*)(ws + pl.bcode_off);
    hipError_t e;
    if (pl.fused) {
        e = launch_score_kernel(pl, a, stream);
    } else {
        const CurvePlanes cp = score_planes(p, pl, ws);
        PlanarArgs q = {};
        q.cur = cur; q.rem = rem; q.inst = inst;
        q.tpm = cp.tpm; q.tl = cp.tl; q.tsm = cp.tsm; q.peak = cp.peak;
        q.sk = cp.sk; q.st = cp.st;
        q.scores = a.scores; q.best_target = a.best_target; q.best_score = a.best_score;
        q.err_word = err_word; q.bbase = a.bbase; q.bcode = a.bcode;
        q.N = lp.n_req; q.n = lp.n_inst; q.b = lp.bucket; q.K = lp.n_buckets; q.lg = pl.lg;
        e = hipSuccess;
        if (!planes_ready) {
            hipLaunchKernelGGL(score_prep_kernel, dim3(lp.n_inst), dim3(PREP_THREADS), 0, stream,
                               load, lp.n_buckets, lp.bucket, cp.sk, cp.st, cp.tpm, cp.tl, cp.tsm,
                               cp.peak);
            e = hipGetLastError();
        }
        if (e == hipSuccess && pl.groups > 0) e = launch_planar(q, pl.groups, planar_tpl(lp.n_inst), stream);
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
    t.magic_n = div_magic((uint32_t)lp.n_inst);
    t.magic_n1 = div_magic((uint32_t)lp.n_inst - 1);
    if (pl.topk_direct) {
        if (pl.topk_rj == 8)
            hipLaunchKernelGGL(topk_direct_kernel<8>, dim3(1), dim3(TK_THREADS), 0, stream, t);
        else
            hipLaunchKernelGGL(topk_direct_kernel<TK_RJ>, dim3(1), dim3(TK_THREADS), 0, stream, t);
        return hipGetLastError();
    }
    t.bbase = a.bbase;
    t.bcode = a.bcode;
    if (pl.topk_reg1) return launch_topk_pruned<kStage1Reg>(t, pl.topk_rj2, stream);
    t.gs = (int64_t*)(ws + pl.gs_off);
    t.gi = (uint32_t*)(ws + pl.gi_off);
    return launch_topk_pruned<kStage1Code>(t, pl.topk_rj2, stream);
}

}  // namespace star
