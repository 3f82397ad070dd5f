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
// complexity analysis in Section 4.2 taken to O(1) per candidate.
//
// Kernels: prep (PM/SM per instance), score (per workgroup: a block of
// requests x all targets; scores, best target, locally sorted top-k list by
// bitonic sort in LDS), merge (one workgroup merges the local lists by
// bitonic merge-and-truncate).  Keys are (score, r*n + t), a total order.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

constexpr int PREP_THREADS = 512;
constexpr int PREP_SEG = 4;
constexpr int SC_THREADS = 256;
constexpr int SC_TARGET_SORT = 512;
constexpr int MG_THREADS = 1024;
constexpr int MG_KEYS = 8192;          // keys held in LDS by the merge kernel

constexpr int64_t kInfS = INT64_MAX;
constexpr uint32_t kInfI = 0xFFFFFFFFu;

__device__ inline int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }

__device__ inline bool key_less(int64_t s0, uint32_t i0, int64_t s1, uint32_t i1) {
    return s0 < s1 || (s0 == s1 && i0 < i1);
}

// ---------------------------------------------------------------------------
// prep: PM_t[0..K] (PM_t[0] unused) and SM_t[0..K] (SM_t[K] unused)
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

    // exclusive prefix max of L[j] + b^2 j
    int64_t carry = INT64_MIN;
    for (int base = 0; base < K; base += CH) {
        const int j0 = base + tid * PREP_SEG;
        int64_t loc = INT64_MIN;
        for (int j = j0; j < j0 + PREP_SEG && j < K; ++j) loc = imax(loc, L[j] + bb * j);
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64(loc, OpMax(), INT64_MIN, tmp, &tot);
        int64_t run = imax(carry, ex);
        for (int j = j0; j < j0 + PREP_SEG && j < K; ++j) {
            pm[j] = run;
            run = imax(run, L[j] + bb * j);
        }
        carry = imax(carry, tot);
    }
    if (tid == 0) pm[K] = carry;

    // inclusive suffix max of L[j]
    carry = INT64_MIN;
    for (int base = 0; base < K; base += CH) {
        // reversed position p = base + tid*SEG + u  <->  j = K - 1 - p
        const int p0 = base + tid * PREP_SEG;
        int64_t loc = INT64_MIN;
        for (int p = p0; p < p0 + PREP_SEG && p < K; ++p) loc = imax(loc, L[K - 1 - p]);
        int64_t tot;
        int64_t ex = block_exclusive_scan_i64(loc, OpMax(), INT64_MIN, tmp, &tot);
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
// LDS bitonic sort (ascending) of n2 keys, n2 a power of two
// ---------------------------------------------------------------------------
__device__ inline void cmp_swap(int64_t* ks, uint32_t* ki, int lo, int hi, bool asc) {
    const int64_t s0 = ks[lo], s1 = ks[hi];
    const uint32_t i0 = ki[lo], i1 = ki[hi];
    if (key_less(s1, i1, s0, i0) == asc) {
        ks[lo] = s1; ks[hi] = s0;
        ki[lo] = i1; ki[hi] = i0;
    }
}

__device__ inline void bitonic_sort_lds(int64_t* ks, uint32_t* ki, int n2) {
    for (int size = 2; size <= n2; size <<= 1)
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int e = threadIdx.x; e < (n2 >> 1); e += blockDim.x) {
                const int lo = 2 * stride * (e / stride) + (e % stride);
                cmp_swap(ks, ki, lo, lo + stride, (lo & size) == 0);
            }
            __syncthreads();
        }
}

// ---------------------------------------------------------------------------
// score
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(SC_THREADS) void score_kernel(
    const int32_t* __restrict__ cur, const int32_t* __restrict__ rem,
    const int32_t* __restrict__ inst, const int64_t* __restrict__ load,
    const int64_t* __restrict__ PM, const int64_t* __restrict__ SM, int N, int n, int b, int K,
    int rpb, int sort_n, int kp, int64_t* __restrict__ scores, int32_t* __restrict__ best_target,
    int64_t* __restrict__ best_score, int64_t* __restrict__ list_s, uint32_t* __restrict__ list_i,
    int32_t* __restrict__ err_word) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    int64_t* ks = (int64_t*)smem;                        // [sort_n]
    uint32_t* ki = (uint32_t*)(ks + sort_n);             // [sort_n]
    int64_t* r_alpha = (int64_t*)(ki + sort_n + (sort_n & 1));   // [rpb]
    int64_t* r_p = r_alpha + rpb;                        // [rpb]
    int32_t* r_ke = (int32_t*)(r_p + rpb);               // [rpb]
    int32_t* r_s = r_ke + rpb;                           // [rpb]; -1 = invalid

    const int tid = threadIdx.x;
    const int row0 = blockIdx.x * rpb;
    const int64_t H = (int64_t)b * K;
    const int64_t bb2 = (int64_t)b * (b - 1) / 2;

    int32_t bad = 0;
    for (int q = tid; q < rpb; q += SC_THREADS) {
        const int r = row0 + q;
        int s = -1;
        if (r < N) {
            s = inst[r];
            const int cr = cur[r];
            const int lr = rem[r];
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
    bad = wave_or_i32(bad);
    if ((tid & 63) == 0) report_error(err_word, bad);
    __syncthreads();

    const int ncand = rpb * n;
    for (int e = tid; e < sort_n; e += SC_THREADS) {
        int64_t key_s = kInfS;
        uint32_t key_i = kInfI;
        if (e < ncand) {
            const int q = e / n, t = e - q * n;
            const int r = row0 + q;
            if (r < N) {
                const int s = r_s[q];
                int64_t sc = -1;
                if (s >= 0) {
                    const int64_t* Lt = load + (int64_t)t * K;
                    const int64_t* sm = SM + (int64_t)t * (K + 1);
                    if (t == s) {
                        sc = sm[0];
                    } else {
                        const int ke = r_ke[q];
                        sc = INT64_MIN;
                        if (ke >= 1) sc = imax(sc, PM[(int64_t)t * (K + 1) + ke] + r_alpha[q]);
                        if (ke < K) sc = imax(sc, Lt[ke] + r_p[q]);
                        if (ke + 1 < K) sc = imax(sc, sm[ke + 1]);
                        key_s = sc;
                        key_i = (uint32_t)((int64_t)r * n + t);
                    }
                }
                if (scores) scores[(int64_t)r * n + t] = sc;
            }
        }
        ks[e] = key_s;
        ki[e] = key_i;
    }
    __syncthreads();

    // best migration per request: smallest (score, t) over t != s
    if (best_target || best_score) {
        for (int q = tid; q < rpb; q += SC_THREADS) {
            const int r = row0 + q;
            if (r >= N) continue;
            int64_t bs = kInfS;
            uint32_t bi = kInfI;
            for (int t = 0; t < n; ++t) {
                const int e = q * n + t;
                if (key_less(ks[e], ki[e], bs, bi)) { bs = ks[e]; bi = ki[e]; }
            }
            const bool none = bi == kInfI;
            if (best_target) best_target[r] = none ? -1 : (int32_t)(bi - (uint32_t)((int64_t)r * n));
            if (best_score) best_score[r] = none ? -1 : bs;
        }
    }
    if (kp == 0) return;
    __syncthreads();

    bitonic_sort_lds(ks, ki, sort_n);
    int64_t* ls = list_s + (int64_t)blockIdx.x * kp;
    uint32_t* li = list_i + (int64_t)blockIdx.x * kp;
    for (int e = tid; e < kp; e += SC_THREADS) {
        ls[e] = ks[e];
        li[e] = ki[e];
    }
}

// ---------------------------------------------------------------------------
// merge: G sorted lists of kp keys -> the kp smallest, sorted
// ---------------------------------------------------------------------------
// a <- the kp smallest of sorted lists a and b, sorted (a, b in LDS).
__device__ inline void merge_truncate_pairs(int64_t* ks, uint32_t* ki, int kp, int n_pairs,
                                            int pair_stride_lists) {
    // step 1: a[i] = min(a[i], b[kp-1-i])  -- a bitonic sequence of the kp smallest
    for (int e = threadIdx.x; e < n_pairs * kp; e += blockDim.x) {
        const int pr = e / kp, i = e - pr * kp;
        const int a = pr * 2 * pair_stride_lists * kp;
        const int bo = a + pair_stride_lists * kp;
        const int j = bo + kp - 1 - i;
        if (key_less(ks[j], ki[j], ks[a + i], ki[a + i])) {
            ks[a + i] = ks[j];
            ki[a + i] = ki[j];
        }
    }
    __syncthreads();
    // step 2: bitonic merge of each a
    for (int stride = kp >> 1; stride > 0; stride >>= 1) {
        for (int e = threadIdx.x; e < n_pairs * (kp >> 1); e += blockDim.x) {
            const int pr = e / (kp >> 1), w = e - pr * (kp >> 1);
            const int a = pr * 2 * pair_stride_lists * kp;
            const int lo = 2 * stride * (w / stride) + (w % stride);
            cmp_swap(ks + a, ki + a, lo, lo + stride, true);
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(MG_THREADS) void merge_kernel(
    const int64_t* __restrict__ list_s, const uint32_t* __restrict__ list_i, int groups, int kp,
    int top_k, int n, int32_t* __restrict__ topk_req, int32_t* __restrict__ topk_tgt,
    int64_t* __restrict__ topk_score) {
    __shared__ int64_t ks[MG_KEYS];
    __shared__ uint32_t ki[MG_KEYS];
    // slot 0 holds the running result; slots 1.. hold a batch of lists
    const int slots = MG_KEYS / kp;              // power of two >= 2
    const int batch = slots / 2;                 // lists per batch (slots batch..2*batch-1 unused pad)
    for (int e = threadIdx.x; e < kp; e += MG_THREADS) {
        ks[e] = kInfS;
        ki[e] = kInfI;
    }
    for (int g0 = 0; g0 < groups; g0 += batch) {
        const int nl = groups - g0 < batch ? groups - g0 : batch;
        // load lists into slots batch .. batch + batch - 1 (pad with +inf)
        for (int e = threadIdx.x; e < batch * kp; e += MG_THREADS) {
            const int l = e / kp, i = e - l * kp;
            const int dst = (batch + l) * kp + i;
            if (l < nl) {
                ks[dst] = list_s[(int64_t)(g0 + l) * kp + i];
                ki[dst] = list_i[(int64_t)(g0 + l) * kp + i];
            } else {
                ks[dst] = kInfS;
                ki[dst] = kInfI;
            }
        }
        __syncthreads();
        // tree over the batch
        for (int w = 1; w < batch; w <<= 1)
            merge_truncate_pairs(ks + batch * kp, ki + batch * kp, kp, batch / (2 * w), w);
        // fold into the running result in slot 0 (slot 'batch' is adjacent at distance batch)
        merge_truncate_pairs(ks, ki, kp, 1, batch);
    }
    for (int q = threadIdx.x; q < top_k; q += MG_THREADS) {
        const bool have = ki[q] != kInfI;
        topk_req[q] = have ? (int32_t)(ki[q] / (uint32_t)n) : -1;
        topk_tgt[q] = have ? (int32_t)(ki[q] % (uint32_t)n) : -1;
        topk_score[q] = have ? ks[q] : -1;
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
static int next_pow2(int x) {
    int p = 1;
    while (p < x) p <<= 1;
    return p;
}

ScorePlan plan_score(const star_score_params& p) {
    ScorePlan pl;
    const int n = p.load.n_inst;
    pl.rpb = SC_TARGET_SORT / n > 1 ? SC_TARGET_SORT / n : 1;
    if (pl.rpb > p.load.n_req && p.load.n_req > 0) pl.rpb = p.load.n_req;
    if (pl.rpb < 1) pl.rpb = 1;
    pl.groups = p.load.n_req > 0 ? (int)ceil_div(p.load.n_req, pl.rpb) : 0;
    pl.kp = p.top_k > 0 ? next_pow2(p.top_k) : 0;
    int sn = next_pow2(pl.rpb * n);
    if (sn < pl.kp) sn = pl.kp;
    pl.sort_n = sn;
    const size_t K1 = (size_t)p.load.n_buckets + 1;
    size_t off = STAR_WS_HEADER_BYTES;
    pl.pm_off = off;
    off = align_up(off + (size_t)n * K1 * 8, 256);
    pl.sm_off = off;
    off = align_up(off + (size_t)n * K1 * 8, 256);
    pl.list_s_off = off;
    off = align_up(off + (size_t)pl.groups * pl.kp * 8, 256);
    pl.list_i_off = off;
    off = align_up(off + (size_t)pl.groups * pl.kp * 4, 256);
    pl.total = off;
    return pl;
}

size_t score_lds_bytes(const ScorePlan& pl) {
    return (size_t)pl.sort_n * 12 + 8 + (size_t)pl.rpb * 24;
}

hipError_t launch_score(const star_score_params& p, const ScorePlan& pl, const int32_t* cur,
                        const int32_t* rem, const int32_t* inst, const int64_t* load,
                        int64_t* scores, int32_t* best_target, int64_t* best_score,
                        int32_t* topk_req, int32_t* topk_tgt, int64_t* topk_score, char* ws,
                        int32_t* err_word, hipStream_t stream) {
    const star_load_params& lp = p.load;
    int64_t* PM = (int64_t*)(ws + pl.pm_off);
    int64_t* SM = (int64_t*)(ws + pl.sm_off);
    int64_t* ls = (int64_t*)(ws + pl.list_s_off);
    uint32_t* li = (uint32_t*)(ws + pl.list_i_off);
    hipLaunchKernelGGL(score_prep_kernel, dim3(lp.n_inst), dim3(PREP_THREADS), 0, stream, load,
                       lp.n_buckets, lp.bucket, PM, SM);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (lp.n_req == 0) {
        if (p.top_k > 0) {
            hipLaunchKernelGGL(merge_kernel, dim3(1), dim3(MG_THREADS), 0, stream, ls, li, 0,
                               pl.kp, p.top_k, lp.n_inst, topk_req, topk_tgt, topk_score);
            return hipGetLastError();
        }
        return hipSuccess;
    }
    const size_t lds = score_lds_bytes(pl);
    hipLaunchKernelGGL(score_kernel, dim3(pl.groups), dim3(SC_THREADS), lds, stream, cur, rem,
                       inst, load, PM, SM, lp.n_req, lp.n_inst, lp.bucket, lp.n_buckets, pl.rpb,
                       pl.sort_n, pl.kp, scores, best_target, best_score, ls, li, err_word);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (p.top_k > 0) {
        hipLaunchKernelGGL(merge_kernel, dim3(1), dim3(MG_THREADS), 0, stream, ls, li, pl.groups,
                           pl.kp, p.top_k, lp.n_inst, topk_req, topk_tgt, topk_score);
        e = hipGetLastError();
    }
    return e;
}

}  // namespace star
