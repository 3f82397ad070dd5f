// (b) Per-instance predicted load curves on gfx950.
//
// Section 5.2 (problem formulation, Eq. 4): request r with N(r) = c current
// tokens and N^(r) = l remaining steps holds c + t tokens at future step
// t < l.  Over a horizon of H = b K steps in buckets of b steps, with
// l' = min(l, H), k_e = l' div b and mu = l' mod b, r contributes
//     b c + b(b-1)/2 + b^2 k          to every full bucket k < k_e,
//     mu c + mu k_e b + mu(mu-1)/2    to the partial bucket k_e (mu > 0),
// i.e. sum_{t in bucket}(c + t).  So an instance's curve is
//     L[k] = S_A(k) + b^2 k S_n(k) + D_P[k],
// with S_A(k) / S_n(k) the sum of alpha_r = b c + b(b-1)/2 / the count over
// its requests with k_e > k (suffix sums of histograms indexed by k_e), and
// D_P the partial-bucket histogram.
//
// Long request streams (16-byte aligned arrays, K <= 1024): one workgroup
// per (instance, slice of the requests) scatters its instance's requests of
// its slice into LDS histograms by k_e and stores them; the last workgroup
// of an instance to finish sums the slices' histograms, runs the suffix scan
// and writes load[i, :].  So each request is read once per instance by a
// few hundred workgroups at once, instead of the whole stream by each of n.
//
// Otherwise one workgroup per (instance, bucket chunk): it streams every
// request (coalesced 16-byte reads of four requests for long streams from
// 16-byte aligned arrays, else int32 reads), scatters its own instance's
// requests into LDS histograms with int64 LDS atomics, runs a block-wide
// suffix scan and writes its chunk of load[i, :].  Requests whose k_e lies
// beyond the chunk are folded into one overflow slot, so chunks are
// independent.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

constexpr int PL_THREADS = 512;
constexpr int PL_CHUNK = 1024;
constexpr int PL_RBATCH = 4;      // loads per thread and array in flight together
// 16-byte reads from this many requests on (the longer kernel costs more
// than it saves on short streams: measured 4.4 -> 5.3 us at 64 requests and
// 4.7 -> 5.2 us at 4096; 15.6 -> 11.5 us at 32768)
constexpr int PL_VEC_MIN_REQ = 8192;

// kVec: requests read four at a time (16-byte loads; the arrays are 16-byte
// aligned), which issues a quarter of the load instructions -- the stream
// of every request through each workgroup is bound by instruction issue to
// the address units, not by bytes (measured at 32768 requests on 64
// instances: loads alone cost as much as the whole kernel).
template <bool kVec>
__global__ __launch_bounds__(PL_THREADS) void project_load_kernel(
    const int32_t* __restrict__ cur, const int32_t* __restrict__ rem,
    const int32_t* __restrict__ inst, int N, int n, int b, int K, int chunk,
    int64_t* __restrict__ load, int32_t* __restrict__ err_word) {
    __shared__ int64_t hA[PL_CHUNK + 1];   // alpha_r by k_e (slot len: k_e >= chunk end)
    __shared__ int64_t hN[PL_CHUNK + 1];   // request count by k_e
    __shared__ int64_t hP[PL_CHUNK];       // partial-bucket contributions
    __shared__ int64_t tmp[PL_THREADS / 64 + 1];

    const int tid = threadIdx.x;
    const int i = blockIdx.x;
    const int c = blockIdx.y;
    const int64_t k0 = (int64_t)c * chunk;
    const int64_t k1 = k0 + chunk < K ? k0 + chunk : K;
    const int len = (int)(k1 - k0);
    const int64_t H = (int64_t)b * K;
    const int64_t alpha0 = (int64_t)b * (b - 1) / 2;

    auto clear_lds = [&]() {
        for (int j = tid; j <= len; j += PL_THREADS) {
            hA[j] = 0;
            hN[j] = 0;
            if (j < len) hP[j] = 0;
        }
        __syncthreads();
    };
    int32_t bad = 0;
    // one request: error flags, then its own instance's histogram entries
    auto take = [&](int s, int cr, int lr) {
        int32_t f = 0;
        if (s < 0 || s >= n) f |= STAR_DEV_BAD_INST;
        if (cr < 1) f |= STAR_DEV_BAD_CUR;
        if (lr < 1) f |= STAR_DEV_BAD_REM;
        bad |= f;
        if (f || s != i) return;
        // l' < 2^31, 1 <= b < 2^31: 32-bit division is exact and cheap
        const uint32_t lp = (uint32_t)((int64_t)lr < H ? (int64_t)lr : H);
        const int64_t ke = (int64_t)(lp / (uint32_t)b);
        const int64_t mu = (int64_t)lp - ke * b;
        if (ke > k0) {
            const int jj = (int)((ke < k1 ? ke : k1) - k0);          // 1..len
            atomicAdd((unsigned long long*)&hA[jj], (unsigned long long)((int64_t)b * cr + alpha0));
            atomicAdd((unsigned long long*)&hN[jj], 1ull);
        }
        if (mu > 0 && ke >= k0 && ke < k1) {
            const int64_t pr = mu * cr + mu * ke * b + mu * (mu - 1) / 2;
            atomicAdd((unsigned long long*)&hP[ke - k0], (unsigned long long)pr);
        }
    };
    // Requests are read PL_RBATCH loads per thread at a time, all issued
    // before the first is used (indices clamped, so the loads are
    // unconditional); the first batch is in flight while LDS is cleared.
    if constexpr (kVec) {
        const int N4 = N >> 2;
        const int4* s4 = (const int4*)inst;
        const int4* c4 = (const int4*)cur;
        const int4* l4 = (const int4*)rem;
        if (N4 == 0) clear_lds();
        for (int base = 0; base < N4; base += PL_THREADS * PL_RBATCH) {
            int4 sv[PL_RBATCH], cv[PL_RBATCH], lv[PL_RBATCH];
#pragma unroll
            for (int j = 0; j < PL_RBATCH; ++j) {
                const int q = base + j * PL_THREADS + tid;
                const int qc = q < N4 ? q : N4 - 1;
                sv[j] = s4[qc];
                cv[j] = c4[qc];
                lv[j] = l4[qc];
            }
            if (base == 0) clear_lds();
#pragma unroll
            for (int j = 0; j < PL_RBATCH; ++j) {
                if (base + j * PL_THREADS + tid >= N4) continue;
                take(sv[j].x, cv[j].x, lv[j].x);
                take(sv[j].y, cv[j].y, lv[j].y);
                take(sv[j].z, cv[j].z, lv[j].z);
                take(sv[j].w, cv[j].w, lv[j].w);
            }
        }
        for (int r = 4 * N4 + tid; r < N; r += PL_THREADS) take(inst[r], cur[r], rem[r]);
    } else {
        if (N == 0) clear_lds();
        for (int base = 0; base < N; base += PL_THREADS * PL_RBATCH) {
            int sv[PL_RBATCH], cv[PL_RBATCH], lv[PL_RBATCH];
#pragma unroll
            for (int j = 0; j < PL_RBATCH; ++j) {
                const int r = base + j * PL_THREADS + tid;
                const int rc = r < N ? r : N - 1;
                sv[j] = inst[rc];
                cv[j] = cur[rc];
                lv[j] = rem[rc];
            }
            if (base == 0) clear_lds();
#pragma unroll
            for (int j = 0; j < PL_RBATCH; ++j) {
                if (base + j * PL_THREADS + tid >= N) continue;
                take(sv[j], cv[j], lv[j]);
            }
        }
    }
    if (i == 0 && c == 0) {
        bad = wave_or_i32(bad);
        if ((tid & 63) == 0) report_error(err_word, bad);
    }
    __syncthreads();

    // Suffix sums over x[q] = h[q + 1], q in [0, len): thread t owns the
    // reversed positions p in [t*seg, (t+1)*seg), q = len - 1 - p.
    const int seg = (len + PL_THREADS - 1) / PL_THREADS;
    const int p0 = tid * seg;
    const int p1 = p0 + seg < len ? p0 + seg : len;
    int64_t la = 0, ln = 0;
    for (int p = p0; p < p1; ++p) {
        const int q = len - 1 - p;
        la += hA[q + 1];
        ln += hN[q + 1];
    }
    int64_t ra = block_exclusive_scan_i64<PL_THREADS>(la, OpAdd(), 0, tmp, (int64_t*)nullptr);
    int64_t rn = block_exclusive_scan_i64<PL_THREADS>(ln, OpAdd(), 0, tmp, (int64_t*)nullptr);
    const int64_t bb = (int64_t)b * b;
    int64_t* out = load + (int64_t)i * K;
    for (int p = p0; p < p1; ++p) {
        const int q = len - 1 - p;
        ra += hA[q + 1];
        rn += hN[q + 1];
        const int64_t k = k0 + q;
        out[k] = ra + bb * k * rn + hP[q];
    }
}

// ---------------------------------------------------------------------------
// split projection
// ---------------------------------------------------------------------------
constexpr int PS_THREADS = 1024;     // one bucket per thread when the slices are summed
constexpr int PS_MAX_K = PS_THREADS;
constexpr int PS_MAX_SLICES = 8;
constexpr int PS_TARGET_GROUPS = 256;  // workgroups the slices aim for (one per CU)
constexpr int PS_MIN_SLICE = 1024;     // requests per slice at least
constexpr int PS_RV = 2;               // 16-byte reads per thread and array in flight
// request streams from which the split is used (at 4096 requests on 16
// instances it took 11.4 us against 4.6 + 4 us for the chunked kernel and
// the separate plane preparation: the meeting's latency dominates)
constexpr int PS_MIN_REQ = 8192;

struct SplitArgs {
    const int32_t* cur;
    const int32_t* rem;
    const int32_t* inst;
    int64_t* load;
    int32_t* err_word;
    int64_t* part;          // [n][slices][3][KP]: the slices' histograms (alpha, count, partial)
    uint32_t* tickets;      // [n] arrival counters (zero between calls)
    CurvePlanes planes;     // written too when planes.tpm is set
    int N, n, b, K, KP, slices, slice_len;
};

__global__ __launch_bounds__(PS_THREADS) void project_split_kernel(SplitArgs a) {
    __shared__ int64_t hA[PS_MAX_K + 2];   // alpha_r by k_e (1..K)
    __shared__ int64_t hN[PS_MAX_K + 2];   // request count by k_e (1..K)
    __shared__ int64_t hP[PS_MAX_K + 2];   // partial-bucket contributions by k_e (0..K-1)
    __shared__ int64_t tmp[2 * PS_THREADS / 64];
    __shared__ uint32_t s_ticket;
    const int tid = threadIdx.x;
    const int i = blockIdx.x, sl = blockIdx.y;
    const int K = a.K, b = a.b, KP = a.KP;
    const int64_t H = (int64_t)b * K;
    const int64_t alpha0 = (int64_t)b * (b - 1) / 2;
    const int r0 = sl * a.slice_len;
    const int r1 = r0 + a.slice_len < a.N ? r0 + a.slice_len : a.N;
    const int q0 = r0 >> 2, q1 = r1 >> 2;           // whole groups of four requests

    int32_t bad = 0;
    auto take = [&](int s, int cr, int lr) {
        int32_t f = 0;
        if (s < 0 || s >= a.n) f |= STAR_DEV_BAD_INST;
        if (cr < 1) f |= STAR_DEV_BAD_CUR;
        if (lr < 1) f |= STAR_DEV_BAD_REM;
        bad |= f;
        if (f || s != i) return;
        // l' < 2^31, 1 <= b < 2^31: 32-bit division is exact
        const uint32_t lp = (uint32_t)((int64_t)lr < H ? (int64_t)lr : H);
        const uint32_t ke = lp / (uint32_t)b;
        const int64_t mu = (int64_t)(lp - ke * (uint32_t)b);
        if (ke > 0) {
            atomicAdd((unsigned long long*)&hA[ke], (unsigned long long)((int64_t)b * cr + alpha0));
            atomicAdd((unsigned long long*)&hN[ke], 1ull);
        }
        if (mu > 0) {                                 // then k_e < K
            const int64_t pr = mu * cr + mu * (int64_t)ke * b + mu * (mu - 1) / 2;
            atomicAdd((unsigned long long*)&hP[ke], (unsigned long long)pr);
        }
    };
    const int4* s4 = (const int4*)a.inst;
    const int4* c4 = (const int4*)a.cur;
    const int4* l4 = (const int4*)a.rem;
    bool cleared = false;
    for (int base = q0; base < q1 || !cleared; base += PS_THREADS * PS_RV) {
        int4 sv[PS_RV], cv[PS_RV], lv[PS_RV];
#pragma unroll
        for (int j = 0; j < PS_RV; ++j) {
            const int q = base + j * PS_THREADS + tid;
            const int qc = q < q1 ? q : (q1 > q0 ? q1 - 1 : q0);
            if (q1 > q0) {
                sv[j] = s4[qc];
                cv[j] = c4[qc];
                lv[j] = l4[qc];
            }
        }
        if (!cleared) {                               // while the first reads are in flight
            for (int j = tid; j < KP; j += PS_THREADS) {
                hA[j] = 0;
                hN[j] = 0;
                hP[j] = 0;
            }
            __syncthreads();
            cleared = true;
        }
#pragma unroll
        for (int j = 0; j < PS_RV; ++j) {
            if (base + j * PS_THREADS + tid >= q1) continue;
            take(sv[j].x, cv[j].x, lv[j].x);
            take(sv[j].y, cv[j].y, lv[j].y);
            take(sv[j].z, cv[j].z, lv[j].z);
            take(sv[j].w, cv[j].w, lv[j].w);
        }
    }
    for (int r = 4 * q1 + tid; r < r1; r += PS_THREADS) take(a.inst[r], a.cur[r], a.rem[r]);
    if (i == 0) {
        bad = wave_or_i32(bad);
        if ((tid & 63) == 0) report_error(a.err_word, bad);
    }
    __syncthreads();

    // this slice's histograms -> the instance's shares, coherent 16-byte stores
    const uint32_t share = 3u * (uint32_t)KP * 8u;            // bytes per slice
    const __amdgpu_buffer_rsrc_t rs =
        xch_rsrc(a.part + (size_t)i * a.slices * 3 * KP, (uint32_t)a.slices * share);
    for (int p = tid; p < 3 * KP / 2; p += PS_THREADS) {
        const int arr = p / (KP / 2), j = 2 * (p - arr * (KP / 2));
        const int64_t* h = arr == 0 ? hA : arr == 1 ? hN : hP;
        const u32x4 v = {(uint32_t)h[j], (uint32_t)(h[j] >> 32), (uint32_t)h[j + 1],
                         (uint32_t)(h[j + 1] >> 32)};
        xch_store(v, rs, (uint32_t)sl * share + (uint32_t)(arr * KP + j) * 8u);
    }
    xch_wait_stores();
    if (!xch_last_arrival(&a.tickets[i], (uint32_t)a.slices, &s_ticket)) return;

    // last arriver: thread t takes bucket q = K-1-t and needs the slices'
    // sums of h_A, h_N at q+1 and of h_P at q; every read is issued first
    const int q = K - 1 - tid;
    const bool live = tid < K;
    int64_t xa = 0, xn = 0, xp = 0;
    {
        u32x2 va[PS_MAX_SLICES], vn[PS_MAX_SLICES], vp[PS_MAX_SLICES];
#pragma unroll
        for (int u = 0; u < PS_MAX_SLICES; ++u) {
            const bool ok = live && u < a.slices;
            const uint32_t o = (uint32_t)u * share;
            va[u] = xch_load_b64(rs, ok ? o + (uint32_t)(q + 1) * 8u : kXchOob);
            vn[u] = xch_load_b64(rs, ok ? o + (uint32_t)(KP + q + 1) * 8u : kXchOob);
            vp[u] = xch_load_b64(rs, ok ? o + (uint32_t)(2 * KP + q) * 8u : kXchOob);
        }
#pragma unroll
        for (int u = 0; u < PS_MAX_SLICES; ++u) {
            xa += (int64_t)(((uint64_t)va[u].y << 32) | va[u].x);
            xn += (int64_t)(((uint64_t)vn[u].y << 32) | vn[u].x);
            xp += (int64_t)(((uint64_t)vp[u].y << 32) | vp[u].x);
        }
    }
    // inclusive prefix in thread order = suffix sums over k_e > q
    block_incl_add2_i64<PS_THREADS>(xa, xn, tmp);
    const int64_t bb = (int64_t)b * b;
    const int64_t Lq = xa + bb * q * xn + xp;
    if (live) a.load[(int64_t)i * K + q] = Lq;
    if (!a.planes.tpm) return;

    // The scoring's planes of this instance (see CurvePlanes):
    // SM (suffix max of L) is the inclusive prefix max in this thread order;
    // PM (max of L[j] + b^2 j over j < k) takes the forward order j = t,
    // with L passed through LDS.
    const CurvePlanes& pl = a.planes;
    if (live) hA[q] = Lq;
    __syncthreads();
    const int j = tid;
    int64_t sm = live ? Lq : INT64_MIN;
    int64_t pm = j < K ? hA[j] + bb * j : INT64_MIN;
    block_incl_max2_i64<PS_THREADS>(sm, pm, tmp);
    hN[j] = pm;                                   // inclusive; PM[j] is thread j-1's
    __syncthreads();
    if (live) {
        pl.tl[q * pl.sk + i * pl.st] = Lq;
        if (q > 0) pl.tsm[(q - 1) * pl.sk + i * pl.st] = sm;
        else pl.peak[i] = sm;
    }
    if (j < K) pl.tpm[j * pl.sk + i * pl.st] = j > 0 ? hN[j - 1] : INT64_MIN;
    if (tid == 0) {
        pl.tpm[K * pl.sk + i * pl.st] = hN[K - 1];
        pl.tl[K * pl.sk + i * pl.st] = INT64_MIN;
        pl.tsm[(K - 1) * pl.sk + i * pl.st] = INT64_MIN;
        pl.tsm[K * pl.sk + i * pl.st] = INT64_MIN;
    }
}

LoadPlan plan_load(const star_load_params& p) {
    LoadPlan pl;
    pl.chunk = p.n_buckets < PL_CHUNK ? p.n_buckets : PL_CHUNK;
    pl.n_chunks = (int)ceil_div(p.n_buckets, pl.chunk);
    pl.split = p.n_req >= PS_MIN_REQ && p.n_buckets <= PS_MAX_K && p.n_inst <= kMaxTickets;
    if (pl.split) {
        int s = (int)ceil_div(PS_TARGET_GROUPS, p.n_inst);
        s = s < PS_MAX_SLICES ? s : PS_MAX_SLICES;
        const int smax = (int)(p.n_req / PS_MIN_SLICE);
        s = s < smax ? s : smax;
        s = s > 1 ? s : 1;
        pl.slice_len = (int)align_up((size_t)ceil_div(p.n_req, s), 4);
        pl.slices = (int)ceil_div(p.n_req, pl.slice_len);
        pl.kp = (int)align_up((size_t)p.n_buckets + 1, 2);
        pl.part_bytes = align_up((size_t)p.n_inst * pl.slices * 3 * pl.kp * 8, 256);
    }
    return pl;
}

hipError_t launch_project_load(const star_load_params& p, const LoadPlan& pl, const int32_t* cur,
                               const int32_t* rem, const int32_t* inst, int64_t* load,
                               char* ws, char* part, const CurvePlanes* planes,
                               bool* planes_written, hipStream_t stream) {
    int32_t* err_word = (int32_t*)(ws + kHdrErrorWord);
    const bool aligned16 = (((uintptr_t)cur | (uintptr_t)rem | (uintptr_t)inst) & 15) == 0;
    if (planes_written) *planes_written = false;
    if (pl.split && aligned16) {
        SplitArgs a;
        a.cur = cur; a.rem = rem; a.inst = inst; a.load = load; a.err_word = err_word;
        a.part = (int64_t*)part;
        a.tickets = (uint32_t*)(ws + kHdrTickets);
        a.planes = planes ? *planes : CurvePlanes{};
        if (planes_written) *planes_written = planes != nullptr;
        a.N = p.n_req; a.n = p.n_inst; a.b = p.bucket; a.K = p.n_buckets; a.KP = pl.kp;
        a.slices = pl.slices; a.slice_len = pl.slice_len;
        hipLaunchKernelGGL(project_split_kernel, dim3(p.n_inst, pl.slices), dim3(PS_THREADS), 0,
                           stream, a);
        return hipGetLastError();
    }
    const bool vec = p.n_req >= PL_VEC_MIN_REQ && aligned16;
    if (vec)
        hipLaunchKernelGGL(project_load_kernel<true>, dim3(p.n_inst, pl.n_chunks), dim3(PL_THREADS),
                           0, stream, cur, rem, inst, p.n_req, p.n_inst, p.bucket, p.n_buckets,
                           pl.chunk, load, err_word);
    else
        hipLaunchKernelGGL(project_load_kernel<false>, dim3(p.n_inst, pl.n_chunks), dim3(PL_THREADS),
                           0, stream, cur, rem, inst, p.n_req, p.n_inst, p.bucket, p.n_buckets,
                           pl.chunk, load, err_word);
    return hipGetLastError();
}

}  // namespace star
