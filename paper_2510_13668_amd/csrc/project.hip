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
// One workgroup per (instance, bucket chunk): it streams every request
// (coalesced 16-byte reads of four requests for long streams from 16-byte
// aligned arrays, else int32 reads), scatters its own instance's requests into LDS
// histograms with int64 LDS atomics, runs a block-wide suffix scan and
// writes its chunk of load[i, :].  Requests whose k_e lies beyond the chunk
// are folded into one overflow slot, so chunks are independent.
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

LoadPlan plan_load(const star_load_params& p) {
    LoadPlan pl;
    pl.chunk = p.n_buckets < PL_CHUNK ? p.n_buckets : PL_CHUNK;
    pl.n_chunks = (int)ceil_div(p.n_buckets, pl.chunk);
    return pl;
}

hipError_t launch_project_load(const star_load_params& p, const LoadPlan& pl, const int32_t* cur,
                               const int32_t* rem, const int32_t* inst, int64_t* load,
                               int32_t* err_word, hipStream_t stream) {
    const bool vec = p.n_req >= PL_VEC_MIN_REQ &&
                     (((uintptr_t)cur | (uintptr_t)rem | (uintptr_t)inst) & 15) == 0;
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
