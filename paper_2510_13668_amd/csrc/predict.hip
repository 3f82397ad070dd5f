// (a) Remaining-length predictor head on gfx950.
//
// Section 3.2 (Eq. 1-2): the last-layer, last-token hidden state of every
// running request goes through a small MLP.  Here: a1 = act(W1 h + b1),
// logits = W2 a1 + b2 over length bins, p = softmax, E = sum p_j v_j, then
// the continuous-prediction smoothing of Section 3.3 and integerisation.
//
// Kernel 1 (gemm1_splitk): Z1 partials = H W1^T over a K-slice, on MFMA.
//   128x128 output tile per 256-thread workgroup (4 waves, 64x64 each as
//   2x2 MFMA 32x32 blocks), 128 bytes of K per LDS row (64 bf16 / 32 fp32),
//   double-buffered LDS fed by 16-byte global loads, split-K so that small
//   batches still launch ~256 workgroups.  Partials are fp32, reduced later
//   in a fixed order (deterministic results).
// Kernel 2 (head): 16 rows per workgroup: fixed-order split-K reduction,
//   bias, activation, the bin GEMM (bf16 MFMA 16x16x32 on a hi/lo split of
//   a1, or fp32 FMA), softmax, expectation, EMA, round-half-even, clamp.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

// ---------------------------------------------------------------------------
// GEMM1
// ---------------------------------------------------------------------------
constexpr int G1_BM = 128;
constexpr int G1_BN = 128;
constexpr int G1_KBYTES = 128;                 // bytes of K per LDS row
constexpr int G1_ROW = G1_KBYTES + 16;         // padded LDS row (bytes)
constexpr int G1_TILE = G1_BM * G1_ROW;        // one operand tile (bytes)
constexpr int G1_THREADS = 256;
constexpr int G1_CHUNKS = G1_BM * G1_KBYTES / 16 / G1_THREADS;   // 16-byte chunks per thread per operand

template <int kElemBytes> struct G1Elem;
template <> struct G1Elem<2> { static constexpr int BK = 64; };   // bf16
template <> struct G1Elem<4> { static constexpr int BK = 32; };   // fp32

// Map blockIdx to a logical tile index so that consecutive logical indices
// run on the same XCD (workgroups are dealt round-robin over the 8 XCDs):
// logical neighbours share operand rows and hence that XCD's L2.
__device__ inline int xcd_logical_block(int bid, int nblk) {
    const int q = nblk / 8, r = nblk % 8;
    const int x = bid % 8;
    return x * q + (x < r ? x : r) + bid / 8;
}

template <int kElemBytes>
__global__ __launch_bounds__(G1_THREADS) void gemm1_splitk_kernel(
    const char* __restrict__ A, const char* __restrict__ W, float* __restrict__ P,
    int M, int N, int Kd, int splits, int tiles_n, int ktiles) {
    constexpr int BK = G1Elem<kElemBytes>::BK;
    __shared__ __attribute__((aligned(16))) char lds[2][2][G1_TILE];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid >> 1, wn = wid & 1;

    const int logical = xcd_logical_block(blockIdx.x, gridDim.x);
    const int tiles = gridDim.x / splits;
    const int split = logical / tiles;
    const int tile = logical % tiles;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int kt0 = (int)((int64_t)split * ktiles / splits);
    const int kt1 = (int)((int64_t)(split + 1) * ktiles / splits);

    const int64_t row_bytes = (int64_t)Kd * kElemBytes;
    const int64_t kd_bytes = row_bytes;

    // global -> register staging for one K-tile (both operands)
    uint4 ra[G1_CHUNKS], rb[G1_CHUNKS];
    auto load_tile = [&](int kt) {
        const int64_t kb = (int64_t)kt * G1_KBYTES;
#pragma unroll
        for (int p = 0; p < G1_CHUNKS; ++p) {
            const int c = tid + p * G1_THREADS;
            const int row = c >> 3;
            const int cb = (c & 7) * 16;
            const int ga = tm * G1_BM + row;
            const int gb = tn * G1_BN + row;
            const bool kin = kb + cb < kd_bytes;
            ra[p] = (ga < M && kin) ? *(const uint4*)(A + (int64_t)ga * row_bytes + kb + cb)
                                    : make_uint4(0, 0, 0, 0);
            rb[p] = (gb < N && kin) ? *(const uint4*)(W + (int64_t)gb * row_bytes + kb + cb)
                                    : make_uint4(0, 0, 0, 0);
        }
    };
    auto store_tile = [&](int buf) {
#pragma unroll
        for (int p = 0; p < G1_CHUNKS; ++p) {
            const int c = tid + p * G1_THREADS;
            const int row = c >> 3;
            const int cb = (c & 7) * 16;
            *(uint4*)(&lds[buf][0][row * G1_ROW + cb]) = ra[p];
            *(uint4*)(&lds[buf][1][row * G1_ROW + cb]) = rb[p];
        }
    };

    f32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int r32 = lane & 31;
    const int khalf = lane >> 5;   // which half of the MFMA's K slice this lane feeds

    if (kt0 < kt1) {
        load_tile(kt0);
        store_tile(0);
        __syncthreads();
        for (int kt = kt0; kt < kt1; ++kt) {
            const int buf = (kt - kt0) & 1;
            const bool more = kt + 1 < kt1;
            if (more) load_tile(kt + 1);
            const char* la = lds[buf][0];
            const char* lb = lds[buf][1];
            if constexpr (kElemBytes == 2) {
                // v_mfma_f32_32x32x16_bf16: lane feeds row (lane%32), k = 8*(lane/32)..+7
#pragma unroll
                for (int kk = 0; kk < BK / 16; ++kk) {
                    const int koff = (kk * 16 + khalf * 8) * 2;
                    bf16x8_t a[2], b[2];
#pragma unroll
                    for (int i = 0; i < 2; ++i)
                        a[i] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(la + (wm * 64 + i * 32 + r32) * G1_ROW + koff));
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        b[j] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(lb + (wn * 64 + j * 32 + r32) * G1_ROW + koff));
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
                }
            } else {
                // v_mfma_f32_32x32x2_f32: lane feeds row (lane%32), k = lane/32
#pragma unroll
                for (int kk = 0; kk < BK / 2; ++kk) {
                    const int koff = (kk * 2 + khalf) * 4;
                    float a[2], b[2];
#pragma unroll
                    for (int i = 0; i < 2; ++i) a[i] = *(const float*)(la + (wm * 64 + i * 32 + r32) * G1_ROW + koff);
#pragma unroll
                    for (int j = 0; j < 2; ++j) b[j] = *(const float*)(lb + (wn * 64 + j * 32 + r32) * G1_ROW + koff);
#pragma unroll
                    for (int i = 0; i < 2; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
                }
            }
            if (more) store_tile(buf ^ 1);
            __syncthreads();
        }
    }

    // epilogue: 32x32 accumulator layout -- element v of lane l is
    // row 8*(v/4) + 4*(l/32) + v%4, column l%32 of the block.
    float* out = P + (int64_t)split * M * N;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int col = tn * G1_BN + wn * 64 + j * 32 + r32;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = tm * G1_BM + wm * 64 + i * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
                if (row < M && col < N) out[(int64_t)row * N + col] = acc[i][j][v];
            }
        }
}

// ---------------------------------------------------------------------------
// head
// ---------------------------------------------------------------------------
constexpr int HD_RB = 16;
constexpr int HD_THREADS = 256;

__device__ inline float apply_act(float x, int act) {
    if (act == STAR_ACT_RELU) return x > 0.0f ? x : 0.0f;
    return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
}

template <bool kBF16>
__global__ __launch_bounds__(HD_THREADS) void head_kernel(
    const float* __restrict__ P, int splits, int B, int m, int nb, const float* __restrict__ b1,
    const void* __restrict__ w2, const float* __restrict__ b2, const float* __restrict__ bins,
    int act, float ema_alpha, int ema_init, float* __restrict__ ema_state,
    float* __restrict__ expected, int32_t* __restrict__ rem_len, int len_max) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int row0 = blockIdx.x * HD_RB;
    const int mpad = (m + 31) & ~31;
    const int astride = mpad + 8;                 // bf16 elements per LDS row
    const int nbpad = (nb + 15) & ~15;

    uint16_t* ahi = (uint16_t*)smem;
    uint16_t* alo = ahi + HD_RB * astride;
    float* a32 = (float*)smem;
    float* z = kBF16 ? (float*)(alo + HD_RB * astride) : (float*)(a32 + HD_RB * m);

    const int64_t plane = (int64_t)B * m;
    // 1) fixed-order split-K reduction, bias, activation
    for (int r = 0; r < HD_RB; ++r) {
        const int gr = row0 + r;
        for (int u = tid; u < (kBF16 ? mpad : m); u += HD_THREADS) {
            float a = 0.0f;
            if (gr < B && u < m) {
                const float* src = P + (int64_t)gr * m + u;
                float s = src[0];
                for (int q = 1; q < splits; ++q) s += src[q * plane];
                if (b1) s += b1[u];
                a = apply_act(s, act);
            }
            if constexpr (kBF16) {
                const uint16_t hi = f32_to_bf16_rne(a);
                ahi[r * astride + u] = hi;
                alo[r * astride + u] = f32_to_bf16_rne(a - bf16_to_f32(hi));
            } else {
                a32[r * m + u] = a;
            }
        }
    }
    __syncthreads();

    // 2) bin logits
    if constexpr (kBF16) {
        // v_mfma_f32_16x16x32_bf16: lane feeds row (lane%16), k = 8*(lane/16)..+7;
        // accumulator element v of lane l is row 4*(l/16)+v, column l%16.
        const uint16_t* W2 = (const uint16_t*)w2;
        const int r16 = lane & 15;
        const int kq = lane >> 4;
        for (int nblk = wid; nblk * 16 < nb; nblk += HD_THREADS / 64) {
            const int j = nblk * 16 + r16;
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
            for (int k0 = 0; k0 < mpad; k0 += 32) {
                const int k = k0 + kq * 8;
                bf16x8 bw = {0, 0, 0, 0, 0, 0, 0, 0};
                if (j < nb && k < m) bw = *(const bf16x8*)(W2 + (int64_t)j * m + k);
                const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, bw);
                const bf16x8_t h = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(ahi + r16 * astride + k));
                const bf16x8_t l = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(alo + r16 * astride + k));
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(h, bv, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(l, bv, acc, 0, 0, 0);
            }
            const int col = nblk * 16 + r16;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 4 * kq + v;
                if (col < nb) z[row * nbpad + col] = acc[v] + (b2 ? b2[col] : 0.0f);
            }
        }
    } else {
        const float* W2 = (const float*)w2;
        for (int e = tid; e < HD_RB * nb; e += HD_THREADS) {
            const int r = e / nb, j = e % nb;
            const float* wrow = W2 + (int64_t)j * m;
            const float* arow = a32 + r * m;
            float s = 0.0f;
            for (int u = 0; u < m; ++u) s = fmaf(arow[u], wrow[u], s);
            z[r * nbpad + j] = s + (b2 ? b2[j] : 0.0f);
        }
    }
    __syncthreads();

    // 3) softmax, expectation, EMA, integerisation: one wave per row
    for (int r = wid; r < HD_RB; r += HD_THREADS / 64) {
        const int gr = row0 + r;
        if (gr >= B) continue;
        float zmax = -INFINITY;
        for (int j = lane; j < nb; j += 64) zmax = fmaxf(zmax, z[r * nbpad + j]);
        zmax = wave_max_f32(zmax);
        float den = 0.0f, num = 0.0f;
        for (int j = lane; j < nb; j += 64) {
            const float e = expf(z[r * nbpad + j] - zmax);
            den += e;
            num += e * bins[j];
        }
        den = wave_sum_f32(den);
        num = wave_sum_f32(num);
        if (lane == 0) {
            const float E = num / den;
            expected[gr] = E;
            float y = E;
            if (ema_alpha > 0.0f) {
                y = ema_init ? E : ema_alpha * E + (1.0f - ema_alpha) * ema_state[gr];
                ema_state[gr] = y;
            }
            if (rem_len) {
                float q = rintf(y);
                int32_t li;
                if (!(q >= 1.0f)) li = 1;
                else if (q >= (float)len_max) li = len_max;
                else li = (int32_t)q;
                rem_len[gr] = li;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
PredictPlan plan_predict(const star_predict_params& p) {
    PredictPlan pl;
    const int elem = p.dtype == STAR_BF16 ? 2 : 4;
    const int bk = G1_KBYTES / elem;
    pl.tiles_m = (int)ceil_div(p.n_req, G1_BM);
    pl.tiles_n = (int)ceil_div(p.d_hidden, G1_BN);
    pl.ktiles = (int)ceil_div(p.d_model, bk);
    const int tiles = pl.tiles_m * pl.tiles_n;
    int s = 1;
    if (tiles > 0 && tiles < 192) {
        s = 256 / tiles;
        if (s > 16) s = 16;
        if (s > pl.ktiles / 2) s = pl.ktiles / 2;
        if (s < 1) s = 1;
    }
    pl.splits = s;
    pl.partial_bytes = (size_t)s * (size_t)p.n_req * (size_t)p.d_hidden * sizeof(float);
    const int mpad = (p.d_hidden + 31) & ~31;
    const int nbpad = (p.n_bins + 15) & ~15;
    if (p.dtype == STAR_BF16)
        pl.head_lds = (size_t)2 * HD_RB * (mpad + 8) * 2 + (size_t)HD_RB * nbpad * 4;
    else
        pl.head_lds = (size_t)HD_RB * p.d_hidden * 4 + (size_t)HD_RB * nbpad * 4;
    return pl;
}

hipError_t launch_predict(const star_predict_params& p, const PredictPlan& pl, const void* hidden,
                          const void* w1, const float* b1, const void* w2, const float* b2,
                          const float* bins, float* ema_state, float* expected, int32_t* rem_len,
                          float* partials, hipStream_t stream) {
    if (p.n_req == 0) return hipSuccess;
    hipEvent_t* ev = (hipEvent_t*)p.timing_events;
    hipError_t e;
    if (ev) {
        e = hipEventRecord(ev[0], stream);
        if (e != hipSuccess) return e;
    }
    const dim3 g1(pl.tiles_m * pl.tiles_n * pl.splits);
    if (p.dtype == STAR_BF16)
        hipLaunchKernelGGL(gemm1_splitk_kernel<2>, g1, dim3(G1_THREADS), 0, stream,
                           (const char*)hidden, (const char*)w1, partials, p.n_req, p.d_hidden,
                           p.d_model, pl.splits, pl.tiles_n, pl.ktiles);
    else
        hipLaunchKernelGGL(gemm1_splitk_kernel<4>, g1, dim3(G1_THREADS), 0, stream,
                           (const char*)hidden, (const char*)w1, partials, p.n_req, p.d_hidden,
                           p.d_model, pl.splits, pl.tiles_n, pl.ktiles);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (ev) {
        e = hipEventRecord(ev[1], stream);
        if (e != hipSuccess) return e;
    }
    const dim3 g2((unsigned)ceil_div(p.n_req, HD_RB));
    if (p.dtype == STAR_BF16) {
        if (pl.head_lds > 64 * 1024) {
            e = hipFuncSetAttribute((const void*)head_kernel<true>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.head_lds);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(head_kernel<true>, g2, dim3(HD_THREADS), pl.head_lds, stream, partials,
                           pl.splits, p.n_req, p.d_hidden, p.n_bins, b1, w2, b2, bins, p.act,
                           p.ema_alpha, p.ema_init, ema_state, expected, rem_len, p.len_max);
    } else {
        if (pl.head_lds > 64 * 1024) {
            e = hipFuncSetAttribute((const void*)head_kernel<false>,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.head_lds);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(head_kernel<false>, g2, dim3(HD_THREADS), pl.head_lds, stream, partials,
                           pl.splits, p.n_req, p.d_hidden, p.n_bins, b1, w2, b2, bins, p.act,
                           p.ema_alpha, p.ema_init, ema_state, expected, rem_len, p.len_max);
    }
    return hipGetLastError();
}

}  // namespace star
