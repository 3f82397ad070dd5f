// (a) Remaining-length predictor head on gfx950.
//
// Section 4.2 (Eq. 1-2): the last-layer, last-token hidden state of every
// running request goes through a small MLP.  Here: a1 = act(W1 h + b1),
// logits = W2 a1 + b2 over length bins, p = softmax, E = sum p_j v_j, then
// the continuous-prediction smoothing of Section 4.3 and integerisation.
//
// Kernel 1 (gemm1_splitk): Z1 partials = H W1^T over a K-slice, on MFMA
//   (32x32 blocks), 128 bytes of K per LDS row (64 bf16 / 32 fp32),
//   double-buffered LDS fed by register-staged 16-byte global loads, split-K
//   so that small batches still fill the CUs.  Tile shapes: 64x64 on 4
//   waves, 128x128 on 8 or 4 waves, 256x256 on 8 waves; a cost model picks
//   one per product.  Partials are fp32, reduced later in a fixed order
//   (deterministic results).
// Kernel 2 (head): 4 rows per workgroup (many workgroups, so the split-K
//   partial reads have plenty of loads in flight), 16 for large batches:
//   fixed-order split-K reduction, bias, activation, the bin GEMM (bf16 MFMA
//   16x16x32 on a hi/lo split of a1, or fp32 FMA), softmax, expectation,
//   EMA, round-half-even, clamp.
#include "star_common.hpp"
#include "star_internal.hpp"

namespace star {

// ---------------------------------------------------------------------------
// GEMM1
// ---------------------------------------------------------------------------
constexpr int G1_KBYTES = 128;                 // bytes of K per LDS row
constexpr int G1_ROW = G1_KBYTES + 16;         // padded LDS row (bytes)
constexpr int G1_CPR = G1_KBYTES / 16;         // 16-byte chunks per row
// K-tiles of global loads in flight ahead of the multiply: three for the
// 128 x 128 shape (one 8-wave workgroup per CU), two for the 64 x 64 one,
// which runs two workgroups per CU that share the CU's load path (measured:
// deeper register staging only lengthens each workgroup there).
constexpr int G1_STAGES_BIG = 3;
constexpr int G1_STAGES_SMALL = 2;
constexpr int G1_STAGES_MID = 2;
constexpr int G1_STAGES_WIDE = 2;
constexpr int G1_WIDE_MIN_TILES = 1024;   // 128 x 128 tiles from which G1Wide replaces G1Big
constexpr int G1_STAGES_HUGE = 1;
constexpr int G1_HUGE_MIN_TILES = 256;    // 256 x 256 tiles (no split) from which G1Huge is used

template <int kElemBytes> struct G1Elem {
    static constexpr int BK = G1_KBYTES / kElemBytes;   // K elements per K-tile
};

// Map blockIdx to a logical tile index so that consecutive logical indices
// run on the same XCD (workgroups are dealt round-robin over the 8 XCDs):
// logical neighbours share operand rows and hence that XCD's L2.
__device__ inline int xcd_logical_block(int bid, int nblk) {
    const int q = nblk / 8, r = nblk % 8;
    const int x = bid % 8;
    return x * q + (x < r ? x : r) + bid / 8;
}

// Tile shape of the split-K product: BM x BN outputs per workgroup, WM x WN
// waves, each wave a (BM/WM) x (BN/WN) slab of 32 x 32 matrix-core blocks.
template <int kBM, int kBN, int kWM, int kWN>
struct G1Shape {
    static constexpr int BM = kBM, BN = kBN, WM = kWM, WN = kWN;
    static constexpr int THREADS = 64 * WM * WN;
    static constexpr int MI = BM / WM / 32, NJ = BN / WN / 32;
    static constexpr int CA = BM * G1_KBYTES / 16 / THREADS;   // 16-byte chunks per thread, A
    static constexpr int CB = BN * G1_KBYTES / 16 / THREADS;   // ... and W
    static constexpr int LDS_A = BM * G1_ROW, LDS_B = BN * G1_ROW;
    static constexpr int OUT_ROW = BN + 8;     // floats per LDS row of the output tile
    static_assert(MI >= 1 && NJ >= 1 && CA >= 1 && CB >= 1, "shape");
    // the output tile goes out through LDS when it fits the operand buffers,
    // else straight from the accumulators
    static constexpr bool LDS_EPI = BM * OUT_ROW * 4 <= 2 * (LDS_A + LDS_B);
};
using G1Big = G1Shape<128, 128, 4, 2>;     // 8 waves, 32 x 64 slabs
using G1Small = G1Shape<64, 64, 2, 2>;     // 4 waves, 32 x 32 slabs
// 8 waves, 32 x 32 slabs of a 128 x 64 tile, for products of at most 128
// rows: twice G1Big's tiles along N, so half its K-splits fill the chip, and
// the partials written and read back halve.  The regression head's first
// layer (2048 x 3584) went from 22.7 to 20.4 us per call at one row and
// from 26.4 to 23.3 us at ten.  With several row tiles the cost model would
// also pick it, but there it measured slower (the regression head's first
// layer at 1024 rows: 29.3 against 33.9 us), so it is offered only here.
using G1Mid = G1Shape<128, 64, 4, 2>;
// 4 waves, 64 x 64 slabs: twice the matrix-core work per LDS byte of G1Big,
// at half its waves per workgroup; it wins once every CU has several
// workgroups queued (measured: 580 against 786 us for 32768 x 1024 x 8192)
using G1Wide = G1Shape<128, 128, 2, 2>;
// 8 waves, 64 x 128 slabs of a 256 x 256 tile: four times G1Big's matrix-core
// work per byte loaded, one workgroup per CU (147 KiB of LDS); one K-tile in
// flight keeps it within 256 registers.  For products with hundreds of such
// tiles (measured at 32768 x 1024 x 8192: 511-715 us per call, 570 us on
// average over 70 calls, 39% of peak, the matrix cores busy half the time).
using G1Huge = G1Shape<256, 256, 4, 2>;

// One K-tile of both operands staged in registers (constant indices only,
// so the stages stay in VGPRs).
template <class SH>
struct G1Stage {
    uint4 a[SH::CA], b[SH::CB];
};

struct G1Ctx {
    const char* A;
    const char* W;
    int M, N, tm, tn, tid, threads, bm, bn;
    int64_t row_bytes;
};

// Loads are unconditional (addresses clamped into the operands) so the
// compiler can count them and wait only for the stage it is about to store;
// out-of-range values are zeroed when they are written to LDS.
__device__ __forceinline__ uint4 g1_load(const G1Ctx& c, const char* base, int rows, int row0,
                                         int p, int64_t kb) {
    const int ch = c.tid + p * c.threads;
    const int row = row0 + ch / G1_CPR;
    const int64_t off = kb + (ch % G1_CPR) * 16;
    const int64_t ko = off < c.row_bytes ? off : 0;
    return *(const uint4*)(base + (int64_t)(row < rows ? row : rows - 1) * c.row_bytes + ko);
}

template <class SH>
__device__ __forceinline__ void g1_load_stage(const G1Ctx& c, int kt, G1Stage<SH>& s) {
    const int64_t kb = (int64_t)kt * G1_KBYTES;
    const int ra = c.tm * SH::BM, rb = c.tn * SH::BN;
#pragma unroll
    for (int p = 0; p < SH::CA; ++p) s.a[p] = g1_load(c, c.A, c.M, ra, p, kb);
#pragma unroll
    for (int p = 0; p < SH::CB; ++p) s.b[p] = g1_load(c, c.W, c.N, rb, p, kb);
}

__device__ __forceinline__ void g1_store_chunk(const G1Ctx& c, char* l, int p, int64_t kb,
                                               int row0, int rows, uint4 v) {
    const int ch = c.tid + p * c.threads;
    const int row = ch / G1_CPR;
    const int cb = (ch % G1_CPR) * 16;
    // bitwise masks, not a select of uint4 structs (which would go through memory)
    const uint32_t m = (kb + cb < c.row_bytes && row0 + row < rows) ? 0xFFFFFFFFu : 0u;
    *(uint4*)(l + row * G1_ROW + cb) = make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
}

template <class SH>
__device__ __forceinline__ void g1_store_stage(const G1Ctx& c, char* la, char* lb, int kt,
                                               const G1Stage<SH>& s) {
    const int64_t kb = (int64_t)kt * G1_KBYTES;
#pragma unroll
    for (int p = 0; p < SH::CA; ++p) g1_store_chunk(c, la, p, kb, c.tm * SH::BM, c.M, s.a[p]);
#pragma unroll
    for (int p = 0; p < SH::CB; ++p) g1_store_chunk(c, lb, p, kb, c.tn * SH::BN, c.N, s.b[p]);
}

// A wave multiplies its (32 MI) x (32 NJ) slab: rows wm * 32 MI..,
// columns wn * 32 NJ..
template <int kElemBytes, class SH>
__device__ __forceinline__ void g1_compute(const char* la, const char* lb, int wm, int wn,
                                           int lane, f32x16 (&acc)[SH::MI][SH::NJ]) {
    constexpr int BK = G1Elem<kElemBytes>::BK;
    constexpr int MI = SH::MI, NJ = SH::NJ;
    const int r32 = lane & 31;
    const int khalf = lane >> 5;   // which half of the MFMA's K slice this lane feeds
    constexpr int KK = BK / 16;
    if constexpr (kElemBytes == 2 && (MI + NJ) * KK <= 12) {
        // every fragment of the K-tile is read from LDS first, so the wave
        // waits for LDS once per K-tile and then issues its MFMAs back to back
        bf16x8_t a[KK][MI], b[KK][NJ];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const int koff = (kk * 16 + khalf * 8) * 2;
#pragma unroll
            for (int i = 0; i < MI; ++i)
                a[kk][i] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(la + (wm * 32 * MI + i * 32 + r32) * G1_ROW + koff));
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                b[kk][j] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(lb + (wn * 32 * NJ + j * 32 + r32) * G1_ROW + koff));
        }
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk][i], b[kk][j], acc[i][j], 0, 0, 0);
        // keep that order: the scheduler would otherwise pair reads with
        // MFMAs to save registers and wait for LDS once per pair
        __builtin_amdgcn_sched_group_barrier(0x100, (MI + NJ) * KK, 0);   // LDS reads
        __builtin_amdgcn_sched_group_barrier(0x008, MI * NJ * KK, 0);     // MFMAs
    } else if constexpr (kElemBytes == 2) {
        // v_mfma_f32_32x32x16_bf16: lane feeds row (lane%32), k = 8*(lane/32)..+7
#pragma unroll
        for (int kk = 0; kk < BK / 16; ++kk) {
            const int koff = (kk * 16 + khalf * 8) * 2;
            bf16x8_t a[MI], b[NJ];
#pragma unroll
            for (int i = 0; i < MI; ++i)
                a[i] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(la + (wm * 32 * MI + i * 32 + r32) * G1_ROW + koff));
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                b[j] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(lb + (wn * 32 * NJ + j * 32 + r32) * G1_ROW + koff));
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    } else {
        // v_mfma_f32_32x32x2_f32: lane feeds row (lane%32), k = lane/32
#pragma unroll
        for (int kk = 0; kk < BK / 2; ++kk) {
            const int koff = (kk * 2 + khalf) * 4;
            float a[MI], b[NJ];
#pragma unroll
            for (int i = 0; i < MI; ++i) a[i] = *(const float*)(la + (wm * 32 * MI + i * 32 + r32) * G1_ROW + koff);
#pragma unroll
            for (int j = 0; j < NJ; ++j) b[j] = *(const float*)(lb + (wn * 32 * NJ + j * 32 + r32) * G1_ROW + koff);
#pragma unroll
            for (int i = 0; i < MI; ++i)
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[j], acc[i][j], 0, 0, 0);
        }
    }
}

// One pipeline step: stage s holds tile i; write it to LDS buffer i % 2,
// barrier, refill s with tile i + NS (or re-read tile i -- a cache hit --
// past the end, so that every step issues exactly one stage of loads), and
// multiply buffer i % 2.  A buffer is rewritten two steps after its last
// use, and every thread has passed the intervening barrier only after
// finishing that use.
template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void g1_step(const G1Ctx& c, char (*lds)[SH::LDS_A + SH::LDS_B],
                                        int kt0, int nk, int i, G1Stage<SH>& s, int wm, int wn,
                                        int lane, f32x16 (&acc)[SH::MI][SH::NJ]) {
    const int buf = i & 1;
    // scheduling fences keep each phase in place: otherwise the compiler
    // hoists the next stage's masking into the multiply, which then waits
    // for loads issued only one step earlier
    __builtin_amdgcn_sched_barrier(0);
    g1_store_stage<SH>(c, lds[buf], lds[buf] + SH::LDS_A, kt0 + i, s);
    __syncthreads();
    g1_load_stage<SH>(c, kt0 + (i + NS < nk ? i + NS : i), s);
    __builtin_amdgcn_sched_barrier(0);
    g1_compute<kElemBytes, SH>(lds[buf], lds[buf] + SH::LDS_A, wm, wn, lane, acc);
}

// The work of one workgroup of the split-K product: tile (tm, tn), K-tiles
// [kt0, kt1).  Workgroups are dealt to the XCDs round-robin; the logical
// order puts one K-slice of neighbouring tiles on each XCD.
struct G1Work {
    int split, tile, tm, tn, kt0, nk;
};
__device__ inline G1Work g1_work(int splits, int tiles_n, int ktiles, int bid, int nblocks) {
    G1Work w;
    const int logical = xcd_logical_block(bid, nblocks);
    const int tiles = nblocks / splits;
    w.split = logical / tiles;
    w.tile = logical % tiles;
    w.tm = w.tile / tiles_n;
    w.tn = w.tile % tiles_n;
    w.kt0 = (int)((int64_t)w.split * ktiles / splits);
    const int kt1 = (int)((int64_t)(w.split + 1) * ktiles / splits);
    w.nk = kt1 - w.kt0;
    return w;
}

// Main loop of one workgroup's product: NS K-tiles of global loads are in
// flight ahead of the tile being multiplied (register staging, two LDS
// buffers, one barrier per K-tile).  acc receives this wave's slab.
template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void g1_mainloop_edge(const G1Ctx& c, const G1Work& w,
                                                 char (*lds)[SH::LDS_A + SH::LDS_B], int wm,
                                                 int wn, int lane, f32x16 (&acc)[SH::MI][SH::NJ]) {
    const int nk = w.nk, kt0 = w.kt0;
    if (nk > 0) {
        G1Stage<SH> st[NS];
#pragma unroll
        for (int u = 0; u < NS; ++u) g1_load_stage<SH>(c, kt0 + (u < nk ? u : 0), st[u]);
        int i = 0;
        for (; i + NS <= nk; i += NS) {
#pragma unroll
            for (int u = 0; u < NS; ++u)
                g1_step<kElemBytes, NS, SH>(c, lds, kt0, nk, i + u, st[u], wm, wn, lane, acc);
        }
#pragma unroll
        for (int u = 0; u < NS - 1; ++u)
            if (i + u < nk) g1_step<kElemBytes, NS, SH>(c, lds, kt0, nk, i + u, st[u], wm, wn, lane, acc);
    }
}

// The same for a tile wholly inside the product whose K is a whole number
// of K-tiles: nothing to clamp or mask.  Each thread's row offsets (32-bit,
// the operands are under 4 GiB) and LDS offsets are computed once; per
// K-tile only the uniform base pointer moves, so the loads take the
// scalar-base form and the loop carries no per-element masks.
template <class SH>
struct G1Fast {
    uint32_t ga[SH::CA], gb[SH::CB];          // global byte offsets within a K-tile column
    uint32_t la[SH::CA], lb[SH::CB];          // LDS byte offsets
};
typedef uint32_t g1u4 __attribute__((ext_vector_type(4)));
template <class SH>
struct G1FStage {                             // one K-tile of both operands in registers
    g1u4 a[SH::CA], b[SH::CB];
};

template <class SH>
__device__ __forceinline__ void g1f_load(const G1Ctx& c, const G1Fast<SH>& f, int kt,
                                         G1FStage<SH>& st) {
    const char* pa = c.A + (int64_t)kt * G1_KBYTES;
    const char* pb = c.W + (int64_t)kt * G1_KBYTES;
#pragma unroll
    for (int p = 0; p < SH::CA; ++p) st.a[p] = *(const g1u4*)(pa + f.ga[p]);
#pragma unroll
    for (int p = 0; p < SH::CB; ++p) st.b[p] = *(const g1u4*)(pb + f.gb[p]);
}

template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void g1f_step(const G1Ctx& c, const G1Fast<SH>& f,
                                         char (*lds)[SH::LDS_A + SH::LDS_B], int kt0, int nk,
                                         int i, G1FStage<SH>& st, int wm, int wn, int lane,
                                         f32x16 (&acc)[SH::MI][SH::NJ]) {
    char* l = lds[i & 1];
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int p = 0; p < SH::CA; ++p) *(g1u4*)(l + f.la[p]) = st.a[p];
#pragma unroll
    for (int p = 0; p < SH::CB; ++p) *(g1u4*)(l + f.lb[p]) = st.b[p];
    __syncthreads();
    g1f_load<SH>(c, f, kt0 + (i + NS < nk ? i + NS : i), st);
    __builtin_amdgcn_sched_barrier(0);
    g1_compute<kElemBytes, SH>(l, l + SH::LDS_A, wm, wn, lane, acc);
}

template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void g1_mainloop_interior(const G1Ctx& c, const G1Work& w,
                                                     char (*lds)[SH::LDS_A + SH::LDS_B], int wm,
                                                     int wn, int lane,
                                                     f32x16 (&acc)[SH::MI][SH::NJ]) {
    G1Fast<SH> f;
#pragma unroll
    for (int p = 0; p < SH::CA; ++p) {
        const int ch = c.tid + p * c.threads;
        f.ga[p] = (uint32_t)((c.tm * SH::BM + ch / G1_CPR) * c.row_bytes + (ch % G1_CPR) * 16);
        f.la[p] = (uint32_t)((ch / G1_CPR) * G1_ROW + (ch % G1_CPR) * 16);
    }
#pragma unroll
    for (int p = 0; p < SH::CB; ++p) {
        const int ch = c.tid + p * c.threads;
        f.gb[p] = (uint32_t)((c.tn * SH::BN + ch / G1_CPR) * c.row_bytes + (ch % G1_CPR) * 16);
        f.lb[p] = (uint32_t)(SH::LDS_A + (ch / G1_CPR) * G1_ROW + (ch % G1_CPR) * 16);
    }
    const int nk = w.nk, kt0 = w.kt0;
    if (nk > 0) {
        G1FStage<SH> st[NS];
#pragma unroll
        for (int u = 0; u < NS; ++u) g1f_load<SH>(c, f, kt0 + (u < nk ? u : 0), st[u]);
        int i = 0;
        for (; i + NS <= nk; i += NS) {
#pragma unroll
            for (int u = 0; u < NS; ++u)
                g1f_step<kElemBytes, NS, SH>(c, f, lds, kt0, nk, i + u, st[u], wm, wn, lane, acc);
        }
#pragma unroll
        for (int u = 0; u < NS - 1; ++u)
            if (i + u < nk)
                g1f_step<kElemBytes, NS, SH>(c, f, lds, kt0, nk, i + u, st[u], wm, wn, lane, acc);
    }
}

template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void g1_mainloop(const char* A, const char* W, int M, int N, int Kd,
                                            const G1Work& w, char (*lds)[SH::LDS_A + SH::LDS_B],
                                            f32x16 (&acc)[SH::MI][SH::NJ]) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid / SH::WN, wn = wid % SH::WN;
    G1Ctx c;
    c.A = A; c.W = W; c.M = M; c.N = N; c.tm = w.tm; c.tn = w.tn; c.tid = tid;
    c.threads = SH::THREADS; c.bm = SH::BM; c.bn = SH::BN;
    c.row_bytes = (int64_t)Kd * kElemBytes;
#pragma unroll
    for (int i = 0; i < SH::MI; ++i)
#pragma unroll
        for (int j = 0; j < SH::NJ; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;
    // uniform over the workgroup: rows and columns in range, K whole tiles,
    // and both operands addressable with 32-bit offsets
    const bool interior = (w.tm + 1) * SH::BM <= M && (w.tn + 1) * SH::BN <= N &&
                          c.row_bytes % G1_KBYTES == 0 &&
                          (int64_t)M * c.row_bytes < ((int64_t)1 << 32) &&
                          (int64_t)N * c.row_bytes < ((int64_t)1 << 32);
    if (interior)
        g1_mainloop_interior<kElemBytes, NS, SH>(c, w, lds, wm, wn, lane, acc);
    else
        g1_mainloop_edge<kElemBytes, NS, SH>(c, w, lds, wm, wn, lane, acc);
}

// Split-K product P[split] = A[:, Ks] W[:, Ks]^T over one BM x BN tile: the
// work of block `bid` of a grid of `nblocks` product blocks.
template <int kElemBytes, int NS, class SH>
__device__ __forceinline__ void gemm1_tile(const char* __restrict__ A, const char* __restrict__ W,
                                           float* __restrict__ P, int M, int N, int Kd,
                                           int splits, int tiles_n, int ktiles, int bid,
                                           int nblocks,
                                           char (*lds)[SH::LDS_A + SH::LDS_B]) {
    constexpr int MI = SH::MI, NJ = SH::NJ;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid / SH::WN, wn = wid % SH::WN;
    const G1Work w = g1_work(splits, tiles_n, ktiles, bid, nblocks);
    const int split = w.split, tm = w.tm, tn = w.tn;
    f32x16 acc[MI][NJ];
    g1_mainloop<kElemBytes, NS, SH>(A, W, M, N, Kd, w, lds, acc);
    const int r32 = lane & 31;
    const int khalf = lane >> 5;

    // epilogue: the 32x32 accumulator layout (element v of lane l is row
    // 8*(v/4) + 4*(l/32) + v%4, column l%32 of its block) goes through LDS
    // (the operand buffers, free now) so that global stores are whole
    // 16-byte row chunks.  LDS rows hold OUT_ROW floats (the padding puts
    // the two 4-row halves of a store on disjoint banks).  Tiles too large
    // for that store each accumulator element directly: 32 lanes write 128
    // contiguous bytes of a row.
    if constexpr (!SH::LDS_EPI) {
        float* outd = P + (int64_t)split * M * N;
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const int gcol = tn * SH::BN + wn * 32 * NJ + j * 32 + r32;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int grow = tm * SH::BM + wm * 32 * MI + i * 32 + 8 * (v >> 2) +
                                     4 * khalf + (v & 3);
                    if (grow < M && gcol < N)
                        __builtin_nontemporal_store(acc[i][j][v], &outd[(int64_t)grow * N + gcol]);
                }
            }
        return;
    }
    __syncthreads();
    float* otile = (float*)&lds[0][0];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int col = wn * 32 * NJ + j * 32 + r32;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = wm * 32 * MI + i * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
                otile[row * SH::OUT_ROW + col] = acc[i][j][v];
            }
        }
    __syncthreads();
    float* out = P + (int64_t)split * M * N;
    constexpr int CH = SH::BM * SH::BN / 4;           // float4 chunks in the tile
#pragma unroll
    for (int it = 0; it < CH / SH::THREADS; ++it) {
        const int ch = it * SH::THREADS + tid;
        const int row = ch / (SH::BN / 4), c4 = ch % (SH::BN / 4);
        const int grow = tm * SH::BM + row, gcol = tn * SH::BN + c4 * 4;
        if (grow < M && gcol < N)                     // N % 4 == 0: chunks never straddle N
            // partials are written once and read once by the next kernel:
            // non-temporal stores stream them out instead of leaving them
            // dirty in L2 for the end-of-kernel writeback (measured: 15.8 ->
            // 12.8 us at 1024 x 512 x 4096 with four splits)
            __builtin_nontemporal_store(*(const f32x4*)&otile[row * SH::OUT_ROW + c4 * 4],
                                        (f32x4*)&out[(int64_t)grow * N + gcol]);
    }
}

template <int kElemBytes, int NS, class SH>
__global__ __launch_bounds__(SH::THREADS) void gemm1_splitk_kernel(
    const char* __restrict__ A, const char* __restrict__ W, float* __restrict__ P,
    int M, int N, int Kd, int splits, int tiles_n, int ktiles) {
    __shared__ __attribute__((aligned(16))) char lds[2][SH::LDS_A + SH::LDS_B];
    gemm1_tile<kElemBytes, NS, SH>(A, W, P, M, N, Kd, splits, tiles_n, ktiles, blockIdx.x,
                                   gridDim.x, lds);
}

// Launch of the split-K product with the plan's tile shape.
template <int NS, class SH>
static void launch_gemm_shape(const GemmPlan& g, bool bf16, const void* A, const void* W,
                              float* P, int M, int N, int K, hipStream_t stream) {
    const dim3 grid(g.tiles_m * g.tiles_n * g.splits);
    if (bf16)
        hipLaunchKernelGGL((gemm1_splitk_kernel<2, NS, SH>), grid, dim3(SH::THREADS), 0, stream,
                           (const char*)A, (const char*)W, P, M, N, K, g.splits, g.tiles_n,
                           g.ktiles);
    else
        hipLaunchKernelGGL((gemm1_splitk_kernel<4, NS, SH>), grid, dim3(SH::THREADS), 0, stream,
                           (const char*)A, (const char*)W, P, M, N, K, g.splits, g.tiles_n,
                           g.ktiles);
}

static hipError_t launch_gemm(const GemmPlan& g, bool bf16, const void* A, const void* W,
                              float* P, int M, int N, int K, hipStream_t stream) {
    switch (g.shape) {
        case GemmPlan::kBig:
            launch_gemm_shape<G1_STAGES_BIG, G1Big>(g, bf16, A, W, P, M, N, K, stream);
            break;
        case GemmPlan::kWide:
            launch_gemm_shape<G1_STAGES_WIDE, G1Wide>(g, bf16, A, W, P, M, N, K, stream);
            break;
        case GemmPlan::kHuge:
            launch_gemm_shape<G1_STAGES_HUGE, G1Huge>(g, bf16, A, W, P, M, N, K, stream);
            break;
        case GemmPlan::kMid:
            launch_gemm_shape<G1_STAGES_MID, G1Mid>(g, bf16, A, W, P, M, N, K, stream);
            break;
        default:
            launch_gemm_shape<G1_STAGES_SMALL, G1Small>(g, bf16, A, W, P, M, N, K, stream);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// head
// ---------------------------------------------------------------------------
// Rows per workgroup: 4, so that the split-K partial reads of a batch have
// plenty of workgroups in flight (large bf16 batches take head_tiled_kernel).
constexpr int HD_RB = 4;
constexpr int HD_THREADS = 256;
// float4 items per thread whose partial loads are in flight together: more
// when there are few split-K planes (registers hold kS x batch float4)
template <int kS> constexpr int hd_batch() { return kS == 1 ? 8 : kS == 2 ? 4 : 2; }
// W2 fragments (K-steps of 32) a wave loads at a time, the first group at
// kernel entry so that its latency overlaps the split-K reads.  A deep group
// costs registers: past two workgroups per CU (more than 512 of them) the
// shallow one, which keeps every workgroup resident, is faster (measured:
// 54.9 -> 50.8 us per call at 4096 rows with two planes; at 1024 rows the
// deep group is 0.2 us and for the regression head 1.2 us faster).
constexpr int HD_W2PF = 16;
constexpr int HD_W2PF_LOW = 2;
constexpr int HD_LOWREG_GROUPS = 512;

// GELU in its erf form, x Phi(x) with Phi the standard normal distribution
// function, without branches: h = Phi(-|x|) = erfc(|x| / sqrt 2) / 2 from the
// rational-times-Gaussian approximation of erfc in Abramowitz & Stegun 7.1.26
// (absolute error under 1.5e-7 in erf; in fp32 the result is within 1.5e-7
// max(1, |x|) of the exact GELU, twenty times below the rounding of the bf16
// hi/lo pair that carries activations into the next product), and
// x Phi(x) = x - x h for x >= 0, x h below.
__device__ inline float gelu_erf(float x) {
    const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, fabsf(x), 1.0f));
    // coefficients a5 .. a1 of 7.1.26, halved
    float q = fmaf(t, 0.5307027145f, -0.7265760135f);
    q = fmaf(t, q, 0.7107068705f);
    q = fmaf(t, q, -0.142248368f);
    q = fmaf(t, q, 0.127414796f);
    // exp(-x^2 / 2) = 2^(-x^2 / (2 ln 2))
    const float h = t * q * __builtin_amdgcn_exp2f(x * x * -0.72134752044448170f);
    const float xh = x * h;
    return x >= 0.0f ? x - xh : xh;
}

__device__ inline float apply_act(float x, int act) {
    if (act == STAR_ACT_RELU) return x > 0.0f ? x : 0.0f;
    return gelu_erf(x);
}

// kS = number of split-K partial planes (compile time, so that all of a
// thread's partial loads are issued before the first is consumed).
// kReg: the regression head's last two layers instead of the binned one
// (the nb "bin logits" are the third layer's outputs, `bins` holds w4 and
// phase 3 computes relu(z) . w4 + b4 in place of the softmax mean).
// The head over rows [blk HD_RB, (blk + 1) HD_RB), its buffers in `smem`
// (head_lds bytes).
template <bool kBF16, int kS, bool kReg, int kPF>
__device__ __forceinline__ void head_rows(
    const float* __restrict__ P, int B, int m, int nb, const float* __restrict__ b1,
    const void* __restrict__ w2, const float* __restrict__ b2, const float* __restrict__ bins,
    int act, float ema_alpha, int ema_init, float* __restrict__ ema_state,
    float* __restrict__ expected, int32_t* __restrict__ rem_len, int len_max, float b4, int blk,
    char* smem) {
    constexpr int kBatch = hd_batch<kS>();
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int row0 = blk * HD_RB;
    const int mpad = (m + 31) & ~31;
    const int astride = mpad + 8;                 // bf16 elements per LDS row
    const int nbpad = (nb + 15) & ~15;

    uint16_t* ahi = (uint16_t*)smem;
    uint16_t* alo = ahi + HD_RB * astride;
    float* a32 = (float*)smem;
    float* z = kBF16 ? (float*)(alo + HD_RB * astride) : (float*)(a32 + HD_RB * m);

    // 0) everything phases 2 and 3 read from global memory is requested now,
    //    so that its latency overlaps the split-K reads
    const int r16 = lane & 15;
    const int kq = lane >> 4;
    const int j0 = wid * 16 + r16;                // this lane's bin in the wave's first block
    bf16x8 wf0[kPF];
    if constexpr (kBF16) {
        const uint16_t* W2 = (const uint16_t*)w2;
        // Loads are unconditional (clamped indices) so none of them is waited
        // for before it is used.  An out-of-range fragment reads W2[0, 0..7]:
        // it only ever meets zero K-padding of a1 or lands in a column >= nb,
        // which is discarded.
#pragma unroll
        for (int u = 0; u < kPF; ++u) {
            const int k = u * 32 + kq * 8;
            const bool in = j0 < nb && k < m;
            wf0[u] = *(const bf16x8*)(W2 + (in ? (int64_t)j0 * m + k : 0));
        }
    }
    float binv[4];                                // used only where lane + 64 i < nb
#pragma unroll
    for (int i = 0; i < 4; ++i) binv[i] = bins[lane + 64 * i < nb ? lane + 64 * i : nb - 1];
    const float b2v = b2 ? b2[j0 < nb ? j0 : nb - 1] : 0.0f;
    const int my_row = row0 + wid;                // the row this wave finishes in phase 3
    const float ema_prev = (ema_alpha > 0.0f && !ema_init) ? ema_state[my_row < B ? my_row : B - 1] : 0.0f;

    // 1) fixed-order split-K reduction, bias, activation (float4 items)
    const int m4 = m >> 2;
    const int items = HD_RB * m4;
    const int64_t plane4 = (int64_t)B * m4;
    const float4* P4 = (const float4*)P;
    for (int base = 0; base < items; base += kBatch * HD_THREADS) {
        float4 v[kBatch][kS];
        float4 bv[kBatch];
        int row[kBatch], c4[kBatch];
        bool ok[kBatch];
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int e = base + i * HD_THREADS + tid;
            row[i] = e / m4;
            c4[i] = e - row[i] * m4;
            ok[i] = e < items && row0 + row[i] < B;
            const int64_t off = ok[i] ? (int64_t)(row0 + row[i]) * m4 + c4[i] : 0;
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                // read once: streamed past L2 (non-temporal), so they do not
                // evict the operands the next product reads
                const f32x4 t = __builtin_nontemporal_load((const f32x4*)&P4[q * plane4 + off]);
                v[i][q] = make_float4(t[0], t[1], t[2], t[3]);
            }
            bv[i] = b1 ? *(const float4*)(b1 + 4 * c4[i]) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            const int e = base + i * HD_THREADS + tid;
            if (e >= items) continue;
            float4 sum = v[i][0];
#pragma unroll
            for (int q = 1; q < kS; ++q) {
                sum.x += v[i][q].x; sum.y += v[i][q].y; sum.z += v[i][q].z; sum.w += v[i][q].w;
            }
            float a[4] = {sum.x + bv[i].x, sum.y + bv[i].y, sum.z + bv[i].z, sum.w + bv[i].w};
#pragma unroll
            for (int j = 0; j < 4; ++j) a[j] = ok[i] ? apply_act(a[j], act) : 0.0f;
            if constexpr (kBF16) {
                uint32_t h0, l0, h1, l1;
                split_bf16x2(a[0], a[1], h0, l0);
                split_bf16x2(a[2], a[3], h1, l1);
                const int o = row[i] * astride + 4 * c4[i];
                *(uint2*)(ahi + o) = make_uint2(h0, h1);
                *(uint2*)(alo + o) = make_uint2(l0, l1);
            } else {
                *(float4*)(a32 + row[i] * m + 4 * c4[i]) = make_float4(a[0], a[1], a[2], a[3]);
            }
        }
    }
    if constexpr (kBF16) {      // zero K padding [m, mpad)
        for (int e = tid; e < HD_RB * (mpad - m); e += HD_THREADS) {
            const int r = e / (mpad - m), u = m + e % (mpad - m);
            ahi[r * astride + u] = 0;
            alo[r * astride + u] = 0;
        }
    }
    __syncthreads();

    // 2) bin logits
    if constexpr (kBF16) {
        // v_mfma_f32_16x16x32_bf16: lane feeds row (lane%16), k = 8*(lane/16)..+7;
        // accumulator element v of lane l is row 4*(l/16)+v, column l%16.  Only
        // rows < HD_RB are real; the other A rows are fed as zeros.
        const uint16_t* W2 = (const uint16_t*)w2;
        const bool arow = r16 < HD_RB;
        for (int nblk = wid; nblk * 16 < nb; nblk += HD_THREADS / 64) {
            const int j = nblk * 16 + r16;
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            for (int kb = 0; kb < mpad; kb += 32 * kPF) {
                bf16x8 wf[kPF];
                if (nblk == wid && kb == 0) {
#pragma unroll
                    for (int u = 0; u < kPF; ++u) wf[u] = wf0[u];
                } else {
#pragma unroll
                    for (int u = 0; u < kPF; ++u) {
                        const int k = kb + u * 32 + kq * 8;
                        wf[u] = (j < nb && k < m) ? *(const bf16x8*)(W2 + (int64_t)j * m + k)
                                                  : bf16x8{0, 0, 0, 0, 0, 0, 0, 0};
                    }
                }
                // all of this chunk's a1 fragments are read from LDS first, so
                // their latencies overlap; rows >= HD_RB read row 0 and are
                // zeroed afterwards (their MFMA rows are discarded anyway)
                bf16x8 hv[kPF], lv[kPF];
                const int arow_off = (arow ? r16 : 0) * astride;
#pragma unroll
                for (int u = 0; u < kPF; ++u) {
                    const int k = (kb + u * 32 < mpad ? kb + u * 32 : 0) + kq * 8;
                    hv[u] = *(const bf16x8*)(ahi + arow_off + k);
                    lv[u] = *(const bf16x8*)(alo + arow_off + k);
                }
                const bf16x8 zero8 = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
                for (int u = 0; u < kPF; ++u) {
                    if (kb + u * 32 >= mpad) break;          // uniform: mpad % 32 == 0
                    const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, wf[u]);
                    const bf16x8 h = arow ? hv[u] : zero8;
                    const bf16x8 l = arow ? lv[u] : zero8;
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, h), bv, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, l), bv, acc, 0, 0, 0);
                }
            }
            const int col = nblk * 16 + r16;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 4 * kq + v;
                const float bias = nblk == wid ? b2v : (b2 && col < nb ? b2[col] : 0.0f);
                if (row < HD_RB && col < nb) z[row * nbpad + col] = acc[v] + bias;
            }
        }
    } else {
        const float* W2 = (const float*)w2;
        for (int e = tid; e < HD_RB * nb; e += HD_THREADS) {
            const int r = e / nb, j = e % nb;
            // m % 4 == 0 and 16-byte aligned rows: float4 reads, the same
            // sequential fma chain
            const float4* wrow = (const float4*)(W2 + (int64_t)j * m);
            const float4* arow = (const float4*)(a32 + r * m);
            float s = 0.0f;
            for (int u = 0; u < (m >> 2); ++u) {
                const float4 a = arow[u], w = wrow[u];
                s = fmaf(a.x, w.x, s);
                s = fmaf(a.y, w.y, s);
                s = fmaf(a.z, w.z, s);
                s = fmaf(a.w, w.w, s);
            }
            z[r * nbpad + j] = s + (b2 ? b2[j] : 0.0f);
        }
    }
    __syncthreads();

    // 3) softmax, expectation, EMA, integerisation: one wave per row
    for (int r = wid; r < HD_RB; r += HD_THREADS / 64) {
        const int gr = row0 + r;
        if (gr >= B) continue;
        float den = 1.0f, num = 0.0f;
        if constexpr (kReg) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = lane + 64 * i;
                if (j < nb) num += fmaxf(z[r * nbpad + j], 0.0f) * binv[i];
            }
            num = wave_sum_f32(num) + b4;
        } else {
            float zmax = -INFINITY;
            for (int j = lane; j < nb; j += 64) zmax = fmaxf(zmax, z[r * nbpad + j]);
            zmax = wave_max_f32(zmax);
            den = 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = lane + 64 * i;
                if (j < nb) {
                    const float e = expf(z[r * nbpad + j] - zmax);
                    den += e;
                    num += e * binv[i];
                }
            }
            den = wave_sum_f32(den);
            num = wave_sum_f32(num);
        }
        if (lane == 0) {
            const float E = kReg ? num : num / den;
            expected[gr] = E;
            float y = E;
            if (ema_alpha > 0.0f) {
                const float prev = r == wid ? ema_prev : ema_state[gr];
                y = ema_init ? E : ema_alpha * E + (1.0f - ema_alpha) * prev;
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

template <bool kBF16, int kS, bool kReg = false, int kPF = HD_W2PF>
__global__ __launch_bounds__(HD_THREADS) void head_kernel(
    const float* __restrict__ P, int B, int m, int nb, const float* __restrict__ b1,
    const void* __restrict__ w2, const float* __restrict__ b2, const float* __restrict__ bins,
    int act, float ema_alpha, int ema_init, float* __restrict__ ema_state,
    float* __restrict__ expected, int32_t* __restrict__ rem_len, int len_max, float b4 = 0.0f) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    head_rows<kBF16, kS, kReg, kPF>(P, B, m, nb, b1, w2, b2, bins, act, ema_alpha, ema_init,
                                    ema_state, expected, rem_len, len_max, b4, blockIdx.x, smem);
}

// ---------------------------------------------------------------------------
// The head for large bf16 batches, K-chunked: 64 rows per workgroup of eight
// waves.  Wave w takes the 16 rows of group w % 4 and the 32-wide half w / 4
// of every chunk of 64 a1 columns.  Each lane loads from HBM exactly the 8
// partials that it feeds to the 16x16x32 MFMA as its A operand (row
// lane % 16 of the group, columns 8 (lane / 16) + 0..7 of the half), reduces
// the planes in a fixed order, adds b1 (staged in LDS once), applies the
// activation and splits the result into the bf16 hi/lo pair in registers:
// a1 never passes through LDS and every activation is computed once.  W2's
// chunk, the B operand the four row groups share, is staged in LDS in two
// stages with one barrier per chunk.  The two halves' logits are summed once
// at the end (lower half first), and the softmax runs on the logits in
// registers: a row's bins are spread over 16 lanes, plus registers.
// W2 is read once per 64 rows (the 4-row head reads it once per 4).
// ---------------------------------------------------------------------------
constexpr int HT_ROWS = 64;
constexpr int HT_KC = 64;                   // a1 columns per chunk
constexpr int HT_ASTR = HT_KC + 8;          // bf16 per LDS row of W2 (padding spreads banks)
constexpr int HT_THREADS = 512;             // 4 row groups x 2 halves of each chunk
constexpr int HT_MIN_REQ = 8192;            // batches from which the tiled head is used
constexpr int HT_MAX_SPLITS = 4;            // its partial registers: 2 float4 per plane

// bin blocks of 16 the tiled head computes: 4, 8 or 16 (compile time, so that
// every loop over them has a fixed trip count; blocks past nb carry zeros)
static int head_tiled_blocks(int nb) { return nb <= 64 ? 4 : nb <= 128 ? 8 : 16; }
// two W2 stages, then b1 (m fp32); the halves' logits meet in the stages
constexpr size_t head_tiled_stage_bytes(int nbb) { return (size_t)nbb * 16 * HT_ASTR * 2; }
static size_t head_tiled_lds(int nb, int m) {
    return 2 * head_tiled_stage_bytes(head_tiled_blocks(nb)) + (size_t)m * 4;
}

struct HtArgs {
    const float4* P4;
    const uint16_t* W2;
    int64_t plane4;
    int B, m, m4, nb;
};

// a lane's 8 partials of one chunk, per plane
template <int kS>
struct HtP {
    float4 v[kS][2];
};
// the thread's 16-byte pieces of a W2 chunk (kNBB x 16 bins x 8 pieces over
// the workgroup)
template <int kNBB>
struct HtW {
    static constexpr int kU = kNBB * 16 * 8 / HT_THREADS;
    static_assert(kU >= 1 && kU * HT_THREADS == kNBB * 128, "whole W2 pieces per thread");
    uint4 v[kU];
};

// partials of row `row`, columns k .. k + 7 (m % 8 == 0: all in range or
// none); rows past B and columns past m read offset 0 and are masked later
template <int kS>
__device__ __forceinline__ void ht_load_p(const HtArgs& a, int row, int k, HtP<kS>& g) {
    const bool ok = row < a.B && k < a.m;
    const int64_t off = ok ? (int64_t)row * a.m4 + (k >> 2) : 0;
#pragma unroll
    for (int q = 0; q < kS; ++q) {
        const f32x4 t0 = __builtin_nontemporal_load((const f32x4*)&a.P4[q * a.plane4 + off]);
        const f32x4 t1 = __builtin_nontemporal_load((const f32x4*)&a.P4[q * a.plane4 + off + 1]);
        g.v[q][0] = make_float4(t0[0], t0[1], t0[2], t0[3]);
        g.v[q][1] = make_float4(t1[0], t1[1], t1[2], t1[3]);
    }
}

template <int kNBB>
__device__ __forceinline__ void ht_load_w(const HtArgs& a, int c, HtW<kNBB>& g) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < HtW<kNBB>::kU; ++u) {
        const int it = u * HT_THREADS + tid;
        const int j = it >> 3, kk = c * HT_KC + (it & 7) * 8;
        const bool ok = j < a.nb && kk < a.m;
        g.v[u] = *(const uint4*)(a.W2 + (ok ? (int64_t)j * a.m + kk : 0));
    }
}

template <int kNBB>
__device__ __forceinline__ void ht_store_w(const HtArgs& a, int c, const HtW<kNBB>& g,
                                           uint16_t* wl) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < HtW<kNBB>::kU; ++u) {
        const int it = u * HT_THREADS + tid;       // row j < kNBB x 16 of the W2 chunk
        const int j = it >> 3, kk = c * HT_KC + (it & 7) * 8;
        const uint32_t z = (j < a.nb && kk < a.m) ? 0xFFFFFFFFu : 0u;
        *(uint4*)(wl + j * HT_ASTR + (it & 7) * 8) =
            make_uint4(g.v[u].x & z, g.v[u].y & z, g.v[u].z & z, g.v[u].w & z);
    }
}

// a1 = act(sum of the planes + b1) for the lane's 8 columns as the bf16
// hi/lo pair (zeros outside the batch and past m)
template <int kS, bool kGelu>
__device__ __forceinline__ void ht_act(const HtP<kS>& g, const float* b1s, int k, bool ok,
                                       bf16x8& hi, bf16x8& lo) {
    float4 s0 = g.v[0][0], s1 = g.v[0][1];
#pragma unroll
    for (int q = 1; q < kS; ++q) {
        s0.x += g.v[q][0].x; s0.y += g.v[q][0].y; s0.z += g.v[q][0].z; s0.w += g.v[q][0].w;
        s1.x += g.v[q][1].x; s1.y += g.v[q][1].y; s1.z += g.v[q][1].z; s1.w += g.v[q][1].w;
    }
    const float4 c0 = *(const float4*)(b1s + (ok ? k : 0));
    const float4 c1 = *(const float4*)(b1s + (ok ? k : 0) + 4);
    const float av[8] = {s0.x + c0.x, s0.y + c0.y, s0.z + c0.z, s0.w + c0.w,
                         s1.x + c1.x, s1.y + c1.y, s1.z + c1.z, s1.w + c1.w};
    uint32_t hw[4], lw[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float y0 = av[2 * e], y1 = av[2 * e + 1];
        const float g0 = kGelu ? gelu_erf(y0) : fmaxf(y0, 0.0f);
        const float g1 = kGelu ? gelu_erf(y1) : fmaxf(y1, 0.0f);
        split_bf16x2(ok ? g0 : 0.0f, ok ? g1 : 0.0f, hw[e], lw[e]);
    }
    hi = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
    lo = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
}

// up to 128 bins and two planes, two workgroups per CU (four waves per
// SIMD, at most 128 VGPRs)
template <int kS, int kNBB, bool kGelu>
__global__ __launch_bounds__(HT_THREADS)
__attribute__((amdgpu_waves_per_eu(kNBB <= 8 && kS <= 2 ? 4 : 1))) void head_tiled_kernel(
    const float* __restrict__ P, int B, int m, int nb, const float* __restrict__ b1,
    const uint16_t* __restrict__ W2, const float* __restrict__ b2,
    const float* __restrict__ bins, float ema_alpha, int ema_init,
    float* __restrict__ ema_state, float* __restrict__ expected, int32_t* __restrict__ rem_len,
    int len_max) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int row0 = blockIdx.x * HT_ROWS;
    constexpr int kStage = (int)(head_tiled_stage_bytes(kNBB) / 2);   // bf16 per stage
    uint16_t* const st0 = (uint16_t*)smem;
    uint16_t* const st1 = st0 + kStage;
    float* const b1s = (float*)(st1 + kStage);
    HtArgs a;
    a.P4 = (const float4*)P;
    a.W2 = W2;
    a.m = m;
    a.m4 = m >> 2;
    a.B = B;
    a.plane4 = (int64_t)B * a.m4;
    a.nb = nb;
    const int nchunk = (m + HT_KC - 1) / HT_KC;
    // wave wid: rows of group rg, K half kh of every chunk
    const int rg = wid & 3;
    const int kh = wid >> 2;
    const int row = row0 + rg * 16 + (lane & 15);   // the lane's A row (MFMA row lane % 16)
    const int kofs = kh * 32 + (lane >> 4) * 8;     // its 8 columns within a chunk
    const bool row_ok = row < B;

    f32x4 acc[kNBB];
#pragma unroll
    for (int j = 0; j < kNBB; ++j) acc[j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

    // the products of one chunk: the lane's A pair x kNBB bin blocks of W2
    auto products = [&](const uint16_t* wl, const bf16x8& h, const bf16x8& l) {
        // per group of 4 blocks, the hi products, then the lo ones:
        // consecutive MFMAs are independent
        constexpr int kG = kNBB < 4 ? kNBB : 4;
#pragma unroll
        for (int j0 = 0; j0 < kNBB; j0 += kG) {
            bf16x8_t wb[kG];
#pragma unroll
            for (int j = 0; j < kG; ++j)
                wb[j] = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(wl + ((j0 + j) * 16 + (lane & 15)) * HT_ASTR + kofs));
#pragma unroll
            for (int j = 0; j < kG; ++j)
                acc[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, h), wb[j], acc[j0 + j], 0, 0, 0);
#pragma unroll
            for (int j = 0; j < kG; ++j)
                acc[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, l), wb[j], acc[j0 + j], 0, 0, 0);
        }
    };

    // The partials and W2's chunks are loaded one chunk ahead (chunk c + 1's
    // partials are requested once chunk c is activated).  Loads complete in
    // issue order for the wait counter, so in each step W2, needed sooner,
    // is requested before the partials.
    // workgroups start at different chunks (block index mod chunks), so that
    // at any time the chip reads every column range of the partial rows, not
    // one 256-byte range of all of them (measured at 32768 x 1024 x 128: 48.9
    // against 51.9 us); the chunks' order in each row's sums changes with it
    const int rot = (int)(blockIdx.x % (unsigned)nchunk);
    auto chunk = [&](int c) { return c + rot < nchunk ? c + rot : c + rot - nchunk; };
    HtP<kS> p0;
    HtW<kNBB> w;
    ht_load_w(a, chunk(0), w);
    ht_load_p(a, row, chunk(0) * HT_KC + kofs, p0);
    for (int i = tid; i < m; i += HT_THREADS) b1s[i] = b1 ? b1[i] : 0.0f;
    ht_store_w(a, chunk(0), w, st0);
    if (nchunk > 1) ht_load_w(a, chunk(1), w);
    __syncthreads();

    // step c: activate chunk c and request chunk c + 1's partials, chunk c's
    // products on stage c % 2, W2 of chunk c + 1 into the other stage (last
    // read before the previous barrier)
    int c = 0;
    for (;; ++c) {
        const int k = chunk(c) * HT_KC + kofs;
        bf16x8 h, l;
        ht_act<kS, kGelu>(p0, b1s, k, row_ok && k < m, h, l);
        if (c + 1 < nchunk) ht_load_p(a, row, chunk(c + 1) * HT_KC + kofs, p0);
        products((c & 1) ? st1 : st0, h, l);
        if (c + 1 == nchunk) break;
        ht_store_w(a, chunk(c + 1), w, (c & 1) ? st0 : st1);
        if (c + 2 < nchunk) ht_load_w(a, chunk(c + 2), w);
        __syncthreads();
    }

    // the upper K half's logits join the lower half's, in that order, through
    // the stages (kNBB x 4 KiB; two stages hold kNBB x 4.5 KiB)
    {
        static_assert(4 * kNBB * 64 * 16 <= 2 * kStage * 2, "exchange fits the stages");
        f32x4* const xs = (f32x4*)smem;
        __syncthreads();                        // every wave's last products are done
        if (kh == 1) {
#pragma unroll
            for (int j = 0; j < kNBB; ++j) xs[(rg * kNBB + j) * 64 + lane] = acc[j];
        }
        __syncthreads();
        if (kh == 1) return;                    // no barrier follows
#pragma unroll
        for (int j = 0; j < kNBB; ++j) {
            const f32x4 o = xs[(rg * kNBB + j) * 64 + lane];
#pragma unroll
            for (int v = 0; v < 4; ++v) acc[j][v] += o[v];
        }
    }

    // softmax over the bins: element v of acc[j] is row 4 (lane / 16) + v of
    // the wave's 16, bin 16 j + lane % 16
    // logits with b2; absent bins (past nb) become -inf
    // and their bin values 0, so that the loops below need no conditions
    float bvl[kNBB];
#pragma unroll
    for (int j = 0; j < kNBB; ++j) {
        const int col = j * 16 + (lane & 15);
        const bool ok = col < nb;
        const int cc = ok ? col : 0;
        bvl[j] = ok ? bins[cc] : 0.0f;
        const float bias = b2 ? b2[cc] : 0.0f;
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[j][v] = ok ? acc[j][v] + bias : -INFINITY;
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < kNBB; ++j) mx = fmaxf(mx, acc[j][v]);
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 16));
        float den = 0.0f, num = 0.0f;
#pragma unroll
        for (int j = 0; j < kNBB; ++j) {
            const float e = expf(acc[j][v] - mx);      // exp(-inf) = 0 for absent bins
            den += e;
            num += e * bvl[j];
        }
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) {
            den += __shfl_xor(den, o, 16);
            num += __shfl_xor(num, o, 16);
        }
        const int gr = row0 + rg * 16 + 4 * (lane >> 4) + v;
        if ((lane & 15) == 0 && gr < B) {
            const float E = num / den;
            expected[gr] = E;
            float y = E;
            if (ema_alpha > 0.0f) {
                y = ema_init ? E : ema_alpha * E + (1.0f - ema_alpha) * ema_state[gr];
                ema_state[gr] = y;
            }
            if (rem_len) {
                const float q = rintf(y);
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
// The whole binned head in one kernel (bf16), for products that take one
// K-slice (no split-K): first product, bias, activation, second product,
// softmax, expectation, EMA and integerisation.
//
// Every workgroup computes one BM x BN tile of z1 = H W1^T over all of K,
// adds b1 and applies the activation.  The second product is linear in a1's
// columns, so the workgroup then multiplies its BN columns of a1 with the
// same BN columns of W2: the tile's share of every bin logit of its BM rows.
// The column tiles of a row block meet through a counter; the last to
// arrive sums the shares in column order (the same fixed order whatever the
// arrival order) and finishes its rows: b2, softmax over the bins, mean over
// the bin values, EMA, round half to even, clamp.  z1 never leaves the chip.
//
// The shares meet through the cache-maintenance-free exchange of the common
// header (device-coherent stores and loads, a counter per row block).
//
// Products that need a K-split take the two-kernel path instead (split-K
// product, then the head kernel): meeting the K-slices in this kernel as
// well put two exchanges and the whole head of the last tile on one
// workgroup's critical path, which measured slower than the kernel boundary.
// ---------------------------------------------------------------------------
constexpr int FU_NB_MAX = 128;            // bins of the fused head (its logits fit the LDS)
constexpr int FU_NBP = FU_NB_MAX + 4;     // fp32 per LDS row of logits (banks spread by rows)
constexpr int FU_MAX_TICKETS = kMaxTickets;

__device__ inline void fu_store(f32x4 v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
    xch_store(__builtin_bit_cast(u32x4, v), r, off);
}
__device__ inline f32x4 fu_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(f32x4, xch_load(r, off));
}

__device__ inline f32x4 fu_chunk(const f32x16& a, int q) {
    return f32x4{a[4 * q], a[4 * q + 1], a[4 * q + 2], a[4 * q + 3]};
}

struct FusedArgs {
    const char* A;            // hidden [M, Kd] bf16
    const char* W;            // w1 [N, Kd] bf16
    const float* b1;          // [N] or null
    const uint16_t* W2;       // [nb, N] bf16
    const float* b2;          // [nb] or null
    const float* bins;        // [nb]
    float* lpart;             // logit shares: [tiles_m][tiles_n][blocks][1024] (tiles_n > 1)
    uint32_t* tix_row;        // [tiles_m]
    float* ema_state;
    float* expected;
    int32_t* rem_len;
    int M, N, Kd, nb, tiles_n, ktiles, act, ema_init, len_max;
    float ema_alpha;
};

template <int NS, class SH>
__global__ __launch_bounds__(SH::THREADS) void predict_fused_kernel(FusedArgs a) {
    constexpr int MI = SH::MI, NJ = SH::NJ, T = SH::THREADS, NW = T / 64;
    constexpr int BM = SH::BM, BN = SH::BN;
    constexpr int ZST = BN * 4 + 16;             // bytes per LDS row of the z1 / a1 tile
    constexpr int C8 = BN / 8;                   // 8-column chunks per row
    static_assert(T % C8 == 0, "a thread keeps its chunk column");
    constexpr int NBI = BM / 32;                 // row blocks of the logit product
    constexpr int MAXB = (NBI * (FU_NB_MAX / 32) + NW - 1) / NW;   // logit blocks per wave
    constexpr int LPR = T / BM;                  // lanes per row in the softmax
    static_assert(LPR >= 1 && (LPR & (LPR - 1)) == 0 && LPR <= 64, "lanes per row");
    // the operand buffers of the main loop, reused for the z1 / a1 tile and
    // then the logits
    constexpr int kMainBytes = 2 * (SH::LDS_A + SH::LDS_B);
    constexpr int kLogitBytes = (BM * FU_NBP + 2 * FU_NB_MAX) * 4;   // logits, bin values, b2
    constexpr int kTileBytes = BM * ZST;
    constexpr int kEpiBytes = kLogitBytes > kTileBytes ? kLogitBytes : kTileBytes;
    __shared__ __attribute__((aligned(16))) char lds_raw[kMainBytes > kEpiBytes ? kMainBytes : kEpiBytes];
    auto lds = reinterpret_cast<char (*)[SH::LDS_A + SH::LDS_B]>(lds_raw);
    __shared__ uint32_t s_ticket;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wid = tid >> 6;
    const int wm = wid / SH::WN, wn = wid % SH::WN;
    const int r32 = lane & 31;
    const int khalf = lane >> 5;
    const G1Work w = g1_work(1, a.tiles_n, a.ktiles, blockIdx.x, gridDim.x);
    f32x16 acc[MI][NJ];
    g1_mainloop<2, NS, SH>(a.A, a.W, a.M, a.N, a.Kd, w, lds, acc);

    // The head's global reads (W2 fragments, b1, b2, bin values, EMA state)
    // are all requested at once: one memory latency instead of one per use.
    const int nbj = (a.nb + 31) >> 5;
    const int nblk = NBI * nbj;
    bf16x8 wf[MAXB][BN / 16];
    f32x4 b1v[2];                                 // b1 of this thread's 8-column chunk
    float binv, b2v, ema_prev;
    const int c8 = tid % C8;
    const int r = tid / LPR, sub = tid % LPR;     // the row this thread finishes in 5)
    const int gr = w.tm * BM + r;
    auto prefetch = [&]() {
#pragma unroll
        for (int u = 0; u < MAXB; ++u) {
            const int blk = wid + u * NW;
            const int jrow = (blk / NBI) * 32 + r32;
#pragma unroll
            for (int ks = 0; ks < BN / 16; ++ks) {
                // clamped, unconditional; m % 8 == 0, so a chunk is wholly in or out
                const int c = w.tn * BN + ks * 16 + 8 * khalf;
                const bool ok = blk < nblk && jrow < a.nb && c < a.N;
                const bf16x8 t = *(const bf16x8*)(a.W2 + (ok ? (int64_t)jrow * a.N + c : 0));
                wf[u][ks] = t & (ok ? (short)-1 : (short)0);
            }
        }
        {
            // m % 8 == 0: the chunk is wholly in or out; b1 is 16-byte aligned
            const int gcol = w.tn * BN + c8 * 8;
            b1v[0] = b1v[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            if (a.b1 && gcol < a.N) {
                b1v[0] = *(const f32x4*)(a.b1 + gcol);
                b1v[1] = *(const f32x4*)(a.b1 + gcol + 4);
            }
        }
        const int jb = tid < a.nb ? tid : 0;
        binv = tid < a.nb ? a.bins[jb] : 0.0f;
        b2v = (a.b2 && tid < a.nb) ? a.b2[jb] : 0.0f;
        ema_prev = (a.ema_alpha > 0.0f && !a.ema_init) ? a.ema_state[gr < a.M ? gr : a.M - 1] : 0.0f;
    };

    prefetch();
    __syncthreads();                         // the last products have read the LDS

    // 1) z1 into LDS rows [BM][ZST bytes] (fp32); then, a chunk of 8 columns
    //    at a time, bias and activation, written back in place as the bf16
    //    pair [hi x 8 | lo x 8].  Element v of lane l of a 32 x 32 block is
    //    row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32.
    char* zt = lds_raw;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const int col = wn * 32 * NJ + j * 32 + r32;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int row = wm * 32 * MI + i * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
                *(float*)(zt + row * ZST + col * 4) = acc[i][j][v];
            }
        }
    __syncthreads();
    {
        const bool cok = w.tn * BN + c8 * 8 < a.N;
#pragma unroll 1
        for (int e = tid; e < BM * C8; e += T) {
            char* pz = zt + (e / C8) * ZST + c8 * 32;
            const f32x4 z0 = *(const f32x4*)pz, z1 = *(const f32x4*)(pz + 16);
            float x[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                x[k] = cok ? apply_act(z0[k] + b1v[0][k], a.act) : 0.0f;
                x[k + 4] = cok ? apply_act(z1[k] + b1v[1][k], a.act) : 0.0f;
            }
            uint32_t hi[4], lo[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) split_bf16x2(x[2 * k], x[2 * k + 1], hi[k], lo[k]);
            *(uint4*)pz = make_uint4(hi[0], hi[1], hi[2], hi[3]);
            *(uint4*)(pz + 16) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        }
    }
    __syncthreads();

    // 2) this tile's share of the bin logits, [BM rows] x [bins] over its BN
    //    columns: v_mfma_f32_32x32x16_bf16 with A = a1 rows (hi, then lo) and
    //    B = W2 rows.  Wave wid takes the blocks wid, wid + NW, ...
    f32x16 lg[MAXB];
#pragma unroll
    for (int u = 0; u < MAXB; ++u) {
#pragma unroll
        for (int e = 0; e < 16; ++e) lg[u][e] = 0.0f;
        const int blk = wid + u * NW;
        if (blk < nblk) {
            const int ib = blk % NBI;
#pragma unroll
            for (int ks = 0; ks < BN / 16; ++ks) {
                const char* pa = zt + (ib * 32 + r32) * ZST + (2 * ks + khalf) * 32;
                const bf16x8_t h = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)pa);
                const bf16x8_t l = __builtin_bit_cast(bf16x8_t, *(const bf16x8*)(pa + 16));
                const bf16x8_t b = __builtin_bit_cast(bf16x8_t, wf[u][ks]);
                lg[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(h, b, lg[u], 0, 0, 0);
                lg[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(l, b, lg[u], 0, 0, 0);
            }
        }
    }

    // 3) the column tiles of the row block meet; the last to arrive sums the
    //    shares in column order (share layout: float4 q of lane l of block
    //    blk at (blk 4 + q) 64 + l).  It reads its own share back too (its
    //    stores have completed), so every load is unconditional; tiles past
    //    the last read 0 (an offset past the buffer); the sum starts at -0,
    //    which adds exactly.
    if (a.tiles_n > 1) {
        const uint32_t share = (uint32_t)nblk * 1024u;            // floats per share
        const __amdgpu_buffer_rsrc_t rl =
            xch_rsrc(a.lpart + (size_t)w.tm * a.tiles_n * share, (uint32_t)a.tiles_n * share * 4u);
#pragma unroll
        for (int u = 0; u < MAXB; ++u) {
            const int blk = wid + u * NW;
            if (blk < nblk)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    fu_store(fu_chunk(lg[u], q), rl,
                             (uint32_t)w.tn * share * 4u + (uint32_t)((blk * 4 + q) * 64 + lane) * 16u);
        }
        xch_wait_stores();
        if (!xch_last_arrival(&a.tix_row[w.tm], (uint32_t)a.tiles_n, &s_ticket)) return;
        constexpr int G = 8;                  // shares loaded together
#pragma unroll
        for (int u = 0; u < MAXB; ++u) {
            const int blk = wid + u * NW;
            if (blk >= nblk) continue;
            f32x4 sum[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) sum[q] = f32x4{-0.0f, -0.0f, -0.0f, -0.0f};
#pragma unroll 1
            for (int t0 = 0; t0 < a.tiles_n; t0 += G) {
                f32x4 v[G][4];
#pragma unroll
                for (int g = 0; g < G; ++g)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int t = t0 + g;
                        const uint32_t off = (uint32_t)t * share * 4u +
                                             (uint32_t)((blk * 4 + q) * 64 + lane) * 16u;
                        v[g][q] = fu_load(rl, t < a.tiles_n ? off : kXchOob);
                    }
#pragma unroll
                for (int g = 0; g < G; ++g)
#pragma unroll
                    for (int q = 0; q < 4; ++q) sum[q] += v[g][q];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int e = 0; e < 4; ++e) lg[u][4 * q + e] = sum[q][e];
        }
    }

    // 4) logits into LDS rows [BM][FU_NBP], the bin values and b2 beside
    //    them; then LPR lanes per row: + b2, softmax, mean over the bin
    //    values, EMA, integerisation
    __syncthreads();                          // every wave has read a1 from LDS
    float* zl = (float*)&lds[0][0];
    float* sbin = zl + BM * FU_NBP;           // [FU_NB_MAX] bin values, then [FU_NB_MAX] b2
    if (tid < FU_NB_MAX) {
        sbin[tid] = binv;
        sbin[FU_NB_MAX + tid] = b2v;
    }
#pragma unroll
    for (int u = 0; u < MAXB; ++u) {
        const int blk = wid + u * NW;
        if (blk >= nblk) continue;
        const int ib = blk % NBI, jb = blk / NBI;
        const int j = jb * 32 + r32;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int row = ib * 32 + 8 * (v >> 2) + 4 * khalf + (v & 3);
            zl[row * FU_NBP + j] = lg[u][v];
        }
    }
    __syncthreads();
    const float* zr = zl + r * FU_NBP;
    float zmax = -INFINITY;
#pragma unroll 4
    for (int j = sub; j < a.nb; j += LPR) zmax = fmaxf(zmax, zr[j] + sbin[FU_NB_MAX + j]);
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) zmax = fmaxf(zmax, __shfl_xor(zmax, o, LPR));
    float den = 0.0f, num = 0.0f;
#pragma unroll 4
    for (int j = sub; j < a.nb; j += LPR) {
        const float e = expf(zr[j] + sbin[FU_NB_MAX + j] - zmax);
        den += e;
        num += e * sbin[j];
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) {
        den += __shfl_xor(den, o, LPR);
        num += __shfl_xor(num, o, LPR);
    }
    if (sub == 0 && gr < a.M) {
        const float E = num / den;
        a.expected[gr] = E;
        float y = E;
        if (a.ema_alpha > 0.0f) {
            y = a.ema_init ? E : a.ema_alpha * E + (1.0f - a.ema_alpha) * ema_prev;
            a.ema_state[gr] = y;
        }
        if (a.rem_len) {
            const float q = rintf(y);
            int32_t li;
            if (!(q >= 1.0f)) li = 1;
            else if (q >= (float)a.len_max) li = a.len_max;
            else li = (int32_t)q;
            a.rem_len[gr] = li;
        }
    }
}

// ---------------------------------------------------------------------------
// (f3) between the regression head's first two layers: fixed-order split-K
// reduction, bias, ReLU, and the operand of the next product (bf16, round
// to nearest even, or fp32)
// ---------------------------------------------------------------------------
constexpr int ACT_THREADS = 256;
constexpr int ACT_BATCH = 4;      // float4 items per thread in flight

template <int kS, bool kBF16>
__global__ __launch_bounds__(ACT_THREADS) void act_kernel(const float* __restrict__ P,
                                                          int64_t items, int m4,
                                                          const float* __restrict__ bias,
                                                          void* __restrict__ out) {
    const float4* P4 = (const float4*)P;
    for (int64_t base = (int64_t)blockIdx.x * ACT_THREADS * ACT_BATCH; base < items;
         base += (int64_t)gridDim.x * ACT_THREADS * ACT_BATCH) {
        float4 v[ACT_BATCH][kS];
#pragma unroll
        for (int i = 0; i < ACT_BATCH; ++i) {
            const int64_t e = base + i * ACT_THREADS + threadIdx.x;
            const int64_t o = e < items ? e : 0;
#pragma unroll
            for (int q = 0; q < kS; ++q) {
                const f32x4 t = __builtin_nontemporal_load((const f32x4*)&P4[q * items + o]);
                v[i][q] = make_float4(t[0], t[1], t[2], t[3]);
            }
        }
#pragma unroll
        for (int i = 0; i < ACT_BATCH; ++i) {
            const int64_t e = base + i * ACT_THREADS + threadIdx.x;
            if (e >= items) break;
            float4 sum = v[i][0];
#pragma unroll
            for (int q = 1; q < kS; ++q) {
                sum.x += v[i][q].x; sum.y += v[i][q].y; sum.z += v[i][q].z; sum.w += v[i][q].w;
            }
            const int c = (int)(e % m4) * 4;
            const float4 bv = bias ? *(const float4*)(bias + c) : make_float4(0.f, 0.f, 0.f, 0.f);
            const float a0 = fmaxf(sum.x + bv.x, 0.0f), a1 = fmaxf(sum.y + bv.y, 0.0f);
            const float a2 = fmaxf(sum.z + bv.z, 0.0f), a3 = fmaxf(sum.w + bv.w, 0.0f);
            if constexpr (kBF16) {
                ((uint2*)out)[e] = make_uint2(pack_bf16x2_rne(a0, a1), pack_bf16x2_rne(a2, a3));
            } else {
                ((float4*)out)[e] = make_float4(a0, a1, a2, a3);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
// Tiles and split-K factor of one product [M, K] x [N, K]^T.  For each tile
// shape the split is a power of two in [1, 16] that brings the workgroups
// near one per CU (128 x 128, 128 x 64) or two per CU (64 x 64).  The shape
// is chosen by a cost model of its two data streams: operand rows read into
// the CUs (every A row once per column of tiles, every W row once per row of
// tiles) at the L2's aggregate ~17 TB/s,
// and the fp32 split-K partials written, flushed out of L2 at the end of
// the kernel and read back at ~2.4 TB/s (both rates measured on MI355X).
GemmPlan plan_gemm(int M, int N, int K, int elem) {
    GemmPlan best;
    double best_cost = 0.0;
    const int bk = G1_KBYTES / elem;
    struct Cand { int shape, bm, bn, slots; };
    const Cand cands[3] = {{GemmPlan::kBig, G1Big::BM, G1Big::BN, 256},
                           {GemmPlan::kSmall, G1Small::BM, G1Small::BN, 512},
                           {GemmPlan::kMid, G1Mid::BM, G1Mid::BN, 256}};
    for (int ci = 0; ci < 3; ++ci) {
        if (cands[ci].shape == GemmPlan::kMid && M > G1Mid::BM) continue;
        GemmPlan g;
        g.shape = cands[ci].shape;
        const int bm = cands[ci].bm, bn = cands[ci].bn;
        g.tiles_m = (int)ceil_div(M, bm);
        g.tiles_n = (int)ceil_div(N, bn);
        g.ktiles = (int)ceil_div(K, bk);
        const int tiles = g.tiles_m * g.tiles_n;
        int s = 1;
        const int slots = cands[ci].slots;
        if (tiles > 0 && tiles < 3 * slots / 4) {
            int want = slots / tiles;
            if (want > 16) want = 16;
            if (want > g.ktiles / 2) want = g.ktiles / 2;
            while (s * 2 <= want) s *= 2;
        }
        g.splits = s;
        const double operands = ((double)g.tiles_n * M + (double)g.tiles_m * N) * K * elem;
        const double partials = (double)s * M * N * 4.0;
        const double cost = operands / 17e12 + 2.0 * partials / 2.4e12;
        if (ci == 0 || cost < best_cost) {
            best = g;
            best_cost = cost;
        }
    }
    if (best.shape == GemmPlan::kBig && best.splits == 1) {
        const int hm = (int)ceil_div(M, G1Huge::BM), hn = (int)ceil_div(N, G1Huge::BN);
        if (hm * hn >= G1_HUGE_MIN_TILES) {       // 256 x 256 tiles, 64 x 128 per wave
            best.shape = GemmPlan::kHuge;
            best.tiles_m = hm;
            best.tiles_n = hn;
            return best;
        }
    }
    if (best.shape == GemmPlan::kBig && best.tiles_m * best.tiles_n >= G1_WIDE_MIN_TILES)
        best.shape = GemmPlan::kWide;             // same tiles and splits, 64 x 64 per wave
    return best;
}

// Products the fused kernel takes: one K-slice (no split-K), a tile shape
// with an LDS epilogue, at most FU_NB_MAX bins, and a counter per row block
// in the workspace header.  Measured against the two-kernel path with one
// slice: 61.1 against 68.3 us at 8192 x 512 x 4096, 62.7 against 73.5 us at
// 4096 x 1024 x 4096, 37.2 against 41.0 us at 16384 x 256 x 2048.
static bool fused_fits(const GemmPlan& g, int nb) {
    if (g.shape != GemmPlan::kSmall && g.shape != GemmPlan::kBig && g.shape != GemmPlan::kMid)
        return false;
    if (nb > FU_NB_MAX || g.splits != 1) return false;
    return g.tiles_n == 1 || g.tiles_m <= FU_MAX_TICKETS;
}

static int gemm_bm(int shape) {
    return shape == GemmPlan::kSmall ? G1Small::BM : shape == GemmPlan::kHuge ? G1Huge::BM : G1Big::BM;
}

PredictPlan plan_predict(const star_predict_params& p, bool tiled_ok, bool fused_ok) {
    PredictPlan pl;
    const GemmPlan g = plan_gemm(p.n_req, p.d_hidden, p.d_model, p.dtype == STAR_BF16 ? 2 : 4);
    pl.gemm = g;
    pl.tiles_m = g.tiles_m;
    pl.tiles_n = g.tiles_n;
    pl.ktiles = g.ktiles;
    const int s = g.splits;
    pl.splits = s;
    if (fused_ok && p.dtype == STAR_BF16 && fused_fits(g, p.n_bins)) {
        pl.fused = true;
        const size_t bm = (size_t)gemm_bm(g.shape);
        const size_t tiles = (size_t)g.tiles_m * g.tiles_n;
        const size_t nb32 = (size_t)((p.n_bins + 31) / 32) * 32;
        pl.lpart_bytes = g.tiles_n > 1 ? align_up(tiles * bm * nb32 * sizeof(float), 256) : 0;
        pl.partial_bytes = pl.lpart_bytes;
        pl.head_rows = (int)bm;
        return pl;
    }
    pl.partial_bytes = (size_t)s * (size_t)p.n_req * (size_t)p.d_hidden * sizeof(float);
    const int mpad = (p.d_hidden + 31) & ~31;
    const int nbpad = (p.n_bins + 15) & ~15;
    pl.head_tiled = tiled_ok && p.dtype == STAR_BF16 && p.n_req >= HT_MIN_REQ &&
                    s <= HT_MAX_SPLITS;
    pl.head_rows = pl.head_tiled ? HT_ROWS : HD_RB;
    const size_t rb = (size_t)pl.head_rows;
    if (pl.head_tiled)
        pl.head_lds = head_tiled_lds(p.n_bins, p.d_hidden);
    else if (p.dtype == STAR_BF16)
        pl.head_lds = 2 * rb * (mpad + 8) * 2 + rb * nbpad * 4;
    else
        pl.head_lds = rb * p.d_hidden * 4 + rb * nbpad * 4;
    return pl;
}

template <int NS, class SH>
static hipError_t launch_fused_shape(const PredictPlan& pl, const FusedArgs& a, hipStream_t stream) {
    const dim3 grid(pl.gemm.tiles_m * pl.gemm.tiles_n);
    hipLaunchKernelGGL((predict_fused_kernel<NS, SH>), grid, dim3(SH::THREADS), 0, stream, a);
    return hipGetLastError();
}

static hipError_t launch_fused(const star_predict_params& p, const PredictPlan& pl,
                               const void* hidden, const void* w1, const float* b1,
                               const void* w2, const float* b2, const float* bins,
                               float* ema_state, float* expected, int32_t* rem_len, char* scratch,
                               uint32_t* tickets, hipStream_t stream) {
    FusedArgs a;
    a.A = (const char*)hidden;
    a.W = (const char*)w1;
    a.b1 = b1;
    a.W2 = (const uint16_t*)w2;
    a.b2 = b2;
    a.bins = bins;
    a.lpart = (float*)scratch;
    a.tix_row = tickets;
    a.ema_state = ema_state;
    a.expected = expected;
    a.rem_len = rem_len;
    a.M = p.n_req;
    a.N = p.d_hidden;
    a.Kd = p.d_model;
    a.nb = p.n_bins;
    a.tiles_n = pl.gemm.tiles_n;
    a.ktiles = pl.gemm.ktiles;
    a.act = p.act;
    a.ema_init = p.ema_init;
    a.len_max = p.len_max;
    a.ema_alpha = p.ema_alpha;
    switch (pl.gemm.shape) {
        case GemmPlan::kSmall: return launch_fused_shape<G1_STAGES_SMALL, G1Small>(pl, a, stream);
        case GemmPlan::kBig: return launch_fused_shape<G1_STAGES_BIG, G1Big>(pl, a, stream);
        case GemmPlan::kMid: return launch_fused_shape<G1_STAGES_MID, G1Mid>(pl, a, stream);
    }
    return hipErrorInvalidValue;
}

template <bool kBF16, int kS, bool kReg, int kPF>
static hipError_t launch_head_rows(const star_predict_params& p, const PredictPlan& pl,
                                   const float* partials, const float* b1, const void* w2,
                                   const float* b2, const float* bins, float* ema_state,
                                   float* expected, int32_t* rem_len, float b4,
                                   hipStream_t stream) {
    if (pl.head_lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)head_kernel<kBF16, kS, kReg, kPF>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)pl.head_lds);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)ceil_div(p.n_req, HD_RB));
    hipLaunchKernelGGL((head_kernel<kBF16, kS, kReg, kPF>), grid, dim3(HD_THREADS), pl.head_lds,
                       stream, partials, p.n_req, p.d_hidden, p.n_bins, b1, w2, b2, bins, p.act,
                       p.ema_alpha, p.ema_init, ema_state, expected, rem_len, p.len_max, b4);
    return hipGetLastError();
}

template <int kS, int kNBB, bool kGelu>
static hipError_t launch_head_tiled_act(const star_predict_params& p, const PredictPlan& pl,
                                    const float* partials, const float* b1, const void* w2,
                                    const float* b2, const float* bins, float* ema_state,
                                    float* expected, int32_t* rem_len, hipStream_t stream) {
    if (pl.head_lds > 64 * 1024) {
        hipError_t e = hipFuncSetAttribute((const void*)head_tiled_kernel<kS, kNBB, kGelu>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)pl.head_lds);
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)ceil_div(p.n_req, HT_ROWS));
    hipLaunchKernelGGL((head_tiled_kernel<kS, kNBB, kGelu>), grid, dim3(HT_THREADS), pl.head_lds, stream,
                       partials, p.n_req, p.d_hidden, p.n_bins, b1, (const uint16_t*)w2, b2, bins,
                       p.ema_alpha, p.ema_init, ema_state, expected, rem_len, p.len_max);
    return hipGetLastError();
}

template <int kS, int kNBB>
static hipError_t launch_head_tiled(const star_predict_params& p, const PredictPlan& pl,
                                    const float* partials, const float* b1, const void* w2,
                                    const float* b2, const float* bins, float* ema_state,
                                    float* expected, int32_t* rem_len, hipStream_t stream) {
    return p.act == STAR_ACT_GELU_ERF
        ? launch_head_tiled_act<kS, kNBB, true>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, stream)
        : launch_head_tiled_act<kS, kNBB, false>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, stream);
}

// The tiled head only for the bf16 binned head with at most HT_MAX_SPLITS
// planes (the plan never picks it elsewhere).
template <bool kBF16, int kS, bool kReg>
static hipError_t launch_head_s(const star_predict_params& p, const PredictPlan& pl,
                                const float* partials, const float* b1, const void* w2,
                                const float* b2, const float* bins, float* ema_state,
                                float* expected, int32_t* rem_len, float b4, hipStream_t stream) {
    if constexpr (kBF16 && !kReg && kS <= HT_MAX_SPLITS) {
        if (pl.head_tiled) {
            const int nbb = head_tiled_blocks(p.n_bins);
            return nbb == 4 ? launch_head_tiled<kS, 4>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, stream)
                 : nbb == 8 ? launch_head_tiled<kS, 8>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, stream)
                            : launch_head_tiled<kS, 16>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, stream);
        }
    }
    if (pl.head_tiled || pl.head_rows != HD_RB) return hipErrorInvalidValue;
    if constexpr (kBF16) {
        if (ceil_div(p.n_req, HD_RB) > HD_LOWREG_GROUPS)
            return launch_head_rows<kBF16, kS, kReg, HD_W2PF_LOW>(p, pl, partials, b1, w2, b2, bins,
                                                                 ema_state, expected, rem_len, b4,
                                                                 stream);
    }
    return launch_head_rows<kBF16, kS, kReg, HD_W2PF>(p, pl, partials, b1, w2, b2, bins, ema_state,
                                                      expected, rem_len, b4, stream);
}

template <bool kBF16, bool kReg = false>
static hipError_t launch_head(const star_predict_params& p, const PredictPlan& pl,
                              const float* partials, const float* b1, const void* w2,
                              const float* b2, const float* bins, float* ema_state,
                              float* expected, int32_t* rem_len, hipStream_t stream,
                              float b4 = 0.0f) {
    switch (pl.splits) {
        case 1: return launch_head_s<kBF16, 1, kReg>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, b4, stream);
        case 2: return launch_head_s<kBF16, 2, kReg>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, b4, stream);
        case 4: return launch_head_s<kBF16, 4, kReg>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, b4, stream);
        case 8: return launch_head_s<kBF16, 8, kReg>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, b4, stream);
        case 16: return launch_head_s<kBF16, 16, kReg>(p, pl, partials, b1, w2, b2, bins, ema_state, expected, rem_len, b4, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_predict(const star_predict_params& p, const PredictPlan& pl, const void* hidden,
                          const void* w1, const float* b1, const void* w2, const float* b2,
                          const float* bins, float* ema_state, float* expected, int32_t* rem_len,
                          char* scratch, uint32_t* tickets, hipStream_t stream) {
    if (p.n_req == 0) return hipSuccess;
    if (pl.fused)
        return launch_fused(p, pl, hidden, w1, b1, w2, b2, bins, ema_state, expected, rem_len,
                            scratch, tickets, stream);
    float* partials = (float*)scratch;
    hipError_t e = launch_gemm(pl.gemm, p.dtype == STAR_BF16, hidden, w1, partials, p.n_req,
                               p.d_hidden, p.d_model, stream);
    if (e != hipSuccess) return e;
    return p.dtype == STAR_BF16 ? launch_head<true>(p, pl, partials, b1, w2, b2, bins,
                                                    ema_state, expected, rem_len, stream)
                                : launch_head<false>(p, pl, partials, b1, w2, b2, bins,
                                                     ema_state, expected, rem_len, stream);
}

// ---------------------------------------------------------------------------
// Two batches in one launch.  Blocks [0, gemm_blocks) compute the next
// batch's first-layer split-K partials (64 x 64 tiles); the blocks after
// them run the previous batch's head from its partials.  The roles share no
// data, and each block takes one role for its whole life, so they need no
// synchronisation.  One launch removes the kernel boundary between the
// previous batch's head and the next batch's product, and the head's
// workgroups take the CUs as the product's workgroups leave them.
// ---------------------------------------------------------------------------
struct OverlapArgs {
    // the next batch's product
    const char* A;
    const char* W1;
    float* Pn;
    int M, N, Kd, splits, tiles_n, ktiles, gemm_blocks;
    // the previous batch's head
    const float* Pp;
    const float* b1;
    const void* w2;
    const float* b2;
    const float* bins;
    float* ema_state;
    float* expected;
    int32_t* rem_len;
    int B, m, nb, act, ema_init, len_max;
    float ema_alpha;
};
constexpr size_t OV_LDS = 2 * (size_t)(G1Small::LDS_A + G1Small::LDS_B);
// W2 fragments the head role prefetches: 4 keeps the kernel at 90 VGPRs, so
// head workgroups fit beside the product's two per CU from the start
// (measured at 1024 x 4096 -> 512 -> 64 bins, per batch: 12.9-13.6 us with
// 4, 13.4-13.8 with 8 (124 VGPRs), 16.6-17.5 with 16 (214 VGPRs, two
// workgroups per CU, heads waiting for products to end), against 18.1-18.2
// for star_predict).
constexpr int OV_W2PF = 4;

template <int kS>
__global__ __launch_bounds__(HD_THREADS) void predict_overlap_kernel(OverlapArgs a) {
    static_assert(G1Small::THREADS == HD_THREADS, "one block size for both roles");
    __shared__ __attribute__((aligned(16))) char lds[2][G1Small::LDS_A + G1Small::LDS_B];
    if ((int)blockIdx.x < a.gemm_blocks)
        gemm1_tile<2, G1_STAGES_SMALL, G1Small>(a.A, a.W1, a.Pn, a.M, a.N, a.Kd, a.splits,
                                                a.tiles_n, a.ktiles, blockIdx.x, a.gemm_blocks,
                                                lds);
    else
        head_rows<true, kS, false, OV_W2PF>(a.Pp, a.B, a.m, a.nb, a.b1, a.w2, a.b2, a.bins,
                                            a.act, a.ema_alpha, a.ema_init, a.ema_state,
                                            a.expected, a.rem_len, a.len_max, 0.0f,
                                            (int)blockIdx.x - a.gemm_blocks, &lds[0][0]);
}

hipError_t launch_predict_overlap(const star_predict_params& p, const PredictPlan& pl,
                                  const void* hidden_next, float* partials_next,
                                  const float* partials_prev, const void* w1, const float* b1,
                                  const void* w2, const float* b2, const float* bins,
                                  float* ema_state, float* expected, int32_t* rem_len,
                                  hipStream_t stream) {
    if (pl.fused) return hipErrorInvalidValue;
    if (p.n_req == 0 || (!hidden_next && !partials_prev)) return hipSuccess;
    const bool bf16 = p.dtype == STAR_BF16;
    const GemmPlan& g = pl.gemm;
    const int head_blocks = (int)ceil_div(p.n_req, HD_RB);
    const bool one = hidden_next && partials_prev && bf16 && g.shape == GemmPlan::kSmall &&
                     !pl.head_tiled && pl.head_rows == HD_RB && pl.head_lds <= OV_LDS &&
                     head_blocks <= HD_LOWREG_GROUPS;
    if (!one) {          // the two kernels one after the other, same results
        if (partials_prev) {
            const hipError_t e =
                bf16 ? launch_head<true>(p, pl, partials_prev, b1, w2, b2, bins, ema_state,
                                         expected, rem_len, stream)
                     : launch_head<false>(p, pl, partials_prev, b1, w2, b2, bins, ema_state,
                                          expected, rem_len, stream);
            if (e != hipSuccess) return e;
        }
        if (hidden_next)
            return launch_gemm(g, bf16, hidden_next, w1, partials_next, p.n_req, p.d_hidden,
                               p.d_model, stream);
        return hipSuccess;
    }
    OverlapArgs a;
    a.A = (const char*)hidden_next;
    a.W1 = (const char*)w1;
    a.Pn = partials_next;
    a.M = p.n_req;
    a.N = p.d_hidden;
    a.Kd = p.d_model;
    a.splits = g.splits;
    a.tiles_n = g.tiles_n;
    a.ktiles = g.ktiles;
    a.gemm_blocks = g.tiles_m * g.tiles_n * g.splits;
    a.Pp = partials_prev;
    a.b1 = b1;
    a.w2 = w2;
    a.b2 = b2;
    a.bins = bins;
    a.ema_state = ema_state;
    a.expected = expected;
    a.rem_len = rem_len;
    a.B = p.n_req;
    a.m = p.d_hidden;
    a.nb = p.n_bins;
    a.act = p.act;
    a.ema_init = p.ema_init;
    a.len_max = p.len_max;
    a.ema_alpha = p.ema_alpha;
    const dim3 grid((unsigned)(a.gemm_blocks + head_blocks));
    switch (g.splits) {
        case 1: hipLaunchKernelGGL(predict_overlap_kernel<1>, grid, dim3(HD_THREADS), 0, stream, a); break;
        case 2: hipLaunchKernelGGL(predict_overlap_kernel<2>, grid, dim3(HD_THREADS), 0, stream, a); break;
        case 4: hipLaunchKernelGGL(predict_overlap_kernel<4>, grid, dim3(HD_THREADS), 0, stream, a); break;
        case 8: hipLaunchKernelGGL(predict_overlap_kernel<8>, grid, dim3(HD_THREADS), 0, stream, a); break;
        case 16: hipLaunchKernelGGL(predict_overlap_kernel<16>, grid, dim3(HD_THREADS), 0, stream, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// (f3) the regression head: GEMM (layer 1) -> act -> GEMM (layer 2) -> head
// (layers 3 and 4, EMA, integerisation)
// ---------------------------------------------------------------------------
// The head kernel's view of the last two layers: a "binned head" whose
// input width is m2, whose nb = m3 outputs get ReLU and are dotted with w4.
static star_predict_params head_view(const star_mlp4_params& p) {
    star_predict_params h;
    h.n_req = p.n_req;
    h.d_model = p.m1;
    h.d_hidden = p.m2;
    h.n_bins = p.m3;
    h.dtype = p.dtype;
    h.act = STAR_ACT_RELU;
    h.ema_alpha = p.ema_alpha;
    h.ema_init = p.ema_init;
    h.len_max = p.len_max;
    return h;
}

Mlp4Plan plan_mlp4(const star_mlp4_params& p) {
    Mlp4Plan pl;
    const int elem = p.dtype == STAR_BF16 ? 2 : 4;
    pl.g1 = plan_gemm(p.n_req, p.m1, p.d_model, elem);
    pl.head = plan_predict(head_view(p), false, false);   // layer 2 and the head
    size_t off = 0;
    pl.p1_off = off;
    off += align_up((size_t)pl.g1.splits * p.n_req * p.m1 * sizeof(float), 256);
    pl.a1_off = off;
    off += align_up((size_t)p.n_req * p.m1 * elem, 256);
    pl.p2_off = off;
    off += align_up(pl.head.partial_bytes, 256);
    pl.total = off;
    return pl;
}

template <bool kBF16>
static hipError_t launch_act(int splits, dim3 grid, const float* P, int64_t items, int m4,
                             const float* bias, void* out, hipStream_t stream) {
    switch (splits) {
        case 1: hipLaunchKernelGGL((act_kernel<1, kBF16>), grid, dim3(ACT_THREADS), 0, stream, P, items, m4, bias, out); break;
        case 2: hipLaunchKernelGGL((act_kernel<2, kBF16>), grid, dim3(ACT_THREADS), 0, stream, P, items, m4, bias, out); break;
        case 4: hipLaunchKernelGGL((act_kernel<4, kBF16>), grid, dim3(ACT_THREADS), 0, stream, P, items, m4, bias, out); break;
        case 8: hipLaunchKernelGGL((act_kernel<8, kBF16>), grid, dim3(ACT_THREADS), 0, stream, P, items, m4, bias, out); break;
        case 16: hipLaunchKernelGGL((act_kernel<16, kBF16>), grid, dim3(ACT_THREADS), 0, stream, P, items, m4, bias, out); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_mlp4(const star_mlp4_params& p, const Mlp4Plan& pl, const void* hidden,
                       const void* w1, const float* b1, const void* w2, const float* b2,
                       const void* w3, const float* b3, const float* w4, float* ema_state,
                       float* expected, int32_t* rem_len, char* ws, hipStream_t stream) {
    if (p.n_req == 0) return hipSuccess;
    const bool bf = p.dtype == STAR_BF16;
    float* P1 = (float*)(ws + pl.p1_off);
    void* A1 = ws + pl.a1_off;
    float* P2 = (float*)(ws + pl.p2_off);
    hipError_t e;
    if ((e = launch_gemm(pl.g1, bf, hidden, w1, P1, p.n_req, p.m1, p.d_model, stream)) !=
        hipSuccess)
        return e;
    const int64_t items = (int64_t)p.n_req * p.m1 / 4;
    int64_t ab = ceil_div(items, (int64_t)ACT_THREADS * ACT_BATCH);
    const dim3 ga((unsigned)(ab > 2048 ? 2048 : ab));
    e = bf ? launch_act<true>(pl.g1.splits, ga, P1, items, p.m1 / 4, b1, A1, stream)
           : launch_act<false>(pl.g1.splits, ga, P1, items, p.m1 / 4, b1, A1, stream);
    if (e != hipSuccess) return e;
    const star_predict_params h = head_view(p);
    if ((e = launch_gemm(pl.head.gemm, bf, A1, w2, P2, p.n_req, p.m2, p.m1, stream)) !=
        hipSuccess)
        return e;
    return bf ? launch_head<true, true>(h, pl.head, P2, b2, w3, b3, w4, ema_state, expected,
                                        rem_len, stream, p.b4)
              : launch_head<false, true>(h, pl.head, P2, b2, w3, b3, w4, ema_state, expected,
                                         rem_len, stream, p.b4);
}

}  // namespace star

