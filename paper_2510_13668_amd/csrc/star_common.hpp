// Internal helpers shared by the gfx950 kernels of libstar.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "star.h"

namespace star {

constexpr int kWave = 64;

// Workspace header layout (STAR_WS_HEADER_BYTES bytes at the start of every
// workspace, never used as scratch: whatever must hold between calls lives
// here, and the calls that use a counter or the histogram leave it at zero).
constexpr size_t kHdrErrorWord = 0;     // int32: sticky OR of STAR_DEV_* bits
constexpr size_t kHdrVarTicket = 64;    // uint32: finished variance-scoring workgroups
constexpr size_t kHdrPlanDone = 72;     // int32: the migration plan has stopped
constexpr size_t kHdrPlanCount = 76;    // int32: moves made by the plan
constexpr size_t kHdrScoreHist = 256;   // uint32[1024]: key-code histogram of the ranking
static_assert(kHdrScoreHist + 1024 * 4 <= STAR_WS_HEADER_BYTES, "header holds the histogram");
// uint32 arrival counters of the calls whose workgroups meet through a
// last-arriver exchange (the fused predictor's row blocks, the split
// projection's instances), to the end of the header
constexpr size_t kHdrTickets = kHdrScoreHist + 1024 * 4;
constexpr int kMaxTickets = (int)((STAR_WS_HEADER_BYTES - kHdrTickets) / 4);

__host__ __device__ inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

typedef short bf16x8 __attribute__((ext_vector_type(8)));     // raw bits, 16 bytes
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));  // MFMA operand type
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// two fp32 -> packed bf16 bits, a in the low half, round to nearest even (one
// packed conversion instruction)
__device__ inline uint32_t pack_bf16x2_rne(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2_t));
}
// a (and b) as a bf16 pair hi + lo, hi = bf16(a), lo = bf16(a - hi): packed
// hi and lo words for two values
__device__ inline void split_bf16x2(float a, float b, uint32_t& hi, uint32_t& lo) {
    hi = pack_bf16x2_rne(a, b);
    lo = pack_bf16x2_rne(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xFFFF0000u));
}

// ---------------------------------------------------------------------------
// wavefront reductions (64 lanes)
// ---------------------------------------------------------------------------
__device__ inline float wave_max_f32(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
    return v;
}
__device__ inline float wave_sum_f32(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}
__device__ inline int32_t wave_or_i32(int32_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v |= __shfl_xor(v, o, kWave);
    return v;
}

// ---------------------------------------------------------------------------
// DPP wavefront scans (gfx9 data-parallel primitives: row shifts within 16
// lanes, then row broadcasts of lanes 15 and 31).  A lane whose source lane
// is out of range or masked off receives `ident`.  DPP moves cost a few
// cycles, against ~80 for a ds_bpermute-based shuffle.
// ---------------------------------------------------------------------------
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;

template <int kCtrl, int kRowMask>
__device__ inline int dpp_i32(int v, int ident) {
    return __builtin_amdgcn_update_dpp(ident, v, kCtrl, kRowMask, 0xF, false);
}

// Inclusive prefix sum over the 64 lanes (lane order).
__device__ inline int wave_incl_add_i32(int v) {
    v += dpp_i32<kDppRowShr1, 0xF>(v, 0);
    v += dpp_i32<kDppRowShr2, 0xF>(v, 0);
    v += dpp_i32<kDppRowShr4, 0xF>(v, 0);
    v += dpp_i32<kDppRowShr8, 0xF>(v, 0);
    v += dpp_i32<kDppRowBcast15, 0xA>(v, 0);
    v += dpp_i32<kDppRowBcast31, 0xC>(v, 0);
    return v;
}

template <int kCtrl, int kRowMask>
__device__ inline int64_t dpp_max_step_i64(int64_t v) {
    const int lo = (int)(uint32_t)v, hi = (int)(v >> 32);
    const int slo = dpp_i32<kCtrl, kRowMask>(lo, lo);   // masked / out-of-range: own value
    const int shi = dpp_i32<kCtrl, kRowMask>(hi, hi);
    const int64_t u = (int64_t)(((uint64_t)(uint32_t)shi << 32) | (uint32_t)slo);
    return u > v ? u : v;
}

// Inclusive prefix max over the 64 lanes (lane order).
__device__ inline int64_t wave_incl_max_i64(int64_t v) {
    v = dpp_max_step_i64<kDppRowShr1, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr2, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr4, 0xF>(v);
    v = dpp_max_step_i64<kDppRowShr8, 0xF>(v);
    v = dpp_max_step_i64<kDppRowBcast15, 0xA>(v);
    v = dpp_max_step_i64<kDppRowBcast31, 0xC>(v);
    return v;
}

// The value of `lane` (wave-uniform) broadcast to every lane.
__device__ inline int64_t readlane_i64(int64_t v, int lane) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), lane);
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// v plus the value of its DPP source lane (0 where there is none).
template <int kCtrl, int kRowMask>
__device__ inline int64_t dpp_add_i64(int64_t v) {
    const int lo = dpp_i32<kCtrl, kRowMask>((int)(uint32_t)v, 0);
    const int hi = dpp_i32<kCtrl, kRowMask>((int)(v >> 32), 0);
    return v + (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Inclusive prefix sum of an int64 over the 64 lanes (lane order).
__device__ inline int64_t wave_incl_add_i64(int64_t v) {
    v = dpp_add_i64<kDppRowShr1, 0xF>(v);
    v = dpp_add_i64<kDppRowShr2, 0xF>(v);
    v = dpp_add_i64<kDppRowShr4, 0xF>(v);
    v = dpp_add_i64<kDppRowShr8, 0xF>(v);
    v = dpp_add_i64<kDppRowBcast15, 0xA>(v);
    v = dpp_add_i64<kDppRowBcast31, 0xC>(v);
    return v;
}

// Inclusive prefix sums of two int64 per thread over a block of kT threads
// (thread order, every thread taking part); tmp: 2 kT/64 int64 of LDS.
template <int kT>
__device__ inline void block_incl_add2_i64(int64_t& x, int64_t& y, int64_t* tmp) {
    constexpr int W = kT / kWave;
    static_assert(W <= kWave, "one wave reads every wave's total");
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    x = wave_incl_add_i64(x);
    y = wave_incl_add_i64(y);
    if (lane == kWave - 1) {
        tmp[wid] = x;
        tmp[W + wid] = y;
    }
    __syncthreads();
    // the totals of the waves before this one: lane w < wid reads wave w's,
    // all at once, and a wave sum adds them
    const int64_t tx = lane < W ? tmp[lane] : 0, ty = lane < W ? tmp[W + lane] : 0;
    x += readlane_i64(wave_incl_add_i64(lane < wid ? tx : 0), kWave - 1);
    y += readlane_i64(wave_incl_add_i64(lane < wid ? ty : 0), kWave - 1);
    __syncthreads();
}

// Inclusive prefix maxima of two int64 per thread over a block of kT threads
// (thread order, every thread taking part); tmp: 2 kT/64 int64 of LDS.
template <int kT>
__device__ inline void block_incl_max2_i64(int64_t& x, int64_t& y, int64_t* tmp) {
    constexpr int W = kT / kWave;
    static_assert(W <= kWave, "one wave reads every wave's maximum");
    const int lane = threadIdx.x & (kWave - 1), wid = threadIdx.x / kWave;
    x = wave_incl_max_i64(x);
    y = wave_incl_max_i64(y);
    if (lane == kWave - 1) {
        tmp[wid] = x;
        tmp[W + wid] = y;
    }
    __syncthreads();
    // the maxima of the waves before this one, read all at once
    const int64_t tx = lane < W ? tmp[lane] : INT64_MIN, ty = lane < W ? tmp[W + lane] : INT64_MIN;
    const int64_t mx = readlane_i64(wave_incl_max_i64(lane < wid ? tx : INT64_MIN), kWave - 1);
    const int64_t my = readlane_i64(wave_incl_max_i64(lane < wid ? ty : INT64_MIN), kWave - 1);
    x = mx > x ? mx : x;
    y = my > y ? my : y;
    __syncthreads();
}

// Inclusive scan across the wave (lane order), for a commutative,
// associative op on int64.
template <class Op>
__device__ inline int64_t wave_inclusive_scan_i64(int64_t v, Op op) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t u = __shfl_up(v, o, kWave);
        if (lane >= o) v = op(v, u);
    }
    return v;
}

// Inclusive max-scan across the wave in reverse lane order (lane 63 first).
__device__ inline int64_t wave_inclusive_scan_rev_i64(int64_t v) {
    const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        int64_t u = __shfl_down(v, o, kWave);
        if (lane + o < kWave) v = v > u ? v : u;
    }
    return v;
}

struct OpAdd { __device__ int64_t operator()(int64_t a, int64_t b) const { return a + b; } };
struct OpMax { __device__ int64_t operator()(int64_t a, int64_t b) const { return a > b ? a : b; } };

// Block-wide exclusive scan of one int64 per thread (thread order) for a
// block of kThreads threads, using `tmp` (>= kThreads/64 + 1 int64 of LDS).
// Returns the exclusive prefix; *total receives the block aggregate.
// `ident` is the op's identity.
template <int kThreads, class Op>
__device__ inline int64_t block_exclusive_scan_i64(int64_t v, Op op, int64_t ident,
                                                   int64_t* tmp, int64_t* total) {
    constexpr int nw = (kThreads + kWave - 1) / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x / kWave;
    int64_t inc = wave_inclusive_scan_i64(v, op);
    if (lane == kWave - 1) tmp[wid] = inc;
    __syncthreads();
    if (wid == 0) {
        int64_t w = lane < nw ? tmp[lane] : ident;
        int64_t wi = wave_inclusive_scan_i64(w, op);
        if (lane < nw) tmp[lane] = wi;              // inclusive totals per wave
    }
    __syncthreads();
    int64_t before = wid > 0 ? tmp[wid - 1] : ident;
    int64_t excl_in_wave = __shfl_up(inc, 1, kWave);
    if (lane == 0) excl_in_wave = ident;
    int64_t res = op(before, excl_in_wave);
    if (total) *total = tmp[nw - 1];
    __syncthreads();
    return res;
}

// Per-request terms of Section 5.2's load model.  With l' = min(l, H),
// k_e = l' div b and mu = l' mod b, request r's own bucketed curve is
// alpha + b^2 k for k < k_e (alpha = b c + b(b-1)/2), p = mu c + mu k_e b +
// mu(mu-1)/2 at k = k_e, and 0 beyond.  Invalid requests (instance out of
// range, c < 1, l < 1) get s = -1 and zero terms.
struct ReqTerms {
    int64_t alpha, p;
    int ke, s;
    int32_t bad;
};
__device__ inline ReqTerms request_terms(int s, int c, int l, int n, int b, int64_t H) {
    ReqTerms q;
    q.bad = 0;
    if (s < 0 || s >= n) q.bad |= STAR_DEV_BAD_INST;
    if (c < 1) q.bad |= STAR_DEV_BAD_CUR;
    if (l < 1) q.bad |= STAR_DEV_BAD_REM;
    // (a 32-bit division here, exact since l' < 2^31, cost the variance
    // scoring kernels an occupancy step and gained nothing measurable)
    const int64_t lp = (int64_t)l < H ? (int64_t)l : H;
    const int64_t ke = lp / b;
    const int64_t mu = lp - ke * b;
    const bool ok = q.bad == 0;
    q.s = ok ? s : -1;
    q.ke = ok ? (int)ke : 0;
    q.alpha = ok ? (int64_t)b * c + (int64_t)b * (b - 1) / 2 : 0;
    q.p = ok ? mu * c + mu * ke * b + mu * (mu - 1) / 2 : 0;
    return q;
}

// ---------------------------------------------------------------------------
// Exchange between the workgroups of one launch without cache maintenance:
// shares are stored and loaded with the device-coherent cache policy (sc1)
// through raw buffer resources, every storer waits for its stores to
// complete before its counter increment, and the last arriver loads only
// after its own increment has returned.  So the shares never need an L2
// write-back (release) or invalidation (acquire), which would also throw out
// what the other workgroups of the XCD are still reading.  The counters live
// in the workspace header, and every call leaves them at zero.
// ---------------------------------------------------------------------------
constexpr int kCpolCoherent = 16;          // buffer cache policy bits: sc1 (device scope)
constexpr uint32_t kXchOob = 0x7FFFFFF0u;  // a buffer offset past every share: reads 0

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline __amdgpu_buffer_rsrc_t xch_rsrc(const void* base, uint32_t bytes) {
    // raw buffer (stride 0); out-of-range accesses read 0 and drop writes
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}
__device__ inline void xch_store(u32x4 v, __amdgpu_buffer_rsrc_t r, uint32_t off) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, kCpolCoherent);
}
__device__ inline u32x4 xch_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kCpolCoherent);
}
__device__ inline u32x2 xch_load_b64(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kCpolCoherent);
}
// every store this thread issued has completed (is visible device-wide)
__device__ inline void xch_wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// One workgroup's arrival at a counter that `expect` workgroups reach: true
// for the last to arrive, which also resets the counter.  Call after the
// workgroup's coherent stores have completed (xch_wait_stores in every thread).
__device__ inline bool xch_last_arrival(uint32_t* counter, uint32_t expect, uint32_t* s_ticket) {
    __syncthreads();
    if (threadIdx.x == 0)
        *s_ticket = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const bool last = *s_ticket == expect - 1;
    if (last && threadIdx.x == 0)
        __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return last;
}

// Device-error reporting: OR `bits` into the workspace error word.
__device__ inline void report_error(int32_t* err_word, int32_t bits) {
    if (bits) atomicOr(err_word, bits);
}

}  // namespace star
