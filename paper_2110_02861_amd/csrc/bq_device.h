// Device helpers shared by the HIP kernels (gfx950): codebook decision tables,
// exact nearest-code search, exact division by the block absmax, wave / group
// max reductions, vector loads and stores.
//
// Exact nearest code (Eq. 3 / Eq. 4 of the paper, ties to the lower index)
//   With T_j the smallest fp32 above the midpoint of codes j and j+1 and
//   T_255 = +inf, the nearest code of y is #{j : y >= T_j}.  The sign, exponent
//   and top 7 mantissa bits of y select a bucket (a run of fp32 bit patterns);
//   a table holds, per bucket, the number of thresholds at or below the
//   bucket's smallest value.  At most K thresholds lie inside any bucket (K is
//   computed with the table; K = 1 for the dynamic maps), so K compares
//   against T finish the count.  This is exact for every strictly increasing
//   map.
//
// Exact division
//   y = x / N is the correctly rounded quotient: per block r = RN(1/N'), per
//   element q = x' r, e = fma(-q, N', x'), y = fma(e, r, q) (Markstein's
//   correction), with x' = x s, N' = N s and s a power of two keeping N' within
//   [2^-64, 2^64].  Exact whenever |y| >= 2^-100, far below any threshold of a
//   map whose nonzero magnitudes are >= 2^-60.  An all-zero block uses r = 0,
//   which sends every element to y = 0.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bq_internal.h"

namespace bq {
namespace dev {

// Bucket index: bits [30:16] of |y| (8 exponent + 7 mantissa bits), clamped to
// the binades [2^-25, 2^1).  Magnitudes below 2^-25 share the first bucket,
// magnitudes of 1 and above the last.
constexpr uint32_t kBucketShift = 16;
constexpr uint32_t kBucketLo = (127u - 25u) << 7;
constexpr uint32_t kBucketHi = (127u << 7) + 127u;
constexpr uint32_t kBuckets = kBucketHi - kBucketLo + 1;  // per sign
static_assert(kBuckets == kPreparedBuckets, "prepared table layout");

// Read-only view of one map's decision tables (in LDS).
struct Tables {
    const float *q;       // 256 codebook values
    const float *t;       // 256 thresholds, t[255] = +inf
    const uint8_t *base;  // [sign * kBuckets + bucket]; only the + half for NONNEG use
    int kmax;             // max thresholds strictly inside one bucket
};

__device__ inline float next_up(float f)
{
    if (f == 0.0f)
        return __uint_as_float(1u);  // smallest positive subnormal
    const uint32_t u = __float_as_uint(f);
    return __uint_as_float(f > 0.0f ? u + 1u : u - 1u);
}

__device__ inline float next_down(float f)
{
    return -next_up(-f);
}

// True when y lies strictly above the exact midpoint of a and b, i.e. when
// 2y > a + b without rounding: for a < b this is "y is strictly nearer b".
// a + b = s + e exactly (two-sum in double); 2y - s is exact when 2y and s are
// within a factor 2 of each other, and otherwise outweighs e.
__device__ inline bool above_midpoint(float y, float a, float b)
{
    const double A = a, Bd = b;
    const double s = A + Bd;
    const double bv = s - A;
    const double e = (A - (s - bv)) + (Bd - bv);
    const double t = 2.0 * (double)y;
    const bool close = (s > 0.0 && t >= 0.5 * s && t <= 2.0 * s) ||
                       (s < 0.0 && t <= 0.5 * s && t >= 2.0 * s);
    return close ? (t - s) > e : t > s;
}

__device__ inline uint32_t bucket_lo_bits(uint32_t b)
{
    return b == 0 ? 0u : (kBucketLo + b) << kBucketShift;
}
__device__ inline uint32_t bucket_hi_bits(uint32_t b)
{
    return b == kBuckets - 1 ? 0x7f7fffffu : ((kBucketLo + b + 1) << kBucketShift) - 1u;
}

// Where threshold v falls among the buckets.  Positive half: base[b] counts
// the thresholds <= lo(b); v counts from bucket pos_pos(v) on (kBuckets: from
// none).  Negative half: base[kBuckets + b] counts the thresholds <= -hi(b); v
// counts for buckets b <= pos_neg(v) (-1: none).  inside_*: the bucket whose
// interior (lo, hi] on the positive half, [-hi, -lo) mirrored (i.e. -hi < v <=
// -lo) on the negative half, holds v, or -1.
__device__ inline uint32_t bucket_clamped(uint32_t abs_bits)
{
    return min(max(abs_bits >> kBucketShift, kBucketLo), kBucketHi) - kBucketLo;
}
__device__ inline int pos_pos(float v)
{
    if (!(v > 0.0f))
        return 0;  // v <= +0 <= lo(b) for every b
    const uint32_t u = __float_as_uint(v);
    const uint32_t b = bucket_clamped(u);
    return (b >= 1 && u == bucket_lo_bits(b)) ? (int)b : (int)b + 1;
}
__device__ inline int inside_pos(float v)
{
    if (!(v > 0.0f))
        return -1;
    const uint32_t u = __float_as_uint(v);
    const uint32_t b = bucket_clamped(u);
    return (b >= 1 && u == bucket_lo_bits(b)) ? -1 : (int)b;
}
__device__ inline int pos_neg(float v)
{
    if (!(v < 0.0f))
        return -1;  // -hi(b) < 0 <= v for every b
    const uint32_t a = __float_as_uint(v) & 0x7fffffffu;
    const uint32_t b = bucket_clamped(a);
    return a == bucket_hi_bits(b) ? (int)b : (int)b - 1;
}
__device__ inline int inside_neg(float v)
{
    if (v > 0.0f)
        return -1;
    if (!(v < 0.0f))
        return 0;  // +-0: -hi(0) < v <= -lo(0) = -0
    const uint32_t a = __float_as_uint(v) & 0x7fffffffu;
    const uint32_t b = bucket_clamped(a);
    return a == bucket_hi_bits(b) ? -1 : (int)b;
}

// Build q, t, base and kmax for one map.  All NT threads of the workgroup take
// part (NT >= 512, a multiple of 64); the function contains barriers.  q and t
// may live in LDS or global memory (t is read back after the first barrier);
// base must be LDS, 4-byte aligned.  kmax_out is an LDS int, set to the maximum
// over the workgroup.
//
// base is a prefix count over the buckets of a sorted threshold list, so it is
// formed without any search: every threshold adds one to a byte histogram at
// the first bucket it counts for (LDS atomics on the dword that holds the
// byte; no byte exceeds 255 thresholds), then a workgroup scan turns the
// histogram into counts, ascending over the positive half and descending over
// the negative half.  Thresholds inside one bucket are consecutive, so kmax is
// the longest run of equal inside_* buckets, counted from each run's start.
template <int NT>
__device__ void build_tables(const float *__restrict__ qmap, float *q, float *t, uint8_t *base,
                             int *kmax_out)
{
    static_assert(NT >= 512 && NT % 64 == 0, "two scan halves of at least 208 threads");
    constexpr int kHalf = NT / 2;
    constexpr int kPerThread = 16;                         // buckets scanned per thread
    constexpr int kScanThreads = (int)kBuckets / kPerThread;  // per half
    static_assert(kScanThreads * kPerThread == (int)kBuckets && kScanThreads <= kHalf,
                  "scan layout");
    __shared__ uint32_t wave_sums[NT / 64];
    uint32_t *hist = reinterpret_cast<uint32_t *>(base);
    const uint32_t j = threadIdx.x;
    float thr = __builtin_inff();
    if (j < 256) {
        const float qj = qmap[j];
        q[j] = qj;
        if (j < 255) {
            // the smallest fp32 strictly above the exact midpoint: start from
            // the double midpoint (exact unless the codes are 2^29 apart in
            // magnitude) and settle it with the exact comparison
            const float qn = qmap[j + 1];
            const double mid = ((double)qj + (double)qn) * 0.5;
            float f = (float)mid;
            if ((double)f <= mid)
                f = next_up(f);
            for (int k = 0; k < 4 && !above_midpoint(f, qj, qn); ++k)
                f = next_up(f);
            for (int k = 0; k < 4 && above_midpoint(next_down(f), qj, qn); ++k)
                f = next_down(f);
            thr = f;
        }
        t[j] = thr;
    }
    for (uint32_t i = j; i < 2 * kBuckets / 4; i += NT)
        hist[i] = 0u;
    if (j == 0)
        *kmax_out = 0;
    __syncthreads();

    // histogram of first counting buckets; runs of thresholds inside a bucket
    if (j < 255) {
        const int pp = pos_pos(thr);
        if (pp < (int)kBuckets)
            atomicAdd(&hist[pp >> 2], 1u << (8 * (pp & 3)));
        const int pn = pos_neg(thr);
        if (pn >= 0) {
            const uint32_t i = kBuckets + (uint32_t)pn;
            atomicAdd(&hist[i >> 2], 1u << (8 * (i & 3)));
        }
        int run = 0;
        const int ip = inside_pos(thr);
        if (ip >= 0 && (j == 0 || inside_pos(t[j - 1]) != ip)) {
            run = 1;
            while (j + run < 255 && inside_pos(t[j + run]) == ip)
                ++run;
        }
        const int in = inside_neg(thr);
        if (in >= 0 && (j == 0 || inside_neg(t[j - 1]) != in)) {
            int r = 1;
            while (j + r < 255 && inside_neg(t[j + r]) == in)
                ++r;
            run = max(run, r);
        }
        if (run > 0)
            atomicMax(kmax_out, run);
    }
    __syncthreads();

    // scan: thread k of a half takes 16 consecutive buckets (scan order: up
    // the positive half, down the negative half); in-thread running sums, a
    // wave scan of the thread totals, then the totals of the earlier waves
    const int side = (int)j / kHalf;
    const int k = (int)j % kHalf;
    const bool active = k < kScanThreads;
    const int b0 = side == 0 ? kPerThread * k : kPerThread * (kScanThreads - 1 - k);
    const int d0 = (side == 0 ? 0 : (int)kBuckets / 4) + b0 / 4;
    uint32_t w[4] = {0u, 0u, 0u, 0u};
    if (active) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            w[i] = hist[d0 + i];
    }
    uint32_t total = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
        total += (w[i] & 0xffu) + ((w[i] >> 8) & 0xffu) + ((w[i] >> 16) & 0xffu) + (w[i] >> 24);
    const int lane = (int)j & 63;
    uint32_t incl = total;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off);
        if (lane >= off)
            incl += v;
    }
    if (lane == 63)
        wave_sums[j >> 6] = incl;
    __syncthreads();
    uint32_t run_sum = incl - total;  // counts of the earlier threads of this wave
    for (int wv = side * (kHalf / 64); wv < (int)(j >> 6); ++wv)
        run_sum += wave_sums[wv];
    if (active) {
        uint32_t o[4];
        if (side == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                uint32_t packed = 0;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    run_sum += (w[i] >> (8 * r)) & 0xffu;
                    packed |= run_sum << (8 * r);
                }
                o[i] = packed;
            }
        } else {
#pragma unroll
            for (int i = 3; i >= 0; --i) {
                uint32_t packed = 0;
#pragma unroll
                for (int r = 3; r >= 0; --r) {
                    run_sum += (w[i] >> (8 * r)) & 0xffu;
                    packed |= run_sum << (8 * r);
                }
                o[i] = packed;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            hist[d0 + i] = o[i];
    }
    __syncthreads();
}

// Bucket of y.  NONNEG: y is +0 or positive.
template <bool NONNEG>
__device__ inline uint32_t bucket_of(float y)
{
    const uint32_t u = __float_as_uint(y);
    if constexpr (NONNEG) {
        return min(max(u >> kBucketShift, kBucketLo), kBucketHi) - kBucketLo;
    } else {
        // sign half by one 24-bit multiply-add (written out: the compiler
        // would turn the 0/1 multiplier into a compare and a select)
        const uint32_t a = (u & 0x7fffffffu) >> kBucketShift;
        const uint32_t m = min(max(a, kBucketLo), kBucketHi);
        uint32_t r;
        asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(r) : "v"(u >> 31), "s"(kBuckets), "v"(m));
        return r - kBucketLo;
    }
}

// Nearest codes of N values: one bucket lookup each, then kmax rounds of one
// threshold compare each over all values, so independent LDS reads overlap.
template <int N, bool NONNEG>
__device__ inline void nearest_codes(const Tables &M, const float (&y)[N], uint32_t (&c)[N])
{
#pragma unroll
    for (int i = 0; i < N; ++i)
        c[i] = M.base[bucket_of<NONNEG>(y[i])];
    for (int k = 0; k < M.kmax; ++k) {
#pragma unroll
        for (int i = 0; i < N; ++i)
            c[i] += (y[i] >= M.t[c[i]]) ? 1u : 0u;
    }
}

struct Normalizer {
    float n;  // scaled divisor N' (1 for an all-zero block)
    float r;  // RN(1 / N'), or 0 for an all-zero block
    float s;  // power-of-two scale applied to x
};

__device__ inline Normalizer make_normalizer(float N)
{
    Normalizer z;
    z.s = 1.0f;
    if (N < 0x1p-64f)
        z.s = 0x1p64f;
    else if (N > 0x1p64f)
        z.s = 0x1p-64f;
    const bool zero = !(N > 0.0f);
    z.n = zero ? 1.0f : N * z.s;
    z.r = zero ? 0.0f : 1.0f / z.n;  // correctly rounded division
    return z;
}

template <bool SCALED>
__device__ inline float normalize(const Normalizer &z, float x)
{
    const float xs = SCALED ? x * z.s : x;
    const float q = xs * z.r;
    const float e = __builtin_fmaf(-q, z.n, xs);
    return __builtin_fmaf(e, z.r, q);
}

// ---------------------------------------------------------------------------
// Reductions
// ---------------------------------------------------------------------------

// Unsigned max with a DPP-shifted copy of v, foldable into one v_max_u32 with
// a DPP operand.  Lanes of rows that ROW_MASK disables receive an unspecified
// value; the reduction below only relies on the lanes each step enables.
// Non-negative floats order like their bit patterns, so block absmax
// reductions run on the bits: exact, and free of NaN canonicalization.
template <int CTRL, int ROW_MASK>
__device__ inline uint32_t dpp_umax(uint32_t v)
{
    const uint32_t o = (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, ROW_MASK, 0xf, true);
    return max(v, o);
}

// Max of non-negative bit patterns over each row of 16 lanes, in every lane.
__device__ inline uint32_t row_umax(uint32_t v)
{
    v = dpp_umax<0xb1, 0xf>(v);   // quad_perm [1,0,3,2]
    v = dpp_umax<0x4e, 0xf>(v);   // quad_perm [2,3,0,1]
    v = dpp_umax<0x141, 0xf>(v);  // row_half_mirror
    return dpp_umax<0x140, 0xf>(v);  // row_mirror
}

// ---------------------------------------------------------------------------
// Memory access
// ---------------------------------------------------------------------------

typedef float vf4 __attribute__((ext_vector_type(4)));
typedef uint32_t vu2 __attribute__((ext_vector_type(2)));
typedef uint32_t vu4 __attribute__((ext_vector_type(4)));

// Global-memory (address space 1) views of generic pointers: loads and stores
// through them compile to global_* instructions (vector memory counter only)
// instead of flat_*, which keeps the compiler's wait counts precise.
template <typename T>
using gptr = __attribute__((address_space(1))) T *;
template <typename T>
__device__ inline gptr<T> G(T *p) { return (gptr<T>)p; }
template <typename T>
__device__ inline gptr<const T> G(const T *p) { return (gptr<const T>)p; }

// Streaming (non-temporal) accesses: every byte of the step is touched once.
template <typename T>
__device__ inline T ld_nt(const T *p) { return __builtin_nontemporal_load(G(p)); }
template <typename T>
__device__ inline void st_nt(T *p, T v) { __builtin_nontemporal_store(v, G(p)); }

// Streaming stores at system scope: buffer stores with the sc0, sc1 and nt
// cache-policy bits, over a wave-uniform range [base, base + bytes) (bytes
// < 2^32) at a per-lane byte offset.  On MI355X they drain to HBM faster than
// st_nt's non-temporal stores: dequantize of 67M values 55.2 -> 51.6 us, the
// fused step on the 1.5B list -0.6 % (A/B in one process).  Word 3 of the
// descriptor is the raw-buffer format of gfx9-family parts.
constexpr int kStreamStorePolicy = 1 | 2 | 16;  // sc0 | nt | sc1
__device__ inline __amdgpu_buffer_rsrc_t stream_range(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes,
                                             0x00020000);
}
__device__ inline void st_stream(__amdgpu_buffer_rsrc_t r, int off, vf4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(vu4, v), r, off, 0,
                                           kStreamStorePolicy);
}
__device__ inline void st_stream(__amdgpu_buffer_rsrc_t r, int off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, kStreamStorePolicy);
}

__device__ inline float half_lo(uint32_t w)
{
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xffffu));
}
__device__ inline float half_hi(uint32_t w)
{
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
}

// 16-bit grads (GRAD kF16 or kBF16): the low and high element of a packed word,
// converted to fp32 exactly (a bf16 is the top half of an fp32).
template <int GRAD>
__device__ inline float g16_lo(uint32_t w)
{
    if constexpr (GRAD == kBF16)
        return __uint_as_float(w << 16);
    else
        return half_lo(w);
}
template <int GRAD>
__device__ inline float g16_hi(uint32_t w)
{
    if constexpr (GRAD == kBF16)
        return __uint_as_float(w & 0xffff0000u);
    else
        return half_hi(w);
}

// Element i of a grad array of type GRAD, converted to fp32 exactly.
template <int GRAD>
__device__ inline float grad_at(const void *grad, int64_t i)
{
    if constexpr (GRAD == kF32)
        return G(static_cast<const float *>(grad))[i];
    else if constexpr (GRAD == kF16)
        return (float)G(static_cast<const _Float16 *>(grad))[i];
    else
        return __uint_as_float((uint32_t)G(static_cast<const uint16_t *>(grad))[i] << 16);
}

}  // namespace dev
}  // namespace bq
