// HIP kernels for gfx950: block-wise quantize / dequantize and the fused
// 8-bit optimizer step (Dettmers et al., "8-bit Optimizers via Block-wise
// Quantization", Sections 2.2, 3, 3.1; Eq. 1-4).
//
// Execution model
//   * Persistent workgroups of 256 threads (4 wave64).  A workgroup first
//     stages each codebook, its decision thresholds and a bucket index in LDS,
//     then walks a strided list of tiles.  A tile is 2048 elements (or one 4096
//     block); each thread owns EPT contiguous elements, moved with 128-bit (or
//     64-bit, for 8 codes) accesses.
//   * A quantization block of B elements is owned by B / EPT consecutive
//     threads: its absmax is a DPP reduction inside a wave plus, when the block
//     spans waves, one LDS exchange behind one barrier.
//   * Tiles never span tensors, so neither do blocks.
//
// Exact nearest code (Eq. 3, ties to the lower index)
//   With T_j the smallest fp32 above the midpoint of codes j and j+1 and
//   T_255 = +inf, the nearest code of y is #{j : y >= T_j}.  Instead of a
//   binary search over T, the sign, exponent and top 7 mantissa bits of y
//   select a bucket (a run of fp32 bit patterns); LDS holds, per bucket, the
//   number of thresholds at or below the bucket's smallest value.  At most K
//   thresholds lie inside any bucket (K is computed in the prologue; K = 1 for
//   the dynamic maps), so K compares against T finish the count.  This is
//   exact for every strictly increasing map.
//
// Exact division
//   y = x / N is the correctly rounded quotient: per block r = RN(1/N'), per
//   element q = x' r, e = fma(-q, N', x'), y = fma(e, r, q) (Markstein's
//   correction), with x' = x s, N' = N s and s a power of two keeping N' within
//   [2^-64, 2^64].  Exact whenever |y| >= 2^-100, far below any threshold of a
//   map whose nonzero magnitudes are >= 2^-60.  An all-zero block uses r = 0,
//   which sends every element to y = 0.
//
// State arithmetic is fp32 without contraction (-ffp-contract=off), in the
// operation order of the update's definition, so codes and absmax are
// reproducible bit for bit.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bq_internal.h"

namespace bq {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// Bucket index: bits [30:16] of |y| (8 exponent + 7 mantissa bits), clamped to
// the binades [2^-25, 2^1).  Magnitudes below 2^-25 share the first bucket,
// magnitudes of 1 and above the last.
constexpr uint32_t kBucketShift = 16;
constexpr uint32_t kBucketLo = (127u - 25u) << 7;
constexpr uint32_t kBucketHi = (127u << 7) + 127u;
constexpr uint32_t kBuckets = kBucketHi - kBucketLo + 1;  // per sign

// ---------------------------------------------------------------------------
// Codebook tables in LDS
// ---------------------------------------------------------------------------

struct MapTables {
    float q[256];                  // codebook values (dequantization)
    float t[256];                  // decision thresholds, t[255] = +inf
    uint8_t base[2 * kBuckets];    // [sign * kBuckets + bucket] -> #{j : t_j <= bucket min}
    int kmax;                      // max thresholds strictly inside one bucket
};

__device__ inline float next_up(float f)
{
    if (f == 0.0f)
        return __uint_as_float(1u);  // smallest positive subnormal
    const uint32_t u = __float_as_uint(f);
    return __uint_as_float(f > 0.0f ? u + 1u : u - 1u);
}

// #{j : t_j <= v} for finite v (at most 255 since t_255 = +inf).
__device__ inline uint32_t count_le(const float *t, float v)
{
    uint32_t c = 0;
#pragma unroll
    for (uint32_t s = 128; s >= 1; s >>= 1)
        c += (t[c + s - 1] <= v) ? s : 0u;
    return c;
}

// Smallest and largest magnitude bit pattern of bucket b.
__device__ inline uint32_t bucket_lo_bits(uint32_t b) { return b == 0 ? 0u : (kBucketLo + b) << kBucketShift; }
__device__ inline uint32_t bucket_hi_bits(uint32_t b)
{
    return b == kBuckets - 1 ? 0x7f7fffffu : ((kBucketLo + b + 1) << kBucketShift) - 1u;
}

// Build the tables of one map; all 256 threads take part.  Contains barriers.
__device__ void stage_map(MapTables &M, const float *__restrict__ qmap)
{
    const uint32_t j = threadIdx.x;
    const float qj = qmap[j];
    M.q[j] = qj;
    float thr = __builtin_inff();
    if (j < 255) {
        // adjacent codes of a valid map are within 2^29 of each other, so the
        // double sum is exact
        const double mid = ((double)qj + (double)qmap[j + 1]) * 0.5;
        float f = (float)mid;
        if ((double)f <= mid)
            f = next_up(f);
        thr = f;
    }
    M.t[j] = thr;
    if (j == 0)
        M.kmax = 0;
    __syncthreads();

    // Each thread walks a contiguous run of buckets on each side in ascending
    // value order, so one binary search plus a forward scan gives every count.
    constexpr uint32_t kPer = (kBuckets + kThreads - 1) / kThreads;
    const uint32_t b0 = j * kPer;
    const uint32_t b1 = b0 + kPer < kBuckets ? b0 + kPer : kBuckets;
    int kmax = 0;
    if (b0 < b1) {
        // positive side: values [lo, hi] rise with b
        uint32_t c = count_le(M.t, __uint_as_float(bucket_lo_bits(b0)));
        for (uint32_t b = b0; b < b1; ++b) {
            const float lo = __uint_as_float(bucket_lo_bits(b));
            const float hi = __uint_as_float(bucket_hi_bits(b));
            while (M.t[c] <= lo)
                ++c;
            M.base[b] = (uint8_t)c;
            uint32_t e = c;
            while (M.t[e] <= hi)
                ++e;
            kmax = max(kmax, (int)(e - c));
            c = e;
        }
        // negative side: values [-hi, -lo] rise as b falls
        c = count_le(M.t, -__uint_as_float(bucket_hi_bits(b1 - 1)));
        for (uint32_t b = b1; b-- > b0;) {
            const float lo = -__uint_as_float(bucket_hi_bits(b));
            const float hi = -__uint_as_float(bucket_lo_bits(b));
            while (M.t[c] <= lo)
                ++c;
            M.base[kBuckets + b] = (uint8_t)c;
            uint32_t e = c;
            while (M.t[e] <= hi)
                ++e;
            kmax = max(kmax, (int)(e - c));
            c = e;
        }
    }
    atomicMax(&M.kmax, kmax);
}

// Bucket of y (index into MapTables::base).  NONNEG: y is +0 or positive.
template <bool NONNEG>
__device__ inline uint32_t bucket_of(float y)
{
    const uint32_t u = __float_as_uint(y);
    if constexpr (NONNEG) {
        return min(max(u >> kBucketShift, kBucketLo), kBucketHi) - kBucketLo;
    } else {
        const uint32_t a = (u & 0x7fffffffu) >> kBucketShift;
        return min(max(a, kBucketLo), kBucketHi) - kBucketLo + (u >> 31) * kBuckets;
    }
}

// Nearest codes of EPT values: one bucket lookup each, then kmax rounds of
// one threshold compare each (the rounds run over all EPT values at once so
// the LDS reads of different values overlap).
template <int EPT, bool NONNEG>
__device__ inline void nearest_codes(const MapTables &M, int kmax, const float (&y)[EPT],
                                     uint32_t (&c)[EPT])
{
#pragma unroll
    for (int i = 0; i < EPT; ++i)
        c[i] = M.base[bucket_of<NONNEG>(y[i])];
    for (int k = 0; k < kmax; ++k) {
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            c[i] += (y[i] >= M.t[c[i]]) ? 1u : 0u;
    }
}

// ---------------------------------------------------------------------------
// Exact division by the block absmax
// ---------------------------------------------------------------------------

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
// Block absmax reduction
// ---------------------------------------------------------------------------

template <int CTRL, int ROW_MASK>
__device__ inline float dpp_max(float v)
{
    const int iv = __builtin_bit_cast(int, v);
    const int o = __builtin_amdgcn_update_dpp(iv, iv, CTRL, ROW_MASK, 0xf, false);
    return fmaxf(v, __builtin_bit_cast(float, o));
}

// Max over each row of 16 lanes, left in every lane of the row.
__device__ inline float row_max(float v)
{
    v = dpp_max<0xb1, 0xf>(v);   // quad_perm [1,0,3,2]
    v = dpp_max<0x4e, 0xf>(v);   // quad_perm [2,3,0,1]
    v = dpp_max<0x141, 0xf>(v);  // row_half_mirror
    v = dpp_max<0x140, 0xf>(v);  // row_mirror
    return v;
}

__device__ inline float lane_f(float v, int lane)
{
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// Max of (x, y) over each group of GROUP consecutive threads (power of two,
// 32..256).  slots: LDS scratch of kWaves float2, double-buffered by caller.
template <int GROUP>
__device__ inline float2 group_max(float2 v, float2 *slots)
{
    v.x = row_max(v.x);
    v.y = row_max(v.y);
    v.x = dpp_max<0x142, 0xa>(v.x);  // row_bcast:15 -> lanes 31, 63 hold half maxima
    v.y = dpp_max<0x142, 0xa>(v.y);
    if constexpr (GROUP == 32) {
        const bool hi = (threadIdx.x & 32) != 0;
        return make_float2(hi ? lane_f(v.x, 63) : lane_f(v.x, 31),
                           hi ? lane_f(v.y, 63) : lane_f(v.y, 31));
    } else {
        v.x = dpp_max<0x143, 0xc>(v.x);  // row_bcast:31 -> lane 63 holds the wave max
        v.y = dpp_max<0x143, 0xc>(v.y);
        const float2 w = make_float2(lane_f(v.x, 63), lane_f(v.y, 63));
        if constexpr (GROUP == 64) {
            return w;
        } else {
            constexpr int WPG = GROUP / 64;
            const int wave = threadIdx.x >> 6;
            if ((threadIdx.x & 63) == 0)
                slots[wave] = w;
            __syncthreads();
            const int first = (wave / WPG) * WPG;
            float2 r = slots[first];
#pragma unroll
            for (int k = 1; k < WPG; ++k) {
                const float2 o = slots[first + k];
                r.x = fmaxf(r.x, o.x);
                r.y = fmaxf(r.y, o.y);
            }
            return r;
        }
    }
}

// ---------------------------------------------------------------------------
// Loads and stores of EPT contiguous elements
// ---------------------------------------------------------------------------

template <int EPT>
__device__ inline void load_f32(const float *__restrict__ p, float (&v)[EPT])
{
#pragma unroll
    for (int i = 0; i < EPT; i += 4) {
        const float4 x = *reinterpret_cast<const float4 *>(p + i);
        v[i] = x.x;
        v[i + 1] = x.y;
        v[i + 2] = x.z;
        v[i + 3] = x.w;
    }
}

template <int EPT>
__device__ inline void store_f32(float *__restrict__ p, const float (&v)[EPT])
{
#pragma unroll
    for (int i = 0; i < EPT; i += 4)
        *reinterpret_cast<float4 *>(p + i) = make_float4(v[i], v[i + 1], v[i + 2], v[i + 3]);
}

template <int EPT>
__device__ inline void load_f16(const _Float16 *__restrict__ p, float (&v)[EPT])
{
#pragma unroll
    for (int i = 0; i < EPT; i += 8) {
        const uint4 x = *reinterpret_cast<const uint4 *>(p + i);
        const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            v[i + 2 * k] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] & 0xffffu));
            v[i + 2 * k + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[k] >> 16));
        }
    }
}

template <int EPT>
__device__ inline void load_codes(const uint8_t *__restrict__ p, uint32_t (&c)[EPT])
{
    static_assert(EPT == 8 || EPT == 16, "codes per thread");
    uint32_t w[EPT / 4];
    if constexpr (EPT == 8) {
        const uint2 x = *reinterpret_cast<const uint2 *>(p);
        w[0] = x.x;
        w[1] = x.y;
    } else {
        const uint4 x = *reinterpret_cast<const uint4 *>(p);
        w[0] = x.x;
        w[1] = x.y;
        w[2] = x.z;
        w[3] = x.w;
    }
#pragma unroll
    for (int i = 0; i < EPT; ++i)
        c[i] = (w[i >> 2] >> (8 * (i & 3))) & 0xffu;
}

template <int EPT>
__device__ inline void store_codes(uint8_t *__restrict__ p, const uint32_t (&c)[EPT])
{
    uint32_t w[EPT / 4];
#pragma unroll
    for (int k = 0; k < EPT / 4; ++k)
        w[k] = c[4 * k] | (c[4 * k + 1] << 8) | (c[4 * k + 2] << 16) | (c[4 * k + 3] << 24);
    if constexpr (EPT == 8)
        *reinterpret_cast<uint2 *>(p) = make_uint2(w[0], w[1]);
    else
        *reinterpret_cast<uint4 *>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}

template <int B>
struct Shape {
    static constexpr int EPT = B >= 2048 ? B / kThreads : 8;  // elements per thread
    static constexpr int TILE = kThreads * EPT;               // elements per tile
    static constexpr int GROUP = B / EPT;                     // threads per block
    static_assert(TILE == tile_elems(B), "tile size");
};

// Requantize EPT values of one thread against map M, block absmax N.
template <int EPT, int GROUP, bool NONNEG>
__device__ inline void requantize(const MapTables &M, int kmax, float N, const float (&x)[EPT],
                                  uint32_t (&c)[EPT])
{
    const Normalizer z = make_normalizer(N);
    bool scaled = (z.s != 1.0f);
    if constexpr (GROUP >= 64)
        scaled = __builtin_amdgcn_readfirstlane((int)scaled) != 0;  // wave-uniform
    float y[EPT];
    if (!scaled) {
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            y[i] = normalize<false>(z, x[i]);
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            y[i] = normalize<true>(z, x[i]);
    }
    nearest_codes<EPT, NONNEG>(M, kmax, y, c);
}

// ---------------------------------------------------------------------------
// Fused 8-bit optimizer step
// ---------------------------------------------------------------------------

template <int OPT, int GRAD, int B>
struct StepTile {
    using S = Shape<B>;
    static constexpr int EPT = S::EPT;
    static constexpr bool kTwo = (OPT != kMomentum);

    // One tile of one tensor: e0 is this thread's first element, valid the
    // number of its elements inside the tensor (EPT on full tiles).
    template <bool FULL>
    __device__ static void run(const StepArgs &a, const TensorDesc &D, const MapTables &T1,
                               const MapTables &T2, int k1, int k2, int64_t e0, int valid,
                               float2 *slots)
    {
        const StepScalars &sc = a.sc;
        const int64_t blk = e0 / B;
        float w[EPT], g[EPT], m[EPT], v[EPT];
        uint32_t c1[EPT], c2[EPT];
        float n1 = 0.0f, n2 = 0.0f;
        if (FULL) {
            load_f32<EPT>(D.param + e0, w);
            if constexpr (GRAD == kF16)
                load_f16<EPT>(static_cast<const _Float16 *>(D.grad) + e0, g);
            else
                load_f32<EPT>(static_cast<const float *>(D.grad) + e0, g);
            load_codes<EPT>(D.s1 + e0, c1);
            if constexpr (kTwo)
                load_codes<EPT>(D.s2 + e0, c2);
            n1 = D.a1[blk];
            if constexpr (kTwo)
                n2 = D.a2[blk];
        } else {
#pragma unroll
            for (int i = 0; i < EPT; ++i) {
                const bool ok = i < valid;
                w[i] = ok ? D.param[e0 + i] : 0.0f;
                if constexpr (GRAD == kF16)
                    g[i] = ok ? (float)static_cast<const _Float16 *>(D.grad)[e0 + i] : 0.0f;
                else
                    g[i] = ok ? static_cast<const float *>(D.grad)[e0 + i] : 0.0f;
                c1[i] = ok ? D.s1[e0 + i] : 0u;
                c2[i] = (kTwo && ok) ? D.s2[e0 + i] : 0u;
            }
            if (valid > 0) {
                n1 = D.a1[blk];
                if constexpr (kTwo)
                    n2 = D.a2[blk];
            }
        }

        if (a.use_wd) {  // L2 term (Adam, Momentum); uniform across the grid
#pragma unroll
            for (int i = 0; i < EPT; ++i)
                g[i] = g[i] + sc.wd * w[i];
        }

        float mx1 = 0.0f, mx2 = 0.0f;
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            float wi = w[i];
            const float gi = g[i];
            float mi = T1.q[c1[i]] * n1;
            if constexpr (OPT == kMomentum) {
                mi = sc.b1 * mi + gi;
                wi = wi - sc.lr * mi;
            } else {
                float vi = T2.q[c2[i]] * n2;
                if constexpr (OPT == kAdamW)
                    wi = wi * sc.decay;
                mi = sc.b1 * mi + sc.omb1 * gi;
                vi = sc.b2 * vi + sc.omb2 * (gi * gi);
                const float denom = __builtin_amdgcn_sqrtf(vi) * sc.inv_sqrt_bc2 + sc.eps;
                wi = wi - sc.step_size * (mi * __builtin_amdgcn_rcpf(denom));
                if (!FULL && i >= valid)
                    vi = 0.0f;
                v[i] = vi;
                mx2 = fmaxf(mx2, vi);  // v' >= 0
            }
            if (!FULL && i >= valid)
                mi = 0.0f;
            m[i] = mi;
            w[i] = wi;
            mx1 = fmaxf(mx1, fabsf(mi));
        }

        const float2 mx = group_max<S::GROUP>(make_float2(mx1, mx2), slots);

        requantize<EPT, S::GROUP, false>(T1, k1, mx.x, m, c1);
        if constexpr (kTwo)
            requantize<EPT, S::GROUP, true>(T2, k2, mx.y, v, c2);

        if (FULL) {
            store_f32<EPT>(D.param + e0, w);
            store_codes<EPT>(D.s1 + e0, c1);
            if constexpr (kTwo)
                store_codes<EPT>(D.s2 + e0, c2);
        } else {
#pragma unroll
            for (int i = 0; i < EPT; ++i) {
                if (i < valid) {
                    D.param[e0 + i] = w[i];
                    D.s1[e0 + i] = (uint8_t)c1[i];
                    if constexpr (kTwo)
                        D.s2[e0 + i] = (uint8_t)c2[i];
                }
            }
        }
        if ((FULL || valid > 0) && (threadIdx.x % S::GROUP) == 0) {
            D.a1[blk] = mx.x;
            if constexpr (kTwo)
                D.a2[blk] = mx.y;
        }
    }
};

template <int OPT, int GRAD, int B>
__global__ __launch_bounds__(kThreads) void step_kernel(const StepArgs a)
{
    using S = Shape<B>;
    using Tile = StepTile<OPT, GRAD, B>;
    constexpr int EPT = S::EPT;

    __shared__ MapTables T1;
    __shared__ MapTables T2;
    __shared__ float2 slots[2][kWaves];

    stage_map(T1, a.q1);
    if constexpr (Tile::kTwo)
        stage_map(T2, a.q2);
    __syncthreads();
    const int k1 = __builtin_amdgcn_readfirstlane(T1.kmax);
    const int k2 = Tile::kTwo ? __builtin_amdgcn_readfirstlane(T2.kmax) : 0;

    int t = 0;
    int parity = 0;
    for (int tile = blockIdx.x; tile < a.total_tiles; tile += gridDim.x, parity ^= 1) {
        while (t + 1 < a.ntensors && tile >= a.d[t + 1].tile_begin)
            ++t;
        const TensorDesc &D = a.d[t];
        const int64_t t0 = (int64_t)(tile - D.tile_begin) * S::TILE;
        const int64_t e0 = t0 + (int64_t)threadIdx.x * EPT;
        if (t0 + S::TILE <= D.numel) {
            Tile::template run<true>(a, D, T1, T2, k1, k2, e0, EPT, slots[parity]);
        } else {
            const int64_t rem = D.numel - e0;
            const int valid = rem <= 0 ? 0 : (rem >= EPT ? EPT : (int)rem);
            Tile::template run<false>(a, D, T1, T2, k1, k2, e0, valid, slots[parity]);
        }
    }
}

// ---------------------------------------------------------------------------
// Standalone block-wise quantize / dequantize
// ---------------------------------------------------------------------------

template <int B>
struct QuantTile {
    using S = Shape<B>;
    static constexpr int EPT = S::EPT;

    template <bool FULL>
    __device__ static void run(const MapTables &T, int kmax, const float *__restrict__ x,
                               uint8_t *__restrict__ codes, float *__restrict__ absmax,
                               int64_t e0, int valid, float2 *slots)
    {
        float v[EPT];
        if (FULL) {
            load_f32<EPT>(x + e0, v);
        } else {
#pragma unroll
            for (int i = 0; i < EPT; ++i)
                v[i] = i < valid ? x[e0 + i] : 0.0f;
        }
        float mx = 0.0f;
#pragma unroll
        for (int i = 0; i < EPT; ++i)
            mx = fmaxf(mx, fabsf(v[i]));
        const float N = group_max<S::GROUP>(make_float2(mx, 0.0f), slots).x;
        uint32_t c[EPT];
        requantize<EPT, S::GROUP, false>(T, kmax, N, v, c);
        if (FULL) {
            store_codes<EPT>(codes + e0, c);
        } else {
#pragma unroll
            for (int i = 0; i < EPT; ++i)
                if (i < valid)
                    codes[e0 + i] = (uint8_t)c[i];
        }
        if ((FULL || valid > 0) && (threadIdx.x % S::GROUP) == 0)
            absmax[e0 / B] = N;
    }
};

template <int B>
__global__ __launch_bounds__(kThreads) void quantize_kernel(const float *__restrict__ qmap,
                                                            const float *__restrict__ x,
                                                            int64_t n, int64_t ntiles,
                                                            uint8_t *__restrict__ codes,
                                                            float *__restrict__ absmax)
{
    using S = Shape<B>;
    constexpr int EPT = S::EPT;
    __shared__ MapTables T;
    __shared__ float2 slots[2][kWaves];
    stage_map(T, qmap);
    __syncthreads();
    const int kmax = __builtin_amdgcn_readfirstlane(T.kmax);

    int parity = 0;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x, parity ^= 1) {
        const int64_t t0 = tile * S::TILE;
        const int64_t e0 = t0 + (int64_t)threadIdx.x * EPT;
        if (t0 + S::TILE <= n) {
            QuantTile<B>::template run<true>(T, kmax, x, codes, absmax, e0, EPT, slots[parity]);
        } else {
            const int64_t rem = n - e0;
            const int valid = rem <= 0 ? 0 : (rem >= EPT ? EPT : (int)rem);
            QuantTile<B>::template run<false>(T, kmax, x, codes, absmax, e0, valid,
                                              slots[parity]);
        }
    }
}

// Dequantize: 8 elements per thread; blocksize >= 256 keeps each thread's 8
// elements inside one block.
__global__ __launch_bounds__(kThreads) void dequantize_kernel(const float *__restrict__ qmap,
                                                              const uint8_t *__restrict__ codes,
                                                              const float *__restrict__ absmax,
                                                              int64_t n, int64_t ntiles,
                                                              int log2_blocksize,
                                                              float *__restrict__ out)
{
    constexpr int EPT = 8;
    __shared__ float q[256];
    q[threadIdx.x] = qmap[threadIdx.x];
    __syncthreads();
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t e0 = tile * (kThreads * EPT) + (int64_t)threadIdx.x * EPT;
        const int64_t rem = n - e0;
        if (rem <= 0)
            continue;
        const float N = absmax[e0 >> log2_blocksize];
        if (rem >= EPT) {
            uint32_t c[EPT];
            float v[EPT];
            load_codes<EPT>(codes + e0, c);
#pragma unroll
            for (int i = 0; i < EPT; ++i)
                v[i] = q[c[i]] * N;
            store_f32<EPT>(out + e0, v);
        } else {
            for (int i = 0; i < (int)rem; ++i)
                out[e0 + i] = q[codes[e0 + i]] * N;
        }
    }
}

// ---------------------------------------------------------------------------
// Launch helpers
// ---------------------------------------------------------------------------

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 256;
    return cus;
}

template <typename K>
int64_t persistent_grid(K kernel, int64_t tiles)
{
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) !=
            hipSuccess ||
        per_cu <= 0)
        per_cu = 1;
    const int64_t cap = (int64_t)per_cu * device_cus();
    return tiles < cap ? tiles : cap;
}

template <int OPT, int GRAD, int B>
hipError_t launch_step_t(const StepArgs &a, hipStream_t stream)
{
    auto k = step_kernel<OPT, GRAD, B>;
    const int64_t grid = persistent_grid(k, a.total_tiles);
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

template <int OPT, int GRAD>
hipError_t launch_step_b(int blocksize, const StepArgs &a, hipStream_t s)
{
    switch (blocksize) {
    case 256: return launch_step_t<OPT, GRAD, 256>(a, s);
    case 512: return launch_step_t<OPT, GRAD, 512>(a, s);
    case 1024: return launch_step_t<OPT, GRAD, 1024>(a, s);
    case 2048: return launch_step_t<OPT, GRAD, 2048>(a, s);
    case 4096: return launch_step_t<OPT, GRAD, 4096>(a, s);
    default: return hipErrorInvalidValue;
    }
}

template <int OPT>
hipError_t launch_step_g(int grad_dtype, int blocksize, const StepArgs &a, hipStream_t s)
{
    return grad_dtype == kF16 ? launch_step_b<OPT, kF16>(blocksize, a, s)
                              : launch_step_b<OPT, kF32>(blocksize, a, s);
}

template <int B>
hipError_t launch_quantize_t(const float *qmap, const float *x, int64_t n, uint8_t *codes,
                             float *absmax, hipStream_t stream)
{
    const int64_t tiles = (n + Shape<B>::TILE - 1) / Shape<B>::TILE;
    auto k = quantize_kernel<B>;
    const int64_t grid = persistent_grid(k, tiles);
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kThreads), 0, stream, qmap, x, n, tiles,
                       codes, absmax);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_step(int opt, int grad_dtype, int blocksize, const StepArgs &a,
                       hipStream_t stream)
{
    switch (opt) {
    case kAdam: return launch_step_g<kAdam>(grad_dtype, blocksize, a, stream);
    case kAdamW: return launch_step_g<kAdamW>(grad_dtype, blocksize, a, stream);
    case kMomentum: return launch_step_g<kMomentum>(grad_dtype, blocksize, a, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_quantize(const float *qmap, const float *x, int64_t n, int blocksize,
                           uint8_t *codes, float *absmax, hipStream_t stream)
{
    switch (blocksize) {
    case 256: return launch_quantize_t<256>(qmap, x, n, codes, absmax, stream);
    case 512: return launch_quantize_t<512>(qmap, x, n, codes, absmax, stream);
    case 1024: return launch_quantize_t<1024>(qmap, x, n, codes, absmax, stream);
    case 2048: return launch_quantize_t<2048>(qmap, x, n, codes, absmax, stream);
    case 4096: return launch_quantize_t<4096>(qmap, x, n, codes, absmax, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_dequantize(const float *qmap, const uint8_t *codes, const float *absmax,
                             int64_t n, int blocksize, float *out, hipStream_t stream)
{
    const int64_t tiles = (n + kThreads * 8 - 1) / (kThreads * 8);
    const int64_t grid = persistent_grid(dequantize_kernel, tiles);
    int lg = 0;
    while ((1 << lg) < blocksize)
        ++lg;
    hipLaunchKernelGGL(dequantize_kernel, dim3((unsigned)grid), dim3(kThreads), 0, stream, qmap,
                       codes, absmax, n, tiles, lg, out);
    return hipGetLastError();
}

}  // namespace bq
