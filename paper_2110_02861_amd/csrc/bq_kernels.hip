// Persistent HIP kernels for gfx950 behind the allocation-free calls
// bq_quantize_blockwise and bq_optimizer8bit_step (Dettmers et al., "8-bit
// Optimizers via Block-wise Quantization", Sections 3, 3.1; Eq. 1-4).
//
// These calls receive raw codebooks and no workspace, so each workgroup builds
// the codebook's decision tables in its own LDS once and then walks a strided
// list of tiles.  A tile is 2048 elements (or one 4096 block) of one tensor;
// each thread owns EPT contiguous elements, moved with 128-bit (or 64-bit, for
// 8 codes) accesses.  A quantization block of B elements belongs to B / EPT
// consecutive threads.  Descriptors of up to 56 tensors travel in the kernel
// arguments.  The prepared-codebook path (bq_oneshot.hip) is the faster one.
#include "bq_device.h"

namespace bq {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

using namespace dev;

struct MapTables {
    float q[256];
    float t[256];
    uint8_t base[2 * kBuckets];
    int kmax;
};

__device__ inline Tables view(const MapTables &M, int kmax)
{
    Tables T;
    T.q = M.q;
    T.t = M.t;
    T.base = M.base;
    T.kmax = kmax;
    return T;
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

// ---------------------------------------------------------------------------
// Fused 8-bit optimizer step
// ---------------------------------------------------------------------------

template <int OPT, int GRAD, int B>
struct StepTile {
    using S = Shape<B>;
    static constexpr int EPT = S::EPT;
    static constexpr bool kTwo = has_two_states(OPT);

    // One tile of one tensor: e0 is this thread's first element, valid the
    // number of its elements inside the tensor (EPT on full tiles).
    template <bool FULL>
    __device__ static void run(const StepArgs &a, const TensorDesc &D, const Tables &T1,
                               const Tables &T2, int64_t e0, int valid,
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
            } else if constexpr (OPT == kAdaGrad) {
                mi = mi + gi * gi;
                const float denom = __builtin_amdgcn_sqrtf(mi) * sc.inv_sqrt_bc2 + sc.eps;
                wi = wi - sc.step_size * (gi * __builtin_amdgcn_rcpf(denom));
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
                mx2 = fmaxf(mx2, fabsf(vi));
            }
            if (!FULL && i >= valid)
                mi = 0.0f;
            m[i] = mi;
            w[i] = wi;
            mx1 = fmaxf(mx1, fabsf(mi));
        }

        const float2 mx = group_max<S::GROUP>(make_float2(mx1, mx2), slots);

        requantize<EPT, S::GROUP, false>(T1, mx.x, m, c1);
        if constexpr (kTwo)
            requantize<EPT, S::GROUP, true>(T2, mx.y, v, c2);

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

    build_tables<kThreads>(a.q1, T1.q, T1.t, T1.base, &T1.kmax);
    if constexpr (Tile::kTwo)
        build_tables<kThreads>(a.q2, T2.q, T2.t, T2.base, &T2.kmax);
    const Tables V1 = view(T1, __builtin_amdgcn_readfirstlane(T1.kmax));
    const Tables V2 = view(T2, Tile::kTwo ? __builtin_amdgcn_readfirstlane(T2.kmax) : 0);

    int t = 0;
    int parity = 0;
    for (int tile = blockIdx.x; tile < a.total_tiles; tile += gridDim.x, parity ^= 1) {
        while (t + 1 < a.ntensors && tile >= a.d[t + 1].tile_begin)
            ++t;
        const TensorDesc &D = a.d[t];
        const int64_t t0 = (int64_t)(tile - D.tile_begin) * S::TILE;
        const int64_t e0 = t0 + (int64_t)threadIdx.x * EPT;
        if (t0 + S::TILE <= D.numel) {
            Tile::template run<true>(a, D, V1, V2, e0, EPT, slots[parity]);
        } else {
            const int64_t rem = D.numel - e0;
            const int valid = rem <= 0 ? 0 : (rem >= EPT ? EPT : (int)rem);
            Tile::template run<false>(a, D, V1, V2, e0, valid, slots[parity]);
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
    __device__ static void run(const Tables &T, const float *__restrict__ x,
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
        requantize<EPT, S::GROUP, false>(T, N, v, c);
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
    build_tables<kThreads>(qmap, T.q, T.t, T.base, &T.kmax);
    const Tables V = view(T, __builtin_amdgcn_readfirstlane(T.kmax));

    int parity = 0;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x, parity ^= 1) {
        const int64_t t0 = tile * S::TILE;
        const int64_t e0 = t0 + (int64_t)threadIdx.x * EPT;
        if (t0 + S::TILE <= n) {
            QuantTile<B>::template run<true>(V, x, codes, absmax, e0, EPT, slots[parity]);
        } else {
            const int64_t rem = n - e0;
            const int valid = rem <= 0 ? 0 : (rem >= EPT ? EPT : (int)rem);
            QuantTile<B>::template run<false>(V, x, codes, absmax, e0, valid,
                                              slots[parity]);
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
    case kAdaGrad: return launch_step_g<kAdaGrad>(grad_dtype, blocksize, a, stream);
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

}  // namespace bq
