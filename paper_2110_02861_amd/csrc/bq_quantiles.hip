// Quantile estimation for the quantile map (App. F.2, App. G, "SRAM-Quantiles"):
// the tensor is cut into chunks of kQChunk values; each chunk is sorted on
// chip (registers, lane shuffles and LDS) by one workgroup, which writes the
// chunk's 257 sample quantiles Q_c(i / 257) = sorted[floor(i L / 257)]; the
// estimate of each quantile is the average of the chunk quantiles, weighted
// by chunk length.
// Instead of the atomic averaging in DRAM that App. G describes, the chunk
// quantiles are summed in a fixed order -- sequentially within groups of
// kQGroup consecutive chunks (one workgroup per group), then sequentially over
// the groups -- so the result is deterministic.  From the averaged quantiles
// Q(p) the map follows Eq. 5: q_i = (Q(i / 257) + Q((i + 1) / 257)) / 2,
// divided by max |q_i|, rounded to fp32, equal entries moved up by one ulp.
#include "bq_device.h"

namespace bq {
namespace {

using namespace dev;

constexpr int kQThreads = 256;                    // threads per chunk sort
constexpr int kQPerThread = kQChunk / kQThreads;  // keys per thread
constexpr int kQWaveKeys = 64 * kQPerThread;      // keys held by one wave
static_assert(kQChunk == kQThreads * kQPerThread && kQPerThread % 4 == 0, "chunk shape");
constexpr int kCombineThreads = 512;              // >= 257

// fp32 bit pattern -> unsigned key with the same order (finite values)
__device__ inline uint32_t order_key(float f)
{
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float key_value(uint32_t k)
{
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// Bitonic sort of kQChunk keys by one workgroup, P = kQPerThread keys per
// thread: thread t holds sorted positions P t .. P t + P - 1 when done.  A
// pass compares position p with p ^ J (the lower position keeps the smaller
// key when (p & K) == 0, the larger otherwise).  Partners at distance J < P
// are in the same thread, at P <= J < 64 P in another lane of the same wave
// (exchanged by lane shuffles), at J >= 64 P in another wave (exchanged
// through LDS).  The whole network is unrolled at compile time so the keys
// stay in registers.

// The key of lane (lane ^ M) of the wave: DPP for M = 1, 2 (quad permutes)
// and 8 (rotation of a 16-lane row by 8), a swizzle within 32 lanes for
// M = 4, 16, a permute through the LDS crossbar for M = 32.
template <int M>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v)
{
    const int x = (int)v;
    if constexpr (M == 1)
        return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0xB1, 0xF, 0xF, false);
    else if constexpr (M == 2)
        return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0x4E, 0xF, 0xF, false);
    else if constexpr (M == 8)
        return (uint32_t)__builtin_amdgcn_mov_dpp(x, 0x128, 0xF, 0xF, false);
    else if constexpr (M == 4 || M == 16)
        return (uint32_t)__builtin_amdgcn_ds_swizzle(x, 0x1F | (M << 10));
    else
        return (uint32_t)__shfl_xor(x, M);
}

// median of three: med3(a, b, 0) = min(a, b), med3(a, b, ~0) = max(a, b), so
// one instruction takes the kept key of a compare-exchange given a per-lane
// selector
__device__ __forceinline__ uint32_t med3u(uint32_t a, uint32_t b, uint32_t s)
{
    uint32_t r;
    asm("v_med3_u32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(s));
    return r;
}

template <int K, int J>
__device__ __forceinline__ void bitonic_pass(uint32_t (&a)[kQPerThread], uint32_t *keys, int tid)
{
    if constexpr (J >= kQWaveKeys) {
        constexpr int m = J / kQPerThread;  // partner thread distance (another wave)
        constexpr int V = kQPerThread / 4;  // 16-byte vectors per thread
#pragma unroll
        for (int v = 0; v < V; ++v)
            reinterpret_cast<vu4 *>(keys)[V * tid + v] =
                vu4{a[4 * v], a[4 * v + 1], a[4 * v + 2], a[4 * v + 3]};
        __syncthreads();
        const int pt = tid ^ m;
        uint32_t b[kQPerThread];
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const vu4 bv = reinterpret_cast<const vu4 *>(keys)[V * pt + v];
            b[4 * v] = bv.x;
            b[4 * v + 1] = bv.y;
            b[4 * v + 2] = bv.z;
            b[4 * v + 3] = bv.w;
        }
        __syncthreads();
        const bool keep_min = ((tid & m) == 0) == (((kQPerThread * tid) & K) == 0);
        const uint32_t sel = keep_min ? 0u : ~0u;
#pragma unroll
        for (int i = 0; i < kQPerThread; ++i)
            a[i] = med3u(a[i], b[i], sel);
    } else if constexpr (J >= kQPerThread) {
        constexpr int m = J / kQPerThread;  // partner lane distance, < 64
        const bool keep_min = ((tid & m) == 0) == (((kQPerThread * tid) & K) == 0);
        const uint32_t sel = keep_min ? 0u : ~0u;
#pragma unroll
        for (int i = 0; i < kQPerThread; ++i)
            a[i] = med3u(a[i], lane_xor<m>(a[i]), sel);
    } else {
#pragma unroll
        for (int i = 0; i < kQPerThread; ++i) {
            if ((i & J) == 0) {
                const bool asc = ((kQPerThread * tid + i) & K) == 0;
                const uint32_t lo = asc ? 0u : ~0u;
                const uint32_t x = a[i], y = a[i | J];
                a[i] = med3u(x, y, lo);
                a[i | J] = med3u(x, y, ~lo);
            }
        }
    }
    if constexpr (J > 1)
        bitonic_pass<K, J / 2>(a, keys, tid);
}

template <int K>
__device__ __forceinline__ void bitonic_sort(uint32_t (&a)[kQPerThread], uint32_t *keys, int tid)
{
    bitonic_pass<K, K / 2>(a, keys, tid);
    if constexpr (K < kQChunk)
        bitonic_sort<2 * K>(a, keys, tid);
}

// One workgroup per chunk: load (padded with the largest key; the network
// sorts any arrangement, so the loads are coalesced: element
// 4t + 4 kQThreads h + r of the chunk goes to slot 4h + r of thread t), sort,
// write the 257 sample quantiles.
__global__ __launch_bounds__(kQThreads) void chunk_quantiles_kernel(const float *__restrict__ x,
                                                                    int64_t n,
                                                                    float *__restrict__ partial)
{
    __shared__ __attribute__((aligned(16))) uint32_t keys[kQChunk];
    const int64_t c0 = (int64_t)blockIdx.x * kQChunk;
    const int64_t rem = n - c0;
    const int L = rem >= kQChunk ? kQChunk : (int)rem;
    const int tid = threadIdx.x;
    // 16-byte loads need x itself 16-byte aligned (c0 is a multiple of 4096
    // values); a view that is only 4-byte aligned takes the scalar loads
    const bool vec = L == kQChunk && (reinterpret_cast<uintptr_t>(x) & 15u) == 0;
    uint32_t a[kQPerThread];
#pragma unroll
    for (int h = 0; h < kQPerThread / 4; ++h) {
        const int e = 4 * tid + 4 * kQThreads * h;
        if (vec) {
            const vf4 v = ld_nt(reinterpret_cast<const vf4 *>(x + c0 + e));
            a[4 * h] = order_key(v.x);
            a[4 * h + 1] = order_key(v.y);
            a[4 * h + 2] = order_key(v.z);
            a[4 * h + 3] = order_key(v.w);
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                a[4 * h + r] = e + r < L ? order_key(G(x)[c0 + e + r]) : 0xffffffffu;
        }
    }
    bitonic_sort<2>(a, keys, tid);
    constexpr int V = kQPerThread / 4;
#pragma unroll
    for (int v = 0; v < V; ++v)
        reinterpret_cast<vu4 *>(keys)[V * tid + v] =
            vu4{a[4 * v], a[4 * v + 1], a[4 * v + 2], a[4 * v + 3]};
    __syncthreads();
    for (int i = tid; i <= 256; i += kQThreads) {
        const int idx = (int)(((int64_t)i * L) / 257);
        G(partial)[(int64_t)blockIdx.x * 257 + i] = key_value(keys[idx]);
    }
}

// One workgroup per group of kQGroup chunks: length-weighted sums of the chunk
// quantiles, in chunk order, in double.  A full group's kQGroup loads are all
// issued before the first add (the adds keep chunk order).
__global__ __launch_bounds__(320) void group_sums_kernel(const float *__restrict__ partial,
                                                         int64_t n, int64_t nchunks,
                                                         double *__restrict__ gsum)
{
    const int tid = threadIdx.x;
    if (tid > 256)
        return;
    const int64_t c0 = (int64_t)blockIdx.x * kQGroup;
    const int64_t c1 = c0 + kQGroup < nchunks ? c0 + kQGroup : nchunks;
    double s = 0.0;
    if (c1 - c0 == kQGroup) {
        float v[kQGroup];
#pragma unroll
        for (int k = 0; k < kQGroup; ++k)
            v[k] = G(partial)[(c0 + k) * 257 + tid];
#pragma unroll
        for (int k = 0; k < kQGroup; ++k) {
            const int64_t rem = n - (c0 + k) * kQChunk;
            const double L = (double)(rem >= kQChunk ? kQChunk : rem);
            s += L * (double)v[k];
        }
    } else {
        for (int64_t c = c0; c < c1; ++c) {
            const int64_t rem = n - c * kQChunk;
            const double L = (double)(rem >= kQChunk ? kQChunk : rem);
            s += L * (double)G(partial)[c * 257 + tid];
        }
    }
    G(gsum)[(int64_t)blockIdx.x * 257 + tid] = s;
}

// One workgroup: sum the group sums in order, average, then Eq. 5.
__global__ __launch_bounds__(kCombineThreads) void combine_quantiles_kernel(
    const double *__restrict__ gsum, int64_t n, int64_t ngroups, float *__restrict__ out)
{
    __shared__ double Q[257];
    __shared__ double q[256];
    __shared__ double red[256];
    __shared__ float map[256];
    __shared__ int tie;
    const int tid = threadIdx.x;
    if (tid == 0)
        tie = 0;
    if (tid <= 256) {
        // in group order; loads issued 32 at a time
        double s = 0.0;
        int64_t g = 0;
        for (; g + 32 <= ngroups; g += 32) {
            double v[32];
#pragma unroll
            for (int k = 0; k < 32; ++k)
                v[k] = G(gsum)[(g + k) * 257 + tid];
#pragma unroll
            for (int k = 0; k < 32; ++k)
                s += v[k];
        }
        for (; g < ngroups; ++g)
            s += G(gsum)[g * 257 + tid];
        Q[tid] = s / (double)n;
    }
    __syncthreads();
    if (tid < 256) {
        q[tid] = (Q[tid] + Q[tid + 1]) * 0.5;
        red[tid] = fabs(q[tid]);
    }
    __syncthreads();
    // max |q_i| by a tree (a maximum is exact in any order)
    for (int h = 128; h > 0; h >>= 1) {
        if (tid < h)
            red[tid] = fmax(red[tid], red[tid + h]);
        __syncthreads();
    }
    const double amax = red[0];
    if (tid < 256)
        map[tid] = (float)(amax > 0.0 ? q[tid] / amax : q[tid]);
    __syncthreads();
    // equal neighbours (ties in the sample) moved up by one ulp, in order; the
    // serial pass runs only when some neighbour is not strictly above its
    // predecessor
    if (tid >= 1 && tid < 256 && !(map[tid] > map[tid - 1]))
        tie = 1;
    __syncthreads();
    if (tid == 0 && tie) {
        for (int i = 1; i < 256; ++i)
            if (!(map[i] > map[i - 1]))
                map[i] = next_up(map[i - 1]);
    }
    __syncthreads();
    if (tid < 256)
        G(out)[tid] = map[tid];
}

}  // namespace

hipError_t launch_quantile_codebook(const float *x, int64_t n, void *workspace, float *out,
                                    hipStream_t stream)
{
    const int64_t nchunks = (n + kQChunk - 1) / kQChunk;
    const int64_t ngroups = (nchunks + kQGroup - 1) / kQGroup;
    float *partial = static_cast<float *>(workspace);
    double *gsum = reinterpret_cast<double *>(static_cast<char *>(workspace) +
                                              quantile_partial_bytes(n));
    hipLaunchKernelGGL(chunk_quantiles_kernel, dim3((unsigned)nchunks), dim3(kQThreads), 0,
                       stream, x, n, partial);
    hipLaunchKernelGGL(group_sums_kernel, dim3((unsigned)ngroups), dim3(320), 0, stream, partial,
                       n, nchunks, gsum);
    hipLaunchKernelGGL(combine_quantiles_kernel, dim3(1), dim3(kCombineThreads), 0, stream, gsum,
                       n, ngroups, out);
    return hipGetLastError();
}

}  // namespace bq
