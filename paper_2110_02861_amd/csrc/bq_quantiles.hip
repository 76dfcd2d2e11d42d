// Quantile estimation for the quantile map (App. F.2, App. G, "SRAM-Quantiles"):
// the tensor is cut into chunks of kQChunk values; each chunk is sorted in
// on-chip memory (LDS) by one workgroup, which writes the chunk's 257 sample
// quantiles Q_c(i / 257) = sorted[floor(i L / 257)]; the estimate of each
// quantile is the average of the chunk quantiles, weighted by chunk length.
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

constexpr int kQThreads = 512;
constexpr int kQPerThread = kQChunk / kQThreads;  // 8
static_assert(kQChunk == kQThreads * kQPerThread, "chunk shape");

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

// One workgroup per chunk: load (pad with the largest key), bitonic sort in
// LDS, write the 257 sample quantiles.
__global__ __launch_bounds__(kQThreads) void chunk_quantiles_kernel(const float *__restrict__ x,
                                                                    int64_t n,
                                                                    float *__restrict__ partial)
{
    __shared__ uint32_t keys[kQChunk];
    const int64_t c0 = (int64_t)blockIdx.x * kQChunk;
    const int64_t rem = n - c0;
    const int L = rem >= kQChunk ? kQChunk : (int)rem;
    const int tid = threadIdx.x;
#pragma unroll
    for (int k = 0; k < kQPerThread; ++k) {
        const int i = tid + k * kQThreads;
        keys[i] = i < L ? order_key(G(x)[c0 + i]) : 0xffffffffu;
    }
    __syncthreads();
    // bitonic network over kQChunk keys: kQChunk / 2 compare-exchanges per pass
    for (int size = 2; size <= kQChunk; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
#pragma unroll
            for (int k = 0; k < kQChunk / 2 / kQThreads; ++k) {
                const int t = tid + k * kQThreads;
                const int i = 2 * t - (t & (stride - 1));
                const int j = i + stride;
                const uint32_t a = keys[i], b = keys[j];
                const bool up = (i & size) == 0;
                if ((a > b) == up) {
                    keys[i] = b;
                    keys[j] = a;
                }
            }
            __syncthreads();
        }
    }
    if (tid <= 256) {
        const int idx = (int)(((int64_t)tid * L) / 257);
        G(partial)[(int64_t)blockIdx.x * 257 + tid] = key_value(keys[idx]);
    }
}

// One workgroup per group of kQGroup chunks: length-weighted sums of the chunk
// quantiles, in chunk order, in double.
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
    for (int64_t c = c0; c < c1; ++c) {
        const int64_t rem = n - c * kQChunk;
        const double L = (double)(rem >= kQChunk ? kQChunk : rem);
        s += L * (double)G(partial)[c * 257 + tid];
    }
    G(gsum)[(int64_t)blockIdx.x * 257 + tid] = s;
}

// One workgroup: sum the group sums in order, average, then Eq. 5.
__global__ __launch_bounds__(kQThreads) void combine_quantiles_kernel(
    const double *__restrict__ gsum, int64_t n, int64_t ngroups, float *__restrict__ out)
{
    __shared__ double Q[257];
    __shared__ double q[256];
    __shared__ float map[256];
    const int tid = threadIdx.x;
    if (tid <= 256) {
        double s = 0.0;
        for (int64_t g = 0; g < ngroups; ++g)
            s += G(gsum)[g * 257 + tid];
        Q[tid] = s / (double)n;
    }
    __syncthreads();
    if (tid < 256)
        q[tid] = (Q[tid] + Q[tid + 1]) * 0.5;
    __syncthreads();
    if (tid == 0) {
        double amax = 0.0;
        for (int i = 0; i < 256; ++i)
            amax = fmax(amax, fabs(q[i]));
        for (int i = 0; i < 256; ++i) {
            float v = (float)(amax > 0.0 ? q[i] / amax : q[i]);
            if (i > 0 && !(v > map[i - 1]))
                v = next_up(map[i - 1]);
            map[i] = v;
        }
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
    hipLaunchKernelGGL(combine_quantiles_kernel, dim3(1), dim3(kQThreads), 0, stream, gsum, n,
                       ngroups, out);
    return hipGetLastError();
}

}  // namespace bq
