// Streaming-ceiling kernel for the benchmark (libbq_stream.so, not part of the
// optimizer library): moves the fused 8-bit Adam step's byte mix -- read fp32
// param, fp16 grad, two uint8 states and two fp32 block absmaxes; write back
// the param, both states and both absmaxes -- with no arithmetic beyond an XOR
// by a caller key, over flat buffers, with 512-thread workgroups, 4 contiguous
// elements per thread and chunk, and non-temporal loads and stores.  Variants
// differ in chunks per thread (1 or 2), in where the absmax read sits (with
// the element loads, or after them), and in whether each workgroup first
// stages a 16 KiB L2-resident table in LDS (as a kernel with decision tables
// does) and reads one entry of it per thread.  With key 0 every buffer keeps
// its contents, so the call can be repeated on the same data.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float vf4 __attribute__((ext_vector_type(4)));
typedef uint32_t vu2 __attribute__((ext_vector_type(2)));
typedef uint32_t vu4 __attribute__((ext_vector_type(4)));

template <typename T>
__device__ inline T ld(const T *p) { return __builtin_nontemporal_load(p); }
template <typename T>
__device__ inline void st(T *p, T v) { __builtin_nontemporal_store(v, p); }

constexpr int kThreads = 512;

constexpr int kTableWords = 4096;  // 16 KiB

template <int CHUNKS, bool EARLY_ABSMAX, bool TABLE>
// (no __restrict__ on the buffers: with it the compiler dropped the
// non-temporal hint from the stores of the one-chunk variants)
__global__ __launch_bounds__(kThreads) void stream_kernel(float *w, const uint16_t *g,
                                                          uint8_t *c1, uint8_t *c2, float *a1,
                                                          float *a2, int lg_block, uint32_t key,
                                                          const uint32_t *table)
{
    __shared__ uint32_t lds[TABLE ? kTableWords : 1];
    if (TABLE) {
        for (int i = threadIdx.x; i < kTableWords; i += kThreads)
            lds[i] = table[i];
        __syncthreads();
    }
    constexpr int kTile = kThreads * 4 * CHUNKS;
    const int64_t t0 = (int64_t)blockIdx.x * kTile;
    const int64_t blocks_per_tile = (int64_t)kTile >> lg_block;
    const bool owner = threadIdx.x < blocks_per_tile;  // one thread per block
    const int64_t b = (t0 >> lg_block) + threadIdx.x;
    float n1 = 0.0f, n2 = 0.0f;
    if (EARLY_ABSMAX && owner) {
        n1 = a1[b];
        n2 = a2[b];
    }
    vu4 wv[CHUNKS];
    vu2 gv[CHUNKS];
    uint32_t k1[CHUNKS], k2[CHUNKS];
#pragma unroll
    for (int c = 0; c < CHUNKS; ++c) {
        const int64_t e = t0 + c * (kThreads * 4) + threadIdx.x * 4;
        wv[c] = ld(reinterpret_cast<const vu4 *>(w + e));
        gv[c] = ld(reinterpret_cast<const vu2 *>(g + e));
        k1[c] = ld(reinterpret_cast<const uint32_t *>(c1 + e));
        k2[c] = ld(reinterpret_cast<const uint32_t *>(c2 + e));
    }
    if (!EARLY_ABSMAX && owner) {
        n1 = a1[b];
        n2 = a2[b];
    }
    const uint32_t tk = TABLE ? lds[k1[0] & (kTableWords - 1)] & key : 0u;
#pragma unroll
    for (int c = 0; c < CHUNKS; ++c) {
        const int64_t e = t0 + c * (kThreads * 4) + threadIdx.x * 4;
        const uint32_t gk = ((gv[c].x ^ gv[c].y) & key) ^ tk;
        st(reinterpret_cast<vu4 *>(w + e), wv[c] ^ gk);
        st(reinterpret_cast<uint32_t *>(c1 + e), k1[c] ^ key);
        st(reinterpret_cast<uint32_t *>(c2 + e), k2[c] ^ key);
    }
    if (owner) {
        a1[b] = __uint_as_float(__float_as_uint(n1) ^ key);
        a2[b] = __uint_as_float(__float_as_uint(n2) ^ key);
    }
}

template <int CHUNKS, bool EARLY, bool TABLE>
hipError_t launch(float *w, const uint16_t *g, uint8_t *c1, uint8_t *c2, float *a1, float *a2,
                  int64_t n, int lg, uint32_t key, const uint32_t *table, hipStream_t stream)
{
    const int64_t tiles = n / (kThreads * 4 * CHUNKS);
    hipLaunchKernelGGL((stream_kernel<CHUNKS, EARLY, TABLE>), dim3((unsigned)tiles),
                       dim3(kThreads), 0, stream, w, g, c1, c2, a1, a2, lg, key, table);
    return hipGetLastError();
}

}  // namespace

extern "C" {

// Number of variants: 0 = 1 chunk, absmax read after the element loads;
// 1 = 1 chunk, absmax read first; 2, 3 = the same with 2 chunks; 4, 5 = 1 and
// 2 chunks (absmax read after the loads) with the staged 16 KiB table.
int bq_stream_variants(void) { return 6; }

// n: elements, a positive multiple of 4096; blocksize: power of two in
// [256, 4096]; buffers 16-byte aligned (absmax: n / blocksize floats each);
// table: 4096 uint32 (read by variants 4 and 5 only).  Returns 0, -1 for a
// bad argument, or the HIP error code of the launch.
int bq_stream_ceiling(int variant, float *w, const uint16_t *g, uint8_t *c1, uint8_t *c2,
                      float *a1, float *a2, int64_t n, int32_t blocksize, uint32_t key,
                      const uint32_t *table, hipStream_t stream)
{
    if (!w || !g || !c1 || !c2 || !a1 || !a2 || n <= 0 || n % 4096 != 0 ||
        n / 2048 > INT32_MAX || blocksize < 256 || blocksize > 4096 ||
        (blocksize & (blocksize - 1)) != 0 || (variant >= 4 && !table))
        return -1;
    int lg = 0;
    while ((1 << lg) < blocksize)
        ++lg;
    hipError_t e;
    switch (variant) {
    case 0: e = launch<1, false, false>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 1: e = launch<1, true, false>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 2: e = launch<2, false, false>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 3: e = launch<2, true, false>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 4: e = launch<1, false, true>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 5: e = launch<2, false, true>(w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    default: return -1;
    }
    return (int)e;
}

}  // extern "C"
