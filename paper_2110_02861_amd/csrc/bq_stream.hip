// Streaming-ceiling kernel for the benchmark (libbq_stream.so, not part of the
// optimizer library): moves the fused 8-bit Adam step's byte mix -- read fp32
// param, fp16 grad, two uint8 states and two fp32 block absmaxes; write back
// the param, both states and both absmaxes -- with no arithmetic beyond an XOR
// by a caller key, over flat buffers, with 512-thread workgroups, 4 contiguous
// elements per thread and chunk, and non-temporal loads and stores.  Variants
// differ in chunks per thread (1 or 2), in where the absmax read sits (with
// the element loads, or after them), and in whether each workgroup first
// stages a 16 KiB L2-resident table in LDS (as a kernel with decision tables
// does) and reads one entry of it per thread.  Further variants take the
// step's own launch shape (2 chunks; 14,080 B of table granules loaded from L2
// before the element loads and written to LDS after them) with the number of
// resident workgroups per CU set by a dynamic LDS pad (3, as the step's
// register use allows, or 2), and one moves the codes and grads 16 B per lane
// through LDS.  With key 0 every buffer keeps its contents, so the call can be
// repeated on the same data.
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

// The step's shape: 2 chunks of 4 elements per thread; the table granules
// are issued first and written to LDS after the element loads (one entry read
// back per thread).  WIDE: codes and grads move 16 B per lane (thread t loads
// 16 codes of state 1 (t < 256) or 2, and 8 grads), exchanged through LDS.
constexpr int kGranules = 880;
template <bool WIDE>
__global__ __launch_bounds__(kThreads) void stream_step_kernel(float *w, const uint16_t *g,
                                                               uint8_t *c1, uint8_t *c2,
                                                               float *a1, float *a2, int lg_block,
                                                               uint32_t key, const vu4 *table)
{
    constexpr int kTile = kThreads * 8;
    __shared__ vu4 tab[kGranules];
    __shared__ vu4 xc[WIDE ? kThreads : 1];  // codes: state 1 then state 2
    __shared__ vu4 xg[WIDE ? kThreads : 1];  // grads
    const int tid = threadIdx.x;
    vu4 gran[2];
    gran[0] = table[tid];
    gran[1] = table[min(tid + kThreads, kGranules - 1)];
    const int64_t t0 = (int64_t)blockIdx.x * kTile;
    uint8_t *cs = tid < kThreads / 2 ? c1 : c2;
    const int64_t ce = t0 + (tid & (kThreads / 2 - 1)) * 16;
    vu4 wv[2], cw, gw;
    vu2 gv[2];
    uint32_t k1[2], k2[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int64_t e = t0 + c * (kThreads * 4) + tid * 4;
        wv[c] = ld(reinterpret_cast<const vu4 *>(w + e));
        if (!WIDE) {
            gv[c] = ld(reinterpret_cast<const vu2 *>(g + e));
            k1[c] = ld(reinterpret_cast<const uint32_t *>(c1 + e));
            k2[c] = ld(reinterpret_cast<const uint32_t *>(c2 + e));
        }
    }
    if (WIDE) {
        cw = ld(reinterpret_cast<const vu4 *>(cs + ce));
        gw = ld(reinterpret_cast<const vu4 *>(g + t0 + tid * 8));
    }
    const int64_t blocks_per_tile = (int64_t)kTile >> lg_block;
    const bool owner = tid < blocks_per_tile;
    const int64_t b = (t0 >> lg_block) + tid;
    float n1 = 0.0f, n2 = 0.0f;
    if (owner) {
        n1 = a1[b];
        n2 = a2[b];
    }
    tab[tid] = gran[0];
    tab[min(tid + kThreads, kGranules - 1)] = gran[1];
    if (WIDE) {
        xc[tid] = cw;
        xg[tid] = gw;
    }
    __syncthreads();
    if (WIDE) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            k1[c] = reinterpret_cast<const uint32_t *>(xc)[c * kThreads + tid];
            k2[c] = reinterpret_cast<const uint32_t *>(xc)[2 * kThreads + c * kThreads + tid];
            gv[c] = reinterpret_cast<const vu2 *>(xg)[c * kThreads + tid];
        }
    }
    const uint32_t tk = reinterpret_cast<const uint32_t *>(tab)[k1[0] % (4 * kGranules)] & key;
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int64_t e = t0 + c * (kThreads * 4) + tid * 4;
        const uint32_t gk = ((gv[c].x ^ gv[c].y) & key) ^ tk;
        st(reinterpret_cast<vu4 *>(w + e), wv[c] ^ gk);
        if (!WIDE) {
            st(reinterpret_cast<uint32_t *>(c1 + e), k1[c] ^ key);
            st(reinterpret_cast<uint32_t *>(c2 + e), k2[c] ^ key);
        }
    }
    if (WIDE) {
        __syncthreads();
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            reinterpret_cast<uint32_t *>(xc)[c * kThreads + tid] = k1[c] ^ key;
            reinterpret_cast<uint32_t *>(xc)[2 * kThreads + c * kThreads + tid] = k2[c] ^ key;
        }
        __syncthreads();
        st(reinterpret_cast<vu4 *>(cs + ce), xc[tid]);
    }
    if (owner) {
        a1[b] = __uint_as_float(__float_as_uint(n1) ^ key);
        a2[b] = __uint_as_float(__float_as_uint(n2) ^ key);
    }
}

// resident workgroups per CU set by the total LDS of one workgroup (160 KiB
// per CU): a total in (160 KiB / (k + 1), 160 KiB / k] admits k
template <bool WIDE>
hipError_t launch_step_shape(int per_cu, float *w, const uint16_t *g, uint8_t *c1, uint8_t *c2,
                             float *a1, float *a2, int64_t n, int lg, uint32_t key,
                             const uint32_t *table, hipStream_t stream)
{
    hipFuncAttributes fa;
    hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(stream_step_kernel<WIDE>));
    if (e != hipSuccess)
        return e;
    const int total = per_cu == 3 ? 48 * 1024 : 72 * 1024;
    const int dyn = total - (int)fa.sharedSizeBytes;
    if (dyn < 0)
        return hipErrorInvalidValue;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(stream_step_kernel<WIDE>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, dyn);
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL((stream_step_kernel<WIDE>), dim3((unsigned)(n / (kThreads * 8))),
                       dim3(kThreads), (unsigned)dyn, stream, w, g, c1, c2, a1, a2, lg, key,
                       reinterpret_cast<const vu4 *>(table));
    return hipGetLastError();
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


// ---------------------------------------------------------------------------
// Access-shape study: the step's byte mix, its reads alone and its writes
// alone, under launch shapes, cache policies, tile orders, 16-byte code and
// grad accesses, added arithmetic and occupancies.  Every variant stages the
// step's 14,080 B of table granules from L2 into LDS as the step does.
// ---------------------------------------------------------------------------

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// raw buffer over [base, base + bytes); word 3 of the descriptor is the
// plain raw-buffer format of gfx9-family parts
__device__ inline rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, bytes,
                                             0x00020000);
}

// i-th workgroup -> tile.  XCD: consecutive workgroups go round-robin to the
// 8 XCDs, so workgroup i of XCD i % 8 takes the (i / 8)-th tile of that XCD's
// contiguous eighth of the tiles
template <bool XCD>
__device__ inline int64_t study_tile(int64_t i, int64_t ntiles)
{
    if (!XCD)
        return i;
    const int64_t q = ntiles >> 3, r = ntiles & 7, x = i & 7, k = i >> 3;
    return x * q + (x < r ? x : r) + k;
}

struct StudyBufs {
    float *w;
    uint16_t *g;
    uint8_t *c1, *c2;
    float *a1, *a2;
};

// Cache-policy bits of the buffer instructions: 1 sc0, 2 nt, 16 sc1.
constexpr int kNT = 2, kSC0 = 1, kSC1 = 16;

// MODE 0: the step's mix; 1: its reads only; 2: its writes only (to `out`,
// values from a hash of the element index).  T threads, CH chunks of 4 T
// elements.  WC / WG: codes / grads 16 B per lane through LDS.  GLB: global
// non-temporal loads and stores (the step's access); else buffer instructions
// with load / store policy LP / SP; GLB 2: global non-temporal loads, buffer
// stores with policy SP (the step's access).  ALU: dependent fma per element between
// loads and stores; SLEEP: one s_sleep of that count there.  ORDER 1: params
// stored first, codes after two barriers (the step's order).
template <int T, int CH, int MODE, bool WC, bool WG, bool XCD, int LP, int SP, int GLB, int ALU,
          int SLEEP, int ORDER>
__global__ __launch_bounds__(T) void study_kernel(StudyBufs in, StudyBufs out, int64_t ntiles,
                                                  int lg_block, uint32_t key, const vu4 *table)
{
    static_assert(GLB == 0 || (!WC && !WG), "wide accesses use buffer instructions");
    constexpr int kTile = 4 * T * CH;
    constexpr int kGPT = (kGranules + T - 1) / T;
    constexpr int kHalf = kTile / 16;       // 16-byte lanes of one code array
    constexpr int kWideC = 2 * kHalf;       // both code arrays
    constexpr int kWideG = kTile * 2 / 16;  // grads
    constexpr int kRC = (kWideC + T - 1) / T;
    constexpr int kRG = (kWideG + T - 1) / T;
    __shared__ vu4 tab[kGranules];
    __shared__ __attribute__((aligned(16))) uint8_t cl[WC ? 2 * kTile : 16];
    __shared__ __attribute__((aligned(16))) uint8_t gl[WG ? 2 * kTile : 16];
    const int tid = threadIdx.x;
    const int64_t t0 = study_tile<XCD>(blockIdx.x, ntiles) * kTile;
    const StudyBufs &B = MODE == 2 ? out : in;

    vu4 gran[kGPT];
#pragma unroll
    for (int k = 0; k < kGPT; ++k)
        gran[k] = table[min(tid + k * T, kGranules - 1)];
    const rsrc_t rw = make_rsrc(B.w + t0, kTile * 4);
    const rsrc_t rg = make_rsrc(B.g + t0, kTile * 2);
    const rsrc_t r1 = make_rsrc(B.c1 + t0, kTile);
    const rsrc_t r2 = make_rsrc(B.c2 + t0, kTile);
    vu4 wv[CH];
    vu2 gv[CH];
    uint32_t k1[CH], k2[CH];
    vu4 cin[kRC], gin[kRG];
    if (MODE != 2) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = c * 4 * T + tid * 4;
            if (GLB != 0) {
                wv[c] = ld(reinterpret_cast<const vu4 *>(B.w + t0 + e));
                gv[c] = ld(reinterpret_cast<const vu2 *>(B.g + t0 + e));
                k1[c] = ld(reinterpret_cast<const uint32_t *>(B.c1 + t0 + e));
                k2[c] = ld(reinterpret_cast<const uint32_t *>(B.c2 + t0 + e));
            } else {
                wv[c] = __builtin_amdgcn_raw_buffer_load_b128(rw, e * 4, 0, LP);
                if (!WG)
                    gv[c] = __builtin_amdgcn_raw_buffer_load_b64(rg, e * 2, 0, LP);
                if (!WC) {
                    k1[c] = __builtin_amdgcn_raw_buffer_load_b32(r1, e, 0, LP);
                    k2[c] = __builtin_amdgcn_raw_buffer_load_b32(r2, e, 0, LP);
                }
            }
        }
        if (WC) {
#pragma unroll
            for (int k = 0; k < kRC; ++k) {
                const int l = tid + k * T;
                if (l < kWideC)
                    cin[k] = __builtin_amdgcn_raw_buffer_load_b128(
                        l < kHalf ? r1 : r2, (l < kHalf ? l : l - kHalf) * 16, 0, LP);
            }
        }
        if (WG) {
#pragma unroll
            for (int k = 0; k < kRG; ++k) {
                const int l = tid + k * T;
                if (l < kWideG)
                    gin[k] = __builtin_amdgcn_raw_buffer_load_b128(rg, l * 16, 0, LP);
            }
        }
    }
    const int64_t bpt = kTile >> lg_block;
    const int64_t b = (t0 >> lg_block) + tid;
    float n1 = 0.0f, n2 = 0.0f;
    if (MODE != 2 && tid < bpt) {
        n1 = B.a1[b];
        n2 = B.a2[b];
    }
#pragma unroll
    for (int k = 0; k < kGPT; ++k)
        tab[min(tid + k * T, kGranules - 1)] = gran[k];
    if (MODE != 2 && WC) {
#pragma unroll
        for (int k = 0; k < kRC; ++k) {
            const int l = tid + k * T;
            if (l < kWideC)
                reinterpret_cast<vu4 *>(cl)[l] = cin[k];
        }
    }
    if (MODE != 2 && WG) {
#pragma unroll
        for (int k = 0; k < kRG; ++k) {
            const int l = tid + k * T;
            if (l < kWideG)
                reinterpret_cast<vu4 *>(gl)[l] = gin[k];
        }
    }
    __syncthreads();
    if (MODE == 2) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const uint32_t e = (uint32_t)(t0 + c * 4 * T + tid * 4);
            const uint32_t h = (e * 0x9E3779B1u) ^ (e >> 7) ^ key;
            wv[c] = vu4{h, h * 3u, h * 5u, h * 7u} & 0xBFFFFFFFu;  // finite floats
            gv[c] = vu2{0u, 0u};
            k1[c] = h * 11u;
            k2[c] = h * 13u;
        }
        n1 = (float)(b & 1023);
        n2 = n1 + 1.0f;
    } else {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = c * 4 * T + tid * 4;
            if (WC) {
                k1[c] = reinterpret_cast<const uint32_t *>(cl)[e / 4];
                k2[c] = reinterpret_cast<const uint32_t *>(cl + kTile)[e / 4];
            }
            if (WG)
                gv[c] = reinterpret_cast<const vu2 *>(gl)[e / 4];
        }
    }
    const uint32_t tk = reinterpret_cast<const uint32_t *>(tab)[k1[0] % (4 * kGranules)] & key;
    if (MODE == 1) {
        uint32_t x = tk ^ __float_as_uint(n1) ^ __float_as_uint(n2);
#pragma unroll
        for (int c = 0; c < CH; ++c)
            x ^= wv[c].x ^ wv[c].y ^ wv[c].z ^ wv[c].w ^ gv[c].x ^ gv[c].y ^ k1[c] ^ k2[c];
        if (key == 0x7fu && tid < bpt)  // never taken at key 0; keeps the loads
            B.a1[b] = __uint_as_float(x);
        return;
    }
    if (SLEEP)
        __builtin_amdgcn_s_sleep(SLEEP);
    if (ALU) {
        const float fa = __uint_as_float(0x3f7ff000u ^ (key << 3));
        const float fb = __uint_as_float(key | 0x33800000u);
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            vf4 x = __builtin_bit_cast(vf4, wv[c]);
            for (int k = 0; k < ALU; ++k) {
                x.x = __builtin_fmaf(x.x, fa, fb);
                x.y = __builtin_fmaf(x.y, fa, fb);
                x.z = __builtin_fmaf(x.z, fa, fb);
                x.w = __builtin_fmaf(x.w, fa, fb);
            }
            wv[c] ^= (__builtin_bit_cast(vu4, x) & key);
        }
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int e = c * 4 * T + tid * 4;
        const uint32_t gk = ((gv[c].x ^ gv[c].y) & key) ^ tk;
        if (GLB == 1)
            st(reinterpret_cast<vu4 *>(B.w + t0 + e), wv[c] ^ gk);
        else
            __builtin_amdgcn_raw_buffer_store_b128(wv[c] ^ gk, rw, e * 4, 0, SP);
    }
    if (ORDER == 1) {
        __syncthreads();
        __syncthreads();
    }
    if (!WC) {
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = c * 4 * T + tid * 4;
            if (GLB == 1) {
                st(reinterpret_cast<uint32_t *>(B.c1 + t0 + e), k1[c] ^ key);
                st(reinterpret_cast<uint32_t *>(B.c2 + t0 + e), k2[c] ^ key);
            } else {
                __builtin_amdgcn_raw_buffer_store_b32(k1[c] ^ key, r1, e, 0, SP);
                __builtin_amdgcn_raw_buffer_store_b32(k2[c] ^ key, r2, e, 0, SP);
            }
        }
    } else {
        __syncthreads();
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int e = c * 4 * T + tid * 4;
            reinterpret_cast<uint32_t *>(cl)[e / 4] = k1[c] ^ key;
            reinterpret_cast<uint32_t *>(cl + kTile)[e / 4] = k2[c] ^ key;
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kRC; ++k) {
            const int l = tid + k * T;
            if (l < kWideC)
                __builtin_amdgcn_raw_buffer_store_b128(reinterpret_cast<const vu4 *>(cl)[l],
                                                       l < kHalf ? r1 : r2,
                                                       (l < kHalf ? l : l - kHalf) * 16, 0, SP);
        }
    }
    if (tid < bpt) {
        B.a1[b] = __uint_as_float(__float_as_uint(n1) ^ key);
        B.a2[b] = __uint_as_float(__float_as_uint(n2) ^ key);
    }
}

typedef void (*study_fn)(StudyBufs, StudyBufs, int64_t, int, uint32_t, const vu4 *);
struct StudyVariant {
    study_fn f;
    int threads, chunks, mode;
    const char *name;
};
#define SV(T, CH, M, WC, WG, X, LP, SP, GLB, ALU, SL, ORD, NAME) \
    {study_kernel<T, CH, M, WC, WG, X, LP, SP, GLB, ALU, SL, ORD>, T, CH, M, NAME}
const StudyVariant kStudy[] = {
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 0, 0, 0, "mix: the step's access (global, nt)"),
    SV(512, 2, 0, false, false, false, kNT, kNT, false, 0, 0, 0, "mix: buffer instructions, nt"),
    SV(512, 2, 0, false, false, false, kNT, kSC0 | kSC1 | kNT, 2, 0, 0, 0,
       "mix: global nt loads, stores sc0 sc1 nt (the step's)"),
    SV(512, 2, 0, false, false, false, kSC0 | kNT, kNT, false, 0, 0, 0, "mix: loads sc0 nt"),
    SV(512, 2, 0, false, false, false, kSC1 | kNT, kNT, false, 0, 0, 0, "mix: loads sc1 nt"),
    SV(512, 2, 0, false, false, false, kSC0 | kSC1 | kNT, kNT, false, 0, 0, 0,
       "mix: loads sc0 sc1 nt"),
    SV(512, 2, 0, false, false, false, kSC0 | kSC1 | kNT, kSC0 | kSC1 | kNT, false, 0, 0, 0,
       "mix: loads and stores sc0 sc1 nt"),
    SV(512, 2, 0, false, false, false, kNT, 0, false, 0, 0, 0, "mix: stores default policy"),
    SV(512, 2, 0, false, false, false, kNT, kSC1 | kNT, false, 0, 0, 0, "mix: stores sc1 nt"),
    SV(512, 2, 0, false, false, false, kNT, kSC0 | kSC1 | kNT, false, 0, 0, 0,
       "mix: stores sc0 sc1 nt"),
    SV(512, 2, 0, false, false, false, kNT, kSC0 | kSC1, false, 0, 0, 0, "mix: stores sc0 sc1"),
    SV(512, 2, 0, false, false, false, kNT, kSC1, false, 0, 0, 0, "mix: stores sc1"),
    SV(512, 2, 0, false, false, false, 0, kNT, false, 0, 0, 0, "mix: loads default policy"),
    SV(512, 2, 0, false, false, true, kNT, kNT, false, 0, 0, 0, "mix: XCD-contiguous tile order"),
    SV(512, 2, 0, true, false, false, kNT, kNT, false, 0, 0, 0, "mix: 16-byte code accesses"),
    SV(512, 2, 0, true, true, false, kNT, kNT, false, 0, 0, 0,
       "mix: 16-byte code and grad accesses"),
    SV(512, 2, 0, true, false, true, kNT, kNT, false, 0, 0, 0, "mix: 16-byte codes, XCD order"),
    SV(512, 1, 0, false, false, false, kNT, kNT, true, 0, 0, 0, "mix: 1 chunk per thread"),
    SV(256, 4, 0, false, false, false, kNT, kNT, true, 0, 0, 0, "mix: 256 threads, 4 chunks"),
    SV(1024, 1, 0, false, false, false, kNT, kNT, true, 0, 0, 0, "mix: 1024 threads, 1 chunk"),
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 0, 0, 1,
       "mix: params first, codes after two barriers"),
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 16, 0, 0, "mix: + 16 fma per element"),
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 48, 0, 0, "mix: + 48 fma per element"),
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 96, 0, 0, "mix: + 96 fma per element"),
    SV(512, 2, 0, false, false, false, kNT, kNT, true, 0, 32, 0, "mix: + sleep 32 before stores"),
    SV(512, 2, 1, false, false, false, kNT, kNT, true, 0, 0, 0, "reads: global, nt"),
    SV(512, 2, 1, false, false, false, 0, kNT, false, 0, 0, 0, "reads: default policy"),
    SV(512, 2, 1, false, false, true, kNT, kNT, false, 0, 0, 0, "reads: XCD order"),
    SV(512, 2, 1, false, false, false, kSC0 | kNT, kNT, false, 0, 0, 0, "reads: sc0 nt"),
    SV(512, 2, 1, false, false, false, kSC1 | kNT, kNT, false, 0, 0, 0, "reads: sc1 nt"),
    SV(512, 2, 1, false, false, false, kSC0 | kSC1 | kNT, kNT, false, 0, 0, 0, "reads: sc0 sc1 nt"),
    SV(512, 2, 2, false, false, false, kNT, kNT, true, 0, 0, 0, "writes: global, nt"),
    SV(512, 2, 2, false, false, false, kNT, 0, false, 0, 0, 0, "writes: default policy"),
    SV(512, 2, 2, false, false, false, kNT, kSC1 | kNT, false, 0, 0, 0, "writes: sc1 nt"),
    SV(512, 2, 2, false, false, false, kNT, kSC0 | kSC1 | kNT, false, 0, 0, 0,
       "writes: sc0 sc1 nt"),
    SV(512, 2, 2, false, false, true, kNT, kNT, false, 0, 0, 0, "writes: XCD order"),
};
#undef SV
constexpr int kStudyVariants = (int)(sizeof(kStudy) / sizeof(kStudy[0]));

}  // namespace

extern "C" {

// Number of variants: 0 = 1 chunk, absmax read after the element loads;
// 1 = 1 chunk, absmax read first; 2, 3 = the same with 2 chunks; 4, 5 = 1 and
// 2 chunks (absmax read after the loads) with the staged 16 KiB table; 6, 7 =
// the step's shape at 3 and 2 workgroups per CU; 8 = the step's shape with
// 16-byte code and grad accesses, 2 workgroups per CU.
int bq_stream_variants(void) { return 9; }

// n: elements, a positive multiple of 4096; blocksize: power of two in
// [256, 4096]; buffers 16-byte aligned (absmax: n / blocksize floats each);
// table: 4096 uint32 (read by variants 4 to 8).  Returns 0, -1 for a
// bad argument, or the HIP error code of the launch.
int bq_stream_ceiling(int variant, float *w, const uint16_t *g, uint8_t *c1, uint8_t *c2,
                      float *a1, float *a2, int64_t n, int32_t blocksize, uint32_t key,
                      const uint32_t *table, hipStream_t stream)
{
    if (!w || !g || !c1 || !c2 || !a1 || !a2 || n <= 0 || n % 4096 != 0 ||
        n / 2048 > INT32_MAX || blocksize < 256 || blocksize > 4096 ||
        (blocksize & (blocksize - 1)) != 0 || (variant >= 4 && !table) || (variant >= 6 && ((uintptr_t)table & 15) != 0))
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
    case 6: e = launch_step_shape<false>(3, w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 7: e = launch_step_shape<false>(2, w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    case 8: e = launch_step_shape<true>(2, w, g, c1, c2, a1, a2, n, lg, key, table, stream); break;
    default: return -1;
    }
    return (int)e;
}


// Access-shape study.  bq_stream_study_variants: the number of variants;
// bq_stream_study_info(v, out[3]): threads, chunks, mode (0 the step's mix:
// 14 B per element + 16 B per block; 1 its reads: 8 + 8; 2 its writes: 6 + 8)
// and returns the variant's name ("" for a bad v).
int bq_stream_study_variants(void) { return kStudyVariants; }
const char *bq_stream_study_info(int v, int *out)
{
    if (v < 0 || v >= kStudyVariants)
        return "";
    if (out) {
        out[0] = kStudy[v].threads;
        out[1] = kStudy[v].chunks;
        out[2] = kStudy[v].mode;
    }
    return kStudy[v].name;
}

// One launch of study variant v over n elements: in / out hold six device
// buffers each (param fp32, grad fp16, two uint8 code arrays of n elements,
// two fp32 absmax arrays of n / blocksize), 16-byte aligned; mode 2 writes
// `out`, the others read and write `in` (key 0 keeps the contents).  table:
// 880 x 16 B.  per_cu 0 leaves occupancy to the hardware; 2, 3 or 4 pads the
// workgroup's LDS so that at most that many reside on a CU.  n: a positive
// multiple of 8192; blocksize a power of two in [256, 4096].  Returns 0, -1
// for a bad argument or a per_cu the variant cannot take, or a HIP error.
int bq_stream_study(int v, void *const *in, void *const *out, int64_t n, int32_t blocksize,
                    uint32_t key, const void *table, int per_cu, hipStream_t stream)
{
    if (v < 0 || v >= kStudyVariants || !in || !out || !table || n <= 0 || n % 8192 != 0 ||
        n / 1024 > INT32_MAX || blocksize < 256 || blocksize > 4096 ||
        (blocksize & (blocksize - 1)) != 0 || ((uintptr_t)table & 15) != 0 ||
        !(per_cu == 0 || (per_cu >= 2 && per_cu <= 4)))
        return -1;
    for (int i = 0; i < 6; ++i)
        if (!in[i] || !out[i] || ((uintptr_t)in[i] & 15) || ((uintptr_t)out[i] & 15))
            return -1;
    const StudyVariant &x = kStudy[v];
    if (per_cu * x.threads > 2048)
        return -1;
    int lg = 0;
    while ((1 << lg) < blocksize)
        ++lg;
    const int64_t tile = 4LL * x.threads * x.chunks;
    if (tile < blocksize)
        return -1;
    hipFuncAttributes fa;
    hipError_t e = hipFuncGetAttributes(&fa, reinterpret_cast<const void *>(x.f));
    if (e != hipSuccess)
        return (int)e;
    // LDS per CU 160 KiB: a workgroup total in (160 / (k + 1), 160 / k] KiB admits k
    const int total = per_cu == 0 ? 0 : (per_cu == 2 ? 72 : per_cu == 3 ? 48 : 38) * 1024;
    const int dyn = per_cu == 0 ? 0 : total - (int)fa.sharedSizeBytes;
    if (dyn < 0)
        return -1;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(x.f),
                            hipFuncAttributeMaxDynamicSharedMemorySize, dyn);
    if (e != hipSuccess)
        return (int)e;
    StudyBufs bi{(float *)in[0], (uint16_t *)in[1], (uint8_t *)in[2], (uint8_t *)in[3],
                 (float *)in[4], (float *)in[5]};
    StudyBufs bo{(float *)out[0], (uint16_t *)out[1], (uint8_t *)out[2], (uint8_t *)out[3],
                 (float *)out[4], (float *)out[5]};
    const int64_t ntiles = n / tile;
    hipLaunchKernelGGL(x.f, dim3((unsigned)ntiles), dim3(x.threads), (unsigned)dyn, stream, bi, bo,
                       ntiles, lg, key, reinterpret_cast<const vu4 *>(table));
    return (int)hipGetLastError();
}

}  // extern "C"
