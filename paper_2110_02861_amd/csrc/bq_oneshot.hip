// Kernels of the fused 8-bit step, block-wise quantize / dequantize and the
// LAMB / LARS norm pass, for gfx950.
//
// One-shot kernels (step plans, prepared codebooks): one workgroup of 512
// threads per tile, chunks of 2048 elements with 4 contiguous elements per
// thread, wave-contiguous non-temporal loads and streaming stores (4096-element tiles
// for the step, 8192 for quantize, 4096 for dequantize).  The decision tables
// of each codebook are built by prepare_kernel into a prepared-codebook buffer
// (once per call, or once for all steps when the caller keeps the buffer) and
// copied from there (L2) into LDS by every workgroup.  On MI355X this shape
// streams the step's byte mix (read 4 + 2 + 1 + 1 B, write 4 + 1 + 1 B per
// element) faster than persistent workgroups, which is why the hot path is
// organised this way.
//
// Persistent kernels (the allocation-free calls, which get only the raw
// maps): every workgroup builds the tables in its own LDS once and then runs
// the same tile code (StepOS::tile, QuantOS::tile) over a grid-stride list of
// tiles.
#include <mutex>

#include "bq.h"
#include "bq_device.h"
#include "bq_scalars.h"

namespace bq {
namespace {

using namespace dev;

// The run's per-step scalars: formed on the device from device-resident
// hyperparameters when the run has them (PlanArgs::dev), else the copy the
// host placed in the kernel arguments.  The device copy does not change while
// a kernel of the run executes, so it is read through the constant address
// space: one scalar load, whose wait does not also wait for the tile's HBM
// loads (a generic load became one vector load per field).
__device__ inline DevScalars load_dev_scalars(const DevScalars *p)
{
    typedef const __attribute__((address_space(4))) uint32_t *cword;
    constexpr int kWords = (int)(sizeof(DevScalars) / 4);
    const cword src = (cword)p;
    uint32_t w[kWords];
#pragma unroll
    for (int i = 0; i < kWords; ++i)
        w[i] = src[i];
    DevScalars d;
    __builtin_memcpy(&d, w, sizeof(d));
    return d;
}
__device__ inline StepScalars run_scalars(const PlanArgs &a)
{
    return a.dev ? load_dev_scalars(a.dev).sc : a.sc;
}
__device__ inline int run_use_wd(const PlanArgs &a)
{
    return a.dev ? load_dev_scalars(a.dev).use_wd : a.use_wd;
}
__device__ inline StepScalars run_scalars(const StepArgs &a) { return a.sc; }
__device__ inline int run_use_wd(const StepArgs &a) { return a.use_wd; }
__device__ inline StepScalars run_scalars(const StaticArgs &a) { return a.sc; }
__device__ inline int run_use_wd(const StaticArgs &a) { return a.use_wd; }

// ---------------------------------------------------------------------------
// Scalars of a run from device-resident hyperparameters (one wave)
// ---------------------------------------------------------------------------

// hp: a bq_hparams in device memory.  With advance, the step is incremented
// first and written back, so that a captured run replays as the next step.
// Every lane forms the same scalars; lane i stores word i, and lanes 0 and 1
// the two halves of the new step count.
__global__ __launch_bounds__(64) void scalars_kernel(bq_hparams *hp, int opt, int advance,
                                                     DevScalars *out)
{
    const bq_hparams h = *hp;
    const int64_t t = h.step + (advance ? 1 : 0);
    DevScalars d;
    d.sc = make_scalars(h.lr, h.beta1, h.beta2, h.eps, h.weight_decay, t, h.trust_coeff, opt);
    d.use_wd = l2_on_grad(h.weight_decay, opt);
    d.pad = 0;
    constexpr int kWords = (int)(sizeof(DevScalars) / 4);
    uint32_t w[kWords];
    __builtin_memcpy(w, &d, sizeof(d));
    const int i = threadIdx.x;
    if (i < kWords)
        G(reinterpret_cast<uint32_t *>(out))[i] = w[i];
    if (advance && i < 2)
        G(reinterpret_cast<uint32_t *>(&hp->step))[i] = (uint32_t)((uint64_t)t >> (32 * i));
}

constexpr int kOS = 512;  // threads per workgroup (quantize, dequantize)
constexpr int kOSWaves = kOS / 64;
constexpr int kST = 512;  // threads per workgroup of the step and its norm pass
constexpr int kSTWaves = kST / 64;

// ---------------------------------------------------------------------------
// Prepare: decision tables of 1 or 2 maps (one workgroup each)
// ---------------------------------------------------------------------------

// kPrepThreads threads per map build its tables (build_tables: the thresholds,
// a byte histogram of where each one starts counting, one workgroup scan).
constexpr int kPrepThreads = 1024;

__global__ __launch_bounds__(kPrepThreads) void prepare_kernel(const float *__restrict__ q1,
                                                               const float *__restrict__ q2,
                                                               uint8_t *__restrict__ out)
{
    __shared__ float q[256];
    __shared__ float t[256];
    __shared__ __attribute__((aligned(16))) uint8_t base[2 * kBuckets];
    __shared__ int kmax;
    const float *qm = blockIdx.x == 0 ? q1 : q2;
    build_tables<kPrepThreads>(qm, q, t, base, &kmax);
    uint8_t *dst = out + (size_t)blockIdx.x * kPreparedBytes;
    const int j = threadIdx.x;
    if (j < 256) {
        reinterpret_cast<float *>(dst + kPreparedOffQ)[j] = q[j];
        reinterpret_cast<float *>(dst + kPreparedOffT)[j] = t[j];
    }
    const uint32_t *bs = reinterpret_cast<const uint32_t *>(base);
    uint32_t *bd = reinterpret_cast<uint32_t *>(dst + kPreparedOffBase);
    for (int i = j; i < (int)(2 * kBuckets / 4); i += kPrepThreads)
        bd[i] = bs[i];
    if (j == 0)
        *reinterpret_cast<int *>(dst + kPreparedOffKmax) = kmax;
}

__device__ inline int prepared_kmax(const uint8_t *tables)
{
    return __builtin_amdgcn_readfirstlane(
        *G(reinterpret_cast<const int *>(tables + kPreparedOffKmax)));
}

// ---------------------------------------------------------------------------
// Per-block normalizers, computed once per block by wave 0
// ---------------------------------------------------------------------------

// Everything requantization needs from a block's new absmax A, for one state.
struct BlockNorm {
    float a;  // the absmax itself (stored to memory)
    float n;  // scaled divisor N' (1 for an all-zero block)
    float r;  // RN(1 / N') (0 for an all-zero block)
    float s;  // power-of-two scale of x (1 unless A is tiny or huge)
};

__device__ inline BlockNorm block_norm(float A)
{
    const Normalizer z = make_normalizer(A);
    BlockNorm b;
    b.a = A;
    b.n = z.n;
    b.r = z.r;
    b.s = z.s;
    return b;
}

// x / A, exactly rounded, for a block that needs no rescale (s == 1).
__device__ inline float normalize_plain(const BlockNorm &b, float x)
{
    const float q = x * b.r;
    const float e = __builtin_fmaf(-q, b.n, x);
    return __builtin_fmaf(e, b.r, q);
}

template <int N, bool NONNEG>
__device__ inline void requantize_norm(const Tables &M, const BlockNorm &b, const float (&x)[N],
                                       uint32_t (&c)[N])
{
    Normalizer z;
    z.n = b.n;
    z.r = b.r;
    z.s = b.s;
    float y[N];
    if (__builtin_amdgcn_readfirstlane(__float_as_int(b.s)) == __float_as_int(1.0f)) {
#pragma unroll
        for (int i = 0; i < N; ++i)
            y[i] = normalize<false>(z, x[i]);
    } else {
#pragma unroll
        for (int i = 0; i < N; ++i)
            y[i] = normalize<true>(z, x[i]);
    }
    nearest_codes<N, NONNEG>(M, y, c);
}

// LDS layout of the one-shot step workgroup: the prepared bytes of map 1 (q, t,
// both bucket halves) followed by those of map 2 (q, t, + half), placed so that
// map 1's bucket table starts at byte kBucketLo: "bucket - kBucketLo" then folds
// into the LDS instruction's immediate offset.  The pad in front holds the
// reduction slots and the per-block normalizers.
constexpr int kMaxBlocksPerTile = step_tile(256) / 256;
constexpr int kLdsSlots = 0;                                    // uint32 slots[blocks][2]
constexpr int kLdsNorms = kMaxBlocksPerTile * 2 * 4;            // BlockNorm norms[blocks][2]
constexpr int kLdsMap1 = (int)kBucketLo - kPreparedOffBase;     // 11008
constexpr int kLdsMap2 = kLdsMap1 + kPreparedSignedBytes;
constexpr int kLdsBytes = kLdsMap2 + kPreparedNonnegBytes;
static_assert(kLdsNorms + kMaxBlocksPerTile * 2 * (int)sizeof(BlockNorm) <= kLdsMap1,
              "LDS layout");
static_assert(kLdsMap1 % 16 == 0 && kLdsMap2 % 16 == 0, "16 B granules");

// ---------------------------------------------------------------------------
// Fused 8-bit optimizer step, one tile per workgroup
// ---------------------------------------------------------------------------

// One tile of the step: 4096 elements, kST threads, chunks of 4 contiguous
// elements per thread (chunk c of thread t starts at element 4 kST c + 4t).
// Element groups of 256 (one wave and chunk) are "segments"; segment
// s = kSTWaves c + w covers tile elements [256 s, 256 s + 256), so block b of
// the tile is made of segments [b B/256, (b+1) B/256).
template <int OPT, int GRAD, int B>
struct StepOS {
    static constexpr int C = step_tile(B) / (kST * 4);  // chunks per thread
    static constexpr int N = 4 * C;                     // elements per thread
    static constexpr int TILE = step_tile(B);
    static_assert(TILE == kST * N, "tile size");
    static constexpr bool kTwo = has_two_states(OPT);
    static constexpr int kBPT = TILE / B;               // blocks per tile
    static constexpr int kSPB = B / 256;                // segments per block
    static constexpr int kGran1 = kPreparedSignedBytes / 16;      // map 1 granules
    static constexpr int kGran = kGran1 + (kTwo ? kPreparedNonnegBytes / 16 : 0);
    static constexpr int kGPT = (kGran + kST - 1) / kST;          // granules per thread

    // One tile.  STAGE (one-shot workgroups): gran holds this thread's
    // decision-table granules, loaded by the caller before anything else so
    // their L2 latency overlaps the HBM loads, and the tile writes them into
    // LDS; kmax comes from a.tables.  Without STAGE (persistent workgroups)
    // the tables are already in LDS and kmax is passed in.  Args: PlanArgs or
    // StepArgs (sc and use_wd are read).
    template <bool FULL, bool STAGE = true, class Args = PlanArgs>
    __device__ static void tile(const Args &a, const TensorDesc &D, int64_t t0, uint8_t *lds,
                                const vu4 (&gran)[kGPT], float lr_r, int km1_in = 0,
                                int km2_in = 0)
    {
        uint32_t *slots = reinterpret_cast<uint32_t *>(lds + kLdsSlots);
        BlockNorm *norms = reinterpret_cast<BlockNorm *>(lds + kLdsNorms);
        const int tid = threadIdx.x;
        const int wave = tid >> 6;

        // the tile's streaming loads, kept raw until the tables are in LDS
        vf4 wr[C], gr32[C];
        vu2 gr16[C];
        uint32_t k1r[C], k2r[C];
        int valid[C];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kST * 4) + tid * 4;
            if (FULL) {
                valid[c] = 4;
                wr[c] = ld_nt(reinterpret_cast<const vf4 *>(D.param + e));
                if constexpr (GRAD != kF32)
                    gr16[c] = ld_nt(reinterpret_cast<const vu2 *>(
                        static_cast<const uint16_t *>(D.grad) + e));
                else
                    gr32[c] = ld_nt(reinterpret_cast<const vf4 *>(
                        static_cast<const float *>(D.grad) + e));
                k1r[c] = ld_nt(reinterpret_cast<const uint32_t *>(D.s1 + e));
                k2r[c] = kTwo ? ld_nt(reinterpret_cast<const uint32_t *>(D.s2 + e)) : 0u;
            } else {
                const int64_t rem = D.numel - e;
                valid[c] = rem <= 0 ? 0 : (rem >= 4 ? 4 : (int)rem);
                float wv[4], gv[4];
                uint32_t a1 = 0, a2 = 0;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const bool ok = r < valid[c];
                    const int64_t i = e + r;
                    wv[r] = ok ? G(D.param)[i] : 0.0f;
                    gv[r] = ok ? grad_at<GRAD>(D.grad, i) : 0.0f;
                    a1 |= (ok ? (uint32_t)G(D.s1)[i] : 0u) << (8 * r);
                    if constexpr (kTwo)
                        a2 |= (ok ? (uint32_t)G(D.s2)[i] : 0u) << (8 * r);
                }
                wr[c] = vf4{wv[0], wv[1], wv[2], wv[3]};
                gr32[c] = vf4{gv[0], gv[1], gv[2], gv[3]};
                k1r[c] = a1;
                k2r[c] = a2;
            }
        }
        // old absmax of the block of each chunk (wave-uniform: a segment lies
        // inside one block); a block exists iff its first element does
        const int blk0 = (int)(t0 / B);
        float n1[C], n2[C];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int seg = kSTWaves * c + wave;
            const int b = seg / kSPB;
            const bool live = FULL || t0 + (int64_t)b * B < D.numel;
            n1[c] = live ? G(D.a1)[blk0 + b] : 0.0f;
            n2[c] = (kTwo && live) ? G(D.a2)[blk0 + b] : 0.0f;
        }
        // the loads are issued: the rest of the tile runs at raised wave
        // priority, so tiles that hold loaded data finish (and free their
        // slot for a new tile's loads) ahead of tiles still waiting
        __builtin_amdgcn_s_setprio(2);
        int km1 = km1_in, km2 = km2_in;
        if constexpr (STAGE) {
            km1 = prepared_kmax(a.tables);
            km2 = kTwo ? prepared_kmax(a.tables + kPreparedBytes) : 0;
            // tables into LDS (threads past the last granule rewrite it, same bytes)
#pragma unroll
            for (int k = 0; k < kGPT; ++k)
                reinterpret_cast<vu4 *>(lds + kLdsMap1)[min((int)threadIdx.x + k * kST,
                                                             kGran - 1)] = gran[k];
        }
        // block max slots cleared
        if (tid < 2 * kBPT)
            slots[tid] = 0u;
        __syncthreads();
        Tables T1, T2;
        T1.q = reinterpret_cast<const float *>(lds + kLdsMap1 + kPreparedOffQ);
        T1.t = reinterpret_cast<const float *>(lds + kLdsMap1 + kPreparedOffT);
        T1.base = lds + kLdsMap1 + kPreparedOffBase;
        T1.kmax = km1;
        T2.q = reinterpret_cast<const float *>(lds + kLdsMap2 + kPreparedOffQ);
        T2.t = reinterpret_cast<const float *>(lds + kLdsMap2 + kPreparedOffT);
        T2.base = lds + kLdsMap2 + kPreparedOffBase;
        T2.kmax = km2;

        // unpack, dequantize, 32-bit update, new absmax per chunk
        float w[N], g[N], m[N], v[N];
        uint32_t c1[N], c2[N];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            w[4 * c] = wr[c].x;
            w[4 * c + 1] = wr[c].y;
            w[4 * c + 2] = wr[c].z;
            w[4 * c + 3] = wr[c].w;
            if (GRAD != kF32 && FULL) {
                g[4 * c] = g16_lo<GRAD>(gr16[c].x);
                g[4 * c + 1] = g16_hi<GRAD>(gr16[c].x);
                g[4 * c + 2] = g16_lo<GRAD>(gr16[c].y);
                g[4 * c + 3] = g16_hi<GRAD>(gr16[c].y);
            } else {
                g[4 * c] = gr32[c].x;
                g[4 * c + 1] = gr32[c].y;
                g[4 * c + 2] = gr32[c].z;
                g[4 * c + 3] = gr32[c].w;
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                c1[4 * c + r] = (k1r[c] >> (8 * r)) & 0xffu;
                c2[4 * c + r] = (k2r[c] >> (8 * r)) & 0xffu;
            }
        }
        const StepScalars sc = run_scalars(a);
        if (run_use_wd(a)) {
#pragma unroll
            for (int i = 0; i < N; ++i)
                g[i] = g[i] + sc.wd * w[i];
        }
        float mx1[C], mx2[C];
#pragma unroll
        for (int c = 0; c < C; ++c) {
            mx1[c] = 0.0f;
            mx2[c] = 0.0f;
        }
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const int c = i / 4;
            const bool ok = FULL || (i & 3) < valid[c];
            float wi = w[i];
            const float gi = g[i];
            float mi = T1.q[c1[i]] * n1[c];
            if constexpr (OPT == kMomentum) {
                mi = sc.b1 * mi + gi;
                wi = wi - sc.lr * mi;
            } else if constexpr (OPT == kLars) {
                mi = sc.b1 * mi + lr_r * gi;  // lr_r: the tensor's lr * trust ratio
                wi = wi - mi;
            } else if constexpr (OPT == kAdaGrad) {
                mi = mi + gi * gi;
                const float denom =
                    __builtin_fmaf(__builtin_amdgcn_sqrtf(mi), sc.sdiv_c, sc.sdiv_eps);
                wi = __builtin_fmaf(-gi, __builtin_amdgcn_rcpf(denom), wi);
            } else {
                float vi = T2.q[c2[i]] * n2[c];
                if constexpr (OPT == kAdamW)
                    wi = wi * sc.decay;
                mi = sc.b1 * mi + sc.omb1 * gi;
                vi = sc.b2 * vi + sc.omb2 * (gi * gi);
                // the param update is not rounded like the oracle's anyway
                // (hardware sqrt and reciprocal), so it may fuse
                if constexpr (OPT == kLamb) {
                    // u = mhat / (sqrt(vhat) + eps) + wd w;  w -= lr_r u
                    const float denom =
                        __builtin_fmaf(__builtin_amdgcn_sqrtf(vi), sc.inv_sqrt_bc2, sc.eps);
                    const float u = __builtin_fmaf(mi * sc.bc1_inv, __builtin_amdgcn_rcpf(denom),
                                                   sc.wd * wi);
                    wi = __builtin_fmaf(-lr_r, u, wi);
                } else {
                    // step_size taken into the denominator
                    const float denom =
                        __builtin_fmaf(__builtin_amdgcn_sqrtf(vi), sc.sdiv_c, sc.sdiv_eps);
                    wi = __builtin_fmaf(-mi, __builtin_amdgcn_rcpf(denom), wi);
                }
                v[i] = ok ? vi : 0.0f;
                mx2[c] = fmaxf(mx2[c], fabsf(v[i]));
            }
            m[i] = ok ? mi : 0.0f;
            w[i] = wi;
            mx1[c] = fmaxf(mx1[c], fabsf(m[i]));
        }

        // the params are final: store them now, so their writes overlap the
        // block reduction
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kST * 4) + tid * 4;
            if (FULL) {
                st_stream(stream_range(D.param + t0, TILE * 4), (int)(e - t0) * 4,
                          vf4{w[4 * c], w[4 * c + 1], w[4 * c + 2], w[4 * c + 3]});
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (r < valid[c])
                        G(D.param)[e + r] = w[4 * c + r];
            }
        }

        // block absmax on the bit patterns of the non-negative maxima: row
        // (16-lane) max by DPP, one LDS max per row and value into the block's
        // slot (zeroed before the table barrier); wave 0 then computes each
        // block's normalizers once and stores the new absmax
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int b = (kSTWaves * c + wave) / kSPB;
            const uint32_t u1 = row_umax(__float_as_uint(mx1[c]));
            const uint32_t u2 = kTwo ? row_umax(__float_as_uint(mx2[c])) : 0u;
            if ((tid & 15) == 0) {
                atomicMax(&slots[2 * b], u1);
                if constexpr (kTwo)
                    atomicMax(&slots[2 * b + 1], u2);
            }
        }
        __syncthreads();
        if (wave == 0 && tid < kBPT) {
            const float A1 = __uint_as_float(slots[2 * tid]);
            const float A2 = kTwo ? __uint_as_float(slots[2 * tid + 1]) : 0.0f;
            norms[2 * tid] = block_norm(A1);
            if constexpr (kTwo)
                norms[2 * tid + 1] = block_norm(A2);
            if (FULL || t0 + (int64_t)tid * B < D.numel) {
                G(D.a1)[blk0 + tid] = A1;
                if constexpr (kTwo)
                    G(D.a2)[blk0 + tid] = A2;
            }
        }
        __syncthreads();

        // requantize.  Common case (every map resolves a bucket with at most
        // one threshold, no block needs the power-of-two rescale): one
        // straight-line pass over all chunks and both states.
        BlockNorm nb1[C], nb2[C];
        bool plain = (km1 == 1) && (!kTwo || km2 == 1);
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int b = (kSTWaves * c + wave) / kSPB;
            nb1[c] = norms[2 * b];
            nb2[c] = kTwo ? norms[2 * b + 1] : nb1[c];
            plain = plain && __builtin_amdgcn_readfirstlane(__float_as_int(nb1[c].s)) ==
                                 __float_as_int(1.0f);
            if constexpr (kTwo)
                plain = plain && __builtin_amdgcn_readfirstlane(__float_as_int(nb2[c].s)) ==
                                     __float_as_int(1.0f);
        }
        if (plain) {
            float y1[N], y2[N];
#pragma unroll
            for (int i = 0; i < N; ++i) {
                y1[i] = normalize_plain(nb1[i / 4], m[i]);
                if constexpr (kTwo)
                    y2[i] = normalize_plain(nb2[i / 4], v[i]);
            }
#pragma unroll
            for (int i = 0; i < N; ++i) {
                c1[i] = T1.base[bucket_of<false>(y1[i])];
                if constexpr (kTwo)
                    c2[i] = T2.base[bucket_of<true>(y2[i])];
            }
#pragma unroll
            for (int i = 0; i < N; ++i) {
                c1[i] += (y1[i] >= T1.t[c1[i]]) ? 1u : 0u;
                if constexpr (kTwo)
                    c2[i] += (y2[i] >= T2.t[c2[i]]) ? 1u : 0u;
            }
        } else {
#pragma unroll
            for (int c = 0; c < C; ++c) {
                float mc[4], vc[4];
                uint32_t q1[4], q2[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    mc[r] = m[4 * c + r];
                    vc[r] = v[4 * c + r];
                }
                requantize_norm<4, false>(T1, nb1[c], mc, q1);
                if constexpr (kTwo)
                    requantize_norm<4, true>(T2, nb2[c], vc, q2);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    c1[4 * c + r] = q1[r];
                    c2[4 * c + r] = kTwo ? q2[r] : 0u;
                }
            }
        }

        // store the codes
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kST * 4) + tid * 4;
            if (FULL) {
                st_stream(stream_range(D.s1 + t0, TILE), (int)(e - t0),
                          c1[4 * c] | (c1[4 * c + 1] << 8) | (c1[4 * c + 2] << 16) |
                              (c1[4 * c + 3] << 24));
                if constexpr (kTwo)
                    st_stream(stream_range(D.s2 + t0, TILE), (int)(e - t0),
                              c2[4 * c] | (c2[4 * c + 1] << 8) | (c2[4 * c + 2] << 16) |
                                  (c2[4 * c + 3] << 24));
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (r < valid[c]) {
                        G(D.s1)[e + r] = (uint8_t)c1[4 * c + r];
                        if constexpr (kTwo)
                            G(D.s2)[e + r] = (uint8_t)c2[4 * c + r];
                    }
                }
            }
        }
    }
};

template <int OPT, int GRAD, int B>
__global__ __launch_bounds__(kST) void step_oneshot_kernel(const PlanArgs a)
{
    using K = StepOS<OPT, GRAD, B>;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsBytes];
    const int tid = threadIdx.x;

    // decision-table granules (L2 resident), issued first: granule g of the
    // LDS image comes from prepared byte 16 g (map 1) or 16 g + 16 (map 2,
    // which starts 16 B after map 1's last staged byte)
    vu4 gran[K::kGPT];
#pragma unroll
    for (int k = 0; k < K::kGPT; ++k) {
        const int gi = min(tid + k * kST, K::kGran - 1);
        const int src = 16 * gi + (gi >= K::kGran1 ? kPreparedBytes - kPreparedSignedBytes : 0);
        gran[k] = *G(reinterpret_cast<const vu4 *>(a.tables + src));
    }

    const gptr<const TensorDesc> dp = G(a.tiles) + blockIdx.x;
    TensorDesc D;
    D.param = dp->param;
    D.grad = dp->grad;
    D.s1 = dp->s1;
    D.s2 = dp->s2;
    D.a1 = dp->a1;
    D.a2 = dp->a2;
    D.numel = dp->numel;
    float lr_r = 0.0f;
    if constexpr (has_trust_ratio(OPT))
        lr_r = G(a.lr_ratio)[dp->tile_begin];  // tile_begin holds the tensor index
    const int64_t t0 = 0;
    if (t0 + K::TILE <= D.numel)
        K::template tile<true>(a, D, t0, lds, gran, lr_r);
    else
        K::template tile<false>(a, D, t0, lds, gran, lr_r);
}

// ---------------------------------------------------------------------------
// Fused 8-bit optimizer step from raw maps, persistent workgroups
// ---------------------------------------------------------------------------

// The allocation-free call receives only the raw maps: every workgroup builds
// both maps' decision tables in its own LDS once (in the layout the one-shot
// kernel stages, plus map 2's unused negative half), then runs the one-shot
// tile code over tiles blockIdx.x, blockIdx.x + gridDim.x, ... of the launch,
// whose tensors travel in the kernel arguments (tile_begin in units of
// step_tile(B)).
constexpr int kLdsPersistBytes = kLdsMap2 + kPreparedSignedBytes;

template <int OPT, int GRAD, int B>
__global__ __launch_bounds__(kST) void step_persistent_kernel(const StepArgs a)
{
    using K = StepOS<OPT, GRAD, B>;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsPersistBytes];
    __shared__ int kmax[2];
    build_tables<kST>(a.q1, reinterpret_cast<float *>(lds + kLdsMap1 + kPreparedOffQ),
                      reinterpret_cast<float *>(lds + kLdsMap1 + kPreparedOffT),
                      lds + kLdsMap1 + kPreparedOffBase, &kmax[0]);
    if constexpr (K::kTwo)
        build_tables<kST>(a.q2, reinterpret_cast<float *>(lds + kLdsMap2 + kPreparedOffQ),
                          reinterpret_cast<float *>(lds + kLdsMap2 + kPreparedOffT),
                          lds + kLdsMap2 + kPreparedOffBase, &kmax[1]);
    const int km1 = __builtin_amdgcn_readfirstlane(kmax[0]);
    const int km2 = K::kTwo ? __builtin_amdgcn_readfirstlane(kmax[1]) : 0;
    const vu4 none[K::kGPT] = {};
    int t = 0;
    for (int tile = blockIdx.x; tile < a.total_tiles; tile += gridDim.x) {
        while (t + 1 < a.ntensors && tile >= a.d[t + 1].tile_begin)
            ++t;
        const TensorDesc &S = a.d[t];
        const int64_t t0 = (int64_t)(tile - S.tile_begin) * K::TILE;
        TensorDesc D;
        D.param = S.param + t0;
        D.grad = static_cast<const char *>(S.grad) + t0 * (GRAD == kF32 ? 4 : 2);
        D.s1 = S.s1 + t0;
        D.s2 = K::kTwo ? S.s2 + t0 : nullptr;
        D.a1 = S.a1 + t0 / B;
        D.a2 = K::kTwo ? S.a2 + t0 / B : nullptr;
        D.numel = S.numel - t0;
        // loads of this tile at normal priority, the rest raised (as one-shot)
        __builtin_amdgcn_s_setprio(0);
        if (K::TILE <= D.numel)
            K::template tile<true, false>(a, D, 0, lds, none, 0.0f, km1, km2);
        else
            K::template tile<false, false>(a, D, 0, lds, none, 0.0f, km1, km2);
    }
}

// ---------------------------------------------------------------------------
// Fused 8-bit step from a static device array (the allocation-free call for
// callers that cannot allocate): the maps' tables and the list's descriptors
// live in `scratch`, and every tile is a one-shot workgroup as in a plan
// ---------------------------------------------------------------------------

// The array is reached from host code only through the device address that
// hipGetSymbolAddress returns (static_scratch below); each GPU holds its own.
static __device__ __attribute__((aligned(256))) uint8_t scratch[kStaticScratchBytes];

// Descriptors of entries [first, first + count) from the kernel arguments
// (all four 16-byte loads of a descriptor issued before its stores).
__global__ __launch_bounds__(64) void static_upload_kernel(const StaticUploadArgs a)
{
    const int i = threadIdx.x;
    if (i < a.count) {
        const TensorDesc d = a.d[i];
        vu4 w[4];
        __builtin_memcpy(w, &d, sizeof(d));
        const gptr<vu4> dst = G(reinterpret_cast<vu4 *>(a.scratch + kStaticOffDesc)) +
                              4 * (int64_t)(a.first + i);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            dst[k] = w[k];
    }
}

// One workgroup per tile.  Its tensor is the last one whose first tile is at
// or below the tile index (empty tensors are left out, so first tiles rise
// strictly): a scalar binary search over the first tiles in the kernel
// arguments, then, when they hold only every stride-th tensor, one ballot over
// the next stride descriptors' first tiles; then one scalar load of the
// descriptor -- the one round trip to memory a plan's tile record also costs.
template <int OPT, int GRAD, int B>
__global__ __launch_bounds__(kST) void step_static_kernel(const StaticArgs a)
{
    using K = StepOS<OPT, GRAD, B>;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsBytes];
    const int tid = threadIdx.x;

    // decision-table granules first, as in the plan kernel
    vu4 gran[K::kGPT];
#pragma unroll
    for (int k = 0; k < K::kGPT; ++k) {
        const int gi = min(tid + k * kST, K::kGran - 1);
        const int src = 16 * gi + (gi >= K::kGran1 ? kPreparedBytes - kPreparedSignedBytes : 0);
        gran[k] = *G(reinterpret_cast<const vu4 *>(a.tables + src));
    }

    const int t = blockIdx.x;
    int k = 0;
#pragma unroll
    for (int s = 512; s >= 1; s >>= 1)
        if (k + s < a.nfirst && a.first_tile[k + s] <= t)
            k += s;
    const gptr<const TensorDesc> descs =
        G(reinterpret_cast<const TensorDesc *>(a.scratch + kStaticOffDesc));
    int idx = k * a.stride;
    if (a.stride > 1) {
        const int lane = tid & 63;
        const int e = idx + lane;
        // lane 0's tensor starts at or below t (the search above)
        const uint64_t m =
            __ballot(lane < a.stride && e < a.ntensors && descs[e].tile_begin <= t);
        idx += 63 - __builtin_clzll(m);
    }
    idx = __builtin_amdgcn_readfirstlane(idx);
    const gptr<const TensorDesc> dp = descs + idx;
    const int64_t t0 = ((int64_t)t - dp->tile_begin) * K::TILE;
    TensorDesc D;
    D.param = dp->param + t0;
    D.grad = static_cast<const char *>(dp->grad) + t0 * (GRAD == kF32 ? 4 : 2);
    D.s1 = dp->s1 + t0;
    D.s2 = K::kTwo ? dp->s2 + t0 : nullptr;
    D.a1 = dp->a1 + t0 / B;
    D.a2 = K::kTwo ? dp->a2 + t0 / B : nullptr;
    D.numel = dp->numel - t0;
    if (K::TILE <= D.numel)
        K::template tile<true, true, StaticArgs>(a, D, 0, lds, gran, 0.0f);
    else
        K::template tile<false, true, StaticArgs>(a, D, 0, lds, gran, 0.0f);
}

// ---------------------------------------------------------------------------
// LAMB / LARS: per-tile partial squared norms, then per-tensor lr * ratio
// ---------------------------------------------------------------------------

// One workgroup per tile, the step kernel's tile shape and access pattern
// (wave-contiguous 4-element chunks, non-temporal vector loads, all issued
// before any arithmetic).  Sums (in double) of w^2 and of u^2 (LAMB: u =
// mhat / (sqrt(vhat) + eps) + wd w from the states the step will compute) or
// g^2 (LARS, g before weight decay); each thread sums its elements in order,
// the waves by a fixed butterfly, the 8 wave sums in order.
template <int OPT, int GRAD, int B>
__global__ __launch_bounds__(kST) void norms_kernel(const PlanArgs a)
{
    using K = StepOS<OPT, GRAD, B>;
    constexpr int C = K::C;
    constexpr bool kIsLamb = OPT == kLamb;
    __shared__ float q1[256], q2[256];
    __shared__ double red[kSTWaves][2];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const gptr<const TensorDesc> dp = G(a.tiles) + blockIdx.x;
    float *const param = dp->param;
    const void *const grad = dp->grad;
    const uint8_t *const s1 = dp->s1;
    const uint8_t *const s2 = dp->s2;
    const float *const a1 = dp->a1;
    const float *const a2 = dp->a2;
    const int64_t numel = dp->numel;
    const bool full = numel >= K::TILE;

    float w[4 * C], g[4 * C];
    uint32_t k1[C], k2[C];
    int valid[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int64_t e0 = c * (kST * 4) + tid * 4;
        const int64_t rem = numel - e0;
        valid[c] = rem <= 0 ? 0 : (rem >= 4 ? 4 : (int)rem);
        if (full) {
            const vf4 wv = ld_nt(reinterpret_cast<const vf4 *>(param + e0));
            w[4 * c] = wv.x;
            w[4 * c + 1] = wv.y;
            w[4 * c + 2] = wv.z;
            w[4 * c + 3] = wv.w;
            if constexpr (GRAD != kF32) {
                const vu2 gv =
                    ld_nt(reinterpret_cast<const vu2 *>(static_cast<const uint16_t *>(grad) + e0));
                g[4 * c] = g16_lo<GRAD>(gv.x);
                g[4 * c + 1] = g16_hi<GRAD>(gv.x);
                g[4 * c + 2] = g16_lo<GRAD>(gv.y);
                g[4 * c + 3] = g16_hi<GRAD>(gv.y);
            } else {
                const vf4 gv =
                    ld_nt(reinterpret_cast<const vf4 *>(static_cast<const float *>(grad) + e0));
                g[4 * c] = gv.x;
                g[4 * c + 1] = gv.y;
                g[4 * c + 2] = gv.z;
                g[4 * c + 3] = gv.w;
            }
            k1[c] = kIsLamb ? ld_nt(reinterpret_cast<const uint32_t *>(s1 + e0)) : 0u;
            k2[c] = kIsLamb ? ld_nt(reinterpret_cast<const uint32_t *>(s2 + e0)) : 0u;
        } else {
            uint32_t b1 = 0, b2 = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool ok = r < valid[c];
                const int64_t e = e0 + r;
                w[4 * c + r] = ok ? G(param)[e] : 0.0f;
                g[4 * c + r] = ok ? grad_at<GRAD>(grad, e) : 0.0f;
                if constexpr (kIsLamb) {
                    b1 |= (ok ? (uint32_t)G(s1)[e] : 0u) << (8 * r);
                    b2 |= (ok ? (uint32_t)G(s2)[e] : 0u) << (8 * r);
                }
            }
            k1[c] = b1;
            k2[c] = b2;
        }
    }
    // old absmax of the block of each chunk (wave-uniform, as in the step)
    float n1[C], n2[C];
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int b = (kSTWaves * c + wave) / K::kSPB;
        const bool live = full || (int64_t)b * B < numel;
        n1[c] = (kIsLamb && live) ? G(a1)[b] : 0.0f;
        n2[c] = (kIsLamb && live) ? G(a2)[b] : 0.0f;
    }
    if constexpr (kIsLamb) {
        if (tid < 256) {
            q1[tid] = G(reinterpret_cast<const float *>(a.tables + kPreparedOffQ))[tid];
            q2[tid] = G(reinterpret_cast<const float *>(a.tables + kPreparedBytes +
                                                        kPreparedOffQ))[tid];
        }
        __syncthreads();
    }
    const StepScalars sc = run_scalars(a);
    double sw = 0.0, sx = 0.0;
#pragma unroll
    for (int i = 0; i < 4 * C; ++i) {
        const int c = i / 4;
        if (!full && (i & 3) >= valid[c])
            continue;
        const float wi = w[i], gi = g[i];
        sw += (double)wi * (double)wi;
        if constexpr (kIsLamb) {
            const float m = q1[(k1[c] >> (8 * (i & 3))) & 0xffu] * n1[c];
            const float v = q2[(k2[c] >> (8 * (i & 3))) & 0xffu] * n2[c];
            const float mn = sc.b1 * m + sc.omb1 * gi;
            const float vn = sc.b2 * v + sc.omb2 * (gi * gi);
            const float denom =
                __builtin_fmaf(__builtin_amdgcn_sqrtf(vn), sc.inv_sqrt_bc2, sc.eps);
            const float u =
                __builtin_fmaf(mn * sc.bc1_inv, __builtin_amdgcn_rcpf(denom), sc.wd * wi);
            sx += (double)u * (double)u;
        } else {
            sx += (double)gi * (double)gi;
        }
    }
    // wave sums, then the 8 wave sums in order
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        sw += __shfl_xor(sw, off);
        sx += __shfl_xor(sx, off);
    }
    if ((tid & 63) == 0) {
        red[wave][0] = sw;
        red[wave][1] = sx;
    }
    __syncthreads();
    if (tid == 0) {
        double tw = 0.0, tx = 0.0;
        for (int k = 0; k < kSTWaves; ++k) {
            tw += red[k][0];
            tx += red[k][1];
        }
        G(a.partials)[2 * (int64_t)blockIdx.x] = tw;
        G(a.partials)[2 * (int64_t)blockIdx.x + 1] = tx;
    }
}

// Per-tensor rates from the per-tile partial sums in two steps, each in a
// fixed order (so the result is deterministic): one workgroup per segment of at
// most kTrustSegTiles tiles of one tensor sums them (thread t takes tiles t,
// t + 256, ... in order, then a fixed tree); one thread per tensor sums its
// segments in order and forms lr * ratio, ratio = |w| / |u| (LAMB) or
// trust |w| / (|g| + wd |w|) (LARS), 1 when either norm is zero.
constexpr int kTrustThreads = 256;

__global__ __launch_bounds__(kTrustThreads) void segment_sums_kernel(const PlanArgs a)
{
    __shared__ double rw[kTrustThreads], rx[kTrustThreads];
    const int64_t sg = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t k0 = G(a.seg_range)[2 * sg], k1 = G(a.seg_range)[2 * sg + 1];
    double sw = 0.0, sx = 0.0;
    for (int64_t k = k0 + tid; k < k1; k += kTrustThreads) {
        sw += G(a.partials)[2 * k];
        sx += G(a.partials)[2 * k + 1];
    }
    rw[tid] = sw;
    rx[tid] = sx;
    __syncthreads();
    for (int h = kTrustThreads / 2; h > 0; h >>= 1) {
        if (tid < h) {
            rw[tid] += rw[tid + h];
            rx[tid] += rx[tid + h];
        }
        __syncthreads();
    }
    if (tid == 0) {
        G(a.seg_partials)[2 * sg] = rw[0];
        G(a.seg_partials)[2 * sg + 1] = rx[0];
    }
}

__global__ __launch_bounds__(kTrustThreads) void trust_ratio_kernel(const PlanArgs a, int lamb)
{
    const int t = blockIdx.x * kTrustThreads + threadIdx.x;
    if (t >= a.ntensors)
        return;
    const int64_t s0 = G(a.first_seg)[t], s1 = G(a.first_seg)[t + 1];
    double sw = 0.0, sx = 0.0;
    int64_t sg = s0;
    for (; sg + 16 <= s1; sg += 16) {  // in order; loads issued 16 at a time
        double vw[16], vx[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            vw[k] = G(a.seg_partials)[2 * (sg + k)];
            vx[k] = G(a.seg_partials)[2 * (sg + k) + 1];
        }
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            sw += vw[k];
            sx += vx[k];
        }
    }
    for (; sg < s1; ++sg) {
        sw += G(a.seg_partials)[2 * sg];
        sx += G(a.seg_partials)[2 * sg + 1];
    }
    const double nw = sqrt(sw), nx = sqrt(sx);
    double ratio = 1.0;
    const StepScalars sc = run_scalars(a);
    if (nw > 0.0 && nx > 0.0)
        ratio = lamb ? nw / nx : (double)sc.trust * nw / (nx + (double)sc.wd * nw);
    G(a.lr_ratio)[t] = (float)((double)sc.lr * ratio);
}

// ---------------------------------------------------------------------------
// Block-wise quantize with a prepared map, one tile per workgroup
// ---------------------------------------------------------------------------

// Tile of quant_tile(B) elements: C chunks of 2048, chunk c of thread t at
// tile element 2048 c + 4 t, so that segment s = 8 c + wave covers tile
// elements [256 s, 256 s + 256) and block b of the tile is made of segments
// [b B / 256, (b + 1) B / 256), as in the step.
template <int B>
struct QuantOS {
    static constexpr int TILE = quant_tile(B);
    static constexpr int C = TILE / 2048;      // chunks per thread
    static constexpr int N = 4 * C;            // elements per thread
    static constexpr int kBPT = TILE / B;      // blocks per tile
    static constexpr int kSPB = B / 256;       // segments per block
    static_assert(kBPT <= 64, "one lane of wave 0 per block");

    // The tile's input values, loaded before any table is needed.
    struct Raw {
        float v[N];
        int valid[C];
    };

    // Issue the loads of the tile starting at element t0.
    template <bool FULL>
    __device__ static void load(const float *x, int64_t n, int64_t t0, Raw &R);

    // The rest of the tile.  STAGE (one-shot workgroups): gran is this
    // thread's table granule, loaded by the caller before the tile's HBM
    // loads, written into LDS here; kmax comes from tables.  Without STAGE
    // (persistent workgroups) the tables are already in LDS and km is passed.
    template <bool FULL, bool STAGE>
    __device__ static void process(const uint8_t *tables, int64_t n, int64_t t0, uint8_t *codes,
                                   float *absmax, uint8_t *lds, const vu4 &gran, int km_in,
                                   const Raw &R);

    // One tile: its loads, then the rest.
    template <bool FULL, bool STAGE>
    __device__ static void tile(const uint8_t *tables, const float *x, int64_t n, int64_t t0,
                                uint8_t *codes, float *absmax, uint8_t *lds, const vu4 &gran,
                                int km_in)
    {
        Raw R;
        load<FULL>(x, n, t0, R);
        process<FULL, STAGE>(tables, n, t0, codes, absmax, lds, gran, km_in, R);
    }
};

// Only the thresholds and both bucket halves are copied (the map values
// themselves are not needed to find a code), placed so that the bucket
// table starts at LDS byte kBucketLo, as in the step.
// In front of them: one max slot and one BlockNorm per block of the tile.
constexpr int kQuantGran = (kPreparedSignedBytes - kPreparedOffT) / 16;   // 480
constexpr int kLdsQSlots = 0;                                             // uint32 [64]
constexpr int kLdsQNorms = 64 * 4;                                        // BlockNorm [64]
constexpr int kLdsQuantBytes = kLdsMap1 + kPreparedSignedBytes;
static_assert(kQuantGran <= kOS, "one granule per thread");
static_assert(kLdsQNorms + 64 * (int)sizeof(BlockNorm) <= kLdsMap1, "LDS layout");

template <int B>
template <bool FULL>
__device__ void QuantOS<B>::load(const float *x, int64_t n, int64_t t0, Raw &R)
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int64_t e = t0 + c * (kOS * 4) + tid * 4;
        const int64_t rem = n - e;
        R.valid[c] = FULL ? 4 : (rem <= 0 ? 0 : (rem >= 4 ? 4 : (int)rem));
        if (FULL) {
            const vf4 y = ld_nt(reinterpret_cast<const vf4 *>(x + e));
            R.v[4 * c] = y.x;
            R.v[4 * c + 1] = y.y;
            R.v[4 * c + 2] = y.z;
            R.v[4 * c + 3] = y.w;
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                R.v[4 * c + r] = r < R.valid[c] ? G(x)[e + r] : 0.0f;
        }
    }
}

template <int B>
template <bool FULL, bool STAGE>
__device__ void QuantOS<B>::process(const uint8_t *tables, int64_t n, int64_t t0, uint8_t *codes,
                                    float *absmax, uint8_t *lds, const vu4 &gran, int km_in,
                                    const Raw &R)
{
    uint32_t *slots = reinterpret_cast<uint32_t *>(lds + kLdsQSlots);
    BlockNorm *norms = reinterpret_cast<BlockNorm *>(lds + kLdsQNorms);
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const float(&v)[N] = R.v;
    const int(&valid)[C] = R.valid;
    int km = km_in;
    if constexpr (STAGE) {
        km = prepared_kmax(tables);
        if (tid < kQuantGran)
            reinterpret_cast<vu4 *>(lds + kLdsMap1 + kPreparedOffT)[tid] = gran;
    }
    if (tid < kBPT)
        slots[tid] = 0u;
    __syncthreads();

    // block absmax: row max by DPP, one LDS max per row into the block's slot
#pragma unroll
    for (int c = 0; c < C; ++c) {
        float mx = 0.0f;
#pragma unroll
        for (int r = 0; r < 4; ++r)
            mx = fmaxf(mx, fabsf(v[4 * c + r]));
        const uint32_t u = row_umax(__float_as_uint(mx));
        if ((tid & 15) == 0)
            atomicMax(&slots[(kOSWaves * c + wave) / kSPB], u);
    }
    __syncthreads();
    if (tid < kBPT) {
        const float A = __uint_as_float(slots[tid]);
        norms[tid] = block_norm(A);
        if (FULL || t0 + (int64_t)tid * B < n)
            G(absmax)[t0 / B + tid] = A;
    }
    __syncthreads();

    Tables T;
    T.q = nullptr;  // not copied: finding a code reads only t and base
    T.t = reinterpret_cast<const float *>(lds + kLdsMap1 + kPreparedOffT);
    T.base = lds + kLdsMap1 + kPreparedOffBase;
    T.kmax = km;
    BlockNorm nb[C];
    bool plain = km == 1;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        nb[c] = norms[(kOSWaves * c + wave) / kSPB];
        plain = plain &&
                __builtin_amdgcn_readfirstlane(__float_as_int(nb[c].s)) == __float_as_int(1.0f);
    }
    uint32_t q[N];
    if (plain) {
        float y[N];
#pragma unroll
        for (int i = 0; i < N; ++i)
            y[i] = normalize_plain(nb[i / 4], v[i]);
#pragma unroll
        for (int i = 0; i < N; ++i)
            q[i] = T.base[bucket_of<false>(y[i])];
#pragma unroll
        for (int i = 0; i < N; ++i)
            q[i] += (y[i] >= T.t[q[i]]) ? 1u : 0u;
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const float vc[4] = {v[4 * c], v[4 * c + 1], v[4 * c + 2], v[4 * c + 3]};
            uint32_t qc[4];
            requantize_norm<4, false>(T, nb[c], vc, qc);
#pragma unroll
            for (int r = 0; r < 4; ++r)
                q[4 * c + r] = qc[r];
        }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int64_t e = t0 + c * (kOS * 4) + tid * 4;
        if (FULL) {
            st_nt(reinterpret_cast<uint32_t *>(codes + e),
                  q[4 * c] | (q[4 * c + 1] << 8) | (q[4 * c + 2] << 16) | (q[4 * c + 3] << 24));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (r < valid[c])
                    G(codes)[e + r] = (uint8_t)q[4 * c + r];
        }
    }
}

// Prepared map: one workgroup per tile; this thread's table granule (L2) is
// loaded first, then the tile's HBM loads.
template <int B>
__global__ __launch_bounds__(kOS) void quantize_oneshot_kernel(const uint8_t *__restrict__ tables,
                                                               const float *__restrict__ x,
                                                               int64_t n,
                                                               uint8_t *__restrict__ codes,
                                                               float *__restrict__ absmax)
{
    using S = QuantOS<B>;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsQuantBytes];
    const int64_t t0 = (int64_t)blockIdx.x * S::TILE;
    vu4 gran = {0u, 0u, 0u, 0u};
    if (threadIdx.x < kQuantGran)
        gran = G(reinterpret_cast<const vu4 *>(tables + kPreparedOffT))[threadIdx.x];
    if (t0 + S::TILE <= n)
        S::template tile<true, true>(tables, x, n, t0, codes, absmax, lds, gran, 0);
    else
        S::template tile<false, true>(tables, x, n, t0, codes, absmax, lds, gran, 0);
}

// Raw map (the allocation-free call): every workgroup builds the decision
// tables in its own LDS once, then walks tiles blockIdx.x, blockIdx.x +
// gridDim.x, ...
template <int B>
__global__ __launch_bounds__(kOS) void quantize_persistent_kernel(const float *__restrict__ qmap,
                                                                  const float *__restrict__ x,
                                                                  int64_t n,
                                                                  uint8_t *__restrict__ codes,
                                                                  float *__restrict__ absmax)
{
    using S = QuantOS<B>;
    __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsQuantBytes];
    __shared__ int kmax;
    // the first tile's loads are issued before the tables are built, so the
    // build overlaps them (loading every next tile ahead instead needed 103
    // VGPRs, two workgroups per CU, and was slower)
    const int64_t tiles = (n + S::TILE - 1) / S::TILE;
    int64_t tile = blockIdx.x;
    bool full = (tile + 1) * S::TILE <= n;
    typename S::Raw cur;
    if (full)
        S::template load<true>(x, n, tile * S::TILE, cur);
    build_tables<kOS>(qmap, reinterpret_cast<float *>(lds + kLdsMap1 + kPreparedOffQ),
                      reinterpret_cast<float *>(lds + kLdsMap1 + kPreparedOffT),
                      lds + kLdsMap1 + kPreparedOffBase, &kmax);
    const int km = __builtin_amdgcn_readfirstlane(kmax);
    const vu4 none = {0u, 0u, 0u, 0u};
    bool first = true;
    for (; tile < tiles; tile += gridDim.x) {
        const int64_t t0 = tile * S::TILE;
        if (!first) {
            full = t0 + S::TILE <= n;
            if (full)
                S::template load<true>(x, n, t0, cur);
        }
        first = false;
        if (full)
            S::template process<true, false>(nullptr, n, t0, codes, absmax, lds, none, km, cur);
        else
            S::template tile<false, false>(nullptr, x, n, t0, codes, absmax, lds, none, km);
    }
}

// ---------------------------------------------------------------------------
// Block-wise dequantize: out = q[code] * absmax, one tile per workgroup
// ---------------------------------------------------------------------------

// Tile of kDequantChunks chunks of 2048 elements laid out as in quantize; the 256
// elements of one wave and chunk lie in one block (B >= 256), so the wave reads
// that block's absmax once.
__global__ __launch_bounds__(kOS) void dequantize_kernel(const float *__restrict__ qmap,
                                                         const uint8_t *__restrict__ codes,
                                                         const float *__restrict__ absmax,
                                                         int64_t n, int log2_blocksize,
                                                         float *__restrict__ out)
{
    constexpr int C = kDequantChunks;
    constexpr int TILE = dequant_tile();
    static_assert(TILE == kOS * 4 * C, "tile size");
    __shared__ float q[256];
    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int64_t t0 = (int64_t)blockIdx.x * TILE;
    const bool full = t0 + TILE <= n;
    uint32_t k[C];
    float A[C];
    if (full) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kOS * 4) + tid * 4;
            k[c] = ld_nt(reinterpret_cast<const uint32_t *>(codes + e));
            const int seg = __builtin_amdgcn_readfirstlane(kOSWaves * c + wave);
            A[c] = G(absmax)[(t0 + (int64_t)seg * 256) >> log2_blocksize];
        }
    }
    if (tid < 256)
        q[tid] = G(qmap)[tid];
    __syncthreads();
    if (full) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kOS * 4) + tid * 4;
            const vf4 y = {q[k[c] & 0xffu] * A[c], q[(k[c] >> 8) & 0xffu] * A[c],
                           q[(k[c] >> 16) & 0xffu] * A[c], q[k[c] >> 24] * A[c]};
            st_stream(stream_range(out + t0, TILE * 4), (int)(e - t0) * 4, y);
        }
    } else {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int64_t e = t0 + c * (kOS * 4) + tid * 4;
            for (int r = 0; r < 4; ++r)
                if (e + r < n)
                    G(out)[e + r] = q[G(codes)[e + r]] * G(absmax)[(e + r) >> log2_blocksize];
        }
    }
}

template <int OPT, int GRAD, int B>
hipError_t launch_persist_t(const StepArgs &a, hipStream_t s)
{
    auto k = step_persistent_kernel<OPT, GRAD, B>;
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kST, 0) != hipSuccess ||
        per_cu <= 0)
        per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    const int64_t cap = (int64_t)per_cu * cus;
    const int64_t grid = a.total_tiles < cap ? a.total_tiles : cap;
    hipLaunchKernelGGL(k, dim3((unsigned)grid), dim3(kST), 0, s, a);
    return hipGetLastError();
}

template <int OPT, int GRAD>
hipError_t launch_persist_b(int blocksize, const StepArgs &a, hipStream_t s)
{
    switch (blocksize) {
    case 256: return launch_persist_t<OPT, GRAD, 256>(a, s);
    case 512: return launch_persist_t<OPT, GRAD, 512>(a, s);
    case 1024: return launch_persist_t<OPT, GRAD, 1024>(a, s);
    case 2048: return launch_persist_t<OPT, GRAD, 2048>(a, s);
    case 4096: return launch_persist_t<OPT, GRAD, 4096>(a, s);
    default: return hipErrorInvalidValue;
    }
}

template <int OPT>
hipError_t launch_persist_g(int grad_dtype, int blocksize, const StepArgs &a, hipStream_t s)
{
    switch (grad_dtype) {
    case kF16: return launch_persist_b<OPT, kF16>(blocksize, a, s);
    case kBF16: return launch_persist_b<OPT, kBF16>(blocksize, a, s);
    default: return launch_persist_b<OPT, kF32>(blocksize, a, s);
    }
}

template <int OPT, int GRAD, int B>
hipError_t launch_os_t(const PlanArgs &a, hipStream_t s)
{
    hipLaunchKernelGGL((step_oneshot_kernel<OPT, GRAD, B>), dim3((unsigned)a.total_tiles),
                       dim3(kST), 0, s, a);
    return hipGetLastError();
}

template <int OPT, int GRAD>
hipError_t launch_os_b(int blocksize, const PlanArgs &a, hipStream_t s)
{
    switch (blocksize) {
    case 256: return launch_os_t<OPT, GRAD, 256>(a, s);
    case 512: return launch_os_t<OPT, GRAD, 512>(a, s);
    case 1024: return launch_os_t<OPT, GRAD, 1024>(a, s);
    case 2048: return launch_os_t<OPT, GRAD, 2048>(a, s);
    case 4096: return launch_os_t<OPT, GRAD, 4096>(a, s);
    default: return hipErrorInvalidValue;
    }
}

template <int OPT>
hipError_t launch_os_g(int grad_dtype, int blocksize, const PlanArgs &a, hipStream_t s)
{
    switch (grad_dtype) {
    case kF16: return launch_os_b<OPT, kF16>(blocksize, a, s);
    case kBF16: return launch_os_b<OPT, kBF16>(blocksize, a, s);
    default: return launch_os_b<OPT, kF32>(blocksize, a, s);
    }
}

template <int OPT, int GRAD>
hipError_t launch_static_b(int blocksize, const StaticArgs &a, hipStream_t s)
{
    const dim3 grid((unsigned)a.total_tiles), block(kST);
    switch (blocksize) {
    case 256: hipLaunchKernelGGL((step_static_kernel<OPT, GRAD, 256>), grid, block, 0, s, a); break;
    case 512: hipLaunchKernelGGL((step_static_kernel<OPT, GRAD, 512>), grid, block, 0, s, a); break;
    case 1024:
        hipLaunchKernelGGL((step_static_kernel<OPT, GRAD, 1024>), grid, block, 0, s, a);
        break;
    case 2048:
        hipLaunchKernelGGL((step_static_kernel<OPT, GRAD, 2048>), grid, block, 0, s, a);
        break;
    case 4096:
        hipLaunchKernelGGL((step_static_kernel<OPT, GRAD, 4096>), grid, block, 0, s, a);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int OPT>
hipError_t launch_static_g(int grad_dtype, int blocksize, const StaticArgs &a, hipStream_t s)
{
    switch (grad_dtype) {
    case kF16: return launch_static_b<OPT, kF16>(blocksize, a, s);
    case kBF16: return launch_static_b<OPT, kBF16>(blocksize, a, s);
    default: return launch_static_b<OPT, kF32>(blocksize, a, s);
    }
}

template <int B>
hipError_t launch_qr_t(const float *qmap, const float *x, int64_t n, uint8_t *codes,
                       float *absmax, hipStream_t s)
{
    auto k = quantize_persistent_kernel<B>;
    int per_cu = 0, dev = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k, kOS, 0) != hipSuccess ||
        per_cu <= 0)
        per_cu = 1;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        cus = 256;
    const int64_t tiles = (n + quant_tile(B) - 1) / quant_tile(B);
    const int64_t cap = (int64_t)per_cu * cus;
    hipLaunchKernelGGL(k, dim3((unsigned)(tiles < cap ? tiles : cap)), dim3(kOS), 0, s, qmap, x,
                       n, codes, absmax);
    return hipGetLastError();
}

template <int B>
hipError_t launch_qp_t(const uint8_t *tables, const float *x, int64_t n, uint8_t *codes,
                       float *absmax, hipStream_t s)
{
    const int64_t tiles = (n + quant_tile(B) - 1) / quant_tile(B);
    hipLaunchKernelGGL((quantize_oneshot_kernel<B>), dim3((unsigned)tiles), dim3(kOS), 0, s,
                       tables, x, n, codes, absmax);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_scalars(int opt, void *hp, int advance, DevScalars *out, hipStream_t stream)
{
    hipLaunchKernelGGL(scalars_kernel, dim3(1), dim3(64), 0, stream, static_cast<bq_hparams *>(hp),
                       opt, advance, out);
    return hipGetLastError();
}

hipError_t launch_prepare(const float *qmap1, const float *qmap2, uint8_t *tables,
                          hipStream_t stream)
{
    const unsigned maps = qmap2 ? 2u : 1u;
    hipLaunchKernelGGL(prepare_kernel, dim3(maps), dim3(kPrepThreads), 0, stream, qmap1,
                       qmap2 ? qmap2 : qmap1, tables);
    return hipGetLastError();
}

template <int OPT, int GRAD>
hipError_t launch_norms_b(int blocksize, const PlanArgs &a, hipStream_t stream)
{
    const dim3 grid((unsigned)a.total_tiles), block(kST);
    switch (blocksize) {
    case 256:
        hipLaunchKernelGGL((norms_kernel<OPT, GRAD, 256>), grid, block, 0, stream, a);
        break;
    case 512:
        hipLaunchKernelGGL((norms_kernel<OPT, GRAD, 512>), grid, block, 0, stream, a);
        break;
    case 1024:
        hipLaunchKernelGGL((norms_kernel<OPT, GRAD, 1024>), grid, block, 0, stream, a);
        break;
    case 2048:
        hipLaunchKernelGGL((norms_kernel<OPT, GRAD, 2048>), grid, block, 0, stream, a);
        break;
    case 4096:
        hipLaunchKernelGGL((norms_kernel<OPT, GRAD, 4096>), grid, block, 0, stream, a);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int OPT>
hipError_t launch_norms_g(int grad_dtype, int blocksize, const PlanArgs &a, hipStream_t stream)
{
    switch (grad_dtype) {
    case kF16: return launch_norms_b<OPT, kF16>(blocksize, a, stream);
    case kBF16: return launch_norms_b<OPT, kBF16>(blocksize, a, stream);
    default: return launch_norms_b<OPT, kF32>(blocksize, a, stream);
    }
}

hipError_t launch_trust_ratios(int opt, int grad_dtype, int blocksize, const PlanArgs &a,
                               hipStream_t stream)
{
    hipError_t e;
    switch (opt) {
    case kLamb: e = launch_norms_g<kLamb>(grad_dtype, blocksize, a, stream); break;
    case kLars: e = launch_norms_g<kLars>(grad_dtype, blocksize, a, stream); break;
    default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess)
        return e;
    hipLaunchKernelGGL(segment_sums_kernel, dim3((unsigned)a.nsegments), dim3(kTrustThreads), 0,
                       stream, a);
    hipLaunchKernelGGL(trust_ratio_kernel,
                       dim3((unsigned)((a.ntensors + kTrustThreads - 1) / kTrustThreads)),
                       dim3(kTrustThreads), 0, stream, a, opt == kLamb ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_step_persistent(int opt, int grad_dtype, int blocksize, const StepArgs &a,
                                 hipStream_t stream)
{
    switch (opt) {
    case kAdam: return launch_persist_g<kAdam>(grad_dtype, blocksize, a, stream);
    case kAdamW: return launch_persist_g<kAdamW>(grad_dtype, blocksize, a, stream);
    case kMomentum: return launch_persist_g<kMomentum>(grad_dtype, blocksize, a, stream);
    case kAdaGrad: return launch_persist_g<kAdaGrad>(grad_dtype, blocksize, a, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t static_scratch(uint8_t **ptr)
{
    // one device address per device, looked up with that device current
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static uint8_t *addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        addr[dev] = static_cast<uint8_t *>(p);
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_static_upload(const StaticUploadArgs &a, hipStream_t stream)
{
    hipLaunchKernelGGL(static_upload_kernel, dim3(1), dim3(64), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_step_static(int opt, int grad_dtype, int blocksize, const StaticArgs &a,
                              hipStream_t stream)
{
    switch (opt) {
    case kAdam: return launch_static_g<kAdam>(grad_dtype, blocksize, a, stream);
    case kAdamW: return launch_static_g<kAdamW>(grad_dtype, blocksize, a, stream);
    case kMomentum: return launch_static_g<kMomentum>(grad_dtype, blocksize, a, stream);
    case kAdaGrad: return launch_static_g<kAdaGrad>(grad_dtype, blocksize, a, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_step_oneshot(int opt, int grad_dtype, int blocksize, const PlanArgs &a,
                               hipStream_t stream)
{
    switch (opt) {
    case kLamb: return launch_os_g<kLamb>(grad_dtype, blocksize, a, stream);
    case kLars: return launch_os_g<kLars>(grad_dtype, blocksize, a, stream);
    case kAdam: return launch_os_g<kAdam>(grad_dtype, blocksize, a, stream);
    case kAdamW: return launch_os_g<kAdamW>(grad_dtype, blocksize, a, stream);
    case kMomentum: return launch_os_g<kMomentum>(grad_dtype, blocksize, a, stream);
    case kAdaGrad: return launch_os_g<kAdaGrad>(grad_dtype, blocksize, a, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_dequantize(const float *qmap, const uint8_t *codes, const float *absmax,
                             int64_t n, int blocksize, float *out, hipStream_t stream)
{
    const int64_t tiles = (n + dequant_tile() - 1) / dequant_tile();
    int lg = 0;
    while ((1 << lg) < blocksize)
        ++lg;
    hipLaunchKernelGGL(dequantize_kernel, dim3((unsigned)tiles), dim3(kOS), 0, stream, qmap,
                       codes, absmax, n, lg, out);
    return hipGetLastError();
}

hipError_t launch_quantize(const float *qmap, const float *x, int64_t n, int blocksize,
                           uint8_t *codes, float *absmax, hipStream_t stream)
{
    switch (blocksize) {
    case 256: return launch_qr_t<256>(qmap, x, n, codes, absmax, stream);
    case 512: return launch_qr_t<512>(qmap, x, n, codes, absmax, stream);
    case 1024: return launch_qr_t<1024>(qmap, x, n, codes, absmax, stream);
    case 2048: return launch_qr_t<2048>(qmap, x, n, codes, absmax, stream);
    case 4096: return launch_qr_t<4096>(qmap, x, n, codes, absmax, stream);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_quantize_prepared(const uint8_t *tables, const float *x, int64_t n,
                                    int blocksize, uint8_t *codes, float *absmax,
                                    hipStream_t stream)
{
    switch (blocksize) {
    case 256: return launch_qp_t<256>(tables, x, n, codes, absmax, stream);
    case 512: return launch_qp_t<512>(tables, x, n, codes, absmax, stream);
    case 1024: return launch_qp_t<1024>(tables, x, n, codes, absmax, stream);
    case 2048: return launch_qp_t<2048>(tables, x, n, codes, absmax, stream);
    case 4096: return launch_qp_t<4096>(tables, x, n, codes, absmax, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace bq
