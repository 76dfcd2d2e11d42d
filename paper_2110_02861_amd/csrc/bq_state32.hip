// Optimizer step with 32-bit states, for tensors whose states stay in fp32
// (Section 3.3: the embedding layer keeps 32-bit optimizer states).  The same
// update as the 8-bit step (Eq. 1, Eq. 2, AdamW, AdaGrad) without quantization: the
// states m, r are fp32 arrays updated in place.  One 256-thread workgroup per
// tile of 1024 elements, 4 contiguous elements per thread; the workgroup finds
// its tensor by a binary search over the launch's descriptors.
#include "bq_device.h"

namespace bq {
namespace {

using namespace dev;

constexpr int kThreads32 = 256;
constexpr int kTile32 = kThreads32 * 4;

template <int OPT, int GRAD>
__global__ __launch_bounds__(kThreads32) void step32_kernel(const State32Args a)
{
    // tensor of this tile: the last descriptor with tile_begin <= tile
    const int tile = blockIdx.x;
    int lo = 0, hi = a.ntensors - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.d[mid].tile_begin <= tile)
            lo = mid;
        else
            hi = mid - 1;
    }
    const Desc32 &D = a.d[lo];
    const int64_t e0 = (int64_t)(tile - D.tile_begin) * kTile32 + threadIdx.x * 4;
    if (e0 >= D.numel)
        return;
    const int nv = D.numel - e0 >= 4 ? 4 : (int)(D.numel - e0);
    constexpr bool kTwo = has_two_states(OPT);
    const StepScalars &sc = a.sc;

    float w[4], g[4], m[4], v[4];
    if (nv == 4) {
        const vf4 wv = ld_nt(reinterpret_cast<const vf4 *>(D.param + e0));
        const vf4 mv = ld_nt(reinterpret_cast<const vf4 *>(D.m + e0));
        w[0] = wv.x; w[1] = wv.y; w[2] = wv.z; w[3] = wv.w;
        m[0] = mv.x; m[1] = mv.y; m[2] = mv.z; m[3] = mv.w;
        if constexpr (kTwo) {
            const vf4 vv = ld_nt(reinterpret_cast<const vf4 *>(D.v + e0));
            v[0] = vv.x; v[1] = vv.y; v[2] = vv.z; v[3] = vv.w;
        }
        if constexpr (GRAD != kF32) {
            const vu2 gv = ld_nt(reinterpret_cast<const vu2 *>(
                static_cast<const uint16_t *>(D.grad) + e0));
            g[0] = g16_lo<GRAD>(gv.x); g[1] = g16_hi<GRAD>(gv.x);
            g[2] = g16_lo<GRAD>(gv.y); g[3] = g16_hi<GRAD>(gv.y);
        } else {
            const vf4 gv =
                ld_nt(reinterpret_cast<const vf4 *>(static_cast<const float *>(D.grad) + e0));
            g[0] = gv.x; g[1] = gv.y; g[2] = gv.z; g[3] = gv.w;
        }
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const bool ok = r < nv;
            w[r] = ok ? G(D.param)[e0 + r] : 0.0f;
            m[r] = ok ? G(D.m)[e0 + r] : 0.0f;
            v[r] = (kTwo && ok) ? G(D.v)[e0 + r] : 0.0f;
            g[r] = ok ? grad_at<GRAD>(D.grad, e0 + r) : 0.0f;
        }
    }

#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float gi = g[r];
        if (a.use_wd)
            gi = gi + sc.wd * w[r];
        if constexpr (OPT == kMomentum) {
            m[r] = sc.b1 * m[r] + gi;
            w[r] = w[r] - sc.lr * m[r];
        } else if constexpr (OPT == kAdaGrad) {
            m[r] = m[r] + gi * gi;
            const float denom =
                __builtin_fmaf(__builtin_amdgcn_sqrtf(m[r]), sc.sdiv_c, sc.sdiv_eps);
            w[r] = __builtin_fmaf(-gi, __builtin_amdgcn_rcpf(denom), w[r]);
        } else {
            if constexpr (OPT == kAdamW)
                w[r] = w[r] * sc.decay;
            m[r] = sc.b1 * m[r] + sc.omb1 * gi;
            v[r] = sc.b2 * v[r] + sc.omb2 * (gi * gi);
            const float denom =
                __builtin_fmaf(__builtin_amdgcn_sqrtf(v[r]), sc.sdiv_c, sc.sdiv_eps);
            w[r] = __builtin_fmaf(-m[r], __builtin_amdgcn_rcpf(denom), w[r]);
        }
    }

    if (nv == 4) {
        st_nt(reinterpret_cast<vf4 *>(D.param + e0), vf4{w[0], w[1], w[2], w[3]});
        st_nt(reinterpret_cast<vf4 *>(D.m + e0), vf4{m[0], m[1], m[2], m[3]});
        if constexpr (kTwo)
            st_nt(reinterpret_cast<vf4 *>(D.v + e0), vf4{v[0], v[1], v[2], v[3]});
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (r < nv) {
                G(D.param)[e0 + r] = w[r];
                G(D.m)[e0 + r] = m[r];
                if constexpr (kTwo)
                    G(D.v)[e0 + r] = v[r];
            }
        }
    }
}

template <int OPT>
hipError_t launch32_g(int grad_dtype, const State32Args &a, hipStream_t stream)
{
    const dim3 grid((unsigned)a.total_tiles), block(kThreads32);
    if (grad_dtype == kF16)
        hipLaunchKernelGGL((step32_kernel<OPT, kF16>), grid, block, 0, stream, a);
    else if (grad_dtype == kBF16)
        hipLaunchKernelGGL((step32_kernel<OPT, kBF16>), grid, block, 0, stream, a);
    else
        hipLaunchKernelGGL((step32_kernel<OPT, kF32>), grid, block, 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_step32(int opt, int grad_dtype, const State32Args &a, hipStream_t stream)
{
    switch (opt) {
    case kAdam: return launch32_g<kAdam>(grad_dtype, a, stream);
    case kAdamW: return launch32_g<kAdamW>(grad_dtype, a, stream);
    case kMomentum: return launch32_g<kMomentum>(grad_dtype, a, stream);
    case kAdaGrad: return launch32_g<kAdaGrad>(grad_dtype, a, stream);
    default: return hipErrorInvalidValue;
    }
}

}  // namespace bq
