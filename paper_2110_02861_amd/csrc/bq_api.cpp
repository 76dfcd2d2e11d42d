// C-ABI entry points of libbq (declared in include/bq.h): argument checks,
// per-step scalar precomputation, packing of tensor descriptors (kernel-argument
// chunks, or a device-resident plan), and launches.  Every check runs before
// the first HIP call, so an error return means nothing was enqueued.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "bq.h"
#include "bq_internal.h"
#include "bq_scalars.h"

namespace {

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool valid_blocksize(int32_t b) { return b >= 256 && b <= 4096 && (b & (b - 1)) == 0; }
// optimizers of the allocation-free calls; LAMB and LARS need per-tensor
// norms and run through plans only
bool valid_opt(bq_optimizer o)
{
    return o == BQ_ADAM || o == BQ_ADAMW || o == BQ_MOMENTUM || o == BQ_ADAGRAD;
}
bool valid_plan_opt(bq_optimizer o) { return valid_opt(o) || o == BQ_LAMB || o == BQ_LARS; }
bool trust_opt(bq_optimizer o) { return o == BQ_LAMB || o == BQ_LARS; }
bool two_states(bq_optimizer o) { return o == BQ_ADAM || o == BQ_ADAMW || o == BQ_LAMB; }
bool valid_dtype(bq_dtype d) { return d == BQ_F32 || d == BQ_F16 || d == BQ_BF16; }

bq::StepScalars make_scalars(const bq_hparams &hp, bq_optimizer opt)
{
    return bq::make_scalars(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, hp.step,
                            hp.trust_coeff, static_cast<int>(opt));
}

bq_status from_hip(hipError_t e) { return e == hipSuccess ? BQ_OK : BQ_ERR_HIP; }

// Checks every descriptor of a tensor list (no HIP call).
bq_status check_tensors(const bq_tensor *tensors, int32_t ntensors, int32_t blocksize, bool two)
{
    const int64_t tile = bq::step_tile(blocksize);
    for (int32_t i = 0; i < ntensors; ++i) {
        const bq_tensor &t = tensors[i];
        if (t.numel < 0)
            return BQ_ERR_SIZE;
        // tiles of one launch are counted in int32
        if (t.numel / tile >= (int64_t)INT32_MAX / 2)
            return BQ_ERR_SIZE;
        if (t.numel == 0)
            continue;
        if (!t.param || !t.grad || !t.state1 || !t.absmax1 ||
            (two && (!t.state2 || !t.absmax2)))
            return BQ_ERR_NULL;
        if (!aligned(t.param, 16) || !aligned(t.grad, 16) || !aligned(t.state1, 16) ||
            !aligned(t.absmax1, 4) ||
            (two && (!aligned(t.state2, 16) || !aligned(t.absmax2, 4))))
            return BQ_ERR_ALIGN;
    }
    return BQ_OK;
}

bq::TensorDesc make_desc(const bq_tensor &t, bool two, int64_t tile_begin)
{
    bq::TensorDesc d;
    d.param = t.param;
    d.grad = t.grad;
    d.s1 = t.state1;
    d.s2 = two ? t.state2 : nullptr;
    d.a1 = t.absmax1;
    d.a2 = two ? t.absmax2 : nullptr;
    d.numel = t.numel;
    d.tile_begin = tile_begin;
    return d;
}

// One-shot launches place one 512-thread workgroup per tile; the grid in
// work-items must stay below 2^32.
constexpr int64_t kMaxOneShotTiles = (int64_t{1} << 32) / 512 - 1;

}  // namespace

struct bq_step_plan_s {
    int device;
    bq_optimizer opt;
    int32_t blocksize;
    bq_dtype grad_dtype;
    int32_t ntensors;      // non-empty tensors
    int64_t total_tiles;
    bq::TensorDesc *tiles;  // device, one record per tile
    uint8_t *tables;        // device, two prepared maps
    // LAMB / LARS: per-tile partial norms, segment tile ranges and partial
    // sums, each tensor's first segment, per-tensor lr * ratio
    double *partials;
    int64_t *seg_range;
    double *seg_partials;
    int64_t *first_seg;
    float *lr_ratio;
    int64_t nsegments;
    bq::DevScalars *dev_scalars;  // device, the scalars of device-hyperparameter runs
};

extern "C" {

const char *bq_status_string(bq_status s)
{
    switch (s) {
    case BQ_OK: return "ok";
    case BQ_ERR_NULL: return "required pointer is NULL";
    case BQ_ERR_SIZE: return "size out of range";
    case BQ_ERR_BLOCKSIZE: return "blocksize must be a power of two in [256, 4096]";
    case BQ_ERR_ENUM: return "unknown codebook kind or optimizer";
    case BQ_ERR_DTYPE: return "unknown gradient dtype";
    case BQ_ERR_ALIGN: return "pointer misaligned (elements 16 B, absmax and codebook 4 B)";
    case BQ_ERR_HIP: return "HIP runtime error";
    case BQ_ERR_ARG: return "scalar argument out of range";
    default: break;
    }
    return "unknown status";
}

bq_status bq_make_dynamic_codebook(bq_codebook_kind kind, float out[256])
{
    if (out == nullptr)
        return BQ_ERR_NULL;
    if (kind != BQ_SIGNED && kind != BQ_UNSIGNED)
        return BQ_ERR_ENUM;
    return bq::build_dynamic_codebook(static_cast<int>(kind), out) == 0 ? BQ_OK : BQ_ERR_ENUM;
}

bq_status bq_make_codebook(bq_codebook_kind kind, float out[256])
{
    if (out == nullptr)
        return BQ_ERR_NULL;
    if (static_cast<int>(kind) < BQ_SIGNED || static_cast<int>(kind) > BQ_LINEAR_UNSIGNED)
        return BQ_ERR_ENUM;
    return bq::build_dynamic_codebook(static_cast<int>(kind), out) == 0 ? BQ_OK : BQ_ERR_ENUM;
}

bq_status bq_make_quantile_codebook(const float *sample, int64_t n, float out[256])
{
    if (!sample || !out)
        return BQ_ERR_NULL;
    if (n < 1)
        return BQ_ERR_SIZE;
    return bq::build_quantile_codebook(sample, n, out) == 0 ? BQ_OK : BQ_ERR_ARG;
}

int64_t bq_quantile_workspace_bytes(int64_t n)
{
    return n < 1 ? 0 : bq::quantile_workspace_bytes(n);
}

bq_status bq_estimate_quantile_codebook(const float *x, int64_t n, void *workspace, float *out,
                                        hipStream_t stream)
{
    if (n < 1)
        return BQ_ERR_SIZE;
    if (!x || !workspace || !out)
        return BQ_ERR_NULL;
    if (!aligned(x, 4) || !aligned(workspace, 8) || !aligned(out, 4))
        return BQ_ERR_ALIGN;
    if ((n + bq::kQChunk - 1) / bq::kQChunk > kMaxOneShotTiles)
        return BQ_ERR_SIZE;
    return from_hip(bq::launch_quantile_codebook(x, n, workspace, out, stream));
}

bq_status bq_quantize_blockwise(const float *qmap, const float *x, int64_t n, int32_t blocksize,
                                uint8_t *codes, float *absmax, hipStream_t stream)
{
    if (n < 0)
        return BQ_ERR_SIZE;
    if (!valid_blocksize(blocksize))
        return BQ_ERR_BLOCKSIZE;
    if (n == 0)
        return BQ_OK;
    if (!qmap || !x || !codes || !absmax)
        return BQ_ERR_NULL;
    if (!aligned(x, 16) || !aligned(codes, 16) || !aligned(absmax, 4) || !aligned(qmap, 4))
        return BQ_ERR_ALIGN;
    return from_hip(bq::launch_quantize(qmap, x, n, blocksize, codes, absmax, stream));
}

bq_status bq_dequantize_blockwise(const float *qmap, const uint8_t *codes, const float *absmax,
                                  int64_t n, int32_t blocksize, float *out, hipStream_t stream)
{
    if (n < 0)
        return BQ_ERR_SIZE;
    if (!valid_blocksize(blocksize))
        return BQ_ERR_BLOCKSIZE;
    if (n == 0)
        return BQ_OK;
    if (!qmap || !codes || !absmax || !out)
        return BQ_ERR_NULL;
    if (!aligned(codes, 16) || !aligned(out, 16) || !aligned(absmax, 4) || !aligned(qmap, 4))
        return BQ_ERR_ALIGN;
    if ((n + bq::dequant_tile() - 1) / bq::dequant_tile() > kMaxOneShotTiles)
        return BQ_ERR_SIZE;
    return from_hip(bq::launch_dequantize(qmap, codes, absmax, n, blocksize, out, stream));
}

}  // extern "C"

namespace {

// Checks of the two allocation-free step calls (no HIP call).
bq_status check_step_call(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                          const bq_tensor *tensors, int32_t ntensors, const bq_hparams *hp,
                          const float *qmap1, const float *qmap2)
{
    if (!valid_opt(opt))
        return BQ_ERR_ENUM;
    if (!valid_dtype(grad_dtype))
        return BQ_ERR_DTYPE;
    if (!valid_blocksize(blocksize))
        return BQ_ERR_BLOCKSIZE;
    if (ntensors < 0)
        return BQ_ERR_SIZE;
    if (ntensors == 0)
        return BQ_OK;
    if (!tensors || !hp || !qmap1)
        return BQ_ERR_NULL;
    const bool two = two_states(opt);
    if (two && !qmap2)
        return BQ_ERR_NULL;
    if (hp->step < 1)
        return BQ_ERR_ARG;
    if (!aligned(qmap1, 4) || (two && !aligned(qmap2, 4)))
        return BQ_ERR_ALIGN;
    return check_tensors(tensors, ntensors, blocksize, two);
}

}  // namespace

extern "C" {

bq_status bq_optimizer8bit_step(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                                const bq_tensor *tensors, int32_t ntensors,
                                const bq_hparams *hp, const float *qmap1, const float *qmap2,
                                hipStream_t stream)
{
    const bq_status st =
        check_step_call(opt, blocksize, grad_dtype, tensors, ntensors, hp, qmap1, qmap2);
    if (st != BQ_OK || ntensors == 0)
        return st;
    const bool two = two_states(opt);

    bq::StepArgs args;
    std::memset(&args, 0, sizeof(args));
    args.q1 = qmap1;
    args.q2 = two ? qmap2 : qmap1;
    args.sc = make_scalars(*hp, opt);
    args.use_wd = bq::l2_on_grad(hp->weight_decay, static_cast<int>(opt));

    // Pack non-empty tensors into launches of at most kMaxDescPerLaunch
    // descriptors, or fewer when a launch's tile count would overflow int32.
    const int64_t tile = bq::step_tile(blocksize);
    int32_t i = 0;
    while (i < ntensors) {
        int32_t k = 0;
        int64_t tiles = 0;
        for (; i < ntensors && k < bq::kMaxDescPerLaunch; ++i) {
            const bq_tensor &t = tensors[i];
            if (t.numel == 0)
                continue;
            const int64_t nt = (t.numel + tile - 1) / tile;
            if (k > 0 && tiles + nt > (int64_t)INT32_MAX / 2)
                break;
            args.d[k++] = make_desc(t, two, tiles);
            tiles += nt;
        }
        if (k == 0)
            continue;
        args.ntensors = k;
        args.total_tiles = static_cast<int32_t>(tiles);
        const hipError_t e = bq::launch_step_persistent(
            static_cast<int>(opt), static_cast<int>(grad_dtype), blocksize, args, stream);
        if (e != hipSuccess)
            return BQ_ERR_HIP;
    }
    return BQ_OK;
}

bq_status bq_optimizer8bit_step_static(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                                       const bq_tensor *tensors, int32_t ntensors,
                                       const bq_hparams *hp, const float *qmap1,
                                       const float *qmap2, hipStream_t stream)
{
    const bq_status st =
        check_step_call(opt, blocksize, grad_dtype, tensors, ntensors, hp, qmap1, qmap2);
    if (st != BQ_OK || ntensors == 0)
        return st;
    const bool two = two_states(opt);
    const int64_t tile = bq::step_tile(blocksize);
    int64_t total = 0;
    int32_t nonempty = 0;
    for (int32_t i = 0; i < ntensors; ++i) {
        if (tensors[i].numel == 0)
            continue;
        total += (tensors[i].numel + tile - 1) / tile;
        if (++nonempty > bq::kStaticMaxTensors || total > kMaxOneShotTiles)
            return BQ_ERR_SIZE;
    }
    if (nonempty == 0)
        return BQ_OK;

    uint8_t *scratch = nullptr;
    hipError_t e = bq::static_scratch(&scratch);
    if (e == hipSuccess)
        e = bq::launch_prepare(qmap1, two ? qmap2 : nullptr, scratch + bq::kStaticOffTables,
                               stream);
    // descriptors of the non-empty tensors, in list order, kMaxDescPerLaunch
    // per upload launch
    bq::StaticUploadArgs up;
    std::memset(&up, 0, sizeof(up));
    up.scratch = scratch;
    int64_t tiles = 0;
    int32_t stored = 0;
    for (int32_t i = 0; i < ntensors && e == hipSuccess; ++i) {
        const bq_tensor &t = tensors[i];
        if (t.numel == 0)
            continue;
        up.d[up.count++] = make_desc(t, two, tiles);
        tiles += (t.numel + tile - 1) / tile;
        if (up.count == bq::kMaxDescPerLaunch || stored + up.count == nonempty) {
            up.first = stored;
            e = bq::launch_static_upload(up, stream);
            stored += up.count;
            up.count = 0;
        }
    }
    if (e == hipSuccess) {
        bq::StaticArgs a;
        std::memset(&a, 0, sizeof(a));
        a.tables = scratch + bq::kStaticOffTables;
        a.scratch = scratch;
        a.sc = make_scalars(*hp, opt);
        a.use_wd = bq::l2_on_grad(hp->weight_decay, static_cast<int>(opt));
        a.ntensors = nonempty;
        a.total_tiles = static_cast<int32_t>(total);
        // first tile of every stride-th non-empty tensor
        a.stride = (nonempty + bq::kStaticArgTiles - 1) / bq::kStaticArgTiles;
        a.nfirst = (nonempty + a.stride - 1) / a.stride;
        int64_t first = 0;
        int32_t k = 0;
        for (int32_t i = 0; i < ntensors; ++i) {
            const bq_tensor &t = tensors[i];
            if (t.numel == 0)
                continue;
            if (k % a.stride == 0)
                a.first_tile[k / a.stride] = static_cast<int32_t>(first);
            first += (t.numel + tile - 1) / tile;
            ++k;
        }
        e = bq::launch_step_static(static_cast<int>(opt), static_cast<int>(grad_dtype), blocksize,
                                   a, stream);
    }
    return from_hip(e);
}

bq_status bq_optimizer32bit_step(bq_optimizer opt, bq_dtype grad_dtype,
                                 const bq_tensor32 *tensors, int32_t ntensors,
                                 const bq_hparams *hp, hipStream_t stream)
{
    if (!valid_opt(opt))
        return BQ_ERR_ENUM;
    if (!valid_dtype(grad_dtype))
        return BQ_ERR_DTYPE;
    if (ntensors < 0)
        return BQ_ERR_SIZE;
    if (ntensors == 0)
        return BQ_OK;
    if (!tensors || !hp)
        return BQ_ERR_NULL;
    if (hp->step < 1)
        return BQ_ERR_ARG;
    const bool two = two_states(opt);
    constexpr int64_t tile = 1024;
    for (int32_t i = 0; i < ntensors; ++i) {
        const bq_tensor32 &t = tensors[i];
        if (t.numel < 0 || t.numel / tile >= (int64_t)INT32_MAX / 2)
            return BQ_ERR_SIZE;
        if (t.numel == 0)
            continue;
        if (!t.param || !t.grad || !t.state1 || (two && !t.state2))
            return BQ_ERR_NULL;
        if (!aligned(t.param, 16) || !aligned(t.grad, 16) || !aligned(t.state1, 16) ||
            (two && !aligned(t.state2, 16)))
            return BQ_ERR_ALIGN;
    }

    bq::State32Args args;
    std::memset(&args, 0, sizeof(args));
    args.sc = make_scalars(*hp, opt);
    args.use_wd = bq::l2_on_grad(hp->weight_decay, static_cast<int>(opt));
    int32_t i = 0;
    while (i < ntensors) {
        int32_t k = 0;
        int64_t tiles = 0;
        for (; i < ntensors && k < bq::kMaxDesc32PerLaunch; ++i) {
            const bq_tensor32 &t = tensors[i];
            if (t.numel == 0)
                continue;
            const int64_t nt = (t.numel + tile - 1) / tile;
            if (k > 0 && tiles + nt > (int64_t)INT32_MAX / 2)
                break;
            bq::Desc32 &d = args.d[k++];
            d.param = t.param;
            d.grad = t.grad;
            d.m = t.state1;
            d.v = two ? t.state2 : nullptr;
            d.numel = t.numel;
            d.tile_begin = tiles;
            tiles += nt;
        }
        if (k == 0)
            continue;
        args.ntensors = k;
        args.total_tiles = static_cast<int32_t>(tiles);
        const hipError_t e = bq::launch_step32(static_cast<int>(opt), static_cast<int>(grad_dtype),
                                               args, stream);
        if (e != hipSuccess)
            return BQ_ERR_HIP;
    }
    return BQ_OK;
}

bq_status bq_prepare_codebook(const float *qmap, void *prepared, hipStream_t stream)
{
    if (!qmap || !prepared)
        return BQ_ERR_NULL;
    if (!aligned(qmap, 4) || !aligned(prepared, 16))
        return BQ_ERR_ALIGN;
    return from_hip(bq::launch_prepare(qmap, nullptr, static_cast<uint8_t *>(prepared), stream));
}

bq_status bq_quantize_blockwise_prepared(const void *prepared, const float *x, int64_t n,
                                         int32_t blocksize, uint8_t *codes, float *absmax,
                                         hipStream_t stream)
{
    if (n < 0)
        return BQ_ERR_SIZE;
    if (!valid_blocksize(blocksize))
        return BQ_ERR_BLOCKSIZE;
    if (n == 0)
        return BQ_OK;
    if (!prepared || !x || !codes || !absmax)
        return BQ_ERR_NULL;
    if (!aligned(prepared, 16) || !aligned(x, 16) || !aligned(codes, 16) || !aligned(absmax, 4))
        return BQ_ERR_ALIGN;
    const int64_t tile = bq::quant_tile(blocksize);
    if ((n + tile - 1) / tile > kMaxOneShotTiles)
        return BQ_ERR_SIZE;
    return from_hip(bq::launch_quantize_prepared(static_cast<const uint8_t *>(prepared), x, n,
                                                 blocksize, codes, absmax, stream));
}

bq_status bq_step_plan_create(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                              const bq_tensor *tensors, int32_t ntensors, bq_step_plan *plan)
{
    if (!plan)
        return BQ_ERR_NULL;
    *plan = nullptr;
    if (!valid_plan_opt(opt))
        return BQ_ERR_ENUM;
    if (!valid_dtype(grad_dtype))
        return BQ_ERR_DTYPE;
    if (!valid_blocksize(blocksize))
        return BQ_ERR_BLOCKSIZE;
    if (ntensors < 0)
        return BQ_ERR_SIZE;
    if (ntensors > 0 && !tensors)
        return BQ_ERR_NULL;
    const bool two = two_states(opt);
    const bq_status st = check_tensors(tensors, ntensors, blocksize, two);
    if (st != BQ_OK)
        return st;

    const int64_t tile = bq::step_tile(blocksize);
    const size_t gbytes = grad_dtype == BQ_F32 ? 4 : 2;
    int64_t total = 0;
    int32_t nonempty = 0;
    for (int32_t i = 0; i < ntensors; ++i) {
        total += (tensors[i].numel + tile - 1) / tile;
        nonempty += tensors[i].numel > 0 ? 1 : 0;
        if (total > kMaxOneShotTiles)
            return BQ_ERR_SIZE;
    }
    std::vector<bq::TensorDesc> recs;
    std::vector<int64_t> first_tile;
    recs.reserve((size_t)total);
    const bool trust = trust_opt(opt);
    for (int32_t i = 0; i < ntensors; ++i) {
        const bq_tensor &t = tensors[i];
        const int64_t nt = (t.numel + tile - 1) / tile;
        if (nt > 0)
            first_tile.push_back((int64_t)recs.size());
        for (int64_t k = 0; k < nt; ++k) {
            const int64_t t0 = k * tile;
            bq::TensorDesc d;
            d.param = t.param + t0;
            d.grad = static_cast<const char *>(t.grad) + t0 * gbytes;
            d.s1 = t.state1 + t0;
            d.s2 = two ? t.state2 + t0 : nullptr;
            d.a1 = t.absmax1 + t0 / blocksize;
            d.a2 = two ? t.absmax2 + t0 / blocksize : nullptr;
            d.numel = t.numel - t0;
            // LAMB / LARS: the tensor's index, for its lr * ratio
            d.tile_begin = trust ? (int64_t)first_tile.size() - 1 : 0;
            recs.push_back(d);
        }
    }
    first_tile.push_back((int64_t)recs.size());
    // segments of at most kTrustSegTiles tiles, never across tensors
    std::vector<int64_t> seg_range, first_seg;
    if (trust) {
        for (size_t t = 0; t + 1 < first_tile.size(); ++t) {
            first_seg.push_back((int64_t)seg_range.size() / 2);
            for (int64_t k = first_tile[t]; k < first_tile[t + 1]; k += bq::kTrustSegTiles) {
                seg_range.push_back(k);
                seg_range.push_back(std::min(k + bq::kTrustSegTiles, first_tile[t + 1]));
            }
        }
        first_seg.push_back((int64_t)seg_range.size() / 2);
    }

    bq_step_plan_s *p = new (std::nothrow) bq_step_plan_s();
    if (!p)
        return BQ_ERR_HIP;
    p->opt = opt;
    p->blocksize = blocksize;
    p->grad_dtype = grad_dtype;
    p->ntensors = nonempty;
    p->total_tiles = (int64_t)recs.size();
    p->nsegments = (int64_t)seg_range.size() / 2;
    hipError_t e = hipGetDevice(&p->device);
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&p->tables), 2 * bq::kPreparedBytes);
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&p->dev_scalars), sizeof(bq::DevScalars));
    if (e == hipSuccess && !recs.empty()) {
        e = hipMalloc(reinterpret_cast<void **>(&p->tiles), recs.size() * sizeof(bq::TensorDesc));
        if (e == hipSuccess)
            e = hipMemcpy(p->tiles, recs.data(), recs.size() * sizeof(bq::TensorDesc),
                          hipMemcpyHostToDevice);
        if (e == hipSuccess && trust) {
            e = hipMalloc(reinterpret_cast<void **>(&p->partials),
                          recs.size() * 2 * sizeof(double));
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&p->lr_ratio),
                              (size_t)nonempty * sizeof(float));
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&p->seg_partials),
                              (size_t)p->nsegments * 2 * sizeof(double));
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&p->seg_range),
                              seg_range.size() * sizeof(int64_t));
            if (e == hipSuccess)
                e = hipMemcpy(p->seg_range, seg_range.data(), seg_range.size() * sizeof(int64_t),
                              hipMemcpyHostToDevice);
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&p->first_seg),
                              first_seg.size() * sizeof(int64_t));
            if (e == hipSuccess)
                e = hipMemcpy(p->first_seg, first_seg.data(), first_seg.size() * sizeof(int64_t),
                              hipMemcpyHostToDevice);
        }
    }
    if (e != hipSuccess) {
        bq_step_plan_destroy(p);
        return BQ_ERR_HIP;
    }
    *plan = p;
    return BQ_OK;
}

}  // extern "C"

namespace {

// Checks shared by the two run calls (no HIP call before the device query).
bq_status check_run(bq_step_plan plan, const bq_hparams *hp)
{
    if (!plan || !hp)
        return BQ_ERR_NULL;
    if (hp->step < 1)
        return BQ_ERR_ARG;
    return BQ_OK;
}

// Launches one run of a plan.  The hyperparameters come from the host (hp)
// or, with hp NULL, from device memory (hp_dev, read by scalars_kernel when
// the run executes; advance increments its step first).  With qmap1 set, the
// plan's own workspace is prepared from the raw maps first; otherwise `tables`
// already holds both prepared codebooks.
bq_status launch_run(bq_step_plan plan, const bq_hparams *hp, bq_hparams *hp_dev, int advance,
                     const uint8_t *tables, const float *qmap1, const float *qmap2,
                     hipStream_t stream)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return BQ_ERR_HIP;
    if (dev != plan->device)
        return BQ_ERR_ARG;

    bq::PlanArgs a;
    std::memset(&a, 0, sizeof(a));
    a.tables = tables;
    a.tiles = plan->tiles;
    a.partials = plan->partials;
    a.seg_range = plan->seg_range;
    a.seg_partials = plan->seg_partials;
    a.first_seg = plan->first_seg;
    a.lr_ratio = plan->lr_ratio;
    a.ntensors = plan->ntensors;
    a.nsegments = (int32_t)plan->nsegments;
    if (hp) {
        a.sc = make_scalars(*hp, plan->opt);
        // decoupled decay for AdamW, inside the update direction for LAMB, an
        // L2 term on the gradient otherwise
        a.use_wd = bq::l2_on_grad(hp->weight_decay, static_cast<int>(plan->opt));
    } else {
        a.dev = plan->dev_scalars;
    }
    a.total_tiles = (int32_t)plan->total_tiles;
    hipError_t e = hipSuccess;
    // a device step advances even for an empty plan, so that step counts stay
    // in line with the caller's other plans
    if (!hp)
        e = bq::launch_scalars(static_cast<int>(plan->opt), hp_dev, advance, plan->dev_scalars,
                               stream);
    if (plan->total_tiles == 0)
        return from_hip(e);
    if (e == hipSuccess && qmap1)
        e = bq::launch_prepare(qmap1, two_states(plan->opt) ? qmap2 : nullptr, plan->tables,
                               stream);
    if (e == hipSuccess && trust_opt(plan->opt))
        e = bq::launch_trust_ratios((int)plan->opt, (int)plan->grad_dtype, plan->blocksize, a,
                                    stream);
    if (e == hipSuccess)
        e = bq::launch_step_oneshot((int)plan->opt, (int)plan->grad_dtype, plan->blocksize, a,
                                    stream);
    return from_hip(e);
}

}  // namespace

extern "C" {

bq_status bq_step_plan_run(bq_step_plan plan, const bq_hparams *hp, const float *qmap1,
                           const float *qmap2, hipStream_t stream)
{
    bq_status st = check_run(plan, hp);
    if (st != BQ_OK)
        return st;
    const bool two = two_states(plan->opt);
    if (!qmap1 || (two && !qmap2))
        return BQ_ERR_NULL;
    if (!aligned(qmap1, 4) || (two && !aligned(qmap2, 4)))
        return BQ_ERR_ALIGN;
    if (plan->total_tiles == 0)
        return BQ_OK;
    return launch_run(plan, hp, nullptr, 0, plan->tables, qmap1, qmap2, stream);
}

bq_status bq_step_plan_run_prepared(bq_step_plan plan, const bq_hparams *hp, const void *prepared,
                                    hipStream_t stream)
{
    bq_status st = check_run(plan, hp);
    if (st != BQ_OK)
        return st;
    if (!prepared)
        return BQ_ERR_NULL;
    if (!aligned(prepared, 16))
        return BQ_ERR_ALIGN;
    if (plan->total_tiles == 0)
        return BQ_OK;
    return launch_run(plan, hp, nullptr, 0, static_cast<const uint8_t *>(prepared), nullptr,
                      nullptr, stream);
}

bq_status bq_step_plan_run_device(bq_step_plan plan, bq_hparams *hp_device, int32_t advance_step,
                                  const void *prepared, hipStream_t stream)
{
    if (!plan || !hp_device || !prepared)
        return BQ_ERR_NULL;
    if (advance_step != 0 && advance_step != 1)
        return BQ_ERR_ARG;
    if (!aligned(hp_device, 8) || !aligned(prepared, 16))
        return BQ_ERR_ALIGN;
    return launch_run(plan, nullptr, hp_device, advance_step,
                      static_cast<const uint8_t *>(prepared), nullptr, nullptr, stream);
}

bq_status bq_step_plan_destroy(bq_step_plan plan)
{
    if (!plan)
        return BQ_OK;
    hipError_t e = hipSuccess;
    for (void *ptr : {static_cast<void *>(plan->tiles), static_cast<void *>(plan->tables),
                      static_cast<void *>(plan->partials), static_cast<void *>(plan->lr_ratio),
                      static_cast<void *>(plan->seg_range), static_cast<void *>(plan->seg_partials),
                      static_cast<void *>(plan->first_seg),
                      static_cast<void *>(plan->dev_scalars)}) {
        if (ptr && hipFree(ptr) != hipSuccess)
            e = hipErrorUnknown;
    }
    delete plan;
    return from_hip(e);
}

}  // extern "C"
