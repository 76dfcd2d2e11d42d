// Internal declarations shared by the C-ABI layer (bq_api.cpp) and the HIP
// kernels (bq_oneshot.hip, bq_state32.hip, bq_quantiles.hip).  Not part of the
// public interface.
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "bq.h"

namespace bq {

// Per-step fp32 scalars, each formed in double and rounded once (make_scalars
// in bq_scalars.h: on the host for the kernel arguments, or on the device).
struct StepScalars {
    float b1, omb1;        // beta1, 1 - beta1
    float b2, omb2;        // beta2, 1 - beta2
    float eps, lr, wd;
    float step_size;       // lr / (1 - beta1^t)
    float inv_sqrt_bc2;    // 1 / sqrt(1 - beta2^t)
    float decay;           // 1 - lr * wd  (AdamW)
    // Adam denominator divided by step_size, so that the param update is
    // w - m / (sqrt(v) * sdiv_c + sdiv_eps) without a separate multiply:
    // sdiv_c = inv_sqrt_bc2 / step_size, sdiv_eps = eps / step_size (each
    // clamped to the finite range; lr = 0 gives 0 and +inf: no update).
    float sdiv_c, sdiv_eps;
    float bc1_inv;         // 1 / (1 - beta1^t)  (LAMB)
    float trust;           // trust coefficient (LARS)
};

// One tensor of a multi-tensor launch.  tile_begin is the index of the
// tensor's first tile in the launch's flat tile list.
struct TensorDesc {
    float *param;
    const void *grad;
    uint8_t *s1;
    uint8_t *s2;
    float *a1;
    float *a2;
    int64_t numel;
    int64_t tile_begin;
};
static_assert(sizeof(TensorDesc) == 64, "descriptor layout");

// Descriptors travel by value in the kernel arguments; a launch carries at
// most this many so that the argument block stays below 4 KiB.
constexpr int kMaxDescPerLaunch = 56;

struct StepArgs {
    const float *q1;
    const float *q2;
    StepScalars sc;
    int32_t ntensors;
    int32_t total_tiles;
    int32_t use_wd;        // L2 term for Adam / Momentum (weight_decay != 0)
    int32_t pad;
    TensorDesc d[kMaxDescPerLaunch];
};
static_assert(sizeof(StepArgs) <= 4096, "kernel argument block must stay below 4 KiB");

// Elements per tile of the prepared-codebook quantize kernel: kQuantChunks
// chunks of 2048 (512 threads x 4 elements), or one block when the block is
// larger; of the dequantize kernel: kDequantChunks chunks of 2048.  (Measured
// on MI355X at 67M elements: quantize streams best with 4 chunks, dequantize,
// whose traffic is mostly writes, with 2.)
constexpr int kQuantChunks = 4;
constexpr int kDequantChunks = 2;
constexpr int quant_tile(int blocksize)
{
    return 2048 * (blocksize > 2048 * kQuantChunks ? blocksize / 2048 : kQuantChunks);
}
constexpr int dequant_tile() { return 2048 * kDequantChunks; }

// Elements per tile of the one-shot step kernel: 512 threads x 4 elements per
// chunk, kStepChunks chunks (two for 4096 blocks, which must fit one tile).
constexpr int kStepChunks = 2;
constexpr int step_tile(int blocksize)
{
    return 2048 * (blocksize > 2048 * kStepChunks ? blocksize / 2048 : kStepChunks);
}

// Prepared codebook: decision tables of one map in device memory, built once
// by the prepare kernel and copied into LDS by every workgroup.
//   [0, 1024)      float q[256]          codebook values
//   [1024, 2048)   float t[256]          thresholds, t[255] = +inf
//   [2048, 5376)   uint8 base[+, 3328]   per bucket of positive values
//   [5376, 8704)   uint8 base[-, 3328]   per bucket of negative values
//   [8704, 8708)   int32 kmax            thresholds inside one bucket, at most
constexpr int kPreparedBuckets = 3328;
constexpr int kPreparedOffQ = 0;
constexpr int kPreparedOffT = 1024;
constexpr int kPreparedOffBase = 2048;
constexpr int kPreparedOffKmax = kPreparedOffBase + 2 * kPreparedBuckets;
constexpr int kPreparedBytes = kPreparedOffKmax + 16;
constexpr int kPreparedSignedBytes = kPreparedOffKmax;            // q, t, both halves
constexpr int kPreparedNonnegBytes = kPreparedOffBase + kPreparedBuckets;  // q, t, + half
static_assert(kPreparedBytes % 16 == 0 && kPreparedNonnegBytes % 16 == 0, "16 B granules");

// Scalars of a plan run formed on the device from device-resident
// hyperparameters (scalars_kernel), read by the run's kernels in place of the
// kernel-argument copy.
struct DevScalars {
    StepScalars sc;
    int32_t use_wd;
    int32_t pad;
};

// Arguments of the one-shot step kernel (one workgroup per tile).
struct PlanArgs {
    const uint8_t *tables;        // prepared map of state 1, then of state 2
    // device array, one record per tile: pointers at the tile's first element
    // (param, grad, states) and first block (absmax), numel = elements from
    // the tile start to the tensor end (a full tile when >= the tile size)
    // (for LAMB / LARS plans tile_begin holds the record's tensor index)
    const TensorDesc *tiles;
    StepScalars sc;
    int32_t use_wd;
    int32_t total_tiles;
    // when set, sc and use_wd are read from here instead (formed on the device)
    const DevScalars *dev;
    // LAMB / LARS only: per-tile partial squared norms (2 doubles per tile);
    // each tensor's tiles cut into segments of at most kTrustSegTiles tiles:
    // per segment its tile range [begin, end) and its 2 partial sums; first
    // segment of each tensor (ntensors + 1); per-tensor lr * trust ratio
    double *partials;
    const int64_t *seg_range;
    double *seg_partials;
    const int64_t *first_seg;
    float *lr_ratio;
    int32_t ntensors;
    int32_t nsegments;
};
constexpr int64_t kTrustSegTiles = 2048;

// One tensor of a 32-bit-state launch (states are fp32 arrays).
struct Desc32 {
    float *param;
    const void *grad;
    float *m;
    float *v;  // nullptr for Momentum
    int64_t numel;
    int64_t tile_begin;  // first tile of the tensor in the launch (1024 elements per tile)
};
constexpr int kMaxDesc32PerLaunch = 72;

struct State32Args {
    StepScalars sc;
    int32_t ntensors;
    int32_t total_tiles;
    int32_t use_wd;
    int32_t pad;
    Desc32 d[kMaxDesc32PerLaunch];
};
static_assert(sizeof(State32Args) <= 4096, "kernel argument block must stay below 4 KiB");

// Allocation-free step from a static device array (bq_optimizer8bit_step_static):
// the two prepared maps, then the descriptors of up to kStaticMaxTensors
// non-empty tensors (tile_begin counted in step tiles over the whole list).
constexpr int kStaticMaxTensors = 4096;
constexpr int64_t kStaticOffTables = 0;
constexpr int64_t kStaticOffDesc = 17664;  // 2 * kPreparedBytes, rounded up to 256
constexpr int64_t kStaticScratchBytes = kStaticOffDesc + kStaticMaxTensors * 64;
static_assert(2 * kPreparedBytes <= kStaticOffDesc, "static scratch layout");
static_assert(kStaticScratchBytes == BQ_STATIC_SCRATCH_BYTES &&
                  kStaticMaxTensors == BQ_STATIC_MAX_TENSORS, "bq.h limits");

// One launch of the descriptor upload: count descriptors (kernel arguments)
// written to entries [first, first + count) of the static array.
struct StaticUploadArgs {
    uint8_t *scratch;
    int32_t first;
    int32_t count;
    TensorDesc d[kMaxDescPerLaunch];
};
static_assert(sizeof(StaticUploadArgs) <= 4096, "kernel argument block must stay below 4 KiB");

// Arguments of the static step kernel (one workgroup per tile of the list).
// The first tile of every stride-th non-empty tensor travels in the arguments
// (stride = ceil(ntensors / kStaticArgTiles): 1 up to 992 tensors), so a
// workgroup finds its tensor by a scalar search there, plus, for stride > 1,
// one ballot over the first tiles of at most stride descriptors.
constexpr int kStaticArgTiles = 992;
struct StaticArgs {
    const uint8_t *tables;   // scratch + kStaticOffTables
    const uint8_t *scratch;  // the static array (device address)
    StepScalars sc;
    int32_t use_wd;
    int32_t ntensors;
    int32_t total_tiles;
    int32_t stride;
    int32_t nfirst;          // entries of first_tile: ceil(ntensors / stride)
    int32_t pad;
    int32_t first_tile[kStaticArgTiles];
};
static_assert(sizeof(StaticArgs) <= 4096, "kernel argument block must stay below 4 KiB");
static_assert((kStaticMaxTensors + kStaticArgTiles - 1) / kStaticArgTiles <= 64,
              "the fine search covers one wave");

// Device address of the static array on the current device (looked up once
// per device, then cached).
hipError_t static_scratch(uint8_t **ptr);
hipError_t launch_static_upload(const StaticUploadArgs &a, hipStream_t stream);
hipError_t launch_step_static(int opt, int grad_dtype, int blocksize, const StaticArgs &a,
                              hipStream_t stream);

// Chunk length of the quantile estimator (values sorted per workgroup in LDS)
// and chunks per first-level summation group.
constexpr int kQChunk = 4096;
constexpr int kQGroup = 64;
// Workspace: 257 fp32 chunk quantiles per chunk (padded to 8 bytes), then 257
// fp64 sums per group.
inline int64_t quantile_partial_bytes(int64_t n)
{
    const int64_t nchunks = (n + kQChunk - 1) / kQChunk;
    return (nchunks * 257 * 4 + 7) / 8 * 8;
}
inline int64_t quantile_workspace_bytes(int64_t n)
{
    const int64_t nchunks = (n + kQChunk - 1) / kQChunk;
    const int64_t ngroups = (nchunks + kQGroup - 1) / kQGroup;
    return quantile_partial_bytes(n) + ngroups * 257 * 8;
}
hipError_t launch_quantile_codebook(const float *x, int64_t n, void *workspace, float *out,
                                    hipStream_t stream);

hipError_t launch_step32(int opt, int grad_dtype, const State32Args &args, hipStream_t stream);

hipError_t launch_prepare(const float *qmap1, const float *qmap2, uint8_t *tables,
                          hipStream_t stream);
// The scalars of optimizer opt from device hyperparameters hp (a bq_hparams;
// with advance, hp's step is incremented first and written back) into out.
hipError_t launch_scalars(int opt, void *hp, int advance, DevScalars *out, hipStream_t stream);
hipError_t launch_step_oneshot(int opt, int grad_dtype, int blocksize, const PlanArgs &args,
                               hipStream_t stream);
// LAMB / LARS: per-tile partial norms, then the per-tensor lr * ratio.
hipError_t launch_trust_ratios(int opt, int grad_dtype, int blocksize, const PlanArgs &args,
                               hipStream_t stream);
hipError_t launch_quantize_prepared(const uint8_t *tables, const float *x, int64_t n,
                                    int blocksize, uint8_t *codes, float *absmax,
                                    hipStream_t stream);

enum { kAdam = 0, kAdamW = 1, kMomentum = 2, kAdaGrad = 3, kLamb = 4, kLars = 5 };
// optimizers with a second state (Adam, AdamW, LAMB)
constexpr bool has_two_states(int opt) { return opt == kAdam || opt == kAdamW || opt == kLamb; }
// optimizers with a per-tensor trust ratio (two passes: norms, then the step)
constexpr bool has_trust_ratio(int opt) { return opt == kLamb || opt == kLars; }
enum { kF32 = 0, kF16 = 1, kBF16 = 2 };

// the fused step from raw maps: the one-shot tile code in persistent
// workgroups (tile_begin in units of step_tile(blocksize))
hipError_t launch_step_persistent(int opt, int grad_dtype, int blocksize, const StepArgs &args,
                                  hipStream_t stream);
hipError_t launch_quantize(const float *qmap, const float *x, int64_t n, int blocksize,
                           uint8_t *codes, float *absmax, hipStream_t stream);
hipError_t launch_dequantize(const float *qmap, const uint8_t *codes, const float *absmax,
                             int64_t n, int blocksize, float *out, hipStream_t stream);

// Host-side codebook construction (bq_codebook.cpp).
int build_dynamic_codebook(int kind, float out[256]);
int build_quantile_codebook(const float *sample, int64_t n, float out[256]);

}  // namespace bq
