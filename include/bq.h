/*
 * bq.h - C ABI of libbq, 8-bit block-wise optimizers for AMD MI355X (gfx950).
 *
 * Implements the hot path of Dettmers, Lewis, Shleifer, Zettlemoyer,
 * "8-bit Optimizers via Block-wise Quantization" (ICLR 2022):
 *   - the dynamic (tree) quantization codebooks          (Sections 2.3, 3.2)
 *   - block-wise quantization and dequantization         (Sections 2.2, 3.1, Eq. 3-4)
 *   - the fused 8-bit Adam / AdamW / Momentum / AdaGrad step (Section 3, Eq. 1-2, App. H),
 *     and LAMB / LARS through step plans (App. E)
 *   - the quantile maps and their GPU estimator                 (App. F.2, App. G)
 *
 * Conventions shared by every call
 *   - Pointers named "device" must point to GPU memory of the current HIP
 *     device; host arrays are read or written only during the call.  The
 *     caller owns all memory; the library keeps no pointer after returning and
 *     allocates no device memory, except bq_step_plan_create (a plan owns the
 *     device copy of its descriptors until bq_step_plan_destroy).
 *   - A block covers flat elements [b*B, min((b+1)*B, n)) of one tensor, so a
 *     tensor of n elements has ceil(n/B) blocks and its last block may be
 *     partial.  Blocks never span tensors.
 *   - blocksize B must be a power of two in [256, 4096] (the paper uses 2048).
 *   - Element arrays (values, codes, params, grads, states) must be 16-byte
 *     aligned; absmax arrays and codebooks 4-byte aligned.
 *   - A codebook is 256 fp32 values in device memory, strictly increasing, so
 *     that a code is the rank of its value, with every nonzero magnitude at
 *     least 2^-60 (for such maps the division below is exact; see Eq. 4 note).
 *   - Calls that take a stream are asynchronous and stream-ordered: they only
 *     enqueue kernels on `stream` (0 = the null stream).  All argument checks
 *     run before anything is enqueued, so on an error return nothing was
 *     launched.  n == 0 (or ntensors == 0) is a no-op returning BQ_OK.
 *   - Non-finite inputs are outside the contract.
 */
#ifndef BQ_H
#define BQ_H

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum bq_status {
    BQ_OK = 0,
    BQ_ERR_NULL = 1,      /* a required pointer is NULL */
    BQ_ERR_SIZE = 2,      /* negative n / numel / ntensors, or too large */
    BQ_ERR_BLOCKSIZE = 3, /* blocksize not a power of two in [256, 4096] */
    BQ_ERR_ENUM = 4,      /* unknown codebook kind or optimizer */
    BQ_ERR_DTYPE = 5,     /* unknown gradient dtype */
    BQ_ERR_ALIGN = 6,     /* a pointer violates the alignment rule above */
    BQ_ERR_HIP = 7,       /* the HIP runtime reported an error at launch */
    BQ_ERR_ARG = 8,       /* a scalar argument is out of range (e.g. step < 1) */
    /* not values: these two make the type span every int, so a call that
     * receives any int in it has defined behavior (and rejects it) */
    BQ_STATUS_RANGE_MIN = -2147483647 - 1,
    BQ_STATUS_RANGE_MAX = 2147483647
} bq_status;

typedef enum bq_codebook_kind {
    BQ_SIGNED = 0,            /* dynamic tree map, signed (Section 2.3) */
    BQ_UNSIGNED = 1,          /* dynamic map, unsigned (Section 3.2) */
    BQ_INVERSE_SIGNED = 2,    /* inverse dynamic map, signed (App. F.1) */
    BQ_INVERSE_UNSIGNED = 3,  /* inverse dynamic map, unsigned (App. F.1) */
    BQ_LINEAR_SIGNED = 4,     /* 256 evenly spaced values in [-1, 1] */
    BQ_LINEAR_UNSIGNED = 5,   /* 256 evenly spaced values in [0, 1] */
    /* not values: these two make the type span every int, so a call that
     * receives any int in it has defined behavior (and rejects it) */
    BQ_CODEBOOK_RANGE_MIN = -2147483647 - 1,
    BQ_CODEBOOK_RANGE_MAX = 2147483647
} bq_codebook_kind;
typedef enum bq_optimizer {
    BQ_ADAM = 0,
    BQ_ADAMW = 1,
    BQ_MOMENTUM = 2,
    BQ_ADAGRAD = 3,
    BQ_LAMB = 4,  /* step plans only */
    BQ_LARS = 5,  /* step plans only */
    /* not values: these two make the type span every int, so a call that
     * receives any int in it has defined behavior (and rejects it) */
    BQ_OPTIMIZER_RANGE_MIN = -2147483647 - 1,
    BQ_OPTIMIZER_RANGE_MAX = 2147483647
} bq_optimizer;
/* Gradient element types.  Every grad is converted to fp32 exactly before the
 * update (Section 3: the update itself runs in 32 bit); the paper's setups use
 * fp16 (mixed precision) and fp32 grads, bfloat16 is the common mixed-precision
 * type on MI355X. */
typedef enum bq_dtype {
    BQ_F32 = 0,
    BQ_F16 = 1,
    BQ_BF16 = 2,
    /* not values: these two make the type span every int, so a call that
     * receives any int in it has defined behavior (and rejects it) */
    BQ_DTYPE_RANGE_MIN = -2147483647 - 1,
    BQ_DTYPE_RANGE_MAX = 2147483647
} bq_dtype;

/*
 * Build a 256-entry dynamic codebook on the host (synchronous, no GPU call).
 * Section 2.3: after a sign bit, a run of E zero bits selects the decade
 * 10^-E, a one bit ends the run and the remaining F bits are a linear fraction;
 * Section 3.2: the unsigned map reuses the sign bit as a fraction bit.  Each
 * decade holds the 2^F values 10^-E * (0.1 + 0.9 j / 2^F), j = 1..2^F, rounded
 * once to fp32 (correctly rounded from the exact rational).
 *   BQ_SIGNED:   E = 0..6, F = 6 - E, both signs (127 magnitudes each), plus 0
 *                and +1e-7; -1 at code 0, 0 at code 127, +1 at code 255.
 *   BQ_UNSIGNED: E = 0..7, F = 7 - E (255 magnitudes), plus 0 at code 0.
 * out: host array of 256 floats, written in ascending order.
 * Errors: BQ_ERR_NULL (out == NULL), BQ_ERR_ENUM (unknown kind).
 */
bq_status bq_make_dynamic_codebook(bq_codebook_kind kind, float out[256]);

/*
 * Any of the fixed codebooks of bq_codebook_kind (host, synchronous), sorted
 * ascending, each entry the exact rational rounded once to fp32.
 *   BQ_SIGNED, BQ_UNSIGNED: as bq_make_dynamic_codebook.
 *   BQ_INVERSE_SIGNED, BQ_INVERSE_UNSIGNED (App. F.1): the dynamic layout with
 *     the exponent run counted from the other end -- E zero bits select decade
 *     10^-(Emax - E) (Emax = 6 signed, 7 unsigned) and keep F = Emax - E
 *     fraction bits, so the smallest decade gets the most values:
 *     signed ±10^-k (0.1 + 0.9 j / 2^k), j = 1..2^k, k = 0..6, plus 0 and
 *     +1e-7; unsigned k = 0..7 plus 0.  Both reach exactly 1.
 *   BQ_LINEAR_SIGNED: (2i - 255) / 255; BQ_LINEAR_UNSIGNED: i / 255.
 * Errors: BQ_ERR_NULL, BQ_ERR_ENUM.
 */
bq_status bq_make_codebook(bq_codebook_kind kind, float out[256]);

/*
 * Quantile map of a sample (App. F.2, lossy minimum-entropy encoding), host,
 * synchronous: with the sample quantile Q(p) = sorted[floor(p n)],
 *   q_i = (Q(i / 257) + Q((i + 1) / 257)) / 2,   i = 0..255,
 * computed in double, divided by max_i |q_i| (so the map spans [-1, 1], or
 * [0, 1] for a non-negative sample) and rounded once to fp32.  Entries that
 * come out equal (ties in the sample) are separated upward by one ulp so the
 * map stays strictly increasing.
 *   sample  host array of n fp32 values (read), all finite
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (n < 1), BQ_ERR_ARG (a non-finite value,
 * or every q_i zero).
 */
bq_status bq_make_quantile_codebook(const float *sample, int64_t n, float out[256]);

/* Values per chunk of the GPU quantile estimator. */
#define BQ_QUANTILE_CHUNK 4096

/* Bytes of device workspace bq_estimate_quantile_codebook needs for n values
 * (0 for n < 1): 257 fp32 per chunk, then 257 fp64 per group of 64 chunks. */
int64_t bq_quantile_workspace_bytes(int64_t n);

/*
 * Quantile map estimated on the GPU (App. F.2 with App. G's chunked
 * estimator): x is cut into chunks of BQ_QUANTILE_CHUNK values (the last one
 * shorter); each chunk is sorted in LDS and gives its sample quantiles
 * Q_c(i / 257) = sorted_c[floor(i L_c / 257)], i = 0..256; the estimate
 * Q(i / 257) is their average weighted by chunk length L_c, summed in double
 * in a fixed order (sequentially within groups of 64 consecutive chunks, then
 * over the groups), so the result is deterministic, unlike atomic averaging;
 * then as bq_make_quantile_codebook: q_i = (Q(i / 257) + Q((i + 1) / 257)) / 2,
 * divided by max |q_i|, rounded to fp32, equal entries moved up by one ulp (an
 * all-zero x gives 0 and then successive subnormals).  Inputs must be finite.
 * Stream-ordered; three launches.
 *   x          device, n fp32 (read), 4-byte aligned (a view such as x + 1
 *              is accepted; 16-byte aligned x is read 16 bytes per lane)
 *   workspace  device, bq_quantile_workspace_bytes(n) bytes, 8-byte aligned,
 *              caller-owned
 *   out        device, 256 fp32 (written)
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (n < 1, or more than 8,388,607 chunks),
 * BQ_ERR_ALIGN, BQ_ERR_HIP.
 */
bq_status bq_estimate_quantile_codebook(const float *x, int64_t n, void *workspace, float *out,
                                        hipStream_t stream);

/*
 * Block-wise quantization (Section 3.1, Eq. 4).  For each block b:
 *   N_b = max_i |x_i|                              -> absmax[b]
 *   code_i = argmin_j |qmap[j] - fl32(x_i / N_b)|  -> codes[i]
 * where fl32(x/N) is the correctly rounded fp32 quotient, ties between two
 * codes go to the lower index, and an all-zero block (N_b == 0) takes the code
 * nearest to 0.
 *   qmap   device, 256 fp32 (read)
 *   x      device, n fp32 (read)
 *   codes  device, n uint8 (written)
 *   absmax device, ceil(n / blocksize) fp32 (written)
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (n < 0), BQ_ERR_BLOCKSIZE, BQ_ERR_ALIGN,
 * BQ_ERR_HIP.
 */
bq_status bq_quantize_blockwise(const float *qmap, const float *x, int64_t n,
                                int32_t blocksize, uint8_t *codes, float *absmax,
                                hipStream_t stream);

/*
 * Block-wise dequantization (Section 2.2): out_i = qmap[codes_i] * absmax[b],
 * one fp32 multiply.
 *   qmap   device, 256 fp32 (read)
 *   codes  device, n uint8 (read)
 *   absmax device, ceil(n / blocksize) fp32 (read)
 *   out    device, n fp32 (written)
 * One workgroup per tile of 4096 elements.
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (n < 0, or more than 8,388,607 tiles),
 * BQ_ERR_BLOCKSIZE, BQ_ERR_ALIGN, BQ_ERR_HIP.
 */
bq_status bq_dequantize_blockwise(const float *qmap, const uint8_t *codes,
                                  const float *absmax, int64_t n, int32_t blocksize,
                                  float *out, hipStream_t stream);

/* One parameter tensor of the step; all pointers are device pointers. */
typedef struct bq_tensor {
    float *param;       /* numel fp32, updated in place */
    const void *grad;   /* numel fp32, fp16 or bf16 (see grad_dtype), read only */
    uint8_t *state1;    /* numel codes of the first state (m), in place */
    uint8_t *state2;    /* numel codes of the second state (r); NULL for Momentum, AdaGrad */
    float *absmax1;     /* ceil(numel / B) block absmax of state 1, in place */
    float *absmax2;     /* ceil(numel / B) block absmax of state 2; NULL for Momentum, AdaGrad */
    int64_t numel;
} bq_tensor;

/* Hyperparameters; step is t >= 1, incremented by the caller. */
typedef struct bq_hparams {
    float lr, beta1, beta2, eps, weight_decay;
    int64_t step;
    float trust_coeff; /* LARS's trust coefficient; unused by the others */
} bq_hparams;

/*
 * The fused 8-bit optimizer step (Section 3, Fig. 1): for every block of every
 * tensor, dequantize the states with the old absmax, apply the 32-bit update,
 * take the new block absmax, and requantize each state to its nearest code
 * (as bq_quantize_blockwise).  The param update uses the unquantized states.
 *   Adam (Eq. 2, with bias correction):
 *       g += wd * w   (only if weight_decay != 0)
 *       m' = b1 m + (1 - b1) g;      r' = b2 r + (1 - b2) g^2
 *       w' = w - (lr / (1 - b1^t)) * m' / (sqrt(r') / sqrt(1 - b2^t) + eps)
 *   AdamW: w *= (1 - lr * wd) first, then Adam without the L2 term.
 *   Momentum (Eq. 1): g += wd * w (if weight_decay != 0); m' = b1 m + g;
 *       w' = w - lr m'  (beta2 and eps unused).
 *   AdaGrad (App. H, textbook form): g += wd * w (if weight_decay != 0);
 *       r' = r + g^2 (state 1, non-negative: pass an unsigned map as qmap1);
 *       w' = w - lr g / (sqrt(r') + eps)  (betas unused; no state 2).
 *   LAMB and LARS (App. E, textbook forms) need per-tensor norms and run
 *   through step plans only; this call returns BQ_ERR_ENUM for them.
 * State 1 uses qmap1 (the signed map), state 2 uses qmap2 (the unsigned map;
 * any map for state 2 must have no negative entries, so that r' >= 0).
 * Momentum and AdaGrad have one state: state2, absmax2 and qmap2 may be NULL.
 * A zero state is every code at the index of 0.0 with absmax 0.
 *   tensors  host array of ntensors descriptors
 *   hp       host pointer to the hyperparameters
 *   qmap1    device, 256 fp32; qmap2 device, 256 fp32 (NULL for Momentum, AdaGrad)
 * Arithmetic of the states is fp32 in a fixed order without contraction, so
 * codes and absmax are reproducible; the param update uses the hardware square
 * root and reciprocal (relative error a few ulp of the update).
 * Allocates nothing: the descriptors of up to 56 non-empty tensors travel in
 * each kernel launch's arguments (so a list takes ceil(count / 56) launches,
 * in list order), and every workgroup builds the maps' decision tables in its
 * own on-chip memory.  A step plan (below) runs the same step in one launch.
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE, BQ_ERR_BLOCKSIZE, BQ_ERR_ENUM, BQ_ERR_DTYPE,
 * BQ_ERR_ALIGN, BQ_ERR_ARG (hp->step < 1), BQ_ERR_HIP.
 */
bq_status bq_optimizer8bit_step(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                                const bq_tensor *tensors, int32_t ntensors,
                                const bq_hparams *hp, const float *qmap1,
                                const float *qmap2, hipStream_t stream);

/*
 * For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): bq_optimizer8bit_step with
 * the same arguments, checks and results bit for bit as a step plan run
 * (bq_step_plan_run) over the same list, without a plan.  The maps' decision
 * tables and the list's descriptors go to a static device array of
 * BQ_STATIC_SCRATCH_BYTES that the library holds on each GPU it runs on until
 * the process ends; then one launch runs every tile of every tensor.
 * Launches: one prepare, ceil(count / 56) descriptor uploads (count = the
 * non-empty tensors, at most BQ_STATIC_MAX_TENSORS), one step.  Allocates
 * nothing and calls no allocating routine.  Every call on one GPU shares that
 * GPU's array: calls that overlap on one GPU (different streams, or different
 * host threads) race and must be ordered by the caller.
 * Errors: as bq_optimizer8bit_step, and BQ_ERR_SIZE for more than
 * BQ_STATIC_MAX_TENSORS non-empty tensors or more than 8,388,607 tiles of
 * 4096 elements in total.
 */
#define BQ_STATIC_MAX_TENSORS 4096
#define BQ_STATIC_SCRATCH_BYTES 279808
bq_status bq_optimizer8bit_step_static(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                                       const bq_tensor *tensors, int32_t ntensors,
                                       const bq_hparams *hp, const float *qmap1,
                                       const float *qmap2, hipStream_t stream);

/* One tensor with 32-bit states; all pointers are device pointers. */
typedef struct bq_tensor32 {
    float *param;       /* numel fp32, updated in place */
    const void *grad;   /* numel fp32, fp16 or bf16 (see grad_dtype), read only */
    float *state1;      /* numel fp32 first state (m), in place */
    float *state2;      /* numel fp32 second state (r); NULL for Momentum, AdaGrad */
    int64_t numel;
} bq_tensor32;

/*
 * The same optimizer step with 32-bit states (Section 3.3 keeps the embedding
 * layer's states in 32 bit): the update of bq_optimizer8bit_step without
 * dequantization and requantization, states fp32 in the same operation order.
 * For tensors exempted from 8-bit states by the caller.
 *   tensors  host array of ntensors descriptors; every non-empty tensor's
 *            pointers 16-byte aligned
 *   hp       host pointer to the hyperparameters (step >= 1)
 * LAMB and LARS are not available here (BQ_ERR_ENUM).
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE, BQ_ERR_ENUM, BQ_ERR_DTYPE, BQ_ERR_ALIGN,
 * BQ_ERR_ARG (step < 1), BQ_ERR_HIP.
 */
bq_status bq_optimizer32bit_step(bq_optimizer opt, bq_dtype grad_dtype,
                                 const bq_tensor32 *tensors, int32_t ntensors,
                                 const bq_hparams *hp, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Prepared codebooks and step plans: the fast path.
 *
 * The calls above build a codebook's decision tables inside every persistent
 * workgroup, because they receive nothing but the raw map.  The calls below
 * keep those tables in caller-visible device memory, so that every tile can
 * run as its own short-lived workgroup (512 threads; 8192 elements for the
 * quantize call, 4096 for the step), which streams HBM markedly faster on
 * MI355X.  Codes and absmax are identical to the calls above, bit for bit.
 * ------------------------------------------------------------------------ */

/* Bytes of device memory one prepared codebook occupies (16-byte aligned). */
#define BQ_PREPARED_CODEBOOK_BYTES 8720

/*
 * Build the decision tables of codebook qmap (256 fp32, device) into
 * `prepared` (device, BQ_PREPARED_CODEBOOK_BYTES, 16-byte aligned, owned by the
 * caller): the map itself, the thresholds halfway between adjacent codes
 * (Eq. 3's argmin boundaries) and a bucket index over fp32 bit patterns.
 * Stream-ordered; re-run it whenever qmap's contents change.
 * Errors: BQ_ERR_NULL, BQ_ERR_ALIGN, BQ_ERR_HIP.
 */
bq_status bq_prepare_codebook(const float *qmap, void *prepared, hipStream_t stream);

/*
 * bq_quantize_blockwise with a prepared codebook (Section 3.1, Eq. 4); same
 * arguments and results, one workgroup per tile of 8192 elements.
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (n < 0, or more than 8,388,607 tiles),
 * BQ_ERR_BLOCKSIZE, BQ_ERR_ALIGN, BQ_ERR_HIP.
 */
bq_status bq_quantize_blockwise_prepared(const void *prepared, const float *x, int64_t n,
                                         int32_t blocksize, uint8_t *codes, float *absmax,
                                         hipStream_t stream);

/* Opaque multi-tensor step plan. */
typedef struct bq_step_plan_s *bq_step_plan;

/*
 * Create a plan for the fused 8-bit step (Section 3, Fig. 1) over a fixed
 * tensor list.  This is the only allocating call: it writes one 64-byte record
 * per tile (4096 elements; pointers at the tile's first element and block) to
 * device memory of the current device -- 16 bytes per 1,024 params -- and
 * reserves space for two prepared codebooks and 64 bytes of step scalars
 * (and, for LAMB and LARS, 16 bytes of partial norms per tile, 32 bytes per
 * segment of up to 2048 tiles of one tensor, and 12 bytes per tensor).
 * Besides the optimizers of bq_optimizer8bit_step, plans run (App. E lists
 * 8-bit versions of both; textbook forms, one trust ratio per tensor, from
 * the norms before the update, 1 when a norm is zero):
 *   LAMB: m' = b1 m + (1 - b1) g;  r' = b2 r + (1 - b2) g^2;
 *         u = (m' / (1 - b1^t)) / (sqrt(r') / sqrt(1 - b2^t) + eps) + wd w;
 *         w' = w - lr (|w| / |u|) u   (states: signed and unsigned maps)
 *   LARS: g' = g + wd w;  m' = b1 m + lr (trust |w| / (|g| + wd |w|)) g';
 *         w' = w - m'   (one state; trust = hp->trust_coeff)
 * Each run first takes the norms in an extra pass over the tensors; the sums
 * are formed in a fixed order, so a run is deterministic.
 * Synchronous.  The tensors' buffers must stay valid while the plan is used.
 *   tensors  host array of ntensors descriptors (as bq_optimizer8bit_step)
 *   plan     receives the handle (NULL on error)
 * Errors: BQ_ERR_NULL, BQ_ERR_SIZE (more than 8,388,607 tiles in total),
 * BQ_ERR_BLOCKSIZE, BQ_ERR_ENUM, BQ_ERR_DTYPE, BQ_ERR_ALIGN, BQ_ERR_HIP.
 */
bq_status bq_step_plan_create(bq_optimizer opt, int32_t blocksize, bq_dtype grad_dtype,
                              const bq_tensor *tensors, int32_t ntensors, bq_step_plan *plan);

/*
 * One step of the plan's optimizer over all its tensors, as
 * bq_optimizer8bit_step with the same hyperparameters and codebooks: one
 * launch that prepares both codebooks, then one launch over every tile of
 * every tensor.  Allocates nothing.  Must be called with the plan's device
 * current (else BQ_ERR_ARG).  A plan holds one codebook workspace: runs of one
 * plan on different streams must not overlap.
 * Errors: BQ_ERR_NULL, BQ_ERR_ALIGN, BQ_ERR_ARG (step < 1, wrong device),
 * BQ_ERR_HIP.
 */
bq_status bq_step_plan_run(bq_step_plan plan, const bq_hparams *hp, const float *qmap1,
                           const float *qmap2, hipStream_t stream);

/*
 * bq_step_plan_run with codebooks prepared beforehand.  An optimizer's maps
 * are fixed (the dynamic maps of Sections 2.3 and 3.2), so their tables can be
 * prepared once and read by every step; the run then skips the prepare launch
 * and leaves the plan's own codebook workspace untouched.  Results are
 * identical, bit for bit, to bq_step_plan_run with the maps the tables were
 * prepared from.
 *   prepared  device, read, 16-byte aligned, owned by the caller: two prepared
 *             codebooks back to back, state 1's map at `prepared` and state
 *             2's at prepared + BQ_PREPARED_CODEBOOK_BYTES (one-state
 *             optimizers read only the first), each written by
 *             bq_prepare_codebook.  It must not change while a run that reads
 *             it is in flight.
 * Errors: BQ_ERR_NULL, BQ_ERR_ALIGN, BQ_ERR_ARG (step < 1, wrong device),
 * BQ_ERR_HIP.
 */
bq_status bq_step_plan_run_prepared(bq_step_plan plan, const bq_hparams *hp, const void *prepared,
                                    hipStream_t stream);

/*
 * bq_step_plan_run_prepared with the hyperparameters read from device memory
 * when the run executes, not when it is enqueued: the run can be captured into
 * a HIP graph once and replayed as successive steps, with the learning rate
 * (or any other field) changed in device memory between replays.  A one-wave
 * launch first forms the per-step scalars from *hp_device, in the same double
 * arithmetic as the host path, so a run gives the same bits as
 * bq_step_plan_run_prepared with the same values.
 *   hp_device     device, one bq_hparams, 8-byte aligned, owned by the caller;
 *                 with advance_step = 1 its step is incremented by one and
 *                 written back before it is used (start from step = 0 for a
 *                 first step); with 0 it is read as is.  step must be >= 1
 *                 when the run uses it (the host cannot check it).
 *   advance_step  0 or 1
 *   prepared      as bq_step_plan_run_prepared
 * The plan's scalar workspace (64 bytes, allocated by bq_step_plan_create) is
 * written by every such run: runs of one plan must not overlap.  An empty
 * plan still advances the step.  Allocates nothing.
 * Errors: BQ_ERR_NULL, BQ_ERR_ALIGN, BQ_ERR_ARG (advance_step not 0 or 1,
 * wrong device), BQ_ERR_HIP.
 */
bq_status bq_step_plan_run_device(bq_step_plan plan, bq_hparams *hp_device, int32_t advance_step,
                                  const void *prepared, hipStream_t stream);

/* Free a plan's device memory (synchronizes with the device).  NULL is a no-op. */
bq_status bq_step_plan_destroy(bq_step_plan plan);

/* Static, human-readable name of a status code (never NULL). */
const char *bq_status_string(bq_status s);

#ifdef __cplusplus
}
#endif

#endif /* BQ_H */
