// Per-step scalars of the optimizer update (bias corrections of Eq. 2, the
// AdamW decay factor, and the fused Adam divisor), formed in double from the
// fp32 hyperparameters and rounded once to fp32.  The same code runs on the
// host (a call's kernel arguments) and on the device (a plan run that reads
// its hyperparameters from device memory), so both give the same bits: every
// operation is an IEEE double +, -, *, / or sqrt, correctly rounded on both.
#pragma once

#include <math.h>
#include <stdint.h>

#include "bq_internal.h"

#if defined(__HIP__)
#define BQ_HD __host__ __device__
#else
#define BQ_HD
#endif

namespace bq {

// beta^t in double by right-to-left binary exponentiation.
BQ_HD inline double beta_pow(double beta, int64_t t)
{
    double acc = 1.0;
    for (double sq = beta; t > 0; t >>= 1, sq *= sq)
        if (t & 1)
            acc *= sq;
    return acc;
}

// Bias-corrected Adam (the paper's Eq. 2 omits the correction constants),
// decoupled AdamW decay, and the L2 weight-decay term; each scalar is formed in
// double from the fp32 inputs and rounded once to fp32.  AdaGrad has neither
// bias correction nor momentum: its update w - lr g / (sqrt(r) + eps) uses
// step_size = lr and inv_sqrt_bc2 = 1.  opt is kAdam .. kLars.
BQ_HD inline StepScalars make_scalars(float lr_f, float beta1, float beta2, float eps, float wd_f,
                                      int64_t step, float trust, int opt)
{
    const double lr = lr_f, b1 = beta1, b2 = beta2, wd = wd_f;
    StepScalars s;
    s.b1 = beta1;
    s.omb1 = static_cast<float>(1.0 - b1);
    s.b2 = beta2;
    s.omb2 = static_cast<float>(1.0 - b2);
    s.eps = eps;
    s.lr = lr_f;
    s.wd = wd_f;
    if (opt == kAdaGrad) {
        s.step_size = lr_f;
        s.inv_sqrt_bc2 = 1.0f;
    } else {
        s.step_size = static_cast<float>(lr / (1.0 - beta_pow(b1, step)));
        s.inv_sqrt_bc2 = static_cast<float>(1.0 / sqrt(1.0 - beta_pow(b2, step)));
    }
    s.decay = static_cast<float>(1.0 - lr * wd);
    s.bc1_inv = static_cast<float>(1.0 / (1.0 - beta_pow(b1, step)));
    s.trust = trust;
    const double ss = static_cast<double>(s.step_size), fmax_f = 3.4028234663852886e38;
    if (ss == 0.0) {
        s.sdiv_c = 0.0f;
        s.sdiv_eps = INFINITY;
    } else {
        s.sdiv_c = static_cast<float>(fmax(-fmax_f, fmin(fmax_f, s.inv_sqrt_bc2 / ss)));
        s.sdiv_eps = static_cast<float>(fmax(-fmax_f, fmin(fmax_f, eps / ss)));
    }
    return s;
}

// The L2 term on the gradient: weight_decay != 0 for every optimizer but AdamW
// (decoupled decay) and LAMB (decay inside the update direction).
BQ_HD inline int32_t l2_on_grad(float wd, int opt)
{
    return (wd != 0.0f && opt != kAdamW && opt != kLamb) ? 1 : 0;
}

}  // namespace bq
