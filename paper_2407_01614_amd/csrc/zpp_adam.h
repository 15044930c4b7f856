// The per-element Adam(W) update shared by the optimizer-step kernels.
#pragma once

#include "zpp_device.h"
#include "zpp_launch.h"

namespace zpp {

// One element, in fp32: decoupled decay (or the L2 term), both moments, and
// the bias-corrected update.  The host folds the bias corrections into
// step_size = lr / (1 - beta1^t) and inv_bc2 = 1 / (1 - beta2^t).  Every
// fused multiply-add is written out and nothing else is contracted, so every
// kernel that inlines the update rounds exactly alike (the compiler would
// otherwise choose per kernel which product of a sum to fuse).
template <bool ADAMW>
__device__ __forceinline__ void adam_update(float &p, float &m, float &v, float g,
                                            const AdamConsts &c) {
#pragma clang fp contract(off)
    if (ADAMW)
        p = __builtin_fmaf(-c.lr_wd, p, p);
    else
        g = __builtin_fmaf(c.wd, p, g);
    m = __builtin_fmaf(c.beta1, m, c.one_minus_beta1 * g);
    v = __builtin_fmaf(c.beta2, v, c.one_minus_beta2 * (g * g));
    const float denom = __builtin_sqrtf(v * c.inv_bc2) + c.eps;
    p = __builtin_fmaf(-c.step_size, m / denom, p);
}

}  // namespace zpp
