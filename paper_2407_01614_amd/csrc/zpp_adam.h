// The per-element Adam(W) update shared by the optimizer-step kernels.
#pragma once

#include "zpp_device.h"
#include "zpp_launch.h"

namespace zpp {

// One element, in fp32: decoupled decay (or the L2 term), both moments, and
// the bias-corrected update.  The host folds the bias corrections into
// step_size = lr / (1 - beta1^t) and inv_bc2 = 1 / (1 - beta2^t).
template <bool ADAMW>
__device__ __forceinline__ void adam_update(float &p, float &m, float &v, float g,
                                            const AdamConsts &c) {
    if (ADAMW)
        p = p - c.lr_wd * p;
    else
        g = g + c.wd * p;
    m = c.beta1 * m + c.one_minus_beta1 * g;
    v = c.beta2 * v + c.one_minus_beta2 * (g * g);
    const float denom = __builtin_sqrtf(v * c.inv_bc2) + c.eps;
    p = p - c.step_size * (m / denom);
}

}  // namespace zpp
