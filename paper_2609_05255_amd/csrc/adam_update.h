// One element of the Adam step (Kingma and Ba, Algorithm 1, with the bias
// corrections moved onto the step size and the denominator), shared by the
// standalone step (adam.hip) and the backward that applies it where each
// gradient is computed (backward.hip): the same fp32 operations, uncontracted,
// so that both give the same bits for the same gradient.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/gsraster.h"

namespace gsr {

// Host-computed constants of one step: per tensor the second-moment terms, per
// row (rows of all tensors in order) the step size lr / (1 - b1^t).
struct AdamStep {
    float b1, omb1, eps;
    float b2[GS_ADAM_MAX_TENSORS], omb2[GS_ADAM_MAX_TENSORS], inv_sqrt_bc2[GS_ADAM_MAX_TENSORS];
    int32_t row0[GS_ADAM_MAX_TENSORS];   // first row of each tensor
    float step_size[GS_ADAM_MAX_ROWS];
};

// m = b1 m + (1 - b1) g; v = b2 v + (1 - b2) g^2;
// p -= step (m / (sqrt(v) / sqrt(1 - b2^t) + eps))
__device__ __forceinline__ void adam_update(float& p, float& m, float& v, float g, float b1, float omb1, float b2,
                                            float omb2, float inv_sqrt_bc2, float eps, float step)
{
#pragma clang fp contract(off)
    m = b1 * m + omb1 * g;
    v = b2 * v + omb2 * (g * g);
    const float denom = sqrtf(v) * inv_sqrt_bc2 + eps;
    p = p - step * (m / denom);
}

// The host constants for `count` tensors (adam.hip).
void adam_step_constants(const gs_adam_tensor* ts, int count, float beta1, float eps, int64_t step, AdamStep& out);

}  // namespace gsr
