// Optimizer arithmetic of the sparse update, shared by tc_sparse_update and
// the fused backward + update so that both round identically: separately
// rounded fp32 operations (the library is built with -ffp-contract=off;
// division and square root are correctly rounded).
#pragma once

#include "tc_internal.h"

namespace tc {

// SGD: W <- W - lr*G (lr*G rounded, then the difference).
__device__ __forceinline__ float sgd_step(float w, float g, float lr) { return w - lr * g; }

// Adagrad, Eq. (2): A <- A + G*G; W <- W - lr * (G / sqrt(eps + A)), epsilon
// inside the square root as the paper writes it.
__device__ __forceinline__ void adagrad_step(float &w, float &a, float g, float lr, float eps) {
    a = a + g * g;
    w = w - lr * (g / sqrtf(eps + a));
}

// RMSprop, Eq. (1): A <- gamma*A + (1 - gamma)*G*G; W <- W - lr * (G /
// sqrt(eps + A)). `omg` is 1 - gamma, rounded once by the caller.
__device__ __forceinline__ void rmsprop_step(float &w, float &a, float g, float lr, float eps,
                                             float gamma, float omg) {
    const float t = gamma * a;
    a = t + omg * (g * g);
    w = w - lr * (g / sqrtf(eps + a));
}

}  // namespace tc
