// Optimizer arithmetic of the sparse update, shared by tc_sparse_update and
// the fused backward + update so that both round identically: separately
// rounded fp32 operations (the library is built with -ffp-contract=off;
// division and square root are correctly rounded).
#pragma once

#include "tc_internal.h"

namespace tc {

// Table and accumulator rows are read and written once per step by the
// update (unique rows are distinct), so those loads and stores are
// non-temporal: they stream through the caches without displacing what the
// caches hold for the gathers (the backward's output-gradient rows, the
// next forward's hot table rows).
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4 stream_load4(const float *p) {
    const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stream_store4(float *p, float4 v) {
    const f32x4_t x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f32x4_t *>(p));
}
__device__ __forceinline__ float stream_load(const float *p) {
    return __builtin_nontemporal_load(p);
}
__device__ __forceinline__ void stream_store(float *p, float v) { __builtin_nontemporal_store(v, p); }

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
