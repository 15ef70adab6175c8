// Device helpers shared by the CHAOS kernels: the activation, wavefront
// reductions and the per-layer push of a weight gradient.
#pragma once

#include "chaos_internal.h"

namespace chaos {

constexpr float kActA = 1.7159f;
constexpr float kActB = 2.0f / 3.0f;

// y = A tanh(B z) and f'(z) = A B (1 - tanh^2(B z)), both from one expm1:
// with m = expm1(-2B|z|), tanh(B|z|) = -m / (2 + m) and
// 1 - tanh^2(B z) = 4 (1 + m) / (2 + m)^2; neither form cancels, so f' keeps
// its relative accuracy for saturated units and y for small |z|.
__device__ __forceinline__ void activation(float z, float &y, float &d) {
    float m = expm1f(-2.0f * kActB * fabsf(z));
    float den = 2.0f + m;
    float t = -m / den;
    y = copysignf(kActA * t, z);
    d = (kActA * kActB * 4.0f) * (1.0f + m) / (den * den);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Where a layer's weight gradient g goes (per element, once per sample):
//   training   W[off] += -lr * g, an atomic fp32 add or a racy load/add/store
//   frozen     each[off] = g (per-sample row) and/or part[off] += g, an atomic
//              add into this worker's own zero-initialised row.  A worker's
//              samples are separated by barriers that wait for its memory
//              operations, so the adds into a row happen in sample order and
//              the partial sums are reproducible bit for bit.
struct Push {
    int mode;
    float *params;
    float neg_lr;
    float *each;  // this sample's gradient row or null
    float *part;  // this worker's partial-sum row or null

    __device__ __forceinline__ void operator()(int off, float g) const {
        if (mode == kTrainAtomic) {
            __hip_atomic_fetch_add(params + off, __fmul_rn(neg_lr, g), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        } else if (mode == kTrainRacy) {
            // same two roundings as the atomic path: w + round(-lr * g)
            // (the library is built without multiply-add contraction)
            float w = __hip_atomic_load(params + off, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(params + off, __fadd_rn(w, __fmul_rn(neg_lr, g)),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (each) each[off] = g;
            if (part)
                __hip_atomic_fetch_add(part + off, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
};

} // namespace chaos
