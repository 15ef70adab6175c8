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
//              add into this worker's own zero-initialised row.  Every
//              wavefront of a worker waits for its memory operations before
//              the worker starts its next sample, so the adds into a row
//              happen in sample order and the partial sums are reproducible
//              bit for bit.
struct Push {
    int mode;
    float *params;
    float neg_lr;
    float *each;  // this sample's gradient row or null
    float *part;  // this worker's partial-sum row or null

    // w_off indexes the shared weights (the kernel's device layout), g_off
    // the gradient rows (canonical layout); they differ only for a net whose
    // device layout pads its rows.
    __device__ __forceinline__ void operator()(int w_off, int g_off, float g) const {
        if (mode == kTrainAtomic) {
            __hip_atomic_fetch_add(params + w_off, __fmul_rn(neg_lr, g), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        } else if (mode == kTrainRacy) {
            // same two roundings as the atomic path: w + round(-lr * g)
            // (the library is built without multiply-add contraction)
            float w = __hip_atomic_load(params + w_off, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(params + w_off, __fadd_rn(w, __fmul_rn(neg_lr, g)),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            if (each) each[g_off] = g;
            if (part)
                __hip_atomic_fetch_add(part + g_off, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __device__ __forceinline__ void operator()(int off, float g) const { (*this)(off, off, g); }

    // The same push, returning the weight it found: the value just before
    // this push (training) or the unchanged weight (frozen).  A layer whose
    // partial derivatives need its own weights can take them from here in
    // one pass instead of reading them before pushing.
    __device__ __forceinline__ float with_old(int w_off, int g_off, float g) const {
        if (mode == kTrainAtomic) {
            return __hip_atomic_fetch_add(params + w_off, __fmul_rn(neg_lr, g), __ATOMIC_RELAXED,
                                          __HIP_MEMORY_SCOPE_AGENT);
        } else if (mode == kTrainRacy) {
            float w = __hip_atomic_load(params + w_off, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(params + w_off, __fadd_rn(w, __fmul_rn(neg_lr, g)), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
            return w;
        } else {
            const float w = params[w_off];
            if (each) each[g_off] = g;
            if (part)
                __hip_atomic_fetch_add(part + g_off, g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return w;
        }
    }
    __device__ __forceinline__ float with_old(int off, float g) const { return with_old(off, off, g); }
};

// Orders the LDS accesses of this wavefront's lanes around this point (a
// read after a write to the same word by another lane of the wavefront sees
// the write).  The LDS serves one wavefront's instructions in issue order, so
// it is enough that the compiler keeps them in program order; unlike a
// workgroup fence this does not wait for outstanding global operations such
// as weight pushes.
__device__ __forceinline__ void wave_lds_order() {
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// Waits until every vector memory operation this wavefront has issued has
// completed (s_waitcnt vmcnt(0)), its fire-and-forget weight pushes
// included.  Workgroup barriers do not wait for them, so a worker that must
// see its own updates (the next sample's weight reads; the next sample's adds
// into a partial-sum row) has every wavefront wait here first.
__device__ __forceinline__ void wait_vector_memory() {
    // simm16: vmcnt 0, expcnt 7, lgkmcnt 15 (no wait on those two)
    __builtin_amdgcn_s_waitcnt(0x0F70);
}

// One ordered step of a col2im scatter in LDS: this lane adds c[j] to
// p[j][off] for every j.  The J reads are issued together, then the J
// writes, with no branch between them: a lane whose column is padding points
// its p[j] at a scratch area instead (of at least off + 1 floats), so the
// targets of one step are distinct across j and across the lanes of an
// instruction.  Steps whose targets overlap stay in program order.
template <int J>
__device__ __forceinline__ void scatter_add(float *const (&p)[J], int off, const float (&c)[J]) {
    float old[J];
#pragma unroll
    for (int j = 0; j < J; ++j) old[j] = p[j][off];
#pragma unroll
    for (int j = 0; j < J; ++j) p[j][off] = old[j] + c[j];
    wave_lds_order();
}

// Start of a Hogwild epoch.  Every worker of a fused kernel is resident from
// the launch, so without care all of them would compute their first gradient
// at the same weights and push it at nearly the same time: a burst of
// concurrent, identically stale updates.  Instead worker b (b > 0) claims its
// first sample once b / kJoinRamp samples have been completed (counter[1]) or
// once every sample has been handed out (counter[0] >= n), so the number of
// workers grows with the completed samples.  Worker 0 never waits, so the
// condition is always reached; the poll count is bounded as well.
constexpr int kJoinRamp = 4;

__device__ __forceinline__ void join_after(int32_t *counter, int64_t n, int target) {
    for (int s = 0; s < (1 << 20); ++s) {
        const int done = __hip_atomic_load(counter + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int claimed = __hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (done >= target || claimed >= n) return;
        __builtin_amdgcn_s_sleep(32);
    }
}

// Workgroup barrier that orders LDS only: the wavefronts' outstanding global
// memory operations (weight pushes) stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

typedef float f4 __attribute__((ext_vector_type(4)));

// 16x16x4 fp32 MFMA: lane l supplies A[l%16][l/16] and B[l/16][l%16] and
// holds C[4(l/16) + r][l%16] in element r.
__device__ __forceinline__ f4 mfma(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 4x4x1 fp32 MFMA, 16 blocks: lane l supplies A[l/4][l%4] and B[l/4][l%4]
// of block l/4 and holds C[l/4][r][l%4] of that block in element r.
__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_4x4x1f32(a, b, c, 0, 0, 0);
}

typedef float f16 __attribute__((ext_vector_type(16)));

// 32x32x2 fp32 MFMA: lane l supplies A[l%32][l/32] and B[l/32][l%32] and
// holds C[8(r/4) + 4(l/32) + r%4][l%32] in element r.
__device__ __forceinline__ f16 mfma32(float a, float b, f16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// scaled tanh without its derivative (forward epilogues)
__device__ __forceinline__ float act_y(float z) {
    float y, d;
    activation(z, y, d);
    return y;
}

// f'(z) from y = f(z): A B (1 - (y/A)^2) = (B/A)(A^2 - y^2)
__device__ __forceinline__ float dact_from_y(float y) {
    return (kActB / kActA) * (kActA * kActA - y * y);
}

// Max over a 2x2 window of activated conv outputs held in one lane's
// accumulator (window elements in row-major order; the first maximum wins).
// The activation is strictly increasing, so the maximum of f(z) is f of the
// maximum of z: the window is compared on z and f is evaluated once.  (Where
// f would round two different z to the same fp32 value, the larger z wins,
// which is the maximum of the exact f.)
__device__ __forceinline__ void pool4(f4 acc, float bias, float &ymax, int &arg) {
    float zmax = acc[0] + bias;
    arg = 0;
#pragma unroll
    for (int r = 1; r < 4; ++r) {
        float z = acc[r] + bias;
        if (z > zmax) { zmax = z; arg = r; }
    }
    ymax = act_y(zmax);
}

// position (row-major index into a map of width `wd`) of element w of the
// 2x2 window of pooled position P on a pooled grid of width `pw`
__device__ __forceinline__ int window_pos(int P, int w, int pw, int wd) {
    int py = P / pw, px = P - py * pw;
    return (2 * py + (w >> 1)) * wd + 2 * px + (w & 1);
}

} // namespace chaos
