// Per-sample CHAOS worker kernel for gfx950 (generic over any layer list).
//
// One workgroup is one worker (Section III-A.1): it repeatedly takes the
// next unprocessed sample, forward-propagates it, computes the error against
// the label and back-propagates layer by layer.  Per layer, the partial
// derivatives of the layer below are computed from the layer's weights first;
// then the layer's weight gradient is formed and pushed to the shared weights
// (Controlled Hogwild, Section III-A.2) without any synchronisation with
// other workers (Arbitrary Order of Synchronization, Section III-A.3).
//
// The same kernel, with the push replaced, gives the frozen-weight
// forward/backward (per-sample gradients or fixed-order partial sums) and
// the forward-only evaluation (Validation/Testing, Section III-A.1).
//
// Per-worker state lives in a private scratch area in global memory (it is
// L2-resident for the nets of Table I); the shared weights are read through
// the caches and are re-validated at the start of every sample.
#include "chaos_internal.h"
#include "device_common.h"

namespace chaos {

namespace {

// Forward of one conv layer: y = f(b + sum w * in) over a valid, stride-1
// cross-correlation with all input maps (Section II-A, Table I).
__device__ void conv_forward(const Layer &ly, const float *__restrict__ in,
                             const float *__restrict__ W, float *__restrict__ y,
                             float *__restrict__ d) {
    const int K = ly.k, KK = K * K, HWo = ly.hout * ly.wout;
    const float *wl = W + ly.w_off, *bl = W + ly.b_off;
    for (int i = threadIdx.x; i < ly.nout; i += blockDim.x) {
        int o = i / HWo, r = i - o * HWo;
        int p = r / ly.wout, q = r - p * ly.wout;
        float s = bl[o];
        const float *wo = wl + o * ly.cin * KK;
        for (int c = 0; c < ly.cin; ++c) {
            const float *ic = in + (c * ly.hin + p) * ly.win + q;
            const float *wc = wo + c * KK;
            for (int u = 0; u < K; ++u)
                for (int v = 0; v < K; ++v) s = fmaf(wc[u * K + v], ic[u * ly.win + v], s);
        }
        activation(s, y[i], d[i]);
    }
}

// Non-overlapping k x k max; the first maximum in row-major window order wins.
__device__ void pool_forward(const Layer &ly, const float *__restrict__ in, float *__restrict__ y,
                             int *__restrict__ arg) {
    const int k = ly.k, HWo = ly.hout * ly.wout;
    for (int i = threadIdx.x; i < ly.nout; i += blockDim.x) {
        int c = i / HWo, r = i - c * HWo;
        int P = r / ly.wout, Q = r - P * ly.wout;
        int best = (c * ly.hin + P * k) * ly.win + Q * k;
        float m = in[best];
        for (int u = 0; u < k; ++u)
            for (int v = 0; v < k; ++v) {
                int idx = (c * ly.hin + P * k + u) * ly.win + Q * k + v;
                float val = in[idx];
                if (val > m) { m = val; best = idx; }
            }
        y[i] = m;
        arg[i] = best;
    }
}

// Fully connected: one wavefront per neuron, lanes across the inputs.
__device__ void fc_forward(const Layer &ly, const float *__restrict__ in,
                           const float *__restrict__ W, float *__restrict__ y,
                           float *__restrict__ d) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
    const float *wl = W + ly.w_off, *bl = W + ly.b_off;
    for (int j = wave; j < ly.cout; j += nwaves) {
        const float *wj = wl + (int64_t)j * ly.cin;
        float s = 0.0f;
        for (int i = lane; i < ly.cin; i += 64) s = fmaf(wj[i], in[i], s);
        s = wave_sum(s);
        if (lane == 0) activation(s + bl[j], y[j], d[j]);
    }
}

// dE/d(input) of a conv layer: e_in[c][r][s] = sum_o sum_{u,v} w[o][c][u][v] *
// delta[o][r-u][s-v] over the in-range terms (gathered, no atomics).
__device__ void conv_backdata(const Layer &ly, const float *__restrict__ W,
                              const float *__restrict__ delta, float *__restrict__ e_in) {
    const int K = ly.k, KK = K * K, HWi = ly.hin * ly.win;
    const float *wl = W + ly.w_off;
    for (int idx = threadIdx.x; idx < ly.nin; idx += blockDim.x) {
        int c = idx / HWi, rr = idx - c * HWi;
        int r = rr / ly.win, s = rr - r * ly.win;
        int u0 = max(0, r - ly.hout + 1), u1 = min(K - 1, r);
        int v0 = max(0, s - ly.wout + 1), v1 = min(K - 1, s);
        float acc = 0.0f;
        for (int o = 0; o < ly.cout; ++o) {
            const float *wc = wl + (o * ly.cin + c) * KK;
            const float *dl = delta + o * ly.hout * ly.wout;
            for (int u = u0; u <= u1; ++u)
                for (int v = v0; v <= v1; ++v)
                    acc = fmaf(wc[u * K + v], dl[(r - u) * ly.wout + (s - v)], acc);
        }
        e_in[idx] = acc;
    }
}

__device__ void fc_backdata(const Layer &ly, const float *__restrict__ W,
                            const float *__restrict__ delta, float *__restrict__ e_in) {
    const float *wl = W + ly.w_off;
    for (int i = threadIdx.x; i < ly.cin; i += blockDim.x) {
        float acc = 0.0f;
        for (int j = 0; j < ly.cout; ++j) acc = fmaf(wl[(int64_t)j * ly.cin + i], delta[j], acc);
        e_in[i] = acc;
    }
}

// Max-pool backward: each input position receives its window's error if it
// is the recorded maximum, else zero.
__device__ void pool_backdata(const Layer &ly, const int *__restrict__ arg,
                              const float *__restrict__ e, float *__restrict__ e_in) {
    const int k = ly.k, HWi = ly.hin * ly.win;
    for (int idx = threadIdx.x; idx < ly.nin; idx += blockDim.x) {
        int c = idx / HWi, rr = idx - c * HWi;
        int r = rr / ly.win, s = rr - r * ly.win;
        int w = (c * ly.hout + r / k) * ly.wout + s / k;
        e_in[idx] = (arg[w] == idx) ? e[w] : 0.0f;
    }
}

// Weight gradient of a conv layer, pushed element by element:
// g[o][c][u][v] = sum_{p,q} delta[o][p][q] in[c][p+u][q+v], g_b[o] = sum delta[o].
__device__ void conv_wgrad(const Layer &ly, const float *__restrict__ in,
                           const float *__restrict__ delta, const Push &push) {
    const int K = ly.k, KK = K * K, CKK = ly.cin * KK;
    for (int widx = threadIdx.x; widx < ly.nw; widx += blockDim.x) {
        int o = widx / CKK, r = widx - o * CKK;
        int c = r / KK, uv = r - c * KK;
        int u = uv / K, v = uv - u * K;
        const float *dl = delta + o * ly.hout * ly.wout;
        const float *ic = in + (c * ly.hin + u) * ly.win + v;
        float g = 0.0f;
        for (int p = 0; p < ly.hout; ++p)
            for (int q = 0; q < ly.wout; ++q) g = fmaf(dl[p * ly.wout + q], ic[p * ly.win + q], g);
        push(ly.w_off + widx, g);
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
    const int HWo = ly.hout * ly.wout;
    for (int o = wave; o < ly.cout; o += nwaves) {
        float g = 0.0f;
        for (int i = lane; i < HWo; i += 64) g += delta[o * HWo + i];
        g = wave_sum(g);
        if (lane == 0) push(ly.b_off + o, g);
    }
}

__device__ void fc_wgrad(const Layer &ly, const float *__restrict__ in,
                         const float *__restrict__ delta, const Push &push) {
    for (int widx = threadIdx.x; widx < ly.nw; widx += blockDim.x) {
        int j = widx / ly.cin, i = widx - j * ly.cin;
        push(ly.w_off + widx, delta[j] * in[i]);
    }
    for (int j = threadIdx.x; j < ly.cout; j += blockDim.x) push(ly.b_off + j, delta[j]);
}

template <int MODE>
__global__ void __launch_bounds__(256, 8) worker_kernel(Net net, WorkArgs a) {
    __shared__ int64_t s_idx;
    __shared__ float s_red[4];
    float *ws = a.scratch + (int64_t)blockIdx.x * net.scratch_floats;
    float *e0 = ws + net.e_off0, *e1 = ws + net.e_off1;
    const float *W = a.params;
    const bool train = (MODE == kTrainAtomic || MODE == kTrainRacy);
    int64_t step = 0;

    for (;; ++step) {
        // Every wavefront waits for its own pushes of the previous sample to
        // complete (a workgroup barrier does not wait for them), so after the
        // barrier below all of this worker's updates have reached memory: the
        // worker sees its own updates and one worker is exact per-sample SGD.
        // In frozen mode the same wait keeps the adds into this worker's
        // partial-sum row in sample order.
        wait_vector_memory();
        if (train) {
            if (threadIdx.x == 0) s_idx = atomicAdd(a.counter, 1);
        } else if (threadIdx.x == 0) {
            s_idx = (int64_t)blockIdx.x + step * gridDim.x;
        }
        __syncthreads();
        const int64_t idx = s_idx;
        __syncthreads();  // everyone has read s_idx before it is rewritten
        if (idx >= a.n) break;
        if (train) {
            // Reads are performed on demand: drop weights cached by this CU
            // during the previous sample so this one sees the pushes made
            // since (by all workers, this one's included) at the agent's
            // coherence point.
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            if (a.claims && threadIdx.x == 0) atomicAdd(a.claims + idx, 1);
        }
        const float *x = a.x + idx * net.in_size;
        const int label = a.labels[idx];

        // ---- forward propagation (Section II-A) ----
        const float *in = x;
        for (int l = 0; l < net.n_layers; ++l) {
            const Layer &ly = net.L[l];
            if (ly.kind == kConv) conv_forward(ly, in, W, ws + ly.y_off, ws + ly.d_off);
            else if (ly.kind == kPool) pool_forward(ly, in, ws + ly.y_off, (int *)(ws + ly.arg_off));
            else fc_forward(ly, in, W, ws + ly.y_off, ws + ly.d_off);
            __syncthreads();
            in = ws + ly.y_off;
        }
        const float *yout = in;
        if (a.out)
            for (int k = threadIdx.x; k < net.n_out; k += blockDim.x) a.out[idx * net.n_out + k] = yout[k];

        if (MODE == kEvaluate) {
            if (threadIdx.x == 0) {
                int best = 0;
                for (int k = 1; k < net.n_out; ++k)
                    if (yout[k] > yout[best]) best = k;
                if (best != label) atomicAdd(a.n_wrong, 1);
            }
            continue;
        }

        // ---- error at the output: E = 1/2 sum (y - t)^2, e = y - t ----
        if (threadIdx.x < 64) {
            float part = 0.0f;
            for (int k = threadIdx.x; k < net.n_out; k += 64) {
                float dk = yout[k] - (k == label ? 1.0f : 0.0f);
                e0[k] = dk;
                part = fmaf(dk, dk, part);
            }
            part = wave_sum(part);
            if (threadIdx.x == 0 && a.loss) a.loss[idx] = 0.5f * part;
        }
        __syncthreads();

        // ---- back-propagation with per-layer push (Section III-A.2) ----
        Push push;
        push.mode = MODE;
        push.params = a.params;
        push.neg_lr = -a.lr;
        push.each = a.grad_each ? a.grad_each + idx * (int64_t)net.n_params : nullptr;
        push.part = a.grad_part ? a.grad_part + (int64_t)blockIdx.x * net.n_params : nullptr;
        float *e = e0, *ep = e1;
        for (int l = net.n_layers - 1; l >= 0; --l) {
            const Layer &ly = net.L[l];
            const float *lin = (l == 0) ? x : ws + net.L[l - 1].y_off;
            if (ly.kind == kPool) {
                if (l > 0) pool_backdata(ly, (const int *)(ws + ly.arg_off), e, ep);
                __syncthreads();
            } else {
                const float *dv = ws + ly.d_off;
                for (int i = threadIdx.x; i < ly.nout; i += blockDim.x) e[i] *= dv[i];
                __syncthreads();
                if (l > 0) {
                    if (ly.kind == kConv) conv_backdata(ly, W, e, ep);
                    else fc_backdata(ly, W, e, ep);
                }
                __syncthreads();  // the layer's weights are no longer read for this sample
                if (ly.kind == kConv) conv_wgrad(ly, lin, e, push);
                else fc_wgrad(ly, lin, e, push);
                __syncthreads();
            }
            float *t = e; e = ep; ep = t;
        }
    }
    (void)s_red;
}

__global__ void fill_i32_kernel(int32_t *p, int32_t v, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

__global__ void fill_f32_kernel(float *p, float v, int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// dst[c] = sum_r part[r][c], r in increasing order, compensated (Kahan)
// summation: the result is a fixed function of the partials.
__global__ void reduce_partials_kernel(const float *__restrict__ part, int64_t rows, int64_t cols,
                                       float *__restrict__ dst) {
    int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= cols) return;
    float s = 0.0f, comp = 0.0f;
    for (int64_t r = 0; r < rows; ++r) {
        float y = part[r * cols + c] - comp;
        float t = s + y;
        comp = (t - s) - y;
        s = t;
    }
    dst[c] = s;
}

// dst[0] = mean of v[0..n) in a fixed order: thread t sums t, t+1024, ...
// sequentially, then a fixed tree over the 1024 partial sums.
__global__ void __launch_bounds__(1024) mean_kernel(const float *__restrict__ v, int64_t n,
                                                    float *__restrict__ dst) {
    __shared__ float part[1024];
    float s = 0.0f;
    for (int64_t i = threadIdx.x; i < n; i += 1024) s += v[i];
    part[threadIdx.x] = s;
    __syncthreads();
    for (int h = 512; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) part[threadIdx.x] += part[threadIdx.x + h];
        __syncthreads();
    }
    if (threadIdx.x == 0) dst[0] = n > 0 ? part[0] / (float)n : 0.0f;
}

__global__ void count_kernel(const int32_t *__restrict__ src, float *__restrict__ dst) {
    if (threadIdx.x == 0) dst[0] = (float)src[0];
}

// dst[c][i] = src[i] for c < copies
__global__ void replicate_kernel(const float *__restrict__ src, float *__restrict__ dst, int64_t n,
                                 int copies) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float v = src[i];
    for (int c = 0; c < copies; ++c) dst[(int64_t)c * n + i] = v;
}

// dst[0] = 1 when *val is not finite or exceeds *ref, else 0
__global__ void above_kernel(const float *__restrict__ val, const float *__restrict__ ref,
                             float *__restrict__ dst) {
    if (threadIdx.x == 0) {
        const float v = val[0];
        dst[0] = (isfinite(v) && v <= ref[0]) ? 0.0f : 1.0f;
    }
}

__global__ void axpy_kernel(float *__restrict__ w, const float *__restrict__ g, float alpha,
                            int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) w[i] = fmaf(alpha, g[i], w[i]);
}

// device index of canonical index i under layout L
__device__ __forceinline__ int64_t dev_index(const ParamLayout &L, int64_t i) {
    for (int s = 0; s < L.n_seg; ++s) {
        const ParamSegment &g = L.seg[s];
        const int64_t r0 = i - g.can_off;
        if (r0 >= 0 && r0 < (int64_t)g.rows * g.len) {
            const int64_t r = r0 / g.len;
            return g.dev_off + r * g.dev_stride + (r0 - r * g.len);
        }
    }
    return -1;  // not reached for i < the layout's canonical size
}

__global__ void convert_params_kernel(const float *__restrict__ src, float *__restrict__ dst,
                                      ParamLayout L, int64_t n_can, int to_device) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_can) return;
    const int64_t d = dev_index(L, i);
    if (d < 0) return;
    if (to_device) dst[d] = src[i];
    else dst[i] = src[d];
}

__global__ void axpy_mapped_kernel(float *__restrict__ w, const float *__restrict__ g, float alpha,
                                   ParamLayout L, int64_t n_can) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n_can) return;
    const int64_t d = dev_index(L, i);
    if (d >= 0) w[d] = fmaf(alpha, g[i], w[d]);
}

inline unsigned blocks_for(int64_t n, int b) { return (unsigned)((n + b - 1) / b); }

} // namespace

hipError_t launch_worker(int mode, const Net &net, const WorkArgs &a, int grid, int block,
                         hipStream_t s) {
    switch (mode) {
    case kTrainAtomic: worker_kernel<kTrainAtomic><<<grid, block, 0, s>>>(net, a); break;
    case kTrainRacy: worker_kernel<kTrainRacy><<<grid, block, 0, s>>>(net, a); break;
    case kForwardBackward: worker_kernel<kForwardBackward><<<grid, block, 0, s>>>(net, a); break;
    case kEvaluate: worker_kernel<kEvaluate><<<grid, block, 0, s>>>(net, a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t *p, int32_t v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_i32_kernel<<<blocks_for(n, 256), 256, 0, s>>>(p, v, n);
    return hipGetLastError();
}

hipError_t launch_fill_f32(float *p, float v, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    fill_f32_kernel<<<blocks_for(n, 256), 256, 0, s>>>(p, v, n);
    return hipGetLastError();
}

hipError_t launch_reduce_partials(const float *part, int64_t rows, int64_t cols, float *dst,
                                  hipStream_t s) {
    if (cols <= 0) return hipSuccess;
    reduce_partials_kernel<<<blocks_for(cols, 256), 256, 0, s>>>(part, rows, cols, dst);
    return hipGetLastError();
}

hipError_t launch_mean(const float *v, int64_t n, float *dst, hipStream_t s) {
    mean_kernel<<<1, 1024, 0, s>>>(v, n, dst);
    return hipGetLastError();
}

hipError_t launch_count(const int32_t *src, float *dst, hipStream_t s) {
    count_kernel<<<1, 64, 0, s>>>(src, dst);
    return hipGetLastError();
}

hipError_t launch_replicate(const float *src, float *dst, int64_t n, int copies, hipStream_t s) {
    if (n <= 0 || copies <= 0) return hipSuccess;
    replicate_kernel<<<blocks_for(n, 256), 256, 0, s>>>(src, dst, n, copies);
    return hipGetLastError();
}

hipError_t launch_above(const float *val, const float *ref, float *dst, hipStream_t s) {
    above_kernel<<<1, 64, 0, s>>>(val, ref, dst);
    return hipGetLastError();
}

hipError_t launch_axpy(float *w, const float *g, float alpha, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    axpy_kernel<<<blocks_for(n, 256), 256, 0, s>>>(w, g, alpha, n);
    return hipGetLastError();
}

hipError_t launch_convert_params(const float *src, float *dst, const ParamLayout &L, int64_t n_can,
                                 bool to_device, hipStream_t s) {
    if (n_can <= 0) return hipSuccess;
    convert_params_kernel<<<blocks_for(n_can, 256), 256, 0, s>>>(src, dst, L, n_can, to_device ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_axpy_mapped(float *w_dev, const float *g_can, float alpha, const ParamLayout &L,
                              int64_t n_can, hipStream_t s) {
    if (n_can <= 0) return hipSuccess;
    axpy_mapped_kernel<<<blocks_for(n_can, 256), 256, 0, s>>>(w_dev, g_can, alpha, L, n_can);
    return hipGetLastError();
}

int worker_blocks_per_cu(int block) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, worker_kernel<kTrainAtomic>, block, 0) !=
        hipSuccess)
        return 0;
    return nb;
}

} // namespace chaos
