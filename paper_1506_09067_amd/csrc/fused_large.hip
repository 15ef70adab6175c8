// Fused per-sample CHAOS worker for the large net on gfx950:
//   1x29x29 -> conv 20@4x4 -> max 2 -> conv 60@3x3 -> conv 100@6x6 -> max 2
//           -> FC 150 -> FC 10, activation 1.7159 tanh(2z/3) on every conv/FC.
//
// One workgroup (4 wavefronts) is one worker and owns one sample at a time
// (Section III-A.1).  All per-sample state stays in LDS.  The three
// convolutions are computed as small implicit GEMMs on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32):
//   forward            rows = output positions, cols = output maps, K = C*k*k
//   weight gradient    rows = output maps, cols = C*k*k, K = output positions
//   backward data      rows = C*k*k, cols = output positions, K = output maps,
//                      followed by a col2im scatter into the input-map errors
// The 2x2 max-pools are fused into the forward epilogues: output rows are
// ordered (pooled position, window element) so that one lane holds the four
// elements of a pooling window in its four accumulator registers.
// The fully connected layers run on the vector ALUs.
//
// Per layer, the partial derivatives of the layer below are computed from the
// layer's weights before the layer's gradient is pushed (Controlled Hogwild,
// Section III-A.2); pushes are lock-free (Section III-A.3).  Every reduction
// has a fixed order, so a worker's results do not depend on timing; with
// frozen weights the whole kernel is deterministic.
#include "chaos_internal.h"
#include "device_common.h"

namespace chaos {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f4 mfma(float a, float b, f4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---- shapes of the large net ---------------------------------------------
constexpr int IN = 29, NX = IN * IN;            // input 1x29x29
constexpr int C1 = 20, K1 = 4, Q1 = 13;         // conv1 20@26x26, pool -> 13x13
constexpr int NP1 = Q1 * Q1;                    // 169
constexpr int C2 = 60, K2 = 3, H2 = 11;         // conv2 60@11x11 on 20@13x13
constexpr int NY2 = H2 * H2;                    // 121
constexpr int KC2 = C1 * K2 * K2;               // 180
constexpr int C3 = 100, K3 = 6;                 // conv3 100@6x6 on 60@11x11
constexpr int KC3 = C2 * K3 * K3;               // 2160
constexpr int NP3 = 9;                          // pool 2 -> 3x3
constexpr int NF1 = C3 * NP3;                   // 900 inputs of FC1
constexpr int F1 = 150, F2 = 10;

// canonical parameter offsets
constexpr int OW1 = 0, OB1 = OW1 + C1 * 16;
constexpr int OW2 = OB1 + C1, OB2 = OW2 + C2 * KC2;
constexpr int OW3 = OB2 + C2, OB3 = OW3 + C3 * KC3;
constexpr int OF1 = OB3 + C3, OBF1 = OF1 + F1 * NF1;
constexpr int OF2 = OBF1 + F1, OBF2 = OF2 + F2 * F1;
constexpr int NPARAM = OBF2 + F2;
static_assert(NPARAM == 363960, "large net parameter count");

constexpr int NT = 256;   // threads per worker
constexpr int NW = NT / 64;

// conv3 output rows m = 4 * P + w (P pooled 3x3 position, w window element)
constexpr int M3 = 36, M3P = 48;                // padded to 3 tiles of 16

struct alignas(16) Smem {
    float x[NX + 3];
    float p1[C1 * NP1];                  // pool1 output
    float y2[C2 * NY2];                  // conv2 output, later its delta
    union {
        struct {
            float s2[C2 * NY2];          // conv3 backward-data sums, then pool1 errors
            float d3[C3 * M3P];          // conv3 output deltas, rows (P, w)
        };
        float red3[2 * 21 * 256];        // conv3 split-K partial sums (forward only)
    };
    float p3[NF1];                       // pool2 output (FC1 input)
    float e3[NF1];                       // dE/d(pool2 output)
    float h[F1 + 10], dh[F1 + 10];
    float o[16], dout[16];
    unsigned char am1[C1 * NP1 + 12];    // pool1 argmax (window element 0..3)
    unsigned char am3[NF1 + 4];          // pool2 argmax
    float red[NW];
    int64_t idx;
};

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

// Max over a 2x2 window held in one lane's accumulator (window elements in
// row-major order); the first maximum wins.
__device__ __forceinline__ void pool4(f4 acc, float bias, float &ymax, int &arg) {
    ymax = act_y(acc[0] + bias);
    arg = 0;
#pragma unroll
    for (int r = 1; r < 4; ++r) {
        float y = act_y(acc[r] + bias);
        if (y > ymax) { ymax = y; arg = r; }
    }
}

// position (row-major index into a map of width `wd`) of element w of the
// 2x2 window of pooled position P on a pooled grid of width `pw`
__device__ __forceinline__ int window_pos(int P, int w, int pw, int wd) {
    int py = P / pw, px = P - py * pw;
    return (2 * py + (w >> 1)) * wd + 2 * px + (w & 1);
}

template <int MODE>
__global__ void __launch_bounds__(NT, 1) fused_large_kernel(WorkArgs a) {
    __shared__ Smem sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lr = lane & 15, lg = lane >> 4;
    const float *W = a.params;
    constexpr bool kTrain = (MODE == kTrainAtomic || MODE == kTrainRacy);
    int64_t step = 0;

    for (;; ++step) {
        // ---- claim a sample (Section III-A.1) ----
        if (tid == 0) sm.idx = kTrain ? (int64_t)atomicAdd(a.counter, 1)
                                      : (int64_t)blockIdx.x + step * gridDim.x;
        __syncthreads();
        const int64_t idx = sm.idx;
        if (idx >= a.n) break;
        if (kTrain) {
            // reads are on demand: drop weights this CU cached for earlier samples
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            if (a.claims && tid == 0) atomicAdd(a.claims + idx, 1);
        }
        const int label = a.labels[idx];
        for (int i = tid; i < NX; i += NT) sm.x[i] = a.x[idx * NX + i];
        __syncthreads();

        // ================= forward propagation =================
        // conv1 + pool1: rows m = 4P + w (P < 169), cols o < 20, K = 16
        {
            float bw[4][2];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    int o = 16 * j + lr;
                    bw[s][j] = (o < C1) ? W[OW1 + o * 16 + 4 * s + lg] : 0.0f;
                }
            float b1[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) b1[j] = (16 * j + lr < C1) ? W[OB1 + 16 * j + lr] : 0.0f;
            for (int i = wave; i < 43; i += NW) {
                int m = 16 * i + lr, P = m >> 2;
                bool valid = P < NP1;
                int base = valid ? window_pos(P, m & 3, Q1, IN) : 0;
                f4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    float av = valid ? sm.x[base + s * IN + lg] : 0.0f;
                    acc0 = mfma(av, bw[s][0], acc0);
                    acc1 = mfma(av, bw[s][1], acc1);
                }
                int Pe = 4 * i + lg;
                if (Pe < NP1) {
                    float ym;
                    int ag;
                    pool4(acc0, b1[0], ym, ag);
                    sm.p1[lr * NP1 + Pe] = ym;
                    sm.am1[lr * NP1 + Pe] = (unsigned char)ag;
                    if (16 + lr < C1) {
                        pool4(acc1, b1[1], ym, ag);
                        sm.p1[(16 + lr) * NP1 + Pe] = ym;
                        sm.am1[(16 + lr) * NP1 + Pe] = (unsigned char)ag;
                    }
                }
            }
        }
        __syncthreads();

        // conv2: rows p < 121 (8 tiles), cols o < 60 (4 tiles), K = 180
        {
            f4 acc[2][4];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[t][j] = f4{0.f, 0.f, 0.f, 0.f};
            int base[2];
            bool valid[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                int p = 16 * (2 * wave + t) + lr;
                valid[t] = p < NY2;
                int py = p / H2, px = p - py * H2;
                base[t] = valid[t] ? py * Q1 + px : 0;
            }
            for (int ks = 0; ks < KC2 / 4; ++ks) {
                int k = 4 * ks + lg;
                int c = k / 9, uv = k - 9 * c, u = uv / 3, v = uv - 3 * u;
                int off = c * NP1 + u * Q1 + v;
                float av[2], bv[4];
#pragma unroll
                for (int t = 0; t < 2; ++t) av[t] = valid[t] ? sm.p1[base[t] + off] : 0.0f;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    int o = 16 * j + lr;
                    bv[j] = (o < C2) ? W[OW2 + o * KC2 + k] : 0.0f;
                }
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[t][j] = mfma(av[t], bv[j], acc[t][j]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int o = 16 * j + lr;
                if (o >= C2) continue;
                float bias = W[OB2 + o];
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int p = 16 * (2 * wave + t) + 4 * lg + r;
                        if (p < NY2) sm.y2[o * NY2 + p] = act_y(acc[t][j][r] + bias);
                    }
            }
        }
        __syncthreads();

        // conv3 + pool2: rows m = 4P + w (36 -> 3 tiles), cols o < 100 (7 tiles),
        // K = 2160 split across the 4 wavefronts (15 input maps each)
        {
            f4 acc[3][7];
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int j = 0; j < 7; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            int base[3];
            bool valid[3];
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                int m = 16 * i + lr;
                valid[i] = m < M3;
                base[i] = valid[i] ? window_pos(m >> 2, m & 3, 3, H2) : 0;
            }
            const int ks0 = wave * (KC3 / 4 / NW), ks1 = ks0 + KC3 / 4 / NW;
            for (int ks = ks0; ks < ks1; ++ks) {
                int k = 4 * ks + lg;
                int c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
                int off = c * NY2 + u * H2 + v;
                float av[3], bv[7];
#pragma unroll
                for (int i = 0; i < 3; ++i) av[i] = valid[i] ? sm.y2[base[i] + off] : 0.0f;
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    int o = 16 * j + lr;
                    bv[j] = (o < C3) ? W[OW3 + o * KC3 + k] : 0.0f;
                }
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 7; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            }
            // fixed-order reduction of the four partial sums through LDS:
            // (w0 + w2) + (w1 + w3)
            float *buf = sm.red3;  // 2 x 21 tiles x 64 lanes x 4 floats
            if (wave >= 2) {
                float *dst = buf + (wave - 2) * (21 * 256);
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 7; ++j)
                        *(f4 *)(dst + ((i * 7 + j) * 64 + lane) * 4) = acc[i][j];
            }
            __syncthreads();
            if (wave < 2) {
                const float *src = buf + wave * (21 * 256);
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 7; ++j)
                        acc[i][j] += *(const f4 *)(src + ((i * 7 + j) * 64 + lane) * 4);
            }
            __syncthreads();
            if (wave == 1) {
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 7; ++j)
                        *(f4 *)(buf + ((i * 7 + j) * 64 + lane) * 4) = acc[i][j];
            }
            __syncthreads();
            if (wave == 0) {
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    int o = 16 * j + lr;
                    if (o >= C3) continue;
                    float bias = W[OB3 + o];
#pragma unroll
                    for (int i = 0; i < 3; ++i) {
                        f4 t = acc[i][j] + *(const f4 *)(buf + ((i * 7 + j) * 64 + lane) * 4);
                        int P = 4 * i + lg;
                        if (P < NP3) {
                            float ym;
                            int ag;
                            pool4(t, bias, ym, ag);
                            sm.p3[o * NP3 + P] = ym;
                            sm.am3[o * NP3 + P] = (unsigned char)ag;
                        }
                    }
                }
            }
        }
        __syncthreads();

        // FC1: one wavefront per neuron, lanes across the 900 inputs
        for (int j = wave; j < F1; j += NW) {
            const float *wj = W + OF1 + j * NF1;
            float s = 0.0f;
            for (int i = lane; i < NF1; i += 64) s = fmaf(wj[i], sm.p3[i], s);
            s = wave_sum(s);
            if (lane == 0) sm.h[j] = act_y(s + W[OBF1 + j]);
        }
        __syncthreads();
        // FC2 (output layer)
        for (int j = wave; j < F2; j += NW) {
            const float *wj = W + OF2 + j * F1;
            float s = 0.0f;
            for (int i = lane; i < F1; i += 64) s = fmaf(wj[i], sm.h[i], s);
            s = wave_sum(s);
            if (lane == 0) sm.o[j] = act_y(s + W[OBF2 + j]);
        }
        __syncthreads();
        if (a.out && tid < F2) a.out[idx * F2 + tid] = sm.o[tid];

        if (MODE == kEvaluate) {
            if (tid == 0) {
                int best = 0;
                for (int k = 1; k < F2; ++k)
                    if (sm.o[k] > sm.o[best]) best = k;
                if (best != label) atomicAdd(a.n_wrong, 1);
            }
            __syncthreads();
            continue;
        }

        // ================= back-propagation =================
        Push push;
        push.mode = MODE;
        push.params = a.params;
        push.neg_lr = -a.lr;
        push.each = a.grad_each ? a.grad_each + idx * (int64_t)NPARAM : nullptr;
        push.part = a.grad_part ? a.grad_part + (int64_t)blockIdx.x * NPARAM : nullptr;
        push.first = (step == 0);

        // output layer: E = 1/2 sum (y - t)^2, delta = (y - t) f'(z)
        if (tid < 64) {
            float e = 0.0f;
            if (tid < F2) {
                float y = sm.o[tid];
                float d = y - (tid == label ? 1.0f : 0.0f);
                e = d * d;
                sm.dout[tid] = d * dact_from_y(y);
            }
            e = wave_sum(e);
            if (tid == 0 && a.loss) a.loss[idx] = 0.5f * e;
        }
        __syncthreads();
        // FC2 backward data (pre-update weights)
        for (int i = tid; i < F1; i += NT) {
            float s = 0.0f;
#pragma unroll
            for (int j = 0; j < F2; ++j) s = fmaf(W[OF2 + j * F1 + i], sm.dout[j], s);
            sm.dh[i] = s * dact_from_y(sm.h[i]);
        }
        __syncthreads();
        // FC2 push; FC1 backward data
        for (int t = tid; t < F2 * F1; t += NT) {
            int j = t / F1, i = t - j * F1;
            push(OF2 + t, sm.dout[j] * sm.h[i]);
        }
        if (tid < F2) push(OBF2 + tid, sm.dout[tid]);
        for (int i = tid; i < NF1; i += NT) {
            float s = 0.0f;
            for (int j = 0; j < F1; ++j) s = fmaf(W[OF1 + j * NF1 + i], sm.dh[j], s);
            sm.e3[i] = s;
        }
        __syncthreads();
        // FC1 push; pool2 backward -> conv3 output deltas d3[o][4P + w]; clear s2
        for (int t = tid; t < F1 * NF1; t += NT) {
            int j = t / NF1, i = t - j * NF1;
            push(OF1 + t, sm.dh[j] * sm.p3[i]);
        }
        if (tid < F1) push(OBF1 + tid, sm.dh[tid]);
        for (int t = tid; t < C3 * M3P; t += NT) {
            int o = t / M3P, m = t - o * M3P;
            float d = 0.0f;
            if (m < M3) {
                int P = m >> 2, w = m & 3, q = o * NP3 + P;
                if (sm.am3[q] == w) d = sm.e3[q] * dact_from_y(sm.p3[q]);
            }
            sm.d3[t] = d;
        }
        for (int t = tid; t < C2 * NY2; t += NT) sm.s2[t] = 0.0f;
        __syncthreads();

        // conv3 backward data: C[k][m] = sum_o W3[o][k] d3[o][m], k = (c,u,v);
        // col2im into s2[c][pos(m) + (u,v)].  Wavefront w owns input maps
        // c in blocks of 4 (144 rows = 9 tiles), so no two wavefronts touch
        // the same s2 entries.
        for (int blk = wave; blk < C2 / 4; blk += NW) {
            f4 acc[9][3];
#pragma unroll
            for (int i = 0; i < 9; ++i)
#pragma unroll
                for (int j = 0; j < 3; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            const int k0 = blk * 144;
            for (int ks = 0; ks < C3 / 4; ++ks) {
                int o = 4 * ks + lg;
                float av[9], bv[3];
#pragma unroll
                for (int i = 0; i < 9; ++i) av[i] = W[OW3 + o * KC3 + k0 + 16 * i + lr];
#pragma unroll
                for (int j = 0; j < 3; ++j) bv[j] = sm.d3[o * M3P + 16 * j + lr];
#pragma unroll
                for (int i = 0; i < 9; ++i)
#pragma unroll
                    for (int j = 0; j < 3; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            }
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                int m = 16 * j + lr;
                if (m >= M3) continue;
                int pos = window_pos(m >> 2, m & 3, 3, H2);
#pragma unroll
                for (int i = 0; i < 9; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int k = k0 + 16 * i + 4 * lg + r;
                        int c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
                        __hip_atomic_fetch_add(&sm.s2[c * NY2 + pos + u * H2 + v], acc[i][j][r],
                                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                    }
            }
        }
        __syncthreads();

        // conv3 weight gradient: G[o][k] = sum_m d3[o][m] y2col[m][k], pushed
        {
            float ad[7][9];
#pragma unroll
            for (int i = 0; i < 7; ++i)
#pragma unroll
                for (int s = 0; s < 9; ++s) {
                    int o = 16 * i + lr;
                    ad[i][s] = (o < C3) ? sm.d3[o * M3P + 4 * s + lg] : 0.0f;
                }
            int pos[9];
#pragma unroll
            for (int s = 0; s < 9; ++s) {
                int m = 4 * s + lg;
                pos[s] = window_pos(m >> 2, m & 3, 3, H2);
            }
            for (int jt = wave; jt < KC3 / 16; jt += NW) {
                int k = 16 * jt + lr;
                int c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
                const float *ycol = sm.y2 + c * NY2 + u * H2 + v;
                f4 acc[7];
#pragma unroll
                for (int i = 0; i < 7; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int s = 0; s < 9; ++s) {
                    float bv = ycol[pos[s]];
#pragma unroll
                    for (int i = 0; i < 7; ++i) acc[i] = mfma(ad[i][s], bv, acc[i]);
                }
#pragma unroll
                for (int i = 0; i < 7; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int o = 16 * i + 4 * lg + r;
                        if (o < C3) push(OW3 + o * KC3 + k, acc[i][r]);
                    }
            }
            if (tid < C3) {
                float g = 0.0f;
                for (int m = 0; m < M3; ++m) g += sm.d3[tid * M3P + m];
                push(OB3 + tid, g);
            }
        }
        __syncthreads();

        // conv2 deltas (in place of y2) and clear the pool1 error buffer
        for (int t = tid; t < C2 * NY2; t += NT) {
            sm.y2[t] = sm.s2[t] * dact_from_y(sm.y2[t]);
            sm.s2[t] = 0.0f;
        }
        __syncthreads();

        // conv2 backward data: C[k][p] = sum_o W2[o][k] d2[o][p], k = (c,u,v) < 180;
        // col2im into e1[c][p + (u,v)] (13x13 maps), wavefront by wavefront
        {
            f4 acc[3][8];
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            for (int ks = 0; ks < C2 / 4; ++ks) {
                int o = 4 * ks + lg;
                float av[3], bv[8];
#pragma unroll
                for (int i = 0; i < 3; ++i) {
                    int k = 16 * (3 * wave + i) + lr;
                    av[i] = (k < KC2) ? W[OW2 + o * KC2 + k] : 0.0f;
                }
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    int p = 16 * j + lr;
                    bv[j] = (p < NY2) ? sm.y2[o * NY2 + p] : 0.0f;
                }
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            }
            float *e1 = sm.s2;
            for (int turn = 0; turn < NW; ++turn) {
                if (wave == turn) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        int p = 16 * j + lr;
                        if (p >= NY2) continue;
                        int py = p / H2, px = p - py * H2;
#pragma unroll
                        for (int i = 0; i < 3; ++i)
#pragma unroll
                            for (int r = 0; r < 4; ++r) {
                                int k = 16 * (3 * wave + i) + 4 * lg + r;
                                if (k >= KC2) continue;
                                int c = k / 9, uv = k - 9 * c, u = uv / 3, v = uv - 3 * u;
                                __hip_atomic_fetch_add(&e1[c * NP1 + (py + u) * Q1 + px + v],
                                                       acc[i][j][r], __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_WORKGROUP);
                            }
                    }
                }
                __syncthreads();
            }
        }

        // conv2 weight gradient: G[o][k] = sum_p d2[o][p] p1col[p][k], pushed;
        // pool1 backward: e1 <- e1 * f'(pool1 value) (delta at each window's max)
        {
            f4 acc[4][3];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 3; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            int boff[3];
            bool kval[3];
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                int k = 16 * (3 * wave + j) + lr;
                kval[j] = k < KC2;
                int c = k / 9, uv = k - 9 * c, u = uv / 3, v = uv - 3 * u;
                boff[j] = kval[j] ? c * NP1 + u * Q1 + v : 0;
            }
            for (int ks = 0; ks < 31; ++ks) {
                int p = 4 * ks + lg;
                bool pv = p < NY2;
                int py = p / H2, px = p - py * H2;
                int pb = pv ? py * Q1 + px : 0;
                float av[4], bv[3];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    int o = 16 * i + lr;
                    av[i] = (pv && o < C2) ? sm.y2[o * NY2 + p] : 0.0f;
                }
#pragma unroll
                for (int j = 0; j < 3; ++j) bv[j] = (pv && kval[j]) ? sm.p1[boff[j] + pb] : 0.0f;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 3; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            }
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                int k = 16 * (3 * wave + j) + lr;
                if (k >= KC2) continue;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int o = 16 * i + 4 * lg + r;
                        if (o < C2) push(OW2 + o * KC2 + k, acc[i][j][r]);
                    }
            }
            if (tid < C2) {
                float g = 0.0f;
                for (int p = 0; p < NY2; ++p) g += sm.y2[tid * NY2 + p];
                push(OB2 + tid, g);
            }
            for (int t = tid; t < C1 * NP1; t += NT) sm.s2[t] *= dact_from_y(sm.p1[t]);
        }
        __syncthreads();

        // conv1 weight gradient from the pool1 deltas at each window's maximum
        for (int t = tid; t < C1 * 16 + C1; t += NT) {
            float g = 0.0f;
            if (t < C1 * 16) {
                int o = t >> 4, u = (t >> 2) & 3, v = t & 3;
                const float *d1 = sm.s2 + o * NP1;
                const unsigned char *am = sm.am1 + o * NP1;
                for (int P = 0; P < NP1; ++P)
                    g = fmaf(d1[P], sm.x[window_pos(P, am[P], Q1, IN) + u * IN + v], g);
                push(OW1 + t, g);
            } else {
                int o = t - C1 * 16;
                for (int P = 0; P < NP1; ++P) g += sm.s2[o * NP1 + P];
                push(OB1 + o, g);
            }
        }
        __syncthreads();
    }
}

} // namespace

bool fused_large_matches(const Net &net) {
    static const int spec[][3] = {{kConv, 20, 4}, {kPool, 0, 2}, {kConv, 60, 3}, {kConv, 100, 6},
                                  {kPool, 0, 2},  {kFc, 150, 0}, {kFc, 10, 0}};
    if (net.n_layers != 7 || net.in_size != NX || net.n_params != NPARAM) return false;
    for (int l = 0; l < 7; ++l) {
        const Layer &ly = net.L[l];
        if (ly.kind != spec[l][0] || ly.k != (spec[l][0] == kFc ? ly.k : spec[l][2])) return false;
        if (ly.kind != kPool && ly.cout != spec[l][1]) return false;
    }
    return net.L[0].hin == IN && net.L[0].win == IN;
}

hipError_t launch_fused_large(int mode, const WorkArgs &a, int grid, hipStream_t s) {
    switch (mode) {
    case kTrainAtomic: fused_large_kernel<kTrainAtomic><<<grid, NT, 0, s>>>(a); break;
    case kTrainRacy: fused_large_kernel<kTrainRacy><<<grid, NT, 0, s>>>(a); break;
    case kForwardBackward: fused_large_kernel<kForwardBackward><<<grid, NT, 0, s>>>(a); break;
    case kEvaluate: fused_large_kernel<kEvaluate><<<grid, NT, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int fused_large_blocks_per_cu() {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fused_large_kernel<kTrainAtomic>, NT, 0) !=
        hipSuccess)
        return 0;
    return nb;
}

} // namespace chaos
