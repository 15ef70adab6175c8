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

// Device layout of the shared weights: the canonical blocks in the same
// order, each starting on a 64-byte boundary, and the rows of conv2, FC1 and
// FC2 padded to whole 64-byte segments (the conv1 and conv3 rows already
// are).  The pushes are fp32 atomic adds performed at the memory side in
// 64-byte requests; a row that starts mid-segment costs one request more per
// 64 consecutive weights, which for the canonical FC1 and conv2 rows is 10 %
// of the update stream.  Padding is never read or written.  get/set/update
// convert (chaos_api.hip); gradients are produced in the canonical layout.
constexpr int align16(int v) { return (v + 15) / 16 * 16; }
constexpr int KC2S = 192, NF1S = 912, F1S = 160;  // padded row strides (floats)
constexpr int DW1 = 0, DB1 = DW1 + C1 * 16;
constexpr int DW2 = align16(DB1 + C1), DB2 = DW2 + C2 * KC2S;
constexpr int DW3 = align16(DB2 + C2), DB3 = DW3 + C3 * KC3;
constexpr int DF1 = align16(DB3 + C3), DBF1 = DF1 + F1 * NF1S;
constexpr int DF2 = align16(DBF1 + F1), DBF2 = DF2 + F2 * F1S;
constexpr int NDEV = align16(DBF2 + F2);
static_assert(KC2S >= KC2 && NF1S >= NF1 && F1S >= F1 && KC2S % 16 == 0 && NF1S % 16 == 0 &&
                  F1S % 16 == 0 && KC3 % 16 == 0,
              "padded rows are whole 64-byte segments; 16-byte loads stay inside a row");

constexpr int NT = 256;   // threads per worker
constexpr int NW = NT / 64;
constexpr int FC1_ROWS = 4;  // FC1 rows a wavefront pushes per step (returning adds)

// conv3 output rows m = 4 * P + w (P pooled 3x3 position, w window element)
constexpr int M3 = 36, M3P = 48;                // padded to 3 tiles of 16

struct alignas(16) Smem {
    float x[NX + 3];
    float p1[C1 * NP1];                  // pool1 output
    float y2[C2 * NY2];                  // conv2 output, later its delta
    union {
        struct {
            float s2[C2 * NY2];          // conv3 backward-data sums, then pool1 errors
            alignas(16) float d3[C3 * M3P];  // conv3 output deltas, rows (P, w)
        };
        float red3[2 * 21 * 256];        // conv3 split-K partial sums (forward only)
        float w2s[KC2 * 65];             // conv2 weights staged as [k][o] (forward only)
    };
    alignas(16) float p3[NF1];           // pool2 output (FC1 input)
    alignas(16) float e3[NF1];           // dE/d(pool2 output)
    float h[F1 + 10], dh[F1 + 10];
    float o[16], dout[16];
    alignas(16) float pushbuf[NW][16 * 65]; // per-wavefront transpose of a 16 x 64 gradient block
    alignas(16) int koff3[KC3];          // im2col offset into y2 of k = (c,u,v), conv3
    alignas(16) int koff2[KC2 + 4];      // im2col offset into p1 of k = (c,u,v), conv2
    unsigned char am1[C1 * NP1 + 12];    // pool1 argmax (window element 0..3)
    unsigned char am3[NF1 + 4];          // pool2 argmax
    float sink[128];                     // scatter target of padding lanes
    float zero[4];                       // a zero operand for K padding (set once)
    int64_t idx;
};
static_assert(sizeof(Smem) <= 160 * 1024, "LDS budget");
static_assert(NW * 16 * 65 >= NW * NF1, "FC1 partial sums fit in the transpose buffer");

template <int MODE>
__global__ void __launch_bounds__(NT, 1) fused_large_kernel(WorkArgs a) {
    __shared__ Smem sm;
    const float *W = a.params;
    constexpr bool kTrain = (MODE == kTrainAtomic || MODE == kTrainRacy);

    // sample-invariant im2col offset tables
    for (int k = threadIdx.x; k < KC3; k += NT) {
        int c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
        sm.koff3[k] = c * NY2 + u * H2 + v;
    }
    for (int k = threadIdx.x; k < KC2 + 4; k += NT) {
        int c = k / 9, uv = k - 9 * c, u = uv / 3, v = uv - 3 * u;
        sm.koff2[k] = (k < KC2) ? c * NP1 + u * Q1 + v : 0;
    }

    if (threadIdx.x < 4) sm.zero[threadIdx.x] = 0.0f;
    for (int64_t step = 0;; ++step) {
        // The thread index is made opaque to the optimizer at the top of each
        // sample: index arithmetic of every phase then stays inside its phase
        // instead of being hoisted out of this loop and kept live throughout.
        int tid_l = threadIdx.x;
        asm volatile("" : "+v"(tid_l));
        const int tid = tid_l, lane = tid_l & 63, lr = lane & 15, lg = lane >> 4;
        const int wave = __builtin_amdgcn_readfirstlane(tid_l >> 6);
        // ---- claim a sample (Section III-A.1) ----
        if (tid == 0) {
            if (kTrain && step == 0 && blockIdx.x > 0)
                join_after(a.counter, a.n, (int)blockIdx.x / kJoinRamp);
            sm.idx = kTrain ? (int64_t)atomicAdd(a.counter, 1) : (int64_t)blockIdx.x + step * gridDim.x;
        }
        // Reads are on demand.  Every wavefront first waits for its own
        // pushes of the previous sample to complete (the worker sees its own
        // updates: one worker is exact per-sample SGD); then one wavefront
        // drops the weights this CU and its L2 hold from earlier samples (an
        // agent-scope acquire: the caches are shared by the workgroup, and
        // the barrier below orders every wavefront's reads after it).
        wait_vector_memory();
        if (kTrain && wave == 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        __syncthreads();
        const int64_t idx = sm.idx;
        if (idx >= a.n) break;
        if (kTrain) {
            if (a.claims && tid == 0) atomicAdd(a.claims + idx, 1);
        }
        const int label = a.labels[idx];
        for (int i = tid; i < NX; i += NT) sm.x[i] = a.x[idx * NX + i];
        // conv2 weights staged in LDS as [k][o] (o padded to 65 to spread
        // banks): every 16-byte load is issued before the first LDS write
        {
            constexpr int N4 = C2 * KC2 / 4, PER = (N4 + NT - 1) / NT;  // 2700 float4
            f4 wv[PER];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                const int o = (4 * t4) / KC2, k = 4 * t4 - o * KC2;  // KC2 % 4 == 0: one row
                wv[q] = (t4 < N4) ? *(const f4 *)(W + DW2 + o * KC2S + k) : f4{0.f, 0.f, 0.f, 0.f};
            }
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                if (t4 < N4) {
                    const int o = (4 * t4) / KC2, k = 4 * t4 - o * KC2;
#pragma unroll
                    for (int e = 0; e < 4; ++e) sm.w2s[(k + e) * 65 + o] = wv[q][e];
                }
            }
        }
        for (int t = tid; t < KC2 * 5; t += NT) {
            int k = t / 5, o = C2 + (t - 5 * k);
            sm.w2s[k * 65 + o] = 0.0f;
        }
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
                    bw[s][j] = (o < C1) ? W[DW1 + o * 16 + 4 * s + lg] : 0.0f;
                }
            float b1[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) b1[j] = (16 * j + lr < C1) ? W[DB1 + 16 * j + lr] : 0.0f;
            // a wavefront's tiles i = wave + 4q, six at a time (12 independent
            // accumulators keep the matrix core busy)
            for (int i0 = wave; i0 < 43; i0 += 6 * NW) {
                f4 acc[6][2];
                int base[6];
                bool valid[6];
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    int m = 16 * (i0 + 4 * q) + lr, P = m >> 2;
                    valid[q] = P < NP1;
                    base[q] = valid[q] ? window_pos(P, m & 3, Q1, IN) : 0;
                    acc[q][0] = f4{0.f, 0.f, 0.f, 0.f};
                    acc[q][1] = acc[q][0];
                }
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int q = 0; q < 6; ++q) {
                        // (base 0 past the map: a valid input, in an output row never used)
                        const float av = sm.x[base[q] + s * IN + lg];
                        acc[q][0] = mfma(av, bw[s][0], acc[q][0]);
                        acc[q][1] = mfma(av, bw[s][1], acc[q][1]);
                    }
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    int Pe = 4 * (i0 + 4 * q) + lg;
                    if (Pe < NP1) {
                        float ym;
                        int ag;
                        pool4(acc[q][0], b1[0], ym, ag);
                        sm.p1[lr * NP1 + Pe] = ym;
                        sm.am1[lr * NP1 + Pe] = (unsigned char)ag;
                        if (16 + lr < C1) {
                            pool4(acc[q][1], b1[1], ym, ag);
                            sm.p1[(16 + lr) * NP1 + Pe] = ym;
                            sm.am1[(16 + lr) * NP1 + Pe] = (unsigned char)ag;
                        }
                    }
                }
            }
        }
        __syncthreads();

        // conv2: rows p < 121 (8 tiles), cols o < 60 (4 tiles), K = 180; all operands in LDS
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
#pragma unroll 3
            for (int ks = 0; ks < KC2 / 4; ++ks) {
                int k = 4 * ks + lg;
                int off = sm.koff2[k];
                float av[2], bv[4];
#pragma unroll
                for (int t = 0; t < 2; ++t) av[t] = sm.p1[base[t] + off];  // padding rows: unused
#pragma unroll
                for (int j = 0; j < 4; ++j) bv[j] = sm.w2s[k * 65 + 16 * j + lr];
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[t][j] = mfma(av[t], bv[j], acc[t][j]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                int o = 16 * j + lr;
                if (o >= C2) continue;
                float bias = W[DB2 + o];
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
        // K = 2160 in 135 super-steps of 16, split 34/34/34/33 over the wavefronts.
        // Within a super-step lane group g holds k = 16S + 4g + s at sub-step s,
        // so each lane reads its four weights of a super-step with one 16-byte
        // load.
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
            const int S0 = wave * 34, S1 = (S0 + 34 < 135) ? S0 + 34 : 135;
            f4 bA[7], bB[7], bC[7], bD[7];
            auto load_b = [&](f4 (&b)[7], int S) {
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    // padding columns (o >= C3) read the last map: their
                    // accumulators are never used, and no branch splits the loads
                    int o = 16 * j + lr;
                    b[j] = *(const f4 *)(W + DW3 + (o < C3 ? o : C3 - 1) * KC3 + 16 * S + 4 * lg);
                }
            };
            auto compute = [&](const f4 (&b)[7], int S) {
                const int4 ko = *(const int4 *)(sm.koff3 + 16 * S + 4 * lg);
                const int offs[4] = {ko.x, ko.y, ko.z, ko.w};
                // the super-step's twelve activations are read at once: the
                // later sub-steps' arrive while the first one computes
                float av[4][3];
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int i = 0; i < 3; ++i) av[s][i] = sm.y2[base[i] + offs[s]];  // padding rows: unused
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int i = 0; i < 3; ++i)
#pragma unroll
                        for (int j = 0; j < 7; ++j) acc[i][j] = mfma(av[s][i], b[j][s], acc[i][j]);
            };
            // weights three super-steps ahead (a ring of four buffers)
            load_b(bA, S0);
            if (S0 + 1 < S1) load_b(bB, S0 + 1);
            if (S0 + 2 < S1) load_b(bC, S0 + 2);
            for (int S = S0; S < S1; S += 4) {
                if (S + 3 < S1) load_b(bD, S + 3);
                compute(bA, S);
                if (S + 1 < S1) {
                    if (S + 4 < S1) load_b(bA, S + 4);
                    compute(bB, S + 1);
                }
                if (S + 2 < S1) {
                    if (S + 5 < S1) load_b(bB, S + 5);
                    compute(bC, S + 2);
                }
                if (S + 3 < S1) {
                    if (S + 6 < S1) load_b(bC, S + 6);
                    compute(bD, S + 3);
                }
            }
            // fixed-order reduction (w0 + w2) + (w1 + w3) through LDS; the
            // epilogue of col tiles 0..3 runs on wavefront 0, of 4..6 on 1
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
            if (wave < 2) {
                // wavefront 0 hands over tiles 4..6, wavefront 1 tiles 0..3
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < 7; ++j)
                        if ((j >= 4) == (wave == 0))
                            *(f4 *)(buf + ((i * 7 + j) * 64 + lane) * 4) = acc[i][j];
            }
            __syncthreads();
            if (wave < 2) {
#pragma unroll
                for (int j = 0; j < 7; ++j) {
                    if ((j >= 4) != (wave == 1)) continue;
                    int o = 16 * j + lr;
                    if (o >= C3) continue;
                    float bias = W[DB3 + o];
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

        // FC1: wavefront w computes neurons [38w, 38w + 38), eight at a time.
        // Lane l holds inputs 4l + 256c (c < 4) and reads four consecutive
        // weights of a row with one 16-byte load; the next eight rows are
        // requested before the current ones are reduced.  The eight partial
        // sums of a lane are reduced by halving: after exchanges with lanes
        // l^32, l^16 and l^8 each lane keeps one neuron, and l^4, l^2, l^1
        // complete its sum.
        {
            f4 xin[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                int i = 4 * lane + 256 * c;
                xin[c] = (i < NF1) ? *(const f4 *)(sm.p3 + i) : f4{0.f, 0.f, 0.f, 0.f};
            }
            const int jb = 38 * wave, je = (jb + 38 < F1) ? jb + 38 : F1;
            f4 wv[8][4];
            auto load_rows = [&](int j0) {
#pragma unroll
                for (int q = 0; q < 8; ++q)
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        int j = j0 + q, i = 4 * lane + 256 * c;
                        wv[q][c] = (j < je && i < NF1) ? *(const f4 *)(W + DF1 + j * NF1S + i)
                                                       : f4{0.f, 0.f, 0.f, 0.f};
                    }
            };
            const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
            load_rows(jb);
            for (int j0 = jb; j0 < je; j0 += 8) {
                float sq[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float t = 0.0f;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        t = fmaf(wv[q][c].x, xin[c].x, t);
                        t = fmaf(wv[q][c].y, xin[c].y, t);
                        t = fmaf(wv[q][c].z, xin[c].z, t);
                        t = fmaf(wv[q][c].w, xin[c].w, t);
                    }
                    sq[q] = t;
                }
                if (j0 + 8 < je) load_rows(j0 + 8);
                float t4[4], t2[2];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    t4[q] = (b5 ? sq[q + 4] : sq[q]) + __shfl_xor(b5 ? sq[q] : sq[q + 4], 32, 64);
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    t2[q] = (b4 ? t4[q + 2] : t4[q]) + __shfl_xor(b4 ? t4[q] : t4[q + 2], 16, 64);
                float t1 = (b3 ? t2[1] : t2[0]) + __shfl_xor(b3 ? t2[0] : t2[1], 8, 64);
                t1 += __shfl_xor(t1, 4, 64);
                t1 += __shfl_xor(t1, 2, 64);
                t1 += __shfl_xor(t1, 1, 64);
                const int j = j0 + ((lane >> 3) & 7);
                if ((lane & 7) == 0 && j < je) sm.h[j] = act_y(t1 + W[DBF1 + j]);
            }
        }
        __syncthreads();
        // FC2 (output layer)
        for (int j = wave; j < F2; j += NW) {
            const float *wj = W + DF2 + j * F1S;
            float s = 0.0f;
#pragma unroll
            for (int it = 0; it < 3; ++it) {
                int i = lane + 64 * it;
                if (i < F1) s = fmaf(wj[i], sm.h[i], s);
            }
            s = wave_sum(s);
            if (lane == 0) sm.o[j] = act_y(s + W[DBF2 + j]);
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
        if (tid < F1) {
            float wv[F2];
#pragma unroll
            for (int j = 0; j < F2; ++j) wv[j] = W[DF2 + j * F1S + tid];
            float s = 0.0f;
#pragma unroll
            for (int j = 0; j < F2; ++j) s = fmaf(wv[j], sm.dout[j], s);
            sm.dh[tid] = s * dact_from_y(sm.h[tid]);
        }
        __syncthreads();
        // FC2 push.  FC1 push and FC1 backward data in one pass: each push
        // returns the weight it updated, which is this layer's pre-update
        // weight (Section III-A.2), so e3[i] = sum_j W[j][i] dh[j] needs no
        // separate read of the 540 KB of FC1 weights.  Wavefront w pushes
        // rows j = w, w + 4, ... (lane l the inputs l + 64c, a push
        // instruction covers 64 consecutive weights) and keeps a partial sum
        // per input; the four partial sums are added in wavefront order.
        for (int t = tid; t < F2 * F1; t += NT) {
            int j = t / F1, i = t - j * F1;
            push(DF2 + j * F1S + i, OF2 + t, sm.dout[j] * sm.h[i]);
        }
        if (tid < F2) push(DBF2 + tid, OBF2 + tid, sm.dout[tid]);
        if (tid < F1) push(DBF1 + tid, OBF1 + tid, sm.dh[tid]);
        if constexpr (MODE == kForwardBackward) {
            // frozen weights: read them (16-byte loads, ten rows per batch,
            // the next batch requested while this one is summed), then push
            if (tid < NF1 / 4) {
                f4 acc = {0.f, 0.f, 0.f, 0.f};
                f4 wa[10], wb[10];
                auto load = [&](f4 (&w)[10], int j0) {
#pragma unroll
                    for (int jj = 0; jj < 10; ++jj)
                        w[jj] = *(const f4 *)(W + DF1 + (j0 + jj) * NF1S + 4 * tid);
                };
                auto comp = [&](const f4 (&w)[10], int j0) {
#pragma unroll
                    for (int jj = 0; jj < 10; ++jj) {
                        float d = sm.dh[j0 + jj];
                        acc.x = fmaf(w[jj].x, d, acc.x);
                        acc.y = fmaf(w[jj].y, d, acc.y);
                        acc.z = fmaf(w[jj].z, d, acc.z);
                        acc.w = fmaf(w[jj].w, d, acc.w);
                    }
                };
                load(wa, 0);
                for (int j0 = 0; j0 < F1; j0 += 20) {
                    if (j0 + 10 < F1) load(wb, j0 + 10);
                    comp(wa, j0);
                    if (j0 + 10 < F1) {
                        if (j0 + 20 < F1) load(wa, j0 + 20);
                        comp(wb, j0 + 10);
                    }
                }
                *(f4 *)(sm.e3 + 4 * tid) = acc;
            }
            if (a.stash) {
                // batched gradient: this sample's FC1 deltas and inputs go to
                // HBM; the FC1 weight gradient is contracted over the batch
                // afterwards
                float *dhs = a.stash + a.n * (int64_t)(C3 * M3 + C2 * NY2) + idx * F1;
                float *p3s = a.stash + a.n * (int64_t)(C3 * M3 + C2 * NY2 + F1) + idx * NF1;
                if (tid < F1) dhs[tid] = sm.dh[tid];
                for (int i = tid; i < NF1; i += NT) p3s[i] = sm.p3[i];
            } else {
                float xv[15];
#pragma unroll
                for (int c = 0; c < 15; ++c) {
                    int i = lane + 64 * c;
                    xv[c] = (i < NF1) ? sm.p3[i] : 0.0f;
                }
                for (int j = wave; j < F1; j += NW) {
                    const float d = sm.dh[j];
#pragma unroll
                    for (int c = 0; c < 15; ++c) {
                        int i = lane + 64 * c;
                        if (i < NF1) push(DF1 + j * NF1S + i, OF1 + j * NF1 + i, d * xv[c]);
                    }
                }
            }
        } else {
            {
                float xv[15], ep[15];
#pragma unroll
                for (int c = 0; c < 15; ++c) {
                    int i = lane + 64 * c;
                    xv[c] = (i < NF1) ? sm.p3[i] : 0.0f;
                    ep[c] = 0.0f;
                }
                // The wavefront's rows j = wave + NW r (r < 38) in half-steps
                // of FC1_ROWS / 2 rows: the next half-step's pushes are issued
                // before the current one's returns are summed, so about
                // 15 FC1_ROWS pushes stay in flight throughout (a row is summed
                // once all its returns are in, rows in increasing order).
                constexpr int HR = FC1_ROWS / 2, NR = (F1 + NW - 1) / NW;
                static_assert(NR % (2 * HR) == HR, "38 rows: pairs of half-steps and a last half-step");
                float oldA[HR][15], oldB[HR][15];
                auto issue = [&](float (&o)[HR][15], int r0) {
#pragma unroll
                    for (int r = 0; r < HR; ++r) {
                        const int jr = wave + NW * (r0 + r);
                        const float d = (jr < F1) ? sm.dh[jr] : 0.0f;
#pragma unroll
                        for (int c = 0; c < 15; ++c) {
                            const int i = lane + 64 * c;
                            o[r][c] = (jr < F1 && i < NF1) ? push.with_old(DF1 + jr * NF1S + i, OF1 + jr * NF1 + i, d * xv[c])
                                                           : 0.0f;
                        }
                    }
                };
                auto consume = [&](const float (&o)[HR][15], int r0) {
#pragma unroll
                    for (int r = 0; r < HR; ++r) {
                        const int jr = wave + NW * (r0 + r);
                        const float d = (jr < F1) ? sm.dh[jr] : 0.0f;
#pragma unroll
                        for (int c = 0; c < 15; ++c) ep[c] = fmaf(o[r][c], d, ep[c]);
                    }
                };
                // (scheduling barriers keep the half-steps in this order)
                issue(oldA, 0);
#pragma unroll 1
                for (int r0 = 0; r0 + 2 * HR < NR; r0 += 2 * HR) {
                    __builtin_amdgcn_sched_barrier(0);
                    issue(oldB, r0 + HR);
                    __builtin_amdgcn_sched_barrier(0);
                    consume(oldA, r0);
                    __builtin_amdgcn_sched_barrier(0);
                    issue(oldA, r0 + 2 * HR);
                    __builtin_amdgcn_sched_barrier(0);
                    consume(oldB, r0 + HR);
                }
                __builtin_amdgcn_sched_barrier(0);
                consume(oldA, NR - HR);
                float *part = sm.pushbuf[0];  // [wavefront][input]
#pragma unroll
                for (int c = 0; c < 15; ++c) {
                    int i = lane + 64 * c;
                    if (i < NF1) part[wave * NF1 + i] = ep[c];
                }
            }
        }
        __syncthreads();
        // e3 = the partial sums in wavefront order (training); pool2
        // backward -> conv3 output deltas d3[o][4P + w]; clear s2
        if constexpr (MODE != kForwardBackward) {
            const float *part = sm.pushbuf[0];
            for (int q = tid; q < NF1; q += NT)
                sm.e3[q] = ((part[q] + part[NF1 + q]) + part[2 * NF1 + q]) + part[3 * NF1 + q];
            __syncthreads();
        }
        // (a thread per pooled output writes its window's four deltas, rows
        // 4P..4P+3 of its map, as one 16-byte store: the delta at the first
        // maximum, zeros elsewhere; rows M3..M3P-1 of every map are zeroed apart)
#pragma unroll 1
        for (int q = tid; q < NF1; q += NT) {
            const int o = q / NP3, P = q - o * NP3, ag = sm.am3[q];
            const float d = sm.e3[q] * dact_from_y(sm.p3[q]);
            *(f4 *)(sm.d3 + o * M3P + 4 * P) = f4{ag == 0 ? d : 0.0f, ag == 1 ? d : 0.0f, ag == 2 ? d : 0.0f,
                                                  ag == 3 ? d : 0.0f};
        }
        static_assert(M3 % 4 == 0 && M3P % 4 == 0, "16-byte delta rows");
        for (int t = tid; t < C3 * (M3P - M3) / 4; t += NT) {
            const int o = t / ((M3P - M3) / 4), r = t - o * ((M3P - M3) / 4);
            *(f4 *)(sm.d3 + o * M3P + M3 + 4 * r) = f4{0.f, 0.f, 0.f, 0.f};
        }
        for (int t = tid; t < C2 * NY2; t += NT) sm.s2[t] = 0.0f;
        __syncthreads();

        // conv3 backward data: C[k][m] = sum_o W3[o][k] d3[o][m], k = (c,u,v);
        // col2im into s2[c][pos(m) + (u,v)].  Wavefront w owns input maps in
        // blocks of 4 (144 rows = 9 tiles), so no two wavefronts touch the
        // same s2 entries.  Row q of tile i holds input map c0 + q/4 at kernel
        // offset uv = 4i + q%4: in the accumulator the four lane groups then
        // hold four different maps at one (u,v), so no scatter instruction
        // has two lanes on one address.
        for (int blk = wave; blk < C2 / 4; blk += NW) {
            f4 acc[9][3];
#pragma unroll
            for (int i = 0; i < 9; ++i)
#pragma unroll
                for (int j = 0; j < 3; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            const int k0 = blk * 144;
            const int arow = k0 + (lr >> 2) * 36 + (lr & 3);
            float aA[9], aB[9], aC[9], aD[9], bA[3], bB[3], bC[3], bD[3];
            auto load = [&](float (&av)[9], float (&bv)[3], int ks) {
                const float *w3 = W + DW3 + (4 * ks + lg) * KC3 + arow;
#pragma unroll
                for (int i = 0; i < 9; ++i) av[i] = w3[4 * i];
                const float *dd = sm.d3 + (4 * ks + lg) * M3P + lr;
#pragma unroll
                for (int j = 0; j < 3; ++j) bv[j] = dd[16 * j];
            };
            auto compute = [&](const float (&av)[9], const float (&bv)[3]) {
                // keeps the weight reads of the steps ahead issued before
                // these matrix instructions wait for this step's
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < 9; ++i)
#pragma unroll
                    for (int j = 0; j < 3; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            };
            // weights and deltas three output-map steps ahead (a ring of four
            // buffers): under the update stream a weight read waits microseconds
            constexpr int NKS = C3 / 4;
            load(aA, bA, 0);
            load(aB, bB, 1);
            load(aC, bC, 2);
            for (int ks = 0; ks < NKS; ks += 4) {
                if (ks + 3 < NKS) load(aD, bD, ks + 3);
                compute(aA, bA);
                if (ks + 1 < NKS) {
                    if (ks + 4 < NKS) load(aA, bA, ks + 4);
                    compute(aB, bB);
                }
                if (ks + 2 < NKS) {
                    if (ks + 5 < NKS) load(aB, bB, ks + 5);
                    compute(aC, bC);
                }
                if (ks + 3 < NKS) {
                    if (ks + 6 < NKS) load(aC, bC, ks + 6);
                    compute(aD, bD);
                }
            }
            float *dst = sm.s2 + (4 * blk + lg) * NY2;
            float *dm[3];
#pragma unroll
            for (int j = 0; j < 3; ++j) {
                int m = 16 * j + lr;
                dm[j] = (m < M3) ? dst + window_pos(m >> 2, m & 3, 3, H2) : sm.sink;
            }
            // scatter grouped by kernel offset uv: inside a group the 3 x 64
            // lanes write distinct addresses; the groups, whose targets
            // overlap, stay in order
#pragma unroll
            for (int i = 0; i < 9; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int uv = 4 * i + r, u = uv / 6, v = uv - 6 * u;
                    const float c[3] = {acc[i][0][r], acc[i][1][r], acc[i][2][r]};
                    scatter_add<3>(dm, u * H2 + v, c);
                }
        }
        __syncthreads();

        // batched gradient (frozen weights, a.stash): this sample's conv3
        // output deltas and conv3 inputs go to HBM, and the conv3 weight
        // gradient is contracted over the batch afterwards; the bias
        // gradient is pushed as usual
        if (MODE == kForwardBackward && a.stash) {
            float *d3s = a.stash + idx * (C3 * M3);
            float *y2s = a.stash + a.n * (int64_t)(C3 * M3) + idx * (C2 * NY2);
            for (int t = tid; t < C3 * M3; t += NT) {
                const int o = t / M3, m = t - o * M3;
                d3s[t] = sm.d3[o * M3P + m];
            }
            for (int t = tid; t < C2 * NY2; t += NT) y2s[t] = sm.y2[t];
            if (tid < C3) {
                float g4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int m = 0; m < M3; ++m) g4[m & 3] += sm.d3[tid * M3P + m];
                push(DB3 + tid, OB3 + tid, (g4[0] + g4[1]) + (g4[2] + g4[3]));
            }
        } else
        // conv3 weight gradient G[o][k] = sum_m d3[o][m] y2col[m][k], pushed.
        // Maps 0..95 on 32x32x2 tiles: element r of a tile holds maps
        // 8(r/4) + r%4 and that + 4 at 32 consecutive k, so a push
        // instruction writes two 128-byte runs of weights.  Maps 96..99 on
        // the 16-block 4x4x1 instruction with block b, column c at
        // k = 4b + c: element r holds map 96 + r at 64 consecutive k.
        // Wavefront w takes the 64-column groups w, w + 4, ... (a column
        // beyond KC3 computes values never pushed).
        {
            float a32[3][18];  // A[o = 32i + l%32][m = 2ms + l/32]
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int ms = 0; ms < 18; ++ms)
                    a32[i][ms] = sm.d3[(32 * i + (lane & 31)) * M3P + 2 * ms + (lane >> 5)];
            const float *a4 = sm.d3 + (96 + (lane & 3)) * M3P;  // A[block][l%4][m]: map 96 + l%4
            for (int grp = wave; grp < (KC3 / 16 + 3) / 4; grp += NW) {
                f16 c32[3][2];
                f4 c4[2];
                const float *y32[2];
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const int k = 64 * grp + 32 * kt + (lane & 31);
                    y32[kt] = sm.y2 + (k < KC3 ? sm.koff3[k] : 0);
                }
                const int k4 = 64 * grp + lane;
                const float *y4 = sm.y2 + (k4 < KC3 ? sm.koff3[k4] : 0);
                // the group's 36 activations are read at once: later steps'
                // arrive while the first ones compute
                float bv[18][2];
#pragma unroll
                for (int ms = 0; ms < 18; ++ms) {
                    const int m = 2 * ms + (lane >> 5), wp = window_pos(m >> 2, m & 3, 3, H2);
#pragma unroll
                    for (int kt = 0; kt < 2; ++kt) bv[ms][kt] = y32[kt][wp];
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int ms = 0; ms < 18; ++ms)
#pragma unroll
                    for (int i = 0; i < 3; ++i)
#pragma unroll
                        for (int kt = 0; kt < 2; ++kt)
                            c32[i][kt] = mfma32(a32[i][ms], bv[ms][kt], ms == 0 ? f16{} : c32[i][kt]);
                // two partial sums (even and odd m) keep the chain short
#pragma unroll
                for (int m = 0; m < M3; ++m) {
                    const float bv = y4[window_pos(m >> 2, m & 3, 3, H2)];
                    c4[m & 1] = mfma4(a4[m], bv, m < 2 ? f4{} : c4[m & 1]);
                }
#pragma unroll
                for (int kt = 0; kt < 2; ++kt) {
                    const int k = 64 * grp + 32 * kt + (lane & 31);
                    if (k < KC3) {
#pragma unroll
                        for (int i = 0; i < 3; ++i)
#pragma unroll
                            for (int r = 0; r < 16; ++r) {
                                const int o = 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                                push(DW3 + o * KC3 + k, OW3 + o * KC3 + k, c32[i][kt][r]);
                            }
                    }
                }
                if (k4 < KC3) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) push(DW3 + (96 + r) * KC3 + k4, OW3 + (96 + r) * KC3 + k4, c4[0][r] + c4[1][r]);
                }
            }
            if (tid < C3) {
                // four partial sums over the window elements, then combined
                float g4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int m = 0; m < M3; ++m) g4[m & 3] += sm.d3[tid * M3P + m];
                push(DB3 + tid, OB3 + tid, (g4[0] + g4[1]) + (g4[2] + g4[3]));
            }
        }
        __syncthreads();

        // conv2 deltas (in place of y2) and clear the pool1 error buffer
        // (four elements per thread and round: their reads are issued together)
        static_assert(C2 * NY2 % 4 == 0, "whole rounds of four");
        for (int t0 = tid; t0 < C2 * NY2 / 4; t0 += NT) {
            float e[4], y[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                e[q] = sm.s2[t0 + q * (C2 * NY2 / 4)];
                y[q] = sm.y2[t0 + q * (C2 * NY2 / 4)];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                sm.y2[t0 + q * (C2 * NY2 / 4)] = e[q] * dact_from_y(y[q]);
                sm.s2[t0 + q * (C2 * NY2 / 4)] = 0.0f;
            }
        }
        __syncthreads();

        // conv2 backward data: C[k][p] = sum_o W2[o][k] d2[o][p], k = (c,u,v);
        // col2im into e1[c][p + (u,v)] (13x13 maps).  Wavefront w owns input
        // maps 5w..5w+4, so col2im needs no ordering between wavefronts.
        // Tiles 0..2 hold maps 5w + q/4 at uv = 4i + q%4 (no two lanes of one
        // scatter instruction on one address, as for conv3); tile 3 holds map
        // 5w + 4 at uv = q and is scattered one lane group at a time.
        {
            f4 acc[4][8];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            const int c0 = 5 * wave;
            // row of this lane in each tile: k index (or -1 when padding)
            int krow[4];
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                int uv = 4 * i + (lr & 3);
                krow[i] = (uv < 9) ? (c0 + (lr >> 2)) * 9 + uv : -1;
            }
            krow[3] = (lr < 9) ? (c0 + 4) * 9 + lr : -1;
            float aA[4], aB[4];
            auto load_a = [&](float (&av)[4], int ks) {
                const float *w2 = W + DW2 + (4 * ks + lg) * KC2S;
#pragma unroll
                for (int i = 0; i < 4; ++i) av[i] = (krow[i] >= 0) ? w2[krow[i]] : 0.0f;
            };
            auto compute = [&](const float (&av)[4], int ks) {
                const float *dd = sm.y2 + (4 * ks + lg) * NY2;
                float bv[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    int p = 16 * j + lr;
                    bv[j] = (p < NY2) ? dd[p] : 0.0f;
                }
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 8; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            };
            load_a(aA, 0);
            for (int ks = 0; ks < C2 / 4; ks += 2) {
                if (ks + 1 < C2 / 4) load_a(aB, ks + 1);
                compute(aA, ks);
                if (ks + 1 < C2 / 4) {
                    if (ks + 2 < C2 / 4) load_a(aA, ks + 2);
                    compute(aB, ks + 1);
                }
            }
            // tiles 0..2: scatter grouped by kernel offset uv (distinct
            // addresses inside a group, groups kept in order); tile 3 (one
            // map, lanes at different uv may meet): one lane group per step
            float *e1 = sm.s2;
            float *dp[8], *dq[8];  // this lane's column in map c0 + lg and in map c0 + 4
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                int p = 16 * j + lr;
                int py = p / H2, px = p - py * H2;
                dp[j] = (p < NY2) ? e1 + (c0 + lg) * NP1 + py * Q1 + px : sm.sink;
                dq[j] = (p < NY2) ? e1 + (c0 + 4) * NP1 + py * Q1 + px : sm.sink;
            }
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int uv = 4 * i + r, u = uv / 3, v = uv - 3 * u;
                    if (uv >= 9) continue;
                    float c[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) c[j] = acc[i][j][r];
                    scatter_add<8>(dp, u * Q1 + v, c);
                }
            // tile 3: the four lane groups hold four (u,v) of the same map, so
            // each scatter step serves one lane group
#pragma unroll
            for (int g = 0; g < 3; ++g)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int uv = 4 * g + r, u = uv / 3, v = uv - 3 * u;
                    if (uv >= 9) continue;
                    if (lg == g) {
                        float c[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) c[j] = acc[3][j][r];
                        scatter_add<8>(dq, u * Q1 + v, c);
                    } else {
                        wave_lds_order();
                    }
                }
        }
        __syncthreads();

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
                boff[j] = kval[j] ? sm.koff2[k] : 0;
            }
            // operands: LDS reads from clamped addresses, the next step's
            // reads while this step's matrix instructions run.  Nothing is
            // zeroed between the matrix instructions: rows past C2 and columns
            // past KC2 only feed outputs never pushed, and a k-step position
            // past the 121 outputs (K padding) reads its deltas from a zero.
            auto load = [&](float (&av)[4], float (&bv)[3], int ks) {
                const int p = 4 * ks + lg, pc = p < NY2 ? p : 0;
                const int py = pc / H2, px = pc - py * H2, pb = py * Q1 + px;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int o = 16 * i + lr;
                    const float *src = (p < NY2) ? sm.y2 + (o < C2 ? o : 0) * NY2 + p : sm.zero;
                    av[i] = *src;
                }
#pragma unroll
                for (int j = 0; j < 3; ++j) bv[j] = sm.p1[boff[j] + pb];  // boff 0 when invalid
            };
            auto step = [&](const float (&av)[4], const float (&bv)[3], int) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 3; ++j) acc[i][j] = mfma(av[i], bv[j], acc[i][j]);
            };
            float aA[4], bA[3], aB[4], bB[3];
            load(aA, bA, 0);
            for (int ks = 0; ks < 31; ks += 2) {
                if (ks + 1 < 31) load(aB, bB, ks + 1);
                step(aA, bA, ks);
                if (ks + 1 < 31) {
                    if (ks + 2 < 31) load(aA, bA, ks + 2);
                    step(aB, bB, ks + 1);
                }
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
                        if (o < C2) push(DW2 + o * KC2S + k, OW2 + o * KC2 + k, acc[i][j][r]);
                    }
            }
            if (tid < C2) {
                float g4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
                for (int p = 0; p < NY2; ++p) g4[p & 3] += sm.y2[tid * NY2 + p];
                push(DB2 + tid, OB2 + tid, (g4[0] + g4[1]) + (g4[2] + g4[3]));
            }
            static_assert(C1 * NP1 % 4 == 0, "whole rounds of four");
            for (int t0 = tid; t0 < C1 * NP1 / 4; t0 += NT) {
                float e[4], y[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    e[q] = sm.s2[t0 + q * (C1 * NP1 / 4)];
                    y[q] = sm.p1[t0 + q * (C1 * NP1 / 4)];
                }
#pragma unroll
                for (int q = 0; q < 4; ++q) sm.s2[t0 + q * (C1 * NP1 / 4)] = e[q] * dact_from_y(y[q]);
            }
        }
        __syncthreads();

        // conv1 weight gradient G[o][uv] = sum over the 26x26 conv1 outputs
        // of the delta (nonzero only at each pooling window's maximum) times
        // the input under the kernel, as a GEMM on the matrix cores: rows o
        // (2 tiles), cols uv = 4u + v, K = 4P + w with the pooled positions
        // P split over the wavefronts; the four partial tiles are summed in
        // wavefront order.
        {
            f4 acc[2][2];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int t = 0; t < 2; ++t) acc[h][t] = f4{0.f, 0.f, 0.f, 0.f};
            const int oa = lr, ob = (16 + lr < C1) ? 16 + lr : 0;
            const bool vb = 16 + lr < C1;
            const int xo = ((lg >> 1) + (lr >> 2)) * IN + (lg & 1) + (lr & 3);
            // operands of four positions (P0 + NW u) read at once, then their
            // selects and matrix instructions; the bias gradients are summed
            // from the same operands (per lane over its positions, then over
            // the lane groups and, after the barrier, the wavefronts in order)
            float bsum[2] = {0.0f, 0.0f};
            for (int P0 = wave; P0 < NP1; P0 += 4 * NW) {
                float bx[4], v0[4], v1[4];
                int m0[4], m1[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int P = (P0 + NW * u < NP1) ? P0 + NW * u : NP1 - 1;
                    const int py = P / Q1, px = P - py * Q1;
                    bx[u] = sm.x[2 * py * IN + 2 * px + xo];
                    // both reads unconditional (ob is 0 when the map is past C1)
                    m0[u] = sm.am1[oa * NP1 + P];
                    m1[u] = sm.am1[ob * NP1 + P];
                    v0[u] = sm.s2[oa * NP1 + P];
                    v1[u] = sm.s2[ob * NP1 + P];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (P0 + NW * u < NP1) {
                        const float a0 = (m0[u] == lg) ? v0[u] : 0.0f;
                        const float a1 = (vb && m1[u] == lg) ? v1[u] : 0.0f;
                        acc[u & 1][0] = mfma(a0, bx[u], acc[u & 1][0]);
                        acc[u & 1][1] = mfma(a1, bx[u], acc[u & 1][1]);
                        bsum[0] += a0;
                        bsum[1] += a1;
                    }
                }
            }
            float *red = sm.pushbuf[0];  // [wavefront][tile][lane][4], then [wavefront][32] bias sums
            float *redb = red + NW * 2 * 256;
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                *(f4 *)(red + ((wave * 2 + t) * 64 + lane) * 4) = acc[0][t] + acc[1][t];
                const float b1 = bsum[t] + __shfl_xor(bsum[t], 16, 64);
                const float b2 = b1 + __shfl_xor(b1, 32, 64);
                if (lg == 0) redb[wave * 32 + 16 * t + lr] = b2;
            }
            static_assert(NW * (2 * 256 + 32) <= NW * 16 * 65, "conv1 partial tiles and bias sums fit the push buffer");
            __syncthreads();
            for (int t = tid; t < C1 * 16 + C1; t += NT) {
                if (t < C1 * 16) {
                    const int o = t >> 4, uv = t & 15, tile = o >> 4, row = o & 15;
                    const int e = ((row >> 2) * 16 + uv) * 4 + (row & 3);
                    float g = red[(0 * 2 + tile) * 256 + e];
#pragma unroll
                    for (int w = 1; w < NW; ++w) g += red[(w * 2 + tile) * 256 + e];
                    push(DW1 + t, OW1 + t, g);
                } else {
                    const int o = t - C1 * 16;
                    float g = redb[o];
#pragma unroll
                    for (int w = 1; w < NW; ++w) g += redb[w * 32 + o];
                    push(DB1 + o, OB1 + o, g);
                }
            }
        }
        if (kTrain && tid == 0) atomicAdd(a.counter + 1, 1);  // samples completed
        __syncthreads();
    }
}

} // namespace

void fused_large_layout(ParamLayout &L) {
    static const ParamSegment seg[] = {
        {OW1, DW1, 1, C1 * 16, C1 * 16}, {OB1, DB1, 1, C1, C1},   {OW2, DW2, C2, KC2, KC2S},
        {OB2, DB2, 1, C2, C2},           {OW3, DW3, 1, C3 * KC3, C3 * KC3},
        {OB3, DB3, 1, C3, C3},           {OF1, DF1, F1, NF1, NF1S}, {OBF1, DBF1, 1, F1, F1},
        {OF2, DF2, F2, F1, F1S},         {OBF2, DBF2, 1, F2, F2}};
    constexpr int n = sizeof(seg) / sizeof(seg[0]);
    static_assert(n <= kMaxSegments, "segment table size");
    L.n_seg = n;
    L.n_dev = NDEV;
    for (int s = 0; s < n; ++s) L.seg[s] = seg[s];
}

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
