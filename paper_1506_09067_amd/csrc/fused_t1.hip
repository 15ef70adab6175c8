// Fused per-sample CHAOS worker for the large net of Table I:
//   1x29x29 -> conv 20@4x4 -> (max 1x1: the identity) -> conv 60@5x5
//           -> max 2 -> conv 100@6x6 -> max 2 -> FC 150 -> FC 10,
// activation 1.7159 tanh(2z/3) on every conv/FC.
//
// Organised like the kernel of the smaller large net (fused_large.hip): one
// workgroup of 4 wavefronts per worker, persistent, every per-sample value in
// LDS, the convolutions as implicit GEMMs on the fp32 matrix cores.  From
// conv3 on the two nets are the same, and so is that part of this kernel.
// What differs is the front: conv1 is not pooled (26x26 maps), conv2 works on
// them with 5x5 kernels (22x22 outputs, 64 % of the MACs) and is pooled 2x2
// in its epilogue.  LDS is reused across phases: region A holds the conv1
// output in the forward pass, then the conv3 split-K partials, the conv3
// backward buffers, the conv1 output again (recomputed for the conv2 weight
// gradient and f'), and last the conv1 partial gradient tiles;
// region B holds the pool2/FC1 values, then the conv1 output errors.
#include <type_traits>

#include "chaos_internal.h"
#include "device_common.h"

namespace chaos {
namespace {

// ---- shapes of the Table I large net ----------------------------------------
constexpr int IN = 29, NX = IN * IN;            // input 1x29x29
constexpr int C1 = 20, H1 = 26, NA1 = H1 * H1;  // conv1 20@26x26 (K = 16)
constexpr int C2 = 60, K2 = 5, H2F = 22;        // conv2 60@22x22 on 20@26x26
constexpr int KC2 = C1 * K2 * K2;               // 500
constexpr int KC2P = 512;                       // K padded to whole 16-k super-steps
constexpr int Q2 = 11, NY2 = Q2 * Q2;           // pool 2 -> 60@11x11 (conv3 input)
constexpr int M2 = 4 * NY2, M2T = 31;           // conv2 outputs in (pooled position, window
                                                // element) order: 484 rows, 31 tiles
constexpr int H2 = Q2;                          // width of the conv3 input maps
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
static_assert(NPARAM == 383160, "Table I large net weight count");

// device layout of the shared weights: every segment starts on a 64-byte
// boundary and the conv2, FC1 and FC2 rows are padded to multiples of 16
// floats, so a wavefront's push of 64 consecutive weights of a row touches
// four 64-byte segments, not five (the padding stays zero)
constexpr int align16(int v) { return (v + 15) / 16 * 16; }
constexpr int KC2S = align16(KC2), NF1S = align16(NF1), F1S = align16(F1);  // 512, 912, 160
constexpr int DW1 = 0, DB1 = DW1 + C1 * 16;
constexpr int DW2 = align16(DB1 + C1), DB2 = DW2 + C2 * KC2S;
constexpr int DW3 = align16(DB2 + C2), DB3 = DW3 + C3 * KC3;
constexpr int DF1 = align16(DB3 + C3), DBF1 = DF1 + F1 * NF1S;
constexpr int DF2 = align16(DBF1 + F1), DBF2 = DF2 + F2 * F1S;
constexpr int NDEV = align16(DBF2 + F2);
static_assert(KC2S == KC2P && KC3 % 16 == 0, "16-byte weight loads stay inside one row");

constexpr int NT = 256;   // threads per worker
constexpr int NW = NT / 64;
constexpr int FC1_ROWS = 4;  // FC1 rows a wavefront pushes per step (returning adds)
// conv2 weight-gradient column tiles of wavefront 0 (which also takes the
// fifth backward-data block) and of wavefronts 1 and 2 (wavefront 3 takes the
// rest of the 32)
constexpr int kT1W0 = 2, kT1W = 10;
// pooled positions whose operands the weight gradient reads at once (121 =
// 11 x 11: no partial batch)
constexpr int kT1Pos = 11;

// conv3 output rows m = 4 * P + w (P pooled 3x3 position, w window element)
constexpr int M3 = 36, M3P = 48;                // padded to 3 tiles of 16

struct alignas(16) Smem {
    float x[NX + 3];
    union {                              // region A
        float a1[C1 * NA1];              // conv1 output
        float red3[2 * 21 * 256];        // conv3 split-K partial sums (forward)
        struct {
            float s2[C2 * NY2];          // conv3 backward-data sums
            alignas(16) float d3[C3 * M3P];  // conv3 output deltas, rows (P, w)
        };
        float red1[NW * 2 * 256];        // conv1 partial gradient tiles
    };
    union {                              // region B
        struct {
            alignas(16) float p3[NF1];   // pool2 output (FC1 input)
            alignas(16) float e3[NF1];   // dE/d(pool2 output)
            float fcpart[NW * NF1];      // FC1 backward partial sums per wavefront
        };
        alignas(16) float e1[C1 * NA1];  // dE/d(conv1 output), then conv1 deltas
    };
    float y2[C2 * NY2];                  // pooled conv2 output (conv3 input), then its deltas
    unsigned char am2[C2 * NY2 + 4];     // pool after conv2: argmax (window element 0..3)
    float h[F1 + 10], dh[F1 + 10];
    float o[16], dout[16];
    alignas(16) int koff3[KC3];          // im2col offset into y2 of k = (c,u,v), conv3
    alignas(16) int koff2[KC2P];         // im2col offset into a1 of k = (c,u,v), conv2 (0 past KC2)
    unsigned char am3[NF1 + 4];          // pool2 argmax
    float sink[128];                     // scatter target of padding lanes
    float b3s[C3];                       // conv3 biases (copied in the conv3 forward)
    int64_t idx;
};
static_assert(sizeof(Smem) <= 160 * 1024, "LDS budget");

template <int MODE>
__global__ void __launch_bounds__(NT, 1) fused_t1_kernel(WorkArgs a) {
    __shared__ Smem sm;
    const float *W = a.params;
    constexpr bool kTrain = (MODE == kTrainAtomic || MODE == kTrainRacy);

    // sample-invariant im2col offset tables
    for (int k = threadIdx.x; k < KC3; k += NT) {
        int c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
        sm.koff3[k] = c * NY2 + u * H2 + v;
    }
    for (int k = threadIdx.x; k < KC2P; k += NT) {
        int c = k / 25, uv = k - 25 * c, u = uv / 5, v = uv - 5 * u;
        sm.koff2[k] = (k < KC2) ? c * NA1 + u * H1 + v : 0;
    }

    // Training: thread 0 claims the worker's next sample as soon as the
    // current one is known (Section III-A.1), so the claim's round trip to
    // the shared counter overlaps a whole sample instead of starting it.
    int next = -1;
    for (int64_t step = 0;; ++step) {
        // opaque thread index: keeps per-phase index arithmetic inside its phase
        int tid_l = threadIdx.x;
        asm volatile("" : "+v"(tid_l));
        const int tid = tid_l, lane = tid_l & 63, lr = lane & 15, lg = lane >> 4;
        const int wave = __builtin_amdgcn_readfirstlane(tid_l >> 6);
        // ---- claim a sample (Section III-A.1) ----
        if (tid == 0) {
            if (kTrain && next < 0 && blockIdx.x > 0)
                join_after(a.counter, a.n, (int)blockIdx.x / kJoinRamp);
            if (kTrain) sm.idx = (next >= 0) ? next : atomicAdd(a.counter, 1);
            else sm.idx = (int64_t)blockIdx.x + step * gridDim.x;
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
        if (kTrain && tid == 0) {
            next = atomicAdd(a.counter, 1);
            if (a.claims) atomicAdd(a.claims + idx, 1);
        }
        const int label = a.labels[idx];
        for (int i = tid; i < NX; i += NT) sm.x[i] = a.x[idx * NX + i];
        __syncthreads();

        // conv1 (no pooling): rows = the 676 output positions (43 tiles), cols
        // o < 20, K = 16; a wavefront's tiles i = wave + 4q, six at a time.
        // Also used to recompute the output for the conv2 weight gradient.
        auto conv1_forward = [&]() {
            // unconditional loads (padding maps read map 19 into outputs that
            // are never stored): a select at a load makes it wait at once
            float bw[4][2], b1[2];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const int o = 16 * j + lr;
                    bw[s][j] = W[DW1 + (o < C1 ? o : C1 - 1) * 16 + 4 * s + lg];
                }
#pragma unroll
            for (int j = 0; j < 2; ++j) b1[j] = W[DB1 + (16 * j + lr < C1 ? 16 * j + lr : C1 - 1)];
            for (int i0 = wave; i0 < 43; i0 += 6 * NW) {
                f4 acc[6][2];
                int base[6];
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    int m = 16 * (i0 + 4 * q) + lr;
                    int my = m / H1, mx = m - my * H1;
                    base[q] = (m < NA1) ? my * IN + mx : 0;
                    acc[q][0] = f4{0.f, 0.f, 0.f, 0.f};
                    acc[q][1] = acc[q][0];
                }
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int q = 0; q < 6; ++q) {
                        float av = sm.x[base[q] + s * IN + lg];
                        acc[q][0] = mfma(av, bw[s][0], acc[q][0]);
                        acc[q][1] = mfma(av, bw[s][1], acc[q][1]);
                    }
#pragma unroll
                for (int q = 0; q < 6; ++q)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int m = 16 * (i0 + 4 * q) + 4 * lg + r;
                        if (m >= NA1) continue;
#pragma unroll
                        for (int j = 0; j < 2; ++j) {
                            int o = 16 * j + lr;
                            if (o < C1) sm.a1[o * NA1 + m] = acc[q][j][r] + b1[j];
                        }
                    }
            }
            // the activation over the 13,520 outputs, one per thread in turn
            // (applied in the tile epilogue, the lanes of map tile 1 past map
            // 19 would idle through it)
            __syncthreads();
            // four outputs per thread and round: their reads are issued
            // together, so the LDS round trip is paid once per four
            static_assert(C1 * NA1 % 4 == 0, "whole rounds of four");
            for (int t0 = tid; t0 < C1 * NA1 / 4; t0 += NT) {
                float v[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) v[q] = sm.a1[t0 + q * (C1 * NA1 / 4)];
#pragma unroll
                for (int q = 0; q < 4; ++q) sm.a1[t0 + q * (C1 * NA1 / 4)] = act_y(v[q]);
            }
        };

        // ================= forward propagation =================
        conv1_forward();
        __syncthreads();

        // conv2 + pool: rows m = 4P + w (P < 121 pooled positions, w window
        // element: one lane's four accumulators are one 2x2 window), 31 tiles;
        // wavefront w takes output maps 16w..16w+15 (one column tile) for all
        // rows; K = 500 (padded to 512) in super-steps of 16, lane group g
        // holding k = 16S + 4g + e at sub-step e, so its four weights of a
        // super-step are one 16-byte load, requested three super-steps ahead.
        {
            const int o = 16 * wave + lr;
            const bool ov = o < C2;
            const float *wrow = W + DW2 + (ov ? o : 0) * KC2S + 4 * lg;
            // the bias, requested now so that the epilogue does not wait for it
            const float bias2 = W[DB2 + (ov ? o : 0)];
            int base[M2T];
#pragma unroll
            for (int i = 0; i < M2T; ++i) {
                const int m = 16 * i + lr, P = m >> 2, w = m & 3;
                const int py = P / Q2, px = P - py * Q2;
                base[i] = (m < M2) ? (2 * py + (w >> 1)) * H1 + 2 * px + (w & 1) : 0;
            }
            f4 acc[M2T];
#pragma unroll
            for (int i = 0; i < M2T; ++i) acc[i] = f4{0.f, 0.f, 0.f, 0.f};
            // weights: unconditional 16-byte loads (the address is in bounds
            // for every lane: padding maps read map 0, whose accumulators are
            // never used).  The zeroing of K padding (k >= 500) is a select
            // at the use, three super-steps later: a select at the load would
            // make the load wait for its data at once.
            auto load = [&](int S) { return *(const f4 *)(wrow + 16 * S); };
            // A operands of a sub-step for every row tile, in two buffers:
            // sub-step e multiplies buffer e % 2 and reads the next sub-step's
            // operands into the other one, each read issued right after the
            // matrix instruction of the same row tile (held there by
            // scheduling barriers).  A read is then consumed a whole sub-step
            // (31 matrix instructions) after it was issued, and no wait for an
            // operand waits for a read issued since.
            float a0[M2T], a1v[M2T];
            auto sub = [&](const float (&cur)[M2T], float (&nxt)[M2T], float bk, int offn) {
#pragma unroll
                for (int i = 0; i < M2T; ++i) {
                    acc[i] = mfma(cur[i], bk, acc[i]);
                    __builtin_amdgcn_sched_barrier(0);
                    nxt[i] = sm.a1[base[i] + offn];
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            // one super-step: buffer a0 holds its first sub-step's operands on
            // entry and the next super-step's first on exit
            auto step = [&](f4 raw, int S) {
                const int4 ko = *(const int4 *)(sm.koff2 + 16 * S + 4 * lg);
                const int4 kn = *(const int4 *)(sm.koff2 + 16 * (S + 1 < KC2P / 16 ? S + 1 : S) + 4 * lg);
                const bool ok = 16 * S + 4 * lg < KC2;
                const f4 b = f4{ok ? raw.x : 0.f, ok ? raw.y : 0.f, ok ? raw.z : 0.f, ok ? raw.w : 0.f};
                sub(a0, a1v, b[0], ko.y);
                sub(a1v, a0, b[1], ko.z);
                sub(a0, a1v, b[2], ko.w);
                sub(a1v, a0, b[3], kn.x);
            };
            constexpr int NS = KC2P / 16;  // 32 super-steps, a ring of four weight buffers
            static_assert(NS % 4 == 0, "whole rounds");
            f4 b0 = load(0), b1 = load(1), b2 = load(2), b3;
            {
                const int off0 = sm.koff2[4 * lg];
#pragma unroll
                for (int i = 0; i < M2T; ++i) a0[i] = sm.a1[base[i] + off0];
            }
            for (int S = 0; S < NS; S += 4) {
                b3 = load(S + 3);
                step(b0, S);
                b0 = load(S + 4 < NS ? S + 4 : NS - 1);
                step(b1, S + 1);
                b1 = load(S + 5 < NS ? S + 5 : NS - 1);
                step(b2, S + 2);
                b2 = load(S + 6 < NS ? S + 6 : NS - 1);
                step(b3, S + 3);
            }
            if (ov) {
                const float bias = bias2;
#pragma unroll
                for (int i = 0; i < M2T; ++i) {
                    const int P = 4 * i + lg;
                    if (P < NY2) {
                        float ym;
                        int ag;
                        pool4(acc[i], bias, ym, ag);
                        sm.y2[o * NY2 + P] = ym;
                        sm.am2[o * NY2 + P] = (unsigned char)ag;
                    }
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
            f4 bA[7], bB[7], bC[7];
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
            // the biases, requested with the first weights and kept in LDS for
            // the epilogue (read there, they would cost it a round trip)
            const float b3pre = W[DB3 + (tid < C3 ? tid : C3 - 1)];
            // weights two super-steps ahead (a ring of three buffers)
            load_b(bA, S0);
            if (S0 + 1 < S1) load_b(bB, S0 + 1);
            if (tid < C3) sm.b3s[tid] = b3pre;
            for (int S = S0; S < S1; S += 3) {
                if (S + 2 < S1) load_b(bC, S + 2);
                compute(bA, S);
                if (S + 1 < S1) {
                    if (S + 3 < S1) load_b(bA, S + 3);
                    compute(bB, S + 1);
                }
                if (S + 2 < S1) {
                    if (S + 4 < S1) load_b(bB, S + 4);
                    compute(bC, S + 2);
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
                    float bias = sm.b3s[o];
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
            // lane l holds the bias of row jb + l, requested with the first
            // rows' weights
            const float bfx = W[DBF1 + (jb + lane < F1 ? jb + lane : F1 - 1)];
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
                const float bias = __shfl(bfx, (j - jb) & 63, 64);
                if ((lane & 7) == 0 && j < je) sm.h[j] = act_y(t1 + bias);
            }
        }
        __syncthreads();
        // FC2 (output layer): wavefront w computes outputs w, w + 4, w + 8;
        // all their weights and biases are requested before the first is used
        // (every load is used unconditionally, a padding lane multiplying a
        // zero, so none is moved into a branch where it would be waited for
        // at once)
        {
            float wf[3][3], bf[3];
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                const int j = (wave + NW * q < F2) ? wave + NW * q : F2 - 1;
#pragma unroll
                for (int it = 0; it < 3; ++it) {
                    const int i = lane + 64 * it;
                    wf[q][it] = W[DF2 + j * F1S + (i < F1 ? i : 0)];
                }
                bf[q] = W[DBF2 + j];
            }
#pragma unroll
            for (int q = 0; q < 3; ++q) {
                const int j = wave + NW * q;
                if (j >= F2) break;
                float s = 0.0f;
#pragma unroll
                for (int it = 0; it < 3; ++it) {
                    const int i = lane + 64 * it;
                    s = fmaf(wf[q][it], (i < F1) ? sm.h[i < F1 ? i : 0] : 0.0f, s);
                }
                s = wave_sum(s);
                if (lane == 0) sm.o[j] = act_y(s + bf[q]);
            }
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
            {
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
                // FC1_ROWS rows per step: 15 FC1_ROWS pushes in flight before
                // their returns are used (a wavefront's rows are still summed
                // in increasing order)
                for (int j = wave; j < F1; j += FC1_ROWS * NW) {
                    float old[FC1_ROWS][15], dr[FC1_ROWS];
#pragma unroll
                    for (int r = 0; r < FC1_ROWS; ++r) {
                        const int jr = j + r * NW;
                        dr[r] = (jr < F1) ? sm.dh[jr] : 0.0f;
                        if (jr < F1) {
#pragma unroll
                            for (int c = 0; c < 15; ++c) {
                                int i = lane + 64 * c;
                                old[r][c] = (i < NF1) ? push.with_old(DF1 + jr * NF1S + i, OF1 + jr * NF1 + i, dr[r] * xv[c])
                                                      : 0.0f;
                            }
                        } else {
#pragma unroll
                            for (int c = 0; c < 15; ++c) old[r][c] = 0.0f;
                        }
                    }
#pragma unroll
                    for (int r = 0; r < FC1_ROWS; ++r)
#pragma unroll
                        for (int c = 0; c < 15; ++c) ep[c] = fmaf(old[r][c], dr[r], ep[c]);
                }
                float *part = sm.fcpart;  // [wavefront][input]
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
            const float *part = sm.fcpart;
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
        static_assert(M3 % 4 == 0 && M3P % 4 == 0 && (C2 * NY2) % 4 == 0, "16-byte delta rows");
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
            float aA[9], aB[9], aC[9], bA[3], bB[3], bC[3];
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
            // weights and deltas two output-map steps ahead (a ring of three
            // buffers)
            constexpr int NKS = C3 / 4;
            load(aA, bA, 0);
            load(aB, bB, 1);
            for (int ks = 0; ks < NKS; ks += 3) {
                if (ks + 2 < NKS) load(aC, bC, ks + 2);
                compute(aA, bA);
                if (ks + 1 < NKS) {
                    if (ks + 3 < NKS) load(aA, bA, ks + 3);
                    compute(aB, bB);
                }
                if (ks + 2 < NKS) {
                    if (ks + 4 < NKS) load(aB, bB, ks + 4);
                    compute(aC, bC);
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
        // (no barrier: the weight gradient below reads what the backward data
        // reads and writes elsewhere, so each wavefront goes on with it; the
        // 15 backward-data blocks leave wavefront 3 one block short, which
        // takes two more column groups: 10 against 8)

        // conv3 weight gradient G[o][k] = sum_m d3[o][m] y2col[m][k], pushed.
        // Maps 0..95 on 32x32x2 tiles: element r of a tile holds maps
        // 8(r/4) + r%4 and that + 4 at 32 consecutive k, so a push
        // instruction writes two 128-byte runs of weights.  Maps 96..99 on
        // the 16-block 4x4x1 instruction with block b, column c at
        // k = 4b + c: element r holds map 96 + r at 64 consecutive k.
        // Wavefront 3 takes the 64-column groups 0..9, wavefront w < 3 the
        // groups 10 + 8w .. 17 + 8w (a column beyond KC3 computes values
        // never pushed).
        {
            float a32[3][18];  // A[o = 32i + l%32][m = 2ms + l/32]
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int ms = 0; ms < 18; ++ms)
                    a32[i][ms] = sm.d3[(32 * i + (lane & 31)) * M3P + 2 * ms + (lane >> 5)];
            const float *a4 = sm.d3 + (96 + (lane & 3)) * M3P;  // A[block][l%4][m]: map 96 + l%4
            static_assert((KC3 / 16 + 3) / 4 == 34 && C2 / 4 == 15, "34 column groups, 15 backward-data blocks");
            const int g0 = (wave == 3) ? 0 : 10 + 8 * wave, g1 = (wave == 3) ? 10 : g0 + 8;
            for (int grp = g0; grp < g1; ++grp) {
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

        // conv2 deltas at the pooled positions (in place of y2); the delta of a
        // conv2 output off its window's maximum is zero.  Clear the conv1
        // error buffer.
        // (four elements per thread and round: their reads are issued together)
        static_assert(C2 * NY2 % 4 == 0 && C1 * NA1 % 4 == 0, "whole rounds of four");
        for (int t0 = tid; t0 < C2 * NY2 / 4; t0 += NT) {
            float e[4], y[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                e[q] = sm.s2[t0 + q * (C2 * NY2 / 4)];
                y[q] = sm.y2[t0 + q * (C2 * NY2 / 4)];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) sm.y2[t0 + q * (C2 * NY2 / 4)] = e[q] * dact_from_y(y[q]);
        }
        for (int t = tid; t < C1 * NA1 / 4; t += NT) *(f4 *)(sm.e1 + 4 * t) = f4{0.f, 0.f, 0.f, 0.f};
        __syncthreads();
        // the conv1 output again (its region held the conv3 buffers meanwhile)
        conv1_forward();
        __syncthreads();

        // conv2 backward data and conv2 weight gradient, which read the same
        // inputs and write different outputs, in one phase so that the work
        // can be balanced over the wavefronts: backward data comes in 5 blocks
        // of 4 input maps (wavefront w takes block w, wavefront 0 also block
        // 4), the weight gradient in 32 column tiles (wavefront 0 takes 2,
        // the others 10 each).
        //
        // Backward data: C[k][m] = sum_o W2[o][k] d2[o][m], k = (c,u,v),
        // col2im into e1[c][pos(m) + (u,v)].  Row q of tile i holds map
        // c0 + q/4 at uv = 4i + q%4 (7 tiles), so the four lane groups of an
        // accumulator element hold four different maps at one (u,v): no
        // scatter instruction has two lanes on one address, and
        // wave_lds_order() keeps the overlapping groups in order.  A block's
        // weights (15 k-steps x 7 tiles) stay in registers while its columns
        // are computed four tiles at a time.
        auto bwd_block = [&](int blk) {
            const int c0 = 4 * blk;
            float av[15][7];
            // (loads are unconditional, from a clamped address, and zeroed by
            // a select: no branch between a load and its use)
#pragma unroll
            for (int ks = 0; ks < 15; ++ks) {
                const float *w2 = W + DW2 + (4 * ks + lg) * KC2S + (c0 + (lr >> 2)) * 25 + (lr & 3);
#pragma unroll
                for (int i = 0; i < 7; ++i) {
                    const bool ok = 4 * i + (lr & 3) < 25;
                    const float v = w2[ok ? 4 * i : 0];
                    av[ks][i] = ok ? v : 0.0f;
                }
            }
            for (int j0 = 0; j0 < M2T; j0 += 4) {
                f4 acc[7][4];
#pragma unroll
                for (int i = 0; i < 7; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
                // B: d2[o][m] for this lane's column m = 16(j0 + j) + lr
                int pq[4], wq[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int m = 16 * (j0 + j) + lr;
                    pq[j] = (m < M2) ? (m >> 2) : -1;
                    wq[j] = m & 3;
                }
                float bv[15][4];
#pragma unroll
                for (int ks = 0; ks < 15; ++ks) {
                    const int o = 4 * ks + lg;
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const int q = o * NY2 + (pq[j] >= 0 ? pq[j] : 0);
                        const int am = sm.am2[q];
                        const float v = sm.y2[q];
                        bv[ks][j] = (pq[j] >= 0 && am == wq[j]) ? v : 0.0f;
                    }
                }
#pragma unroll
                for (int ks = 0; ks < 15; ++ks)
#pragma unroll
                    for (int i = 0; i < 7; ++i)
#pragma unroll
                        for (int j = 0; j < 4; ++j) acc[i][j] = mfma(av[ks][i], bv[ks][j], acc[i][j]);
                // scatter: element r of tile i is (u,v) = uv 4i + r of map
                // c0 + lg; column m = 4P + w is conv2 output (2py + w/2, 2px + w%2)
                float *dp[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int m = 16 * (j0 + j) + lr, P = m >> 2, w = m & 3;
                    const int py = P / Q2, px = P - py * Q2;
                    dp[j] = (m < M2) ? sm.e1 + (c0 + lg) * NA1 + (2 * py + (w >> 1)) * H1 + 2 * px + (w & 1)
                                     : sm.sink;
                }
#pragma unroll
                for (int i = 0; i < 7; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int uv = 4 * i + r, u = uv / 5, v = uv - 5 * u;
                        if (uv >= 25) continue;
                        const float c[4] = {acc[i][0][r], acc[i][1][r], acc[i][2][r], acc[i][3][r]};
                        scatter_add<4>(dp, u * H1 + v, c);
                    }
            }
        };
        // Weight gradient G[o][k] = sum_m d2[o][m] a1col[m][k], pushed: rows o
        // (4 tiles), NTT column tiles of k = (c,u,v) per pass (NTT fixed at
        // compile time: a pass computes no padding tile), K = the 484 outputs
        // in (P, w) order, one pooled position per k-step; d2[o][(P, w)] is
        // the pooled delta where w is the window's maximum and 0 elsewhere.
        auto wgrad_tiles = [&](int jt0, auto ntt_c) {
            constexpr int NTT = decltype(ntt_c)::value;
            f4 acc[4][NTT];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int q = 0; q < NTT; ++q) acc[i][q] = f4{0.f, 0.f, 0.f, 0.f};
            int ko[NTT];
#pragma unroll
            for (int q = 0; q < NTT; ++q) ko[q] = sm.koff2[16 * (jt0 + q) + lr];
            int orow[4];
            bool ovv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                ovv[i] = 16 * i + lr < C2;
                orow[i] = (ovv[i] ? 16 * i + lr : 0) * NY2;
            }
            const int wy = lg >> 1, wx = lg & 1;
            // operands of pooled position P: raw reads, the selects in
            // compute behind a scheduling barrier
            auto operands = [&](int P, int (&am)[4], float (&av)[4], float (&bv)[NTT]) {
                const int py = P / Q2, px = P - py * Q2;
                const int base = (2 * py + wy) * H1 + 2 * px + wx;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    am[i] = sm.am2[orow[i] + P];
                    av[i] = sm.y2[orow[i] + P];
                }
#pragma unroll
                for (int q = 0; q < NTT; ++q) bv[q] = sm.a1[base + ko[q]];
            };
            // the A operands of a position: each row tile's pooled delta
            // where this lane group's window element is the maximum
            auto select = [&](const int (&am)[4], const float (&av)[4], float (&as)[4]) {
#pragma unroll
                for (int i = 0; i < 4; ++i) as[i] = (ovv[i] && am[i] == lg) ? av[i] : 0.0f;
            };
            // kT1Pos positions per iteration: all their reads first, then their
            // matrix instructions in position order (no read crosses the
            // loop's back edge, where the register allocator's copies would
            // wait for all of them).  A position's selects are formed under
            // the previous position's matrix instructions, into registers
            // that no instruction still in the matrix pipeline reads: a
            // select that rewrites the operand of the instruction just issued
            // waits for that instruction to read it.
            static_assert(NY2 % kT1Pos == 0, "whole batches of positions");
            for (int P0 = 0; P0 < NY2; P0 += kT1Pos) {
                int am[kT1Pos][4];
                float av[kT1Pos][4], bv[kT1Pos][NTT], as[kT1Pos][4];
#pragma unroll
                for (int u = 0; u < kT1Pos; ++u) operands(P0 + u, am[u], av[u], bv[u]);
                __builtin_amdgcn_sched_barrier(0);
                select(am[0], av[0], as[0]);
#pragma unroll
                for (int u = 0; u < kT1Pos; ++u)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                        for (int q = 0; q < NTT; ++q) acc[i][q] = mfma(as[u][i], bv[u][q], acc[i][q]);
                        if (i == 1 && u + 1 < kT1Pos) {
                            __builtin_amdgcn_sched_barrier(0);
                            select(am[u + 1], av[u + 1], as[u + 1]);
                            // the operand just issued stays live across the
                            // selects, so none of them is given its register
                            asm volatile("" ::"v"(as[u][1]));
                        }
                    }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < NTT; ++q) {
                const int k = 16 * (jt0 + q) + lr;
                if (k >= KC2) continue;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int o = 16 * i + 4 * lg + r;
                        if (o < C2) push(DW2 + o * KC2S + k, OW2 + o * KC2 + k, acc[i][q][r]);
                    }
            }
        };
        // this wavefront's column tiles [t0, t1): passes of four, then one of
        // the remainder
        auto wgrad_range = [&](int t0, int t1) {
            int jt = t0;
            for (; jt + 4 <= t1; jt += 4) wgrad_tiles(jt, std::integral_constant<int, 4>{});
            if (t1 - jt == 3) wgrad_tiles(jt, std::integral_constant<int, 3>{});
            else if (t1 - jt == 2) wgrad_tiles(jt, std::integral_constant<int, 2>{});
            else if (t1 - jt == 1) wgrad_tiles(jt, std::integral_constant<int, 1>{});
        };
        {
            bwd_block(wave);
            if (wave == 0) bwd_block(4);
            // column tiles [t0, t1) of this wavefront
            const int t0 = (wave == 0) ? 0 : kT1W0 + kT1W * (wave - 1);
            const int t1 = (wave == 0) ? kT1W0 : (wave == 3 ? 32 : t0 + kT1W);
            wgrad_range(t0, t1);
            if (tid < C2) {
                float g4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
                for (int P = 0; P < NY2; ++P) g4[P & 3] += sm.y2[tid * NY2 + P];
                push(DB2 + tid, OB2 + tid, (g4[0] + g4[1]) + (g4[2] + g4[3]));
            }
        }
        __syncthreads();
        // conv1 deltas: e1 * f'(conv1 output)
        for (int t0 = tid; t0 < C1 * NA1 / 4; t0 += NT) {
            float e[4], y[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                e[q] = sm.e1[t0 + q * (C1 * NA1 / 4)];
                y[q] = sm.a1[t0 + q * (C1 * NA1 / 4)];
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) sm.e1[t0 + q * (C1 * NA1 / 4)] = e[q] * dact_from_y(y[q]);
        }
        __syncthreads();

        // conv1 weight gradient G[o][uv] = sum over the 676 outputs of the
        // delta times the input under the kernel: rows o (2 tiles), cols
        // uv = 4u + v, K = outputs (k-step ks covers outputs 4ks..4ks+3) split
        // over the wavefronts, the partial tiles summed in wavefront order.
        // Bias gradient: the deltas summed per map.
        {
            f4 acc[2][2];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int t = 0; t < 2; ++t) acc[h][t] = f4{0.f, 0.f, 0.f, 0.f};
            const int oa = lr, ob = (16 + lr < C1) ? 16 + lr : 0;
            const bool vb = 16 + lr < C1;
            const int xo = (lr >> 2) * IN + (lr & 3);
            auto step = [&](int ks, f4 (&c)[2]) {
                const int m = 4 * ks + lg, my = m / H1, mx = m - my * H1;
                const float bx = sm.x[my * IN + mx + xo];
                const float a0 = sm.e1[oa * NA1 + m];
                const float a1v = vb ? sm.e1[ob * NA1 + m] : 0.0f;
                c[0] = mfma(a0, bx, c[0]);
                c[1] = mfma(a1v, bx, c[1]);
            };
            int ks = wave;
            for (; ks + NW < NA1 / 4; ks += 2 * NW) {
                step(ks, acc[0]);
                step(ks + NW, acc[1]);
            }
            if (ks < NA1 / 4) step(ks, acc[0]);
#pragma unroll
            for (int t = 0; t < 2; ++t)
                *(f4 *)(sm.red1 + ((wave * 2 + t) * 64 + lane) * 4) = acc[0][t] + acc[1][t];
            __syncthreads();
            for (int t = tid; t < C1 * 16 + C1; t += NT) {
                if (t < C1 * 16) {
                    const int o = t >> 4, uv = t & 15, tile = o >> 4, row = o & 15;
                    const int e = ((row >> 2) * 16 + uv) * 4 + (row & 3);
                    float g = sm.red1[(0 * 2 + tile) * 256 + e];
#pragma unroll
                    for (int w = 1; w < NW; ++w) g += sm.red1[(w * 2 + tile) * 256 + e];
                    push(DW1 + t, OW1 + t, g);
                } else {
                    const int o = t - C1 * 16;
                    float g4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
                    for (int q = 0; q < NA1; ++q) g4[q & 3] += sm.e1[o * NA1 + q];
                    push(DB1 + o, OB1 + o, (g4[0] + g4[1]) + (g4[2] + g4[3]));
                }
            }
        }
        if (kTrain && tid == 0) atomicAdd(a.counter + 1, 1);  // samples completed
        __syncthreads();
    }
}

} // namespace

bool fused_t1_matches(const Net &net) {
    static const int spec[][3] = {{kConv, 20, 4}, {kPool, 0, 1}, {kConv, 60, 5}, {kPool, 0, 2},
                                  {kConv, 100, 6}, {kPool, 0, 2}, {kFc, 150, 0}, {kFc, 10, 0}};
    if (net.n_layers != 8 || net.in_size != NX || net.n_params != NPARAM) return false;
    for (int l = 0; l < 8; ++l) {
        const Layer &ly = net.L[l];
        if (ly.kind != spec[l][0]) return false;
        if (ly.kind != kFc && ly.k != spec[l][2]) return false;
        if (ly.kind != kPool && ly.cout != spec[l][1]) return false;
    }
    return net.L[0].hin == IN && net.L[0].win == IN;
}

void fused_t1_layout(ParamLayout &L) {
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

hipError_t launch_fused_t1(int mode, const WorkArgs &a, int grid, hipStream_t s) {
    switch (mode) {
    case kTrainAtomic: fused_t1_kernel<kTrainAtomic><<<grid, NT, 0, s>>>(a); break;
    case kTrainRacy: fused_t1_kernel<kTrainRacy><<<grid, NT, 0, s>>>(a); break;
    case kForwardBackward: fused_t1_kernel<kForwardBackward><<<grid, NT, 0, s>>>(a); break;
    case kEvaluate: fused_t1_kernel<kEvaluate><<<grid, NT, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int fused_t1_blocks_per_cu() {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fused_t1_kernel<kTrainAtomic>, NT, 0) !=
        hipSuccess)
        return 0;
    return nb;
}

} // namespace chaos
