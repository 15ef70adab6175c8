// Fused per-sample CHAOS worker for the Table I small and medium nets:
//   1x29x29 -> conv C1@4x4 -> max 2 -> conv C2@5x5 -> max 3 -> FC F1 -> FC 10
//   small: C1 = 5, C2 = 10, F1 = 50;  medium: C1 = 20, C2 = 40, F1 = 150.
//
// Same organisation as the large-net kernel: one workgroup (4 wavefronts) is
// one worker owning one sample at a time (Section III-A.1); every per-sample
// value stays in LDS; conv1 forward (with the 2x2 pool fused into its
// epilogue), conv2 forward, conv2 weight gradient and conv2 backward data are
// implicit GEMMs on v_mfma_f32_16x16x4_f32; the 3x3 pool and the fully
// connected layers run on the vector ALUs.  Per layer the partial derivatives
// of the layer below are computed from the layer's weights before the layer's
// gradient is pushed (Section III-A.2), lock-free (III-A.3).  A separate
// instantiation for the small net keeps each worker's gradient sum in LDS and
// pushes it every few samples instead (delayed pushes).
#include "chaos_internal.h"
#include "device_common.h"

namespace chaos {
namespace {

constexpr int pad16(bool pad, int v) { return pad ? (v + 15) / 16 * 16 : v; }

template <int C1_, int C2_, int F1_>
struct Cpcp {
    static constexpr int C1 = C1_, C2 = C2_, F1 = F1_, F2 = 10;
    static constexpr int IN = 29, NX = IN * IN;
    static constexpr int Q1 = 13, NP1 = Q1 * Q1;        // pool1 output 13x13
    static constexpr int H2 = 9, NY2 = H2 * H2;         // conv2 output 9x9
    static constexpr int NP2 = 9;                       // pool2 output 3x3
    static constexpr int NF1 = C2 * NP2;                // FC1 inputs
    static constexpr int KC2 = C1 * 25;                 // conv2 K = (c,u,v)
    static constexpr int KC2P = (KC2 + 15) / 16 * 16;   // padded to whole tiles
    static constexpr int KQ2 = (KC2 + 31) / 32 * 8;     // conv2 forward K padded to 4 KQ2
    static constexpr int CT1 = (C1 + 15) / 16;          // conv1 col tiles
    static constexpr int CT2 = (C2 + 15) / 16;          // conv2 map tiles
    static constexpr int C2P = CT2 * 16;
    static constexpr int OKS = (C2 + 3) / 4;            // k-steps over output maps
    static_assert(4 * OKS <= C2P, "every k-step's delta rows lie in the delta buffer");
    // canonical parameter offsets
    static constexpr int OW1 = 0, OB1 = C1 * 16;
    static constexpr int OW2 = OB1 + C1, OB2 = OW2 + C2 * KC2;
    static constexpr int OF1 = OB2 + C2, OBF1 = OF1 + F1 * NF1;
    static constexpr int OF2 = OBF1 + F1, OBF2 = OF2 + F2 * F1;
    static constexpr int NPARAM = OBF2 + F2;
    // A weight vector of at most 8K floats (the small net: 27.6 KB in its
    // device layout) is copied into LDS once per sample and every later
    // weight read of the sample is served from there: one round trip to
    // memory per sample instead of one per layer and pass.
    static constexpr bool STAGE = NPARAM <= 8192;
    // Device layout of the shared weights: every segment starts on a 64-byte
    // boundary and the conv2, FC1 and FC2 rows are padded to multiples of 16
    // floats (the padding stays zero), so the pushes of a row cover whole
    // 64-byte segments and no segment is shared by two rows.  The memory-side
    // atomic units process one request per segment and serialize requests to
    // one line; the small net, whose every line takes a read and an add from
    // every sample, is bound by exactly that.
    static constexpr bool PAD = true;
    static constexpr int KC2S = pad16(PAD, KC2), NF1S = pad16(PAD, NF1), F1S = pad16(PAD, F1);
    static constexpr int DW1 = 0, DB1 = C1 * 16;
    static constexpr int DW2 = pad16(PAD, DB1 + C1), DB2 = DW2 + C2 * KC2S;
    static constexpr int DF1 = pad16(PAD, DB2 + C2), DBF1 = DF1 + F1 * NF1S;
    static constexpr int DF2 = pad16(PAD, DBF1 + F1), DBF2 = DF2 + F2 * F1S;
    static constexpr int NDEV = pad16(PAD, DBF2 + F2);
    static_assert(PAD || NDEV == NPARAM, "the unpadded layout is the canonical one");
    static_assert(NDEV % 4 == 0, "whole 16-byte loads of the device vector");
    // FC1 rows read with 16-byte loads when every row start is 16-byte aligned
    static constexpr int FC1_VEC = (DF1 % 4 == 0 && NF1S % 4 == 0 && NF1 % 4 == 0) ? 4 : 1;
    // Otherwise the conv2 weights (80 KB for the medium net), read by the
    // conv2 forward pass and again by its backward-data pass, are copied into
    // LDS once per sample (one worker per CU then fits), rows of KC2 floats.
    static constexpr int NW2 = C2 * KC2;
    static constexpr bool STAGE2 = !STAGE && NW2 <= 20480 && DW2 % 4 == 0 && KC2 % 4 == 0;
    // row stride of the conv2 weights as the kernel reads them
    static constexpr int W2S = STAGE2 ? KC2 : KC2S;
    // Such a net copies its small segments into LDS with them: the conv1
    // weights and biases [DW1, DB1 + C1), the conv2 biases, and everything
    // from the FC1 biases on (the FC2 weights and biases), so that no read of
    // the sample but the FC1 rows goes to memory.
    static constexpr int NLO = DB1 + C1, NTAIL = NDEV - DBF1;
    static constexpr int NSMALL = STAGE2 ? NLO + C2 + NTAIL : 4;
    static_assert(!STAGE2 || (DW1 == 0 && NLO % 4 == 0 && DB2 % 4 == 0 && C2 % 4 == 0 && DBF1 % 4 == 0),
                  "the small segments are copied with 16-byte loads");
    // 16-byte loads of conv2 weight rows need 16-byte aligned row starts (the
    // LDS copies are 16-byte aligned; a row's padding reads as zero)
    static constexpr bool W2_ALIGNED16 = ((STAGE2 ? 0 : DW2) % 4 == 0) && (W2S % 4 == 0);
};

constexpr int NT = 256, NW = 4;
constexpr int RT2 = 6;  // conv2 output positions 81 -> 6 tiles of 16
// Row stride of the conv2 delta buffer (96 positions read, 81 nonzero): 100
// puts the 16 rows that one matrix operand read takes (lanes over rows) in
// distinct LDS banks, where a stride of 96 folds them onto one or two.
constexpr int D2S = 100;

template <class S, bool DELAY = false>
struct alignas(16) SmemCpcp {
    float x[S::NX + 3];
    float p1[S::C1 * S::NP1];            // pool1 output, later pool1 errors/deltas in e1
    float e1[S::C1 * S::NP1];            // dE/d(pool1 output)
    float y2[S::C2 * S::NY2];            // conv2 output before the activation
    alignas(16) float d2[S::C2P * D2S];   // conv2 output deltas (dense, zero off the argmax);
                                         // conv2 forward partial sums before that
    alignas(16) float p2[S::NF1];        // pool2 output
    float e2[S::NF1], e2b[S::NF1];       // its errors (two partial sums over FC1 rows)
    float h[S::F1 + 16], dh[S::F1 + 16];
    float o[16], dout[16];
    alignas(16) int koff2[4 * S::KQ2];   // im2col offset into p1 of k = (c,u,v) (0 past KC2)
    unsigned char am1[S::C1 * S::NP1 + 16];
    unsigned char am2[S::NF1 + 16];
    alignas(16) float w[S::STAGE ? S::NDEV : 4];  // the weights read at the start of the sample
    alignas(16) float w2[S::STAGE2 ? S::NW2 : 4];    // the conv2 weights read at the start of the sample
    alignas(16) float ws[S::NSMALL];                 // and the small segments (STAGE2)
    float sink[64];                      // scatter target of padding lanes
    float ones[128];                     // the conv2 weight gradient's ones column (bias)
    // delayed pushes: this worker's gradient sum since its last push (device layout)
    alignas(16) float gacc[DELAY ? S::NDEV : 4];
    int64_t idx;
    int rep_refresh;  // this sample's worker refreshes its replica
};

// DELAY (training with atomic pushes, nets whose whole weight vector fits in
// LDS): instead of pushing each layer's gradient after its backward pass,
// the worker adds it to a private sum in LDS and pushes the sum after every
// a.push_delay samples it processes, and after its last (a variant of the
// per-layer update, Section III-A.2, with the delayed sharing of locally
// accumulated updates); its own unpushed updates are not in the weights it
// reads.
template <class S, int MODE, int MINB, bool DELAY = false>
__global__ void __launch_bounds__(NT, MINB) fused_cpcp_kernel(WorkArgs a) {
    static_assert(!DELAY || (MODE == kTrainAtomic && S::STAGE),
                  "delayed pushes: atomic training of a net copied whole into LDS");
    __shared__ SmemCpcp<S, DELAY> sm;
    const float *Wg = a.params;
    // every weight read below goes through W: the LDS copy or the shared vector
    const float *W = S::STAGE ? (const float *)sm.w : Wg;
    const float *W2 = S::STAGE2 ? (const float *)sm.w2 : W + S::DW2;  // conv2 weights [o][k], rows W2S apart
    const float *Wlo = S::STAGE2 ? (const float *)sm.ws : W;                      // conv1 weights and biases
    const float *Wb2 = S::STAGE2 ? (const float *)sm.ws + S::NLO : W + S::DB2;   // conv2 biases
    const float *Wt = S::STAGE2 ? (const float *)sm.ws + S::NLO + S::C2 : W + S::DBF1;  // from the FC1 biases on
    constexpr bool kTrain = (MODE == kTrainAtomic || MODE == kTrainRacy);
    // the FC1 partial derivatives come from a separate read of the weights
    // (frozen weights, or the LDS copy) instead of the values returned by the
    // FC1 pushes
    constexpr bool kFc1Read = (MODE == kForwardBackward) || S::STAGE;
    // Replicated weights (atomic training of a net copied whole into LDS):
    // worker b reads replica b % n_replicas and pushes every update to the
    // shared weights and to that replica, which is refreshed from the shared
    // weights after every refresh_every-th sample completed on it.  Per-line
    // contention at the memory side (every sample reads and adds into every
    // line of the vector) is then spread over the replicas.
    const bool kReplicas = (MODE == kTrainAtomic) && !DELAY && S::STAGE && a.replicas != nullptr;

    for (int k = threadIdx.x; k < 128; k += NT) sm.ones[k] = 1.0f;
    for (int k = threadIdx.x; k < 4 * S::KQ2; k += NT) {
        int c = k / 25, uv = k - 25 * c, u = uv / 5, v = uv - 5 * u;
        sm.koff2[k] = (k < S::KC2) ? c * S::NP1 + u * S::Q1 + v : 0;
    }
    int nproc = 0;  // samples this worker has processed (delayed pushes)
    if constexpr (DELAY) {
        for (int i = threadIdx.x; i < S::NDEV; i += NT) sm.gacc[i] = 0.0f;
    }
    // pushes this worker's gradient sum (W += -lr * sum, the rounding of the
    // per-layer push) and clears it; after a barrier
    auto flush = [&]() {
        if constexpr (DELAY) {
            Push fp;
            fp.mode = kTrainAtomic;
            fp.params = a.params;
            fp.neg_lr = -a.lr;
            fp.each = nullptr;
            fp.part = nullptr;
            // the whole device vector, padding included (its sums stay zero)
            for (int i = threadIdx.x; i < S::NDEV; i += NT) {
                fp(i, sm.gacc[i]);
                sm.gacc[i] = 0.0f;
            }
        }
    };

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
        if (idx >= a.n) {
            if constexpr (DELAY) {
                if (nproc % a.push_delay) flush();
            }
            break;
        }
        if (kTrain && tid == 0) {
            next = atomicAdd(a.counter, 1);
            if (a.claims) atomicAdd(a.claims + idx, 1);
        }
        const int label = a.labels[idx];
        if constexpr (S::STAGE) {
            // the weights of this sample: all 16-byte loads are issued before
            // the first LDS write (the vector starts 16-byte aligned); from
            // this worker's replica when the shared weights are replicated
            const float *Wsrc = kReplicas ? a.replicas + (int64_t)(blockIdx.x % a.n_replicas) * S::NDEV : Wg;
            constexpr int N4 = S::NDEV / 4, PER = (N4 + NT - 1) / NT, TAIL = S::NDEV - 4 * N4;
            f4 wv[PER];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                wv[q] = (t4 < N4) ? *(const f4 *)(Wsrc + 4 * t4) : f4{0.f, 0.f, 0.f, 0.f};
            }
            const float wt = (tid < TAIL) ? Wsrc[4 * N4 + tid] : 0.0f;
            for (int i = tid; i < S::NX; i += NT) sm.x[i] = a.x[idx * S::NX + i];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                if (t4 < N4) *(f4 *)(sm.w + 4 * t4) = wv[q];
            }
            if (tid < TAIL) sm.w[4 * N4 + tid] = wt;
        } else if constexpr (S::STAGE2) {
            constexpr int N4 = S::NW2 / 4, PER = (N4 + NT - 1) / NT;
            static_assert(S::NW2 % 4 == 0, "whole 16-byte loads");
            f4 wv[PER];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                const int o = 4 * t4 / S::KC2, k = 4 * t4 - o * S::KC2;  // a row holds whole 16-byte groups
                wv[q] = (t4 < N4) ? *(const f4 *)(Wg + S::DW2 + o * S::KC2S + k) : f4{0.f, 0.f, 0.f, 0.f};
            }
            constexpr int N4L = S::NLO / 4, N4B = S::C2 / 4, N4S = (S::NLO + S::C2 + S::NTAIL) / 4;
            constexpr int PS = (N4S + NT - 1) / NT;
            f4 sv[PS];
#pragma unroll
            for (int q = 0; q < PS; ++q) {
                const int t4 = tid + NT * q;
                const float *src = (t4 < N4L) ? Wg + 4 * t4
                                   : (t4 < N4L + N4B) ? Wg + S::DB2 + 4 * (t4 - N4L)
                                                      : Wg + S::DBF1 + 4 * (t4 - N4L - N4B);
                sv[q] = (t4 < N4S) ? *(const f4 *)src : f4{0.f, 0.f, 0.f, 0.f};
            }
            for (int i = tid; i < S::NX; i += NT) sm.x[i] = a.x[idx * S::NX + i];
#pragma unroll
            for (int q = 0; q < PER; ++q) {
                const int t4 = tid + NT * q;
                if (t4 < N4) *(f4 *)(sm.w2 + 4 * t4) = wv[q];
            }
#pragma unroll
            for (int q = 0; q < PS; ++q) {
                const int t4 = tid + NT * q;
                if (t4 < N4S) *(f4 *)(sm.ws + 4 * t4) = sv[q];
            }
        } else {
            for (int i = tid; i < S::NX; i += NT) sm.x[i] = a.x[idx * S::NX + i];
        }
        __syncthreads();

        // ---- conv1 + pool1: rows (P, w) P < 169, cols o < C1, K = 16 ----
        {
            float bw[4][S::CT1];
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int j = 0; j < S::CT1; ++j) {
                    int o = 16 * j + lr;
                    bw[s][j] = (o < S::C1) ? Wlo[S::DW1 + o * 16 + 4 * s + lg] : 0.0f;
                }
            float b1[S::CT1];
#pragma unroll
            for (int j = 0; j < S::CT1; ++j) b1[j] = (16 * j + lr < S::C1) ? Wlo[S::DB1 + 16 * j + lr] : 0.0f;
            // a wavefront's tiles i = wave + 4q, six at a time
            for (int i0 = wave; i0 < 43; i0 += 6 * NW) {
                f4 acc[6][S::CT1];
                int base[6];
                bool valid[6];
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    int m = 16 * (i0 + 4 * q) + lr, P = m >> 2;
                    valid[q] = P < S::NP1;
                    base[q] = valid[q] ? window_pos(P, m & 3, S::Q1, S::IN) : 0;
#pragma unroll
                    for (int j = 0; j < S::CT1; ++j) acc[q][j] = f4{0.f, 0.f, 0.f, 0.f};
                }
                // the pass's 24 inputs are read at once, ahead of the matrix
                // instructions
                float xv[4][6];
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int q = 0; q < 6; ++q) xv[s][q] = sm.x[base[q] + s * S::IN + lg];  // base 0 when invalid
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int s = 0; s < 4; ++s)
#pragma unroll
                    for (int q = 0; q < 6; ++q) {
                        // (a row past the map reads a valid input; its output
                        // row is never used)
#pragma unroll
                        for (int j = 0; j < S::CT1; ++j) acc[q][j] = mfma(xv[s][q], bw[s][j], acc[q][j]);
                    }
#pragma unroll
                for (int q = 0; q < 6; ++q) {
                    int Pe = 4 * (i0 + 4 * q) + lg;
                    if (Pe < S::NP1) {
#pragma unroll
                        for (int j = 0; j < S::CT1; ++j) {
                            int o = 16 * j + lr;
                            if (o < S::C1) {
                                float ym;
                                int ag;
                                pool4(acc[q][j], b1[j], ym, ag);
                                sm.p1[o * S::NP1 + Pe] = ym;
                                sm.am1[o * S::NP1 + Pe] = (unsigned char)ag;
                            }
                        }
                    }
                }
            }
        }
        __syncthreads();

        // ---- conv2: rows p < 81 (6 tiles), cols o < C2, K = C1*25 ----
        // K in blocks of 16: at sub-step e of block b lane group g holds
        // k = 16b + 4g + e, so a lane's four weights of a block are
        // consecutive and the four lane groups of a row cover 64 contiguous
        // bytes.  Wavefront w takes row tiles 3(w%2)..3(w%2)+2 and half of
        // the blocks (w/2); the halves are added in a fixed order through LDS
        // (the delta buffer is free during the forward pass).  Weights are
        // requested two blocks ahead.
        {
            constexpr int NB = S::KQ2 / 8;  // blocks per half
            const int rt0 = 3 * (wave & 1), half = wave >> 1;
            f4 acc[3][S::CT2];
#pragma unroll
            for (int i = 0; i < 3; ++i)
#pragma unroll
                for (int j = 0; j < S::CT2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
            int base[3];
            bool pv[3];
#pragma unroll
            for (int i = 0; i < 3; ++i) {
                int p = 16 * (rt0 + i) + lr;
                pv[i] = p < S::NY2;
                int py = p / S::H2, px = p - py * S::H2;
                base[i] = pv[i] ? py * S::Q1 + px : 0;
            }
            const int kb = 16 * NB * half + 4 * lg;  // this lane's first k
            const float *wrow[S::CT2];
            bool ov[S::CT2];
#pragma unroll
            for (int j = 0; j < S::CT2; ++j) {
                int o = 16 * j + lr;
                ov[j] = o < S::C2;
                wrow[j] = W2 + (ov[j] ? o : 0) * S::W2S + kb;
            }
            float bw[3][S::CT2][4];
            auto load = [&](float (&b)[S::CT2][4], int blk) {
#pragma unroll
                for (int j = 0; j < S::CT2; ++j) {
                    if (S::W2_ALIGNED16) {
                        f4 v = (ov[j] && kb + 16 * blk < S::KC2) ? *(const f4 *)(wrow[j] + 16 * blk)
                                                                : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int e = 0; e < 4; ++e) b[j][e] = v[e];
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            int k = kb + 16 * blk + e;
                            b[j][e] = (ov[j] && k < S::KC2) ? wrow[j][16 * blk + e] : 0.0f;
                        }
                    }
                }
            };
            auto compute = [&](const float (&b)[S::CT2][4], int blk) {
                const int4 ko = *(const int4 *)(sm.koff2 + kb + 16 * blk);
                const int offs[4] = {ko.x, ko.y, ko.z, ko.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
#pragma unroll
                    for (int i = 0; i < 3; ++i) {
                        // base 0 past the map: a valid input, in an output row never used
                        const float v = sm.p1[base[i] + offs[e]];
#pragma unroll
                        for (int j = 0; j < S::CT2; ++j) acc[i][j] = mfma(v, b[j][e], acc[i][j]);
                    }
                }
            };
            load(bw[0], 0);
            if (NB > 1) load(bw[1], 1);
            for (int blk = 0; blk < NB; blk += 3) {
                if (blk + 2 < NB) load(bw[2], blk + 2);
                compute(bw[0], blk);
                if (blk + 1 < NB) {
                    if (blk + 3 < NB) load(bw[0], blk + 3);
                    compute(bw[1], blk + 1);
                }
                if (blk + 2 < NB) {
                    if (blk + 4 < NB) load(bw[1], blk + 4);
                    compute(bw[2], blk + 2);
                }
            }
            float *red = sm.d2 + (wave & 1) * (3 * S::CT2 * 256);
            if (half == 1) {
#pragma unroll
                for (int i = 0; i < 3; ++i)
#pragma unroll
                    for (int j = 0; j < S::CT2; ++j)
                        *(f4 *)(red + ((i * S::CT2 + j) * 64 + lane) * 4) = acc[i][j];
            }
            __syncthreads();
            if (half == 0) {
#pragma unroll
                for (int j = 0; j < S::CT2; ++j) {
                    int o = 16 * j + lr;
                    if (o >= S::C2) continue;
                    float bias = Wb2[o];
#pragma unroll
                    for (int i = 0; i < 3; ++i) {
                        f4 t = acc[i][j] + *(const f4 *)(red + ((i * S::CT2 + j) * 64 + lane) * 4);
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            int pe = 16 * (rt0 + i) + 4 * lg + r;
                            if (pe < S::NY2) sm.y2[o * S::NY2 + pe] = t[r] + bias;
                        }
                    }
                }
            }
        }
        __syncthreads();

        // ---- FC1: wavefront w computes neurons [JW w, JW w + JW), eight at a
        //      time, lanes over the inputs (16-byte loads when the rows are
        //      16-byte aligned); the eight partial sums of a lane are reduced
        //      by halving (exchanges with lanes l^32, l^16, l^8 leave one
        //      neuron per lane, l^4, l^2, l^1 complete it).  The next eight
        //      rows are requested before the current ones are reduced. ----
        {
            constexpr int VEC = S::FC1_VEC, IC = (S::NF1 + 64 * VEC - 1) / (64 * VEC);
            constexpr int JW = (S::F1 + NW - 1) / NW;
            const int jb = JW * wave, je = (jb + JW < S::F1) ? jb + JW : S::F1;
            float wv[8][IC][VEC];
            auto load_rows = [&](int j0) {
#pragma unroll
                for (int q = 0; q < 8; ++q)
#pragma unroll
                    for (int c = 0; c < IC; ++c) {
                        const int j = j0 + q, i = VEC * lane + 64 * VEC * c;
                        const bool v = j < je && i < S::NF1;
                        const float *src = W + S::DF1 + (v ? j * S::NF1S + i : 0);
                        if (VEC == 4) {
                            f4 t = v ? *(const f4 *)src : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                            for (int e = 0; e < VEC; ++e) wv[q][c][e] = t[e];
                        } else {
                            wv[q][c][0] = v ? *src : 0.0f;
                        }
                    }
            };
            // the first rows are requested before the pool2 phase, whose
            // maxima and the barrier after it then hide part of their wait
            if (jb < je) load_rows(jb);
            // ---- pool2: 3x3 windows of the 9x9 maps, first maximum wins.  y2
            //      holds the conv2 outputs before the activation; f is strictly
            //      increasing, so the window's maximum is taken on z and f is
            //      applied to it alone. ----
            for (int t = tid; t < S::NF1; t += NT) {
                int o = t / S::NP2, P = t - o * S::NP2;
                int py = P / 3, px = P - 3 * py;
                const float *zo = sm.y2 + o * S::NY2 + 3 * py * S::H2 + 3 * px;
                float m = zo[0];
                int ag = 0;
#pragma unroll
                for (int w = 1; w < 9; ++w) {
                    float v = zo[(w / 3) * S::H2 + (w % 3)];
                    if (v > m) { m = v; ag = w; }
                }
                sm.p2[t] = act_y(m);
                sm.am2[t] = (unsigned char)ag;
            }
            __syncthreads();

            float xin[IC][VEC];
#pragma unroll
            for (int c = 0; c < IC; ++c)
#pragma unroll
                for (int e = 0; e < VEC; ++e) {
                    int i = VEC * lane + 64 * VEC * c + e;
                    xin[c][e] = (i < S::NF1) ? sm.p2[i] : 0.0f;
                }
            const bool b5 = lane & 32, b4 = lane & 16, b3 = lane & 8;
            for (int j0 = jb; j0 < je; j0 += 8) {
                float sq[8];
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float t = 0.0f;
#pragma unroll
                    for (int c = 0; c < IC; ++c)
#pragma unroll
                        for (int e = 0; e < VEC; ++e) t = fmaf(wv[q][c][e], xin[c][e], t);
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
                if ((lane & 7) == 0 && j < je) sm.h[j] = act_y(t1 + Wt[j]);
            }
        }
        __syncthreads();
        for (int j = wave; j < S::F2; j += NW) {
            float s = 0.0f;
#pragma unroll
            for (int it = 0; it < (S::F1 + 63) / 64; ++it) {
                int i = lane + 64 * it;
                if (i < S::F1) s = fmaf(Wt[S::DF2 - S::DBF1 + j * S::F1S + i], sm.h[i], s);
            }
            s = wave_sum(s);
            if (lane == 0) sm.o[j] = act_y(s + Wt[S::DBF2 - S::DBF1 + j]);
        }
        __syncthreads();
        if (a.out && tid < S::F2) a.out[idx * S::F2 + tid] = sm.o[tid];

        if (MODE == kEvaluate) {
            if (tid == 0) {
                int best = 0;
                for (int k = 1; k < S::F2; ++k)
                    if (sm.o[k] > sm.o[best]) best = k;
                if (best != label) atomicAdd(a.n_wrong, 1);
            }
            __syncthreads();
            continue;
        }

        // ================= back-propagation =================
        Push push_now;
        push_now.mode = MODE;
        push_now.params = a.params;
        push_now.neg_lr = -a.lr;
        push_now.each = a.grad_each ? a.grad_each + idx * (int64_t)S::NPARAM : nullptr;
        push_now.part = a.grad_part ? a.grad_part + (int64_t)blockIdx.x * S::NPARAM : nullptr;
        // a layer's gradient element (each weight once per sample, by one
        // thread): pushed now, or added to the worker's sum
        float *const rep = kReplicas ? a.replicas + (int64_t)(blockIdx.x % a.n_replicas) * S::NDEV : nullptr;
        auto push = [&](int w_off, int g_off, float g) {
            if constexpr (DELAY) {
                sm.gacc[w_off] += g;
            } else {
                push_now(w_off, g_off, g);
                // the same update, rounded the same way, into this worker's replica
                if (rep) __hip_atomic_fetch_add(rep + w_off, __fmul_rn(push_now.neg_lr, g), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
            }
        };

        if (tid < 64) {
            float e = 0.0f;
            if (tid < S::F2) {
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
        for (int i = tid; i < S::F1; i += NT) {
            float wv[S::F2];
#pragma unroll
            for (int j = 0; j < S::F2; ++j) wv[j] = Wt[S::DF2 - S::DBF1 + j * S::F1S + i];
            float s = 0.0f;
#pragma unroll
            for (int j = 0; j < S::F2; ++j) s = fmaf(wv[j], sm.dout[j], s);
            sm.dh[i] = s * dact_from_y(sm.h[i]);
        }
        __syncthreads();
        // FC2 push; FC1 push and FC1 backward data
        for (int t = tid; t < S::F2 * S::F1; t += NT) {
            int j = t / S::F1, i = t - j * S::F1;
            push(S::DF2 + j * S::F1S + i, S::OF2 + t, sm.dout[j] * sm.h[i]);
        }
        if (tid < S::F2) push(S::DBF2 + tid, S::OBF2 + tid, sm.dout[tid]);
        if constexpr (kFc1Read) {
            // read the weights (frozen, or this sample's LDS copy), then push
            // FC1 backward data (pre-update weights), summed over the rows in
            // row order: thread t owns VEC inputs (one 16-byte load per row when
            // aligned); with 16-byte loads the rows are split in two halves whose
            // sums are added in the pool2 backward below.  Ten rows per batch,
            // the next batch requested while this one is summed.
            {
                constexpr int VEC = S::FC1_VEC, NI = S::NF1 / VEC, NPART = (VEC == 4) ? 2 : 1;
                constexpr int RP = (S::F1 + NPART - 1) / NPART;
                if (tid < NI * NPART) {
                    const int i0 = VEC * (tid % NI), part = tid / NI;
                    const int r0 = part * RP, r1 = (r0 + RP < S::F1) ? r0 + RP : S::F1;
                    float acc[VEC];
#pragma unroll
                    for (int e = 0; e < VEC; ++e) acc[e] = 0.0f;
                    float wa[10][VEC], wb[10][VEC];
                    auto load = [&](float (&w)[10][VEC], int j0) {
#pragma unroll
                        for (int jj = 0; jj < 10; ++jj) {
                            const int j = j0 + jj;
                            const float *src = W + S::DF1 + (j < r1 ? j : r0) * S::NF1S + i0;
                            if (VEC == 4) {
                                f4 t = *(const f4 *)src;
#pragma unroll
                                for (int e = 0; e < VEC; ++e) w[jj][e] = t[e];
                            } else {
                                w[jj][0] = *src;
                            }
                        }
                    };
                    auto comp = [&](const float (&w)[10][VEC], int j0) {
#pragma unroll
                        for (int jj = 0; jj < 10; ++jj) {
                            if (j0 + jj < r1) {
                                const float d = sm.dh[j0 + jj];
#pragma unroll
                                for (int e = 0; e < VEC; ++e) acc[e] = fmaf(w[jj][e], d, acc[e]);
                            }
                        }
                    };
                    load(wa, r0);
                    for (int j0 = r0; j0 < r1; j0 += 20) {
                        if (j0 + 10 < r1) load(wb, j0 + 10);
                        comp(wa, j0);
                        if (j0 + 10 < r1) {
                            if (j0 + 20 < r1) load(wa, j0 + 20);
                            comp(wb, j0 + 10);
                        }
                    }
                    float *dst = (part == 0) ? sm.e2 : sm.e2b;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) dst[i0 + e] = acc[e];
                }
            }
            __syncthreads();
            // (wavefront w pushes rows j = w, w + 4, ...; lane l the inputs
            // l + 64c, so a push instruction covers up to 64 consecutive weights)
            {
                constexpr int IC = (S::NF1 + 63) / 64;
                float xv[IC];
#pragma unroll
                for (int c = 0; c < IC; ++c) {
                    int i = lane + 64 * c;
                    xv[c] = (i < S::NF1) ? sm.p2[i] : 0.0f;
                }
                for (int j = wave; j < S::F1; j += NW) {
                    const float d = sm.dh[j];
#pragma unroll
                    for (int c = 0; c < IC; ++c) {
                        int i = lane + 64 * c;
                        if (i < S::NF1) push(S::DF1 + j * S::NF1S + i, S::OF1 + j * S::NF1 + i, d * xv[c]);
                    }
                }
            }
            if (tid < S::F1) push(S::DBF1 + tid, S::OBF1 + tid, sm.dh[tid]);
        } else {
            // One pass: each FC1 push returns the weight it updated, this
            // layer's pre-update weight (Section III-A.2), so the errors
            // e2[i] = sum_j W[j][i] dh[j] need no separate read of the FC1
            // weights.  Wavefront w pushes rows j = w, w + 4, ... (lane l the
            // inputs l + 64c) and keeps a partial sum per input in the free
            // conv2 output buffer; the pool2 backward below adds the four in
            // wavefront order.
            constexpr int IC = (S::NF1 + 63) / 64;
            float xv[IC], ep[IC];
#pragma unroll
            for (int c = 0; c < IC; ++c) {
                int i = lane + 64 * c;
                xv[c] = (i < S::NF1) ? sm.p2[i] : 0.0f;
                ep[c] = 0.0f;
            }
            // The wavefront's rows j = wave + NW r in half-steps of HR rows
            // (IC HR returning pushes each): the next half-step's pushes are
            // issued before the current one's returns are summed, so about
            // 2 IC HR stay in flight throughout (a row is summed once all its
            // returns are in, rows in increasing order; scheduling barriers
            // keep the half-steps in this order).
            constexpr int R = (64 / IC < 16) ? 64 / IC : 16, HR = R / 2;
            constexpr int NR = (S::F1 + NW - 1) / NW, NH = (NR + HR - 1) / HR;
            static_assert(HR >= 1 && NH >= 2, "at least two half-steps");
            float oA[HR][IC], oB[HR][IC];
            auto issue = [&](float (&o)[HR][IC], int r0) {
#pragma unroll
                for (int r = 0; r < HR; ++r) {
                    const int jr = wave + NW * (r0 + r);
                    const float d = (jr < S::F1) ? sm.dh[jr] : 0.0f;
#pragma unroll
                    for (int c = 0; c < IC; ++c) {
                        const int i = lane + 64 * c;
                        o[r][c] = (jr < S::F1 && i < S::NF1)
                                      ? push_now.with_old(S::DF1 + jr * S::NF1S + i, S::OF1 + jr * S::NF1 + i, d * xv[c])
                                      : 0.0f;
                    }
                }
            };
            auto consume = [&](const float (&o)[HR][IC], int r0) {
#pragma unroll
                for (int r = 0; r < HR; ++r) {
                    const int jr = wave + NW * (r0 + r);
                    const float d = (jr < S::F1) ? sm.dh[jr] : 0.0f;
#pragma unroll
                    for (int c = 0; c < IC; ++c) ep[c] = fmaf(o[r][c], d, ep[c]);
                }
            };
            issue(oA, 0);
            int h = 0;
#pragma unroll 1
            for (; h + 2 < NH; h += 2) {
                __builtin_amdgcn_sched_barrier(0);
                issue(oB, (h + 1) * HR);
                __builtin_amdgcn_sched_barrier(0);
                consume(oA, h * HR);
                __builtin_amdgcn_sched_barrier(0);
                issue(oA, (h + 2) * HR);
                __builtin_amdgcn_sched_barrier(0);
                consume(oB, (h + 1) * HR);
            }
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (NH % 2 == 0) {
                issue(oB, (NH - 1) * HR);
                __builtin_amdgcn_sched_barrier(0);
                consume(oA, (NH - 2) * HR);
                __builtin_amdgcn_sched_barrier(0);
                consume(oB, (NH - 1) * HR);
            } else {
                consume(oA, (NH - 1) * HR);
            }
#pragma unroll
            for (int c = 0; c < IC; ++c) {
                int i = lane + 64 * c;
                if (i < S::NF1) sm.y2[wave * S::NF1 + i] = ep[c];
            }
            if (tid < S::F1) push(S::DBF1 + tid, S::OBF1 + tid, sm.dh[tid]);
        }
        __syncthreads();
        // pool2 backward -> dense conv2 deltas: a thread per pooled output
        // writes its whole 3x3 window (the delta at the first maximum, zeros
        // elsewhere; the windows tile the 9x9 map); the buffer's padding
        // (positions 81..D2S-1 of every map, maps C2..C2P-1) is zeroed apart.
        // Then clear e1.
        for (int q = tid; q < S::NF1; q += NT) {
            const int o = q / S::NP2, P = q - o * S::NP2, py = P / 3, px = P - 3 * py;
            float e;
            if constexpr (kFc1Read)
                e = (S::FC1_VEC == 4) ? sm.e2[q] + sm.e2b[q] : sm.e2[q];
            else
                e = ((sm.y2[q] + sm.y2[S::NF1 + q]) + sm.y2[2 * S::NF1 + q]) + sm.y2[3 * S::NF1 + q];
            const float d = e * dact_from_y(sm.p2[q]);
            const int ag = sm.am2[q];
            float *dst = sm.d2 + o * D2S + 3 * py * S::H2 + 3 * px;
#pragma unroll
            for (int w = 0; w < 9; ++w) dst[(w / 3) * S::H2 + w % 3] = (w == ag) ? d : 0.0f;
        }
        {
            constexpr int TAIL = D2S - S::NY2, NPAD = S::C2 * TAIL + (S::C2P - S::C2) * D2S;
            for (int t = tid; t < NPAD; t += NT) {
                const int o = t / TAIL;
                sm.d2[(t < S::C2 * TAIL) ? o * D2S + S::NY2 + (t - o * TAIL) : S::C2 * D2S + (t - S::C2 * TAIL)] = 0.0f;
            }
        }
        for (int t = tid; t < S::C1 * S::NP1; t += NT) sm.e1[t] = 0.0f;
        __syncthreads();

        // ---- conv2 backward data: C[(c,u,v)][p] = sum_o W2[o][c][u][v] d2[o][p],
        //      col2im into e1[c][p + (u,v)]. ----
        // One input map alone: rows uv = 16t + q (two tiles).  The four
        // lane groups of an accumulator element then hold four (u,v) of
        // the same map, so each scatter step is done one lane group at a
        // time (plain read-add-write, groups kept in order).
        auto map1 = [&](const int c) {
            f4 acc[2][RT2];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int j = 0; j < RT2; ++j) acc[t][j] = f4{0.f, 0.f, 0.f, 0.f};
            // a step's weights and deltas are read a step ahead, from clamped
            // addresses (the matrix instructions, behind a scheduling barrier,
            // wait for their own step's reads alone).  No operand needs
            // zeroing: a weight row past 25 feeds an output row never
            // scattered, and the deltas of maps C2..C2P-1 are zero.
            float aA[2], aB[2], bA[RT2], bB[RT2];
            auto load = [&](float (&av)[2], float (&bv)[RT2], int ks) {
                const int o = 4 * ks + lg;
                const float *w2 = W2 + (o < S::C2 ? o : 0) * S::W2S + c * 25;
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int uv = 16 * t + lr;
                    av[t] = w2[uv < 25 ? uv : 0];
                }
#pragma unroll
                for (int j = 0; j < RT2; ++j) bv[j] = sm.d2[o * D2S + 16 * j + lr];  // o < C2P: in the buffer
            };
            auto compute = [&](const float (&av)[2], const float (&bv)[RT2]) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int j = 0; j < RT2; ++j) acc[t][j] = mfma(av[t], bv[j], acc[t][j]);
            };
            load(aA, bA, 0);
#pragma unroll
            for (int ks = 0; ks < S::OKS; ks += 2) {
                if (ks + 1 < S::OKS) load(aB, bB, ks + 1);
                compute(aA, bA);
                if (ks + 1 < S::OKS) {
                    if (ks + 2 < S::OKS) load(aA, bA, ks + 2);
                    compute(aB, bB);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            float *dp[RT2];
#pragma unroll
            for (int j = 0; j < RT2; ++j) {
                const int p = 16 * j + lr;
                const int py = p / S::H2, px = p - py * S::H2;
                dp[j] = (p < S::NY2) ? sm.e1 + c * S::NP1 + py * S::Q1 + px : sm.sink;
            }
            // each step serves one lane group
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int uv = 16 * t + 4 * g + r, u = uv / 5, v = uv - 5 * u;
                        if (uv >= 25) continue;
                        if (lg == g) {
                            float cv[RT2];
#pragma unroll
                            for (int j = 0; j < RT2; ++j) cv[j] = acc[t][j][r];
                            scatter_add<RT2>(dp, u * S::Q1 + v, cv);
                        } else {
                            wave_lds_order();
                        }
                    }
        };
        // Input maps in blocks of 4, a block owned by one wavefront.  Row q of
        // tile i holds map c0 + q/4 at uv = 4i + q%4, so the four lane groups
        // of an accumulator element hold four different maps at one (u,v): a
        // scatter instruction never has two lanes on one address, and
        // wave_lds_order() keeps the overlapping groups in order (plain
        // read-add-write, no atomics).  Seven row tiles per block.
        // (passes of four tiles; of two for the small net, whose three
        // workers per CU have a third of the registers)
        auto block4 = [&](const int c0) {
            constexpr int TI = S::STAGE ? 2 : 4, NPASS = (7 + TI - 1) / TI;
#pragma unroll
            for (int pass = 0; pass < NPASS; ++pass) {
                const int i0 = TI * pass, nt = (7 - i0 < TI) ? 7 - i0 : TI;
                f4 acc[TI][RT2];
#pragma unroll
                for (int t = 0; t < TI; ++t)
#pragma unroll
                    for (int j = 0; j < RT2; ++j) acc[t][j] = f4{0.f, 0.f, 0.f, 0.f};
                int wo[TI];  // offset of this lane's row in a weight row, or -1
#pragma unroll
                for (int t = 0; t < TI; ++t) {
                    const int uv = 4 * (i0 + t) + (lr & 3);
                    wo[t] = (t < nt && uv < 25) ? (c0 + (lr >> 2)) * 25 + uv : -1;
                }
                // the next output maps' weights and deltas are read while the
                // current ones compute (as in map1: no operand needs zeroing)
                float aA[TI], aB[TI], bA[RT2], bB[RT2];
                auto load = [&](float (&av)[TI], float (&bv)[RT2], int ks) {
                    const int o = 4 * ks + lg;
                    const float *w2 = W2 + (o < S::C2 ? o : 0) * S::W2S;
#pragma unroll
                    for (int t = 0; t < TI; ++t) av[t] = w2[wo[t] >= 0 ? wo[t] : 0];
#pragma unroll
                    for (int j = 0; j < RT2; ++j) bv[j] = sm.d2[o * D2S + 16 * j + lr];  // o < C2P: in the buffer
                };
                auto compute = [&](const float (&av)[TI], const float (&bv)[RT2]) {
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int t = 0; t < TI; ++t)
#pragma unroll
                        for (int j = 0; j < RT2; ++j) acc[t][j] = mfma(av[t], bv[j], acc[t][j]);
                };
                load(aA, bA, 0);
#pragma unroll
                for (int ks = 0; ks < S::OKS; ks += 2) {
                    if (ks + 1 < S::OKS) load(aB, bB, ks + 1);
                    compute(aA, bA);
                    if (ks + 1 < S::OKS) {
                        if (ks + 2 < S::OKS) load(aA, bA, ks + 2);
                        compute(aB, bB);
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
                float *dp[RT2];
#pragma unroll
                for (int j = 0; j < RT2; ++j) {
                    const int p = 16 * j + lr;
                    const int py = p / S::H2, px = p - py * S::H2;
                    dp[j] = (p < S::NY2) ? sm.e1 + (c0 + lg) * S::NP1 + py * S::Q1 + px : sm.sink;
                }
#pragma unroll
                for (int t = 0; t < TI; ++t)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int uv = 4 * (i0 + t) + r, u = uv / 5, v = uv - 5 * u;
                        if (t >= nt || uv >= 25) continue;
                        float c[RT2];
#pragma unroll
                        for (int j = 0; j < RT2; ++j) c[j] = acc[t][j][r];
                        scatter_add<RT2>(dp, u * S::Q1 + v, c);
                    }
            }
        };

        // The conv2 bias gradients are collected in gb, the FC activations'
        // buffer (free once the FC gradients are pushed), and pushed together
        // by consecutive threads: one push instruction per bias block, as for
        // every other block of weights (single-lane pushes to the same few
        // lines would queue behind each other at the memory side).
        float *gb = sm.h;  // the conv2 bias gradients
        static_assert(S::C2 <= S::F1 + 16, "bias sums fit in the FC activations' buffer");

        // ---- conv2 weight gradient: G[o][k] = sum_p d2[o][p] p1col[p][k],
        //      pushed, in passes of JW column tiles of 16 k (JW * CT2
        //      accumulators keep the matrix core busy).  The first padding
        //      column k = KC2 multiplies the deltas by ones: its entries are
        //      the bias gradients, each map's deltas summed over the 81
        //      positions. ----
        constexpr int NJT = S::KC2P / 16, JW = 4;
        static_assert(NJT % JW == 0, "whole passes");
        static_assert(S::KC2 < S::KC2P, "a padding column holds the bias gradients");
        // input offset of output position p = 4s + lg (or -1 past the map)
        auto pb = [&](int s) {
            const int p = 4 * s + lg, py = p / S::H2, px = p - py * S::H2;
            return (p < S::NY2) ? py * S::Q1 + px : -1;
        };
        auto wgrad_pass = [&](const int jt0, const float (&ad)[S::CT2][21]) {
            const float *pc[JW];
            bool kv[JW], one[JW];
#pragma unroll
            for (int b = 0; b < JW; ++b) {
                const int k = 16 * (jt0 + b) + lr;
                kv[b] = k < S::KC2;
                one[b] = k == S::KC2;
                // the ones column reads ones; the other padding columns read
                // valid inputs into outputs never pushed
                pc[b] = one[b] ? (const float *)sm.ones : sm.p1 + (kv[b] ? sm.koff2[k] : 0);
            }
            f4 acc[JW][S::CT2];
#pragma unroll
            for (int b = 0; b < JW; ++b)
#pragma unroll
                for (int i = 0; i < S::CT2; ++i) acc[b][i] = f4{0.f, 0.f, 0.f, 0.f};
            // operands: LDS reads from a clamped address (a position past the
            // map reads a valid input, and its deltas, the A operand, are the
            // zeros of the delta rows' padding); the next step's reads are
            // issued before this step's matrix instructions, which then wait
            // for this step's alone
            auto load = [&](float (&bv)[JW], int s) {
                const int q = pb(s);  // -1 past the map
#pragma unroll
                for (int b = 0; b < JW; ++b) bv[b] = pc[b][q >= 0 ? q : 0];
            };
            auto step = [&](const float (&bv)[JW], int s) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int b = 0; b < JW; ++b)
#pragma unroll
                    for (int i = 0; i < S::CT2; ++i) acc[b][i] = mfma(ad[i][s], bv[b], acc[b][i]);
            };
            float bA[JW], bB[JW];
            load(bA, 0);
#pragma unroll
            for (int s = 0; s < 21; s += 2) {
                if (s + 1 < 21) load(bB, s + 1);
                step(bA, s);
                if (s + 1 < 21) {
                    if (s + 2 < 21) load(bA, s + 2);
                    step(bB, s + 1);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int b = 0; b < JW; ++b) {
                const int k = 16 * (jt0 + b) + lr;
                if (kv[b]) {
#pragma unroll
                    for (int i = 0; i < S::CT2; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            int o = 16 * i + 4 * lg + r;
                            if (o < S::C2) push(S::DW2 + o * S::KC2S + k, S::OW2 + o * S::KC2 + k, acc[b][i][r]);
                        }
                } else if (one[b]) {
#pragma unroll
                    for (int i = 0; i < S::CT2; ++i)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            int o = 16 * i + 4 * lg + r;
                            if (o < S::C2) gb[o] = acc[b][i][r];
                        }
                }
            }
        };
        // this wavefront's weight-gradient passes (every jt0 = first + step * n)
        auto conv2_wgrad = [&](const int first, const int step) {
            float ad[S::CT2][21];
#pragma unroll
            for (int i = 0; i < S::CT2; ++i)
#pragma unroll
                for (int s = 0; s < 21; ++s) ad[i][s] = sm.d2[(16 * i + lr) * D2S + 4 * s + lg];
            for (int jt0 = first; jt0 < NJT; jt0 += step) wgrad_pass(jt0, ad);
        };
        if constexpr (S::STAGE) {
            // Small net: backward data and weight gradient in one phase.  They
            // read the same deltas and write different places: backward data
            // the pool1 errors in LDS, from this sample's LDS copy of the
            // weights (which the pushes do not touch); the weight gradient the
            // shared weights.  Wavefront 0 takes input maps 0..3 as a block,
            // wavefront 1 map 4 alone, wavefronts 2 and 3 the weight
            // gradient's column tiles and the biases.
            static_assert(S::C1 == 5 && NJT == 2 * JW, "small net: 5 input maps, two passes");
            if (wave == 0) block4(0);
            else if (wave == 1) map1(4);
            else conv2_wgrad(JW * (wave - 2), 2 * JW);
        } else {
            if constexpr (S::C1 == 5 * NW) {
                // five maps per wavefront: a 4-map block and one map alone
                block4(5 * wave);
                map1(5 * wave + 4);
            } else if constexpr (S::C1 % 4 == 0) {
                for (int blk = wave; blk < S::C1 / 4; blk += NW) block4(4 * blk);
            } else {
                // wavefront w owns input maps w, w + 4, ...
                for (int c = wave; c < S::C1; c += NW) map1(c);
            }
            conv2_wgrad(JW * wave, NW * JW);
        }
        __syncthreads();

        // ---- conv1 weight gradient G[o][uv] = sum over the 26x26 conv1 outputs
        //      of the delta times the input under the kernel, on the matrix
        //      cores: rows o, cols uv = 4u + v, K = 4P + w with the pooled
        //      positions P split over the wavefronts; the partial tiles are
        //      summed in wavefront order (through the free delta buffer).  The
        //      delta is nonzero only at each pooling window's maximum, where it
        //      is the pool1 error times f' of the pool1 value (pool1 backward,
        //      formed as the operands are read). ----
        {
            f4 acc[2][S::CT1];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int t = 0; t < S::CT1; ++t) acc[h][t] = f4{0.f, 0.f, 0.f, 0.f};
            int orow[S::CT1];
            bool ov[S::CT1];
#pragma unroll
            for (int t = 0; t < S::CT1; ++t) {
                ov[t] = 16 * t + lr < S::C1;
                orow[t] = (ov[t] ? 16 * t + lr : 0) * S::NP1;
            }
            const int xo = ((lg >> 1) + (lr >> 2)) * S::IN + (lg & 1) + (lr & 3);
            // operands of pooled position P, read a position ahead of their use
            auto operands = [&](int P, float &bx, float (&av)[S::CT1]) {
                const int py = P / S::Q1, px = P - py * S::Q1;
                bx = sm.x[2 * py * S::IN + 2 * px + xo];
#pragma unroll
                for (int t = 0; t < S::CT1; ++t) {
                    const int am = sm.am1[orow[t] + P];  // orow 0 when the map is past C1
                    const float e = sm.e1[orow[t] + P], y = sm.p1[orow[t] + P];
                    av[t] = (ov[t] && am == lg) ? e * dact_from_y(y) : 0.0f;
                }
            };
            auto compute = [&](const float bx, const float (&av)[S::CT1], f4 (&c)[S::CT1]) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < S::CT1; ++t) c[t] = mfma(av[t], bx, c[t]);
            };
            // acc[0] takes positions wave, wave + 2 NW, ...; acc[1] wave + NW,
            // ...; the operands of the next four positions are read while the
            // current four compute.  The conv1 bias gradients are summed from
            // the same operands: per lane over its positions, then over the
            // four lane groups and (after the barrier) the wavefronts in order.
            float bxC[4], avC[4][S::CT1], bxN[4], avN[4][S::CT1], bsum[S::CT1];
#pragma unroll
            for (int t = 0; t < S::CT1; ++t) bsum[t] = 0.0f;
            auto load4 = [&](int P0, float (&bx)[4], float (&av)[4][S::CT1]) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int P = P0 + NW * u;
                    operands(P < S::NP1 ? P : S::NP1 - 1, bx[u], av[u]);
                }
            };
            load4(wave, bxC, avC);
            for (int P0 = wave; P0 < S::NP1; P0 += 4 * NW) {
                load4(P0 + 4 * NW, bxN, avN);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (P0 + NW * u < S::NP1) {
                        compute(bxC[u], avC[u], acc[u & 1]);
#pragma unroll
                        for (int t = 0; t < S::CT1; ++t) bsum[t] += avC[u][t];
                    }
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    bxC[u] = bxN[u];
#pragma unroll
                    for (int t = 0; t < S::CT1; ++t) avC[u][t] = avN[u][t];
                }
            }
            // the conv2 biases summed in the previous phase
            if (tid < S::C2) push(S::DB2 + tid, S::OB2 + tid, gb[tid]);
            float *red = sm.d2;  // [wavefront][tile][lane][4], then [wavefront][CT1 * 16] bias sums
            float *redb = red + NW * S::CT1 * 256;
#pragma unroll
            for (int t = 0; t < S::CT1; ++t) {
                *(f4 *)(red + ((wave * S::CT1 + t) * 64 + lane) * 4) = acc[0][t] + acc[1][t];
                const float b1 = bsum[t] + __shfl_xor(bsum[t], 16, 64);
                const float b2 = b1 + __shfl_xor(b1, 32, 64);
                if (lg == 0) redb[wave * S::CT1 * 16 + 16 * t + lr] = b2;
            }
            __syncthreads();
            // weights and biases of conv1, consecutive in memory, one block
            for (int t = tid; t < S::C1 * 16 + S::C1; t += NT) {
                if (t < S::C1 * 16) {
                    const int o = t >> 4, uv = t & 15, tile = o >> 4, row = o & 15;
                    const int e = ((row >> 2) * 16 + uv) * 4 + (row & 3);
                    float g = red[(0 * S::CT1 + tile) * 256 + e];
#pragma unroll
                    for (int w = 1; w < NW; ++w) g += red[(w * S::CT1 + tile) * 256 + e];
                    push(S::DW1 + t, S::OW1 + t, g);
                } else {
                    const int o = t - S::C1 * 16;
                    float g = redb[o];
#pragma unroll
                    for (int w = 1; w < NW; ++w) g += redb[w * S::CT1 * 16 + o];
                    push(S::DB1 + o, S::OB1 + o, g);
                }
            }
        }
        if constexpr (DELAY) {
            if (++nproc % a.push_delay == 0) {
                __syncthreads();
                flush();
            }
        }
        if (kTrain && tid == 0) atomicAdd(a.counter + 1, 1);  // samples completed
        if (kReplicas) {
            // every refresh_every-th sample completed on this replica: once
            // this worker's pushes have landed, copy the shared weights into it
            // (relaxed agent-scope stores, performed where the pushes are; a
            // concurrent push to the replica that the copy overwrites is in the
            // shared weights and returns with the next copy)
            if (tid == 0) {
                const int r = blockIdx.x % a.n_replicas;
                sm.rep_refresh = (atomicAdd(a.rep_counter + r, 1) % a.refresh_every) == a.refresh_every - 1;
            }
            __syncthreads();
            if (sm.rep_refresh) {
                wait_vector_memory();
                __syncthreads();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                for (int i = tid; i < S::NDEV; i += NT)
                    __hip_atomic_store(rep + i, __hip_atomic_load(Wg + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        __syncthreads();
    }
}

using Small = Cpcp<5, 10, 50>;
using Medium = Cpcp<20, 40, 150>;
static_assert(Small::NPARAM == 6405 && Medium::NPARAM == 76040, "Table I weight counts");
static_assert(NW * Small::NF1 <= Small::C2 * Small::NY2 && NW * Medium::NF1 <= Medium::C2 * Medium::NY2,
              "FC1 partial sums fit in the conv2 output buffer");
static_assert(NW * Small::CT1 * 272 <= Small::C2P * D2S && NW * Medium::CT1 * 272 <= Medium::C2P * D2S,
              "conv1 partial tiles and bias sums fit in the delta buffer");

template <class S, int MINB>
hipError_t launch_cpcp(int mode, const WorkArgs &a, int grid, hipStream_t s) {
    switch (mode) {
    case kTrainAtomic: fused_cpcp_kernel<S, kTrainAtomic, MINB><<<grid, NT, 0, s>>>(a); break;
    case kTrainRacy: fused_cpcp_kernel<S, kTrainRacy, MINB><<<grid, NT, 0, s>>>(a); break;
    case kForwardBackward: fused_cpcp_kernel<S, kForwardBackward, MINB><<<grid, NT, 0, s>>>(a); break;
    case kEvaluate: fused_cpcp_kernel<S, kEvaluate, MINB><<<grid, NT, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <class S, int MINB>
int cpcp_blocks_per_cu() {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &nb, fused_cpcp_kernel<S, kTrainAtomic, MINB>, NT, 0) != hipSuccess)
        return 0;
    return nb;
}

constexpr int kSmallMinBlocks = 3, kMediumMinBlocks = Medium::STAGE2 ? 1 : 2;
constexpr int kSmallDelayMinBlocks = 2;  // the gradient sum takes another 25.6 KB
static_assert(sizeof(SmemCpcp<Small>) * kSmallMinBlocks <= 160 * 1024 &&
                  sizeof(SmemCpcp<Medium>) * kMediumMinBlocks <= 160 * 1024 &&
                  sizeof(SmemCpcp<Small, true>) * kSmallDelayMinBlocks <= 160 * 1024,
              "resident workers per CU fit in the LDS");

bool matches(const Net &net, int c1, int c2, int f1) {
    const int spec[6][3] = {{kConv, c1, 4}, {kPool, 0, 2}, {kConv, c2, 5},
                            {kPool, 0, 3},  {kFc, f1, 0},  {kFc, 10, 0}};
    if (net.n_layers != 6 || net.in_size != 29 * 29) return false;
    if (net.L[0].hin != 29 || net.L[0].win != 29) return false;
    for (int l = 0; l < 6; ++l) {
        const Layer &ly = net.L[l];
        if (ly.kind != spec[l][0]) return false;
        if (ly.kind != kFc && ly.k != spec[l][2]) return false;
        if (ly.kind != kPool && ly.cout != spec[l][1]) return false;
    }
    return true;
}

} // namespace

int fused_cpcp_variant(const Net &net) {
    if (matches(net, Small::C1, Small::C2, Small::F1)) return 1;
    if (matches(net, Medium::C1, Medium::C2, Medium::F1)) return 2;
    return 0;
}

namespace {
template <class S>
bool cpcp_layout(ParamLayout &L) {
    if (!S::PAD) return false;
    const ParamSegment seg[] = {
        {S::OW1, S::DW1, 1, S::C1 * 16, S::C1 * 16}, {S::OB1, S::DB1, 1, S::C1, S::C1},
        {S::OW2, S::DW2, S::C2, S::KC2, S::KC2S},    {S::OB2, S::DB2, 1, S::C2, S::C2},
        {S::OF1, S::DF1, S::F1, S::NF1, S::NF1S},    {S::OBF1, S::DBF1, 1, S::F1, S::F1},
        {S::OF2, S::DF2, S::F2, S::F1, S::F1S},      {S::OBF2, S::DBF2, 1, S::F2, S::F2}};
    constexpr int n = sizeof(seg) / sizeof(seg[0]);
    static_assert(n <= kMaxSegments, "segment table size");
    L.n_seg = n;
    L.n_dev = S::NDEV;
    for (int s = 0; s < n; ++s) L.seg[s] = seg[s];
    return true;
}
} // namespace

bool fused_cpcp_layout(int variant, ParamLayout &L) {
    if (variant == 1) return cpcp_layout<Small>(L);
    if (variant == 2) return cpcp_layout<Medium>(L);
    return false;
}

hipError_t launch_fused_cpcp(int variant, int mode, const WorkArgs &a, int grid, hipStream_t s) {
    if (variant == 1 && mode == kTrainAtomic && a.push_delay > 1) {
        fused_cpcp_kernel<Small, kTrainAtomic, kSmallDelayMinBlocks, true><<<grid, NT, 0, s>>>(a);
        return hipGetLastError();
    }
    if (variant == 1) return launch_cpcp<Small, kSmallMinBlocks>(mode, a, grid, s);
    if (variant == 2) return launch_cpcp<Medium, kMediumMinBlocks>(mode, a, grid, s);
    return hipErrorInvalidValue;
}

int fused_cpcp_blocks_per_cu(int variant) {
    if (variant == 1) return cpcp_blocks_per_cu<Small, kSmallMinBlocks>();
    if (variant == 2) return cpcp_blocks_per_cu<Medium, kMediumMinBlocks>();
    return 0;
}

bool fused_cpcp_supports_replicas(int variant) { return variant == 1 && Small::STAGE; }

int fused_cpcp_delay_blocks_per_cu(int variant) {
    if (variant != 1) return 0;
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &nb, fused_cpcp_kernel<Small, kTrainAtomic, kSmallDelayMinBlocks, true>, NT, 0) !=
        hipSuccess)
        return 0;
    return nb;
}

} // namespace chaos
