// Batched weight gradients of the large net's conv3 and FC1 layers, for the
// frozen-weight gradient sum over a batch (the per-sample gradients of
// Section II-A, summed).  The per-sample kernel leaves, for every sample n,
// the conv3 output deltas d3[n][o][m], the conv3 inputs y2[n][c][p], the FC1
// deltas dh[n][j] and the FC1 inputs p3[n][i] in HBM; here the two weight
// gradients are contracted over the samples on the fp32 matrix cores:
//   conv3  G[o][k] = sum_n sum_m d3[n][o][m] * y2[n][koff(k) + pos(m)]
//          (k = (c,u,v), koff(k) = 121c + 11u + v, pos(m) the conv3 output
//          position of m = 4P + w: pooled position P, window element w)
//   FC1    G[j][i] = sum_n dh[n][j] * p3[n][i]
// The samples are split into fixed chunks (their size a function of the
// batch size only); each chunk's sums go to their own partial rows, which
// are added in chunk order afterwards, so the result does not depend on
// timing.
#include "chaos_internal.h"
#include "device_common.h"

namespace chaos {
namespace {

constexpr int C2 = 60, NY2 = 121, H2 = 11;  // conv3 input: 60 maps of 11x11
constexpr int C3 = 100, M3 = 36;            // conv3 output: 100 maps, 36 positions
constexpr int KC3 = C2 * 36;                // conv3 weights per map (c, u, v)
constexpr int F1 = 150, NF1 = 900;          // FC1 neurons and inputs
constexpr int NT = 256;

// ---- conv3 -----------------------------------------------------------------
// Workgroup: a block of all 100 maps (padded to 128) x 128 columns k, over
// one chunk of samples.  Wavefront w owns rows 64(w/2)..+63 and columns
// 64(w%2)..+63: 2 x 2 tiles of v_mfma_f32_32x32x2_f32.  Per sample the
// operands are staged in LDS: A[m][o] (the deltas, transposed) and B[m][j]
// (the inputs under column k0 + j at output position m), in two buffers:
// the next sample's are read from HBM and written to the other buffer while
// this one's matrix instructions run.
constexpr int BN3 = 128, RP3 = 128;
// row stride of the transposed deltas in LDS: the staging writes go down a
// column (consecutive m), and an odd stride spreads them over the banks
constexpr int RS3 = RP3 + 1;
constexpr int NB3 = (KC3 + BN3 - 1) / BN3;  // 17 column blocks

struct alignas(16) Smem3 {
    float a[2][M3][RS3];  // a[buf][m][o]: zero for C3 <= o < RP3
    float b[2][M3][BN3];  // b[buf][m][j]: zero for k0 + j >= KC3
    int koff[BN3];
};

__global__ void __launch_bounds__(NT) conv3_wgrad_batch(const float *__restrict__ d3,
                                                        const float *__restrict__ y2, int64_t n,
                                                        int chunk, float *__restrict__ part) {
    __shared__ Smem3 sm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int k0 = blockIdx.x * BN3;
    const int64_t s0 = (int64_t)blockIdx.y * chunk;
    const int64_t s1 = (s0 + chunk < n) ? s0 + chunk : n;
    for (int j = tid; j < BN3; j += NT) {
        const int k = k0 + j, c = k / 36, uv = k - 36 * c, u = uv / 6, v = uv - 6 * u;
        sm.koff[j] = (k < KC3) ? c * NY2 + u * H2 + v : -1;
    }
    // the padding rows of A stay zero
    for (int t = tid; t < 2 * M3 * (RP3 - C3); t += NT) {
        const int bm = t / (RP3 - C3), o = C3 + t - bm * (RP3 - C3);
        sm.a[bm / M3][bm % M3][o] = 0.0f;
    }
    __syncthreads();
    // this thread's staged elements: A entries t = tid + 256q (o-major as
    // stored: o = t / 36, m = t % 36); B entries e = tid + 256q (m-major)
    constexpr int QA = (C3 * M3 + NT - 1) / NT, QB = (M3 * BN3 + NT - 1) / NT;  // 15, 18
    int bo[QB];
#pragma unroll
    for (int q = 0; q < QB; ++q) {
        const int e = tid + NT * q, m = e / BN3, j = e - m * BN3;
        const int P = m >> 2, w = m & 3, py = P / 3, px = P - 3 * py;
        const int pos = (2 * py + (w >> 1)) * H2 + 2 * px + (w & 1);
        const int ko = sm.koff[j];
        bo[q] = (e < M3 * BN3 && ko >= 0) ? ko + pos : -1;
    }
    float ra[QA], rb[QB];
    auto fetch = [&](int64_t s) {
        const float *ds = d3 + s * (C3 * M3);
        const float *ys = y2 + s * (C2 * NY2);
#pragma unroll
        for (int q = 0; q < QA; ++q) {
            const int t = tid + NT * q;
            ra[q] = (t < C3 * M3) ? ds[t] : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) rb[q] = (bo[q] >= 0) ? ys[bo[q]] : 0.0f;
    };
    auto stage = [&](int buf) {
#pragma unroll
        for (int q = 0; q < QA; ++q) {
            const int t = tid + NT * q;
            if (t < C3 * M3) {
                const int o = t / M3, m = t - o * M3;
                sm.a[buf][m][o] = ra[q];
            }
        }
#pragma unroll
        for (int q = 0; q < QB; ++q) {
            const int e = tid + NT * q;
            if (e < M3 * BN3) (&sm.b[buf][0][0])[e] = rb[q];
        }
    };
    f16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f16{};
    const int r0 = 64 * (wave >> 1), c0 = 64 * (wave & 1);
    if (s0 < s1) {
        fetch(s0);
        stage(0);
    }
    __syncthreads();
    for (int64_t s = s0; s < s1; ++s) {
        const int buf = (int)(s - s0) & 1;
        if (s + 1 < s1) fetch(s + 1);
#pragma unroll
        for (int ks = 0; ks < M3 / 2; ++ks) {
            const int m = 2 * ks + (lane >> 5);
            float av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) av[i] = sm.a[buf][m][r0 + 32 * i + (lane & 31)];
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = sm.b[buf][m][c0 + 32 * j + (lane & 31)];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(av[i], bv[j], acc[i][j]);
        }
        // the other buffer was last read in the previous step, before the
        // barrier that ended it
        if (s + 1 < s1) stage(buf ^ 1);
        __syncthreads();
    }
    // part[chunk][o][k] for o < C3, k < KC3
    float *dst = part + (int64_t)blockIdx.y * (C3 * KC3);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int k = k0 + c0 + 32 * j + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int o = r0 + 32 * i + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
                if (o < C3 && k < KC3) dst[o * KC3 + k] = acc[i][j][r];
            }
        }
}

// ---- FC1 -------------------------------------------------------------------
// Wavefront: one 32 x 32 tile of G (rows j, columns i) over one chunk of
// samples, two samples per v_mfma_f32_32x32x2_f32 step, operands straight
// from HBM (32 consecutive floats per half-wavefront), eight steps ahead.
constexpr int TM1 = (F1 + 31) / 32, TN1 = (NF1 + 31) / 32;  // 5 x 29 tiles

__global__ void __launch_bounds__(64) fc1_wgrad_batch(const float *__restrict__ dh,
                                                      const float *__restrict__ p3, int64_t n,
                                                      int chunk, float *__restrict__ part) {
    const int lane = threadIdx.x;
    const int tm = blockIdx.x / TN1, tn = blockIdx.x - tm * TN1;
    const int j = 32 * tm + (lane & 31), i = 32 * tn + (lane & 31);
    const bool jv = j < F1, iv = i < NF1;
    const int64_t s0 = (int64_t)blockIdx.y * chunk;
    const int64_t s1 = (s0 + chunk < n) ? s0 + chunk : n;
    f16 acc = f16{};
    constexpr int D = 8;
    float a[D], b[D];
    auto fetch = [&](int q, int64_t s) {  // samples s (lanes 0-31) and s + 1 (lanes 32-63)
        const int64_t sl = s + (lane >> 5);
        const bool ok = sl < s1;
        a[q] = (ok && jv) ? dh[sl * F1 + j] : 0.0f;
        b[q] = (ok && iv) ? p3[sl * NF1 + i] : 0.0f;
    };
#pragma unroll
    for (int q = 0; q < D; ++q) fetch(q, s0 + 2 * q);
    for (int64_t s = s0; s < s1; s += 2 * D) {
#pragma unroll
        for (int q = 0; q < D; ++q) {
            acc = mfma32(a[q], b[q], acc);
            fetch(q, s + 2 * D + 2 * q);
        }
    }
    float *dst = part + (int64_t)blockIdx.y * (F1 * NF1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int jj = 32 * tm + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (jj < F1 && iv) dst[jj * NF1 + i] = acc[r];
    }
}

} // namespace

// Samples per chunk: about 30 chunks, so that the conv3 grid (17 column
// blocks per chunk, two workgroups per CU) fills the GPU in one round; at
// least kBatchChunk.  A function of n only, so the result is reproducible.
int64_t batch_grad_chunk(int64_t n) {
    const int64_t c = (n + 29) / 30;
    return c > kBatchChunk ? c : kBatchChunk;
}

int64_t batch_grad_chunks(int64_t n) {
    const int64_t c = batch_grad_chunk(n);
    return (n + c - 1) / c;
}

hipError_t launch_batch_grad(const float *stash, int64_t n, float *part3, float *partf,
                             hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t nc = batch_grad_chunks(n), chunk = batch_grad_chunk(n);
    if (nc > 65535 || chunk > INT32_MAX) return hipErrorInvalidValue;
    const float *d3 = stash;
    const float *y2 = stash + n * (int64_t)(C3 * M3);
    const float *dh = y2 + n * (int64_t)(C2 * NY2);
    const float *p3 = dh + n * (int64_t)F1;
    conv3_wgrad_batch<<<dim3(NB3, (unsigned)nc), NT, 0, s>>>(d3, y2, n, (int)chunk, part3);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    fc1_wgrad_batch<<<dim3(TM1 * TN1, (unsigned)nc), 64, 0, s>>>(dh, p3, n, (int)chunk, partf);
    return hipGetLastError();
}

} // namespace chaos
