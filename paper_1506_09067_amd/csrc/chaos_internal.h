// Internal descriptors shared by the host API (chaos_api.hip) and the kernels.
// Plain data only: the net descriptor is passed to kernels by value.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace chaos {

constexpr int kMaxLayers = 16;
enum LayerKind { kConv = 1, kPool = 2, kFc = 3 };

// One layer after the shape walk.  Offsets index the shared parameter vector
// (w_off, b_off) or one worker's scratch area (y_off, d_off, arg_off), in
// floats.
struct Layer {
    int kind, k;
    int cin, hin, win;    // input shape; FC: cin = flattened size, hin = win = 1
    int cout, hout, wout; // output shape; FC: cout = neurons, hout = wout = 1
    int nin, nout;        // element counts of input and output
    int w_off, b_off, nw, nb;
    int y_off;            // layer output values y
    int d_off;            // conv/FC: f'(z) of the outputs
    int arg_off;          // pool: flat input index of each window's maximum
};

struct Net {
    int n_layers;
    int in_size;          // in_h * in_w
    int n_out;            // size of the last layer's output
    int n_params;
    int e_max;            // largest layer input/output size
    int e_off0, e_off1;   // two error buffers of e_max floats
    int scratch_floats;   // per-worker scratch size
    Layer L[kMaxLayers];
};

enum Mode { kTrainAtomic = 0, kTrainRacy = 1, kForwardBackward = 2, kEvaluate = 3 };

struct WorkArgs {
    float *params;
    const float *x;
    const int32_t *labels;
    int64_t n;
    float lr;
    int32_t *counter;      // training: [0] samples claimed, [1] samples completed
    float *scratch;        // [workers][scratch_floats]
    float *loss;           // [n] optional
    float *out;            // [n][n_out] optional
    float *grad_each;      // [n][n_params] optional
    float *grad_part;      // [workers][n_params] optional (frozen-weight sums)
    int32_t *n_wrong;      // [1] evaluation
    int32_t *claims;       // [n] optional debug claim counter
    int32_t push_delay;    // training: samples between a worker's pushes (1 = per layer)
    float *stash;          // frozen weights, large net: per-sample operands of the
                           // batched conv3 / FC1 weight gradients, or null
    float *replicas;       // atomic training, small net: [n_replicas][device floats]
                           // copies of the weights the workers read, or null
    int32_t *rep_counter;  // [n_replicas] samples completed per replica
    int32_t n_replicas;    // worker b reads replica b % n_replicas
    int32_t refresh_every; // a replica is copied from the shared weights after
                           // every refresh_every-th sample completed on it
};

// Device layout of a net's shared weights, as segments of the canonical
// vector: segment s holds rows r < rows of len floats, at can_off + r * len
// in the canonical layout and at dev_off + r * dev_stride on the device.
// The identity layout is one segment.  Device floats outside every segment
// are padding.
struct ParamSegment {
    int can_off, dev_off, rows, len, dev_stride;
};
constexpr int kMaxSegments = 12;
struct ParamLayout {
    int n_seg;
    int n_dev;  // device floats
    ParamSegment seg[kMaxSegments];
};

// Launchers (worker.hip).  Each returns the hipError_t of the launch.
hipError_t launch_worker(int mode, const Net &net, const WorkArgs &a, int grid, int block,
                         hipStream_t s);
hipError_t launch_fill_i32(int32_t *p, int32_t v, int64_t n, hipStream_t s);
hipError_t launch_fill_f32(float *p, float v, int64_t n, hipStream_t s);
hipError_t launch_reduce_partials(const float *part, int64_t rows, int64_t cols, float *dst,
                                  hipStream_t s);
hipError_t launch_axpy(float *w, const float *g, float alpha, int64_t n, hipStream_t s);
// canonical <-> device copies, and w_dev += alpha * g_canonical, under a layout
hipError_t launch_convert_params(const float *src, float *dst, const ParamLayout &L, int64_t n_can,
                                 bool to_device, hipStream_t s);
hipError_t launch_axpy_mapped(float *w_dev, const float *g_can, float alpha, const ParamLayout &L,
                              int64_t n_can, hipStream_t s);
hipError_t launch_mean(const float *v, int64_t n, float *dst, hipStream_t s);
hipError_t launch_count(const int32_t *src, float *dst, hipStream_t s);
// dst[c * n + i] = src[i] for every copy c < copies
hipError_t launch_replicate(const float *src, float *dst, int64_t n, int copies, hipStream_t s);
// dst[0] = 1 if val[0] is not finite or val[0] > ref[0], else 0 (all device scalars)
hipError_t launch_above(const float *val, const float *ref, float *dst, hipStream_t s);
// Occupancy of the worker kernel: resident blocks per CU for a given block size.
int worker_blocks_per_cu(int block);

// Fused MFMA worker for the large net (conv20k4, max2, conv60k3, conv100k6,
// max2, FC150, FC10 on 29x29 inputs); 256 threads per worker, no scratch.
bool fused_large_matches(const Net &net);
void fused_large_layout(ParamLayout &L);  // its padded device layout
hipError_t launch_fused_large(int mode, const WorkArgs &a, int grid, hipStream_t s);
int fused_large_blocks_per_cu();

// Fused MFMA worker for the large net of Table I (conv20k4, max1, conv60k5,
// max2, conv100k6, max2, FC150, FC10 on 29x29 inputs); 256 threads, no scratch.
bool fused_t1_matches(const Net &net);
void fused_t1_layout(ParamLayout &L);  // its padded device layout
hipError_t launch_fused_t1(int mode, const WorkArgs &a, int grid, hipStream_t s);
int fused_t1_blocks_per_cu();

// Batched conv3 and FC1 weight gradients of the large net over a frozen-
// weight batch (batch_grad.hip).  stash holds, for n samples, d3 [n][100][36],
// y2 [n][60][121], dh [n][150] and p3 [n][900] one after the other; part3
// receives batch_grad_chunks(n) partial rows of 100 x 2160 floats, partf as
// many of 150 x 900, one per chunk of samples (at least kBatchChunk).
constexpr int kBatchChunk = 64;
constexpr int64_t kStashFloats = 100 * 36 + 60 * 121 + 150 + 900;  // per sample
int64_t batch_grad_chunks(int64_t n);
hipError_t launch_batch_grad(const float *stash, int64_t n, float *part3, float *partf,
                             hipStream_t s);

// Fused MFMA workers for the Table I small (variant 1) and medium (variant 2)
// nets: conv C1@4x4, max2, conv C2@5x5, max3, FC F1, FC10 on 29x29 inputs.
int fused_cpcp_variant(const Net &net);  // 0 when the net is neither
// the variant's device layout; false (L untouched) when it is the canonical one
bool fused_cpcp_layout(int variant, ParamLayout &L);
hipError_t launch_fused_cpcp(int variant, int mode, const WorkArgs &a, int grid, hipStream_t s);
int fused_cpcp_blocks_per_cu(int variant);
// resident workers per CU of the small net's delayed-push kernel (0 for others)
int fused_cpcp_delay_blocks_per_cu(int variant);
// whether the variant's atomic training kernel can read weight replicas
bool fused_cpcp_supports_replicas(int variant);

} // namespace chaos
