/*
 * chaos.h -- C ABI of libchaos.so, the MI355X (gfx950) implementation of the
 * CHAOS per-sample back-propagation hot path (Controlled Hogwild with
 * Arbitrary Order of Synchronization; Viebke & Pllana, HPCC 2015).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every function returns an int status: CHAOS_OK (0) or a negative code.
 *    Nothing aborts or throws.  chaos_last_error() gives a message for the
 *    last failing call of the calling thread.
 *  - Argument and shape errors are detected on the host and returned before
 *    any work is enqueued.  Launch failures are reported as CHAOS_EDEVICE.
 *  - Pointers named *_dev are device pointers (hipMalloc'd or torch CUDA
 *    tensors) owned by the caller; *_host are host pointers.  All device
 *    work is enqueued on `stream` and is asynchronous: the caller
 *    synchronises (hipStreamSynchronize / torch.cuda.synchronize) before it
 *    reads results.  stream = NULL means the null stream.
 *  - One call at a time per chaos_net; different nets are independent.
 *  - Images are fp32, row-major [n][in_h * in_w]; labels int32 in
 *    [0, n_classes) where n_classes is the output size of the last layer.
 *    Labels live in device memory and are not range-checked: a label
 *    outside that range only ever enters comparisons (its one-hot target
 *    is all zeros and an evaluation counts the sample as wrong).
 *  - Canonical parameter layout (get/set, init, gradients): layers in order;
 *    conv: W[o][i][u][v] row-major then b[o]; fully connected: W[j][i] (i over
 *    the map-major flattened input) then b[j]; pooling layers hold nothing.
 */
#ifndef CHAOS_H
#define CHAOS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    CHAOS_OK = 0,
    CHAOS_EINVAL = -1,      /* null pointer, n < 0, unknown kind/mode, bad worker count  */
    CHAOS_ESHAPE = -2,      /* kernel > map, pool not dividing the map, n_params mismatch */
    CHAOS_ENOMEM = -3,      /* device or host allocation failed                          */
    CHAOS_EDEVICE = -4,     /* a HIP runtime error; text in chaos_last_error()            */
    CHAOS_EUNSUPPORTED = -5 /* a shape beyond the library's limits                      */
};

/* Layer kinds (Section II-A, Table I). */
enum { CHAOS_CONV = 1, CHAOS_MAXPOOL = 2, CHAOS_FC = 3 };

/* One layer of the architecture (Table I rows).
 *   CHAOS_CONV:    maps output maps, kernel x kernel weights per (output map,
 *                  input map) pair, valid cross-correlation, stride 1, every
 *                  output map connected to every input map, one bias per map.
 *   CHAOS_MAXPOOL: non-overlapping kernel x kernel max (stride = kernel; the
 *                  kernel must divide the map); maps is ignored; kernel 1 is
 *                  the identity.
 *   CHAOS_FC:      maps neurons, each connected to every input value, one bias.
 * Every conv and FC layer, the output layer included, applies the activation
 * f(z) = 1.7159 tanh(2z/3).  The first layer reads the image directly. */
typedef struct {
    int32_t kind;
    int32_t maps;
    int32_t kernel;
} chaos_layer;

/* Training modes of chaos_train_epoch (Section III-A).
 *   CHAOS_SEQUENTIAL      one worker, samples in index order: per-sample SGD.
 *   CHAOS_HOGWILD_ATOMIC  `workers` concurrent workers claim samples from a
 *                         shared counter (dynamic work-sharing, III-A.1) and
 *                         add their per-layer updates to the shared weights
 *                         with atomic fp32 adds (III-A.2, III-A.3).
 *   CHAOS_HOGWILD_RACY    as above, but each update is a plain load, fma and
 *                         store: concurrent updates to one weight may be lost. */
enum { CHAOS_SEQUENTIAL = 0, CHAOS_HOGWILD_ATOMIC = 1, CHAOS_HOGWILD_RACY = 2 };

typedef struct chaos_net chaos_net; /* opaque; owned by the library */

/* Build a net (Section II-A, Table I): walks the layer list from a 1 x in_h x
 * in_w input, allocates the shared weights on the current device and copies
 * init_params_host (n_params floats, canonical layout) into them.
 * n_params must equal the architecture's weight count (Table I "Weights"
 * summed over layers), else CHAOS_ESHAPE.  *out receives the handle.  The
 * library may hold the weights on the device in a padded layout of its own
 * (rows starting on 64-byte boundaries); every weight or gradient buffer
 * that crosses this interface is in the canonical layout. */
int chaos_create_net(int32_t in_h, int32_t in_w, const chaos_layer *layers, int32_t n_layers,
                     const float *init_params_host, int64_t n_params, chaos_net **out);

/* Free the net and every device buffer it owns.  NULL is accepted. */
int chaos_destroy_net(chaos_net *net);

/* Number of weights incl. biases (the Table I total), or a negative code. */
int64_t chaos_num_params(const chaos_net *net);

/* Output size of the last layer (the class count), or a negative code. */
int32_t chaos_num_outputs(const chaos_net *net);

/* Copy the shared weights to / from a device buffer of chaos_num_params()
 * floats in the canonical layout, on `stream`.  These are the network
 * instances' shared weights of Section III-A.1 (one copy that every worker
 * reads and updates); get is also how the intermediate results of a session
 * are serialized (the time model's term d, Section III-B), set how a run is
 * resumed from them.  dst_dev / src_dev: caller-owned, NULL is CHAOS_EINVAL. */
int chaos_get_params(const chaos_net *net, float *dst_dev, hipStream_t stream);
int chaos_set_params(chaos_net *net, const float *src_dev, hipStream_t stream);

/* Frozen-weight forward and back-propagation of n samples (Section II-A):
 * the weights are not modified.  Optional outputs, NULL = skip:
 *   out_dev        [n][n_classes]  last-layer outputs y
 *   loss_dev       [n]             E_i = 1/2 sum_k (y_k - t_k)^2, t one-hot
 *   grad_sum_dev   [n_params]      sum_i dE_i/dW, accumulated in a fixed
 *                                  order: bitwise reproducible run to run
 *   grad_each_dev  [n][n_params]   per-sample gradients
 * n = 0 writes zeros into grad_sum_dev and nothing else.  A gradient sum
 * uses net-owned partial sums allocated on first use (grown when a call
 * needs more); for the large net without grad_each_dev also 47.6 KB per
 * sample of per-sample operands, whose conv3 and FC1 weight gradients are
 * then contracted over the batch (CHAOS_ENOMEM if they cannot be had). */
int chaos_forward_backward(chaos_net *net, const float *x_dev, const int32_t *labels_dev,
                           int64_t n, float *out_dev, float *loss_dev, float *grad_sum_dev,
                           float *grad_each_dev, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * computation and outputs as chaos_forward_backward, with no hipMalloc,
 * hipFree or other allocating call.  A gradient sum keeps its per-worker
 * partial sums in a fixed 32 MiB array of device memory that the library
 * holds on every device it runs on until the process ends, instead of
 * net-owned buffers allocated on first use; it therefore runs at most
 * 32 MiB / (4 n_params) workers (small net 512, medium 110, large 23) and
 * the large net's conv3 and FC1 gradients are pushed per sample rather than
 * contracted over the batch.  The sum is bitwise reproducible from call to
 * call; it equals chaos_forward_backward's to rounding (a different fixed
 * order), outputs and losses are identical.  A net with more than 8,388,608
 * weights cannot take a gradient sum here (CHAOS_EUNSUPPORTED).  Every call
 * on one device shares that array: calls that overlap in time on one device
 * (different streams, threads or nets) race and give wrong sums; calls
 * ordered on one stream are safe.  The array is cleared by a kernel at the
 * start of each call (no memset node when captured). */
int chaos_forward_backward_noalloc(chaos_net *net, const float *x_dev, const int32_t *labels_dev,
                                   int64_t n, float *out_dev, float *loss_dev, float *grad_sum_dev,
                                   float *grad_each_dev, hipStream_t stream);

/* The weight update of Section II-A: each weight moves against its partial
 * derivative of the error, scaled by the factor the paper calls the decay
 * (lambda) and this library the learning rate: W <- W - lr * grad_dev.
 * grad_dev: n_params floats, canonical layout, caller-owned (for example a
 * gradient sum from chaos_forward_backward, which makes one step of
 * mini-batch SGD); NULL is CHAOS_EINVAL.  Each weight is rounded to fp32 once
 * (one fused multiply-add). */
int chaos_apply_update(chaos_net *net, const float *grad_dev, float lr, hipStream_t stream);

/* One Training pass over x[0..n) (Section III-A.1 "Training"): each worker
 * repeatedly claims the next unprocessed sample (in index order), forward-
 * propagates it, computes the error against its label and back-propagates;
 * after each layer's gradients and the partial derivatives below it are
 * computed, that layer's shared weights receive W <- W - lr * g (Controlled
 * Hogwild, III-A.2) with no synchronisation between workers (Arbitrary Order
 * of Synchronization, III-A.3).  workers: number of concurrent workers for
 * the Hogwild modes (0 = chaos_default_workers(net)); ignored by
 * CHAOS_SEQUENTIAL.  Up to chaos_max_workers() the net's own kernel runs,
 * and the workers of an epoch join as its first samples complete (worker b
 * claims its first sample after b/4 samples have been completed), so that
 * their first gradients are not all taken at the same weights; above it, up
 * to chaos_worker_limit(), every worker is one 64-thread wavefront of the
 * generic kernel (per-worker state in HBM, allocated on first use), all
 * starting at once.  Larger values are CHAOS_EINVAL.
 * loss_dev [n] (optional): each sample's loss at the time it was processed. */
int chaos_train_epoch(chaos_net *net, const float *x_dev, const int32_t *labels_dev, int64_t n,
                      float lr, int32_t mode, int32_t workers, float *loss_dev,
                      hipStream_t stream);

/* Validation / Testing (Section III-A.1, Table II): forward only.
 * out_dev [n][n_classes] optional; n_wrong_dev [1] receives the number of
 * samples whose predicted class (lowest index among maximal outputs) differs
 * from the label (it is overwritten, not accumulated). */
int chaos_evaluate(chaos_net *net, const float *x_dev, const int32_t *labels_dev, int64_t n,
                   float *out_dev, int32_t *n_wrong_dev, hipStream_t stream);

/* A training session (Section III-A.1): for each epoch e = 0..epochs-1,
 * Training over x_train[0..n_train) (as chaos_train_epoch, with
 * lr = lr0 * decay^e computed in double and rounded to float), then
 * Validation on the training set and Testing on x_test[0..n_test) (forward
 * only, as chaos_evaluate).  stats_dev [epochs][5] floats receives per epoch:
 *   [0] mean training loss (each sample's loss when it was processed)
 *   [1] wrong predictions on the training set after the epoch (Validation)
 *   [2] wrong predictions on the test set (Testing, the Table II count)
 *   [3] mean test loss
 *   [4] divergence flag: 1 when the epoch's mean test loss (its mean
 *       training loss if n_test = 0) is not finite or above the mean loss of
 *       the same set at the session's starting weights, else 0.  A Hogwild
 *       run whose outputs saturate (the tanh units stuck at +-1.7159) is
 *       flagged instead of passing silently.
 * ckpt_dev (optional, NULL = skip) [epochs][n_params] receives the weights
 * after each epoch's Training, canonical layout: the per-epoch serialization
 * of intermediate results of the paper's time model (Section III-B, term d).
 * n_test may be 0 (then [2] and [3] are 0).  Before the first epoch one
 * forward/backward pass at the starting weights over the test set (the
 * training set if n_test = 0) gives the flag's reference.  Uses net-owned
 * buffers of max(n_train, n_test) floats, allocated on first use. */
int chaos_train_session(chaos_net *net, const float *x_train_dev, const int32_t *labels_train_dev,
                        int64_t n_train, const float *x_test_dev, const int32_t *labels_test_dev,
                        int64_t n_test, int32_t epochs, float lr0, float decay, int32_t mode,
                        int32_t workers, float *stats_dev, float *ckpt_dev, hipStream_t stream);

/* Concurrent Hogwild workers the net's own kernel keeps resident: the
 * counterpart of the paper's thread count, one
 * network instance per hardware thread (Section III-A.1; 244 threads on its
 * Xeon Phi), here one workgroup per in-flight sample.  Negative code on a
 * NULL net. */
int32_t chaos_max_workers(const chaos_net *net);

/* The worker count of chaos_train_epoch(workers = 0): one worker per compute
 * unit, at most chaos_max_workers().  Hogwild's updates are computed at
 * weights that miss the updates of every other sample in flight, and a net
 * whose every weight is touched by every sample (the small net of Table I)
 * trains stably at lr 1e-3 with 256 samples in flight but not always with
 * 512-768 (its early loss spikes and, in a few runs in a hundred, the tanh
 * outputs saturate for good); one sample per compute unit is the
 * concurrency at which every net here passes its acceptance.  Larger counts
 * up to chaos_max_workers() stay available explicitly.  Negative code on a
 * NULL net. */
int32_t chaos_default_workers(const chaos_net *net);

/* Largest accepted worker count: one-wavefront workers of the generic kernel,
 * up to 32 per compute unit (>= chaos_max_workers).  It bounds the thread
 * count sweep of Section IV-B (the paper runs 1 to 244 threads; the worker
 * counts above the resident ones are what the performance model of Section
 * III-C is asked to predict).  Negative code on a NULL net. */
int32_t chaos_worker_limit(const chaos_net *net);

/* Delayed pushes (a variant of the per-layer update, Section III-A.2, with
 * delayed sharing of locally accumulated updates): with k > 1, every worker
 * of a CHAOS_HOGWILD_ATOMIC epoch adds its per-layer gradients to a private
 * sum and pushes W <- W - lr * sum after every k-th sample it processes and
 * after its last; a worker does not see its own unpushed updates, so one
 * worker is mini-batch SGD with batches of k consecutive samples.  k = 1
 * (the default) is the per-layer push.  CHAOS_SEQUENTIAL and
 * CHAOS_HOGWILD_RACY epochs ignore the setting.  Only the small net of
 * Table I supports k > 1 (its weights and the sum fit in LDS), else
 * CHAOS_EUNSUPPORTED; k < 1 is CHAOS_EINVAL.  While k > 1,
 * chaos_max_workers() reports the delayed kernel's capacity and larger
 * worker counts are CHAOS_EINVAL. */
int chaos_set_push_delay(chaos_net *net, int32_t k);

/* Weight replicas (an update-path variant for nets whose every weight is
 * touched by every sample, Controlled Hogwild's delayed sharing applied to
 * the reads, Section III-A.2): with r > 1, each worker of a
 * CHAOS_HOGWILD_ATOMIC epoch reads its weights from replica (worker index
 * mod r) instead of the shared weights, pushes every update to the shared
 * weights and to that replica, and the replica is copied from the shared
 * weights after every m-th sample completed on it.  A worker then sees the
 * updates of workers on its replica at once and the others' after at most
 * about r * m further samples.  Every replica equals the shared weights at the
 * start of each epoch; the shared weights stay the result.  With one worker
 * this is sequential per-sample SGD bit for bit.  The memory side serializes
 * requests to one cache line, and every sample reads and adds into every
 * line of such a net's weights: r replicas spread those requests.  r = 1 (the
 * default) turns replicas off.  Only the small net of Table I supports r > 1
 * (its weights fit in LDS), else CHAOS_EUNSUPPORTED; r outside [1, 64] or
 * m < 1 is CHAOS_EINVAL, as is combining r > 1 with a push delay k > 1.
 * Allocates r copies of the weights (device memory owned by the net).
 * CHAOS_SEQUENTIAL and CHAOS_HOGWILD_RACY epochs ignore the setting, as do
 * worker counts above chaos_max_workers(). */
int chaos_set_replicas(chaos_net *net, int32_t r, int32_t m);

/* Debug aid: when claims_dev (int32 [n] of the next chaos_train_epoch) is not
 * NULL, every processed sample index i adds 1 to claims_dev[i]; NULL turns it
 * off.  The buffer must hold at least n entries for each later call. */
int chaos_set_claim_counter(chaos_net *net, int32_t *claims_dev);

/* Message of the last failing call on this thread ("" if none). */
const char *chaos_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CHAOS_H */
