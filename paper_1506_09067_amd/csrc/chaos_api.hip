// Host side of libchaos.so: argument validation, the shape walk of Table I,
// device memory owned by a net, and the launches behind every entry point
// declared in include/chaos.h.
#include "../../include/chaos.h"
#include "chaos_internal.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using chaos::Layer;
using chaos::Net;

struct chaos_net {
    int device = 0;
    Net desc{};
    int64_t n_params = 0;
    float *params = nullptr;      // shared weights, in the layout of the net's kernel
    chaos::ParamLayout layout{};  // canonical <-> device layout of params
    bool padded = false;          // layout is not the identity
    float *canon = nullptr;       // canonical copy for the generic kernel (padded nets)
    int block = 256;              // threads per worker
    bool fused = false;           // the fused large-net kernel serves this net
    bool t1 = false;              // the fused kernel of Table I's large net serves this net
    int cpcp = 0;                 // fused small (1) / medium (2) kernel serves this net
    int max_workers = 0;          // resident workers of the training kernel
    int cus = 0;                  // compute units of the device
    float *scratch = nullptr;     // [max_workers][scratch_floats]
    int32_t *counter = nullptr;   // [0] samples claimed, [1] samples completed (training)
    int fb_workers = 0;           // rows of grad_part
    float *grad_part = nullptr;   // [fb_workers][n_params]
    int32_t *claims = nullptr;    // debug claim counter (caller-owned)
    int worker_limit = 0;         // one-wavefront generic workers the device keeps resident
    float *wide_scratch = nullptr;  // [worker_limit][scratch_floats], allocated on first use
    float *sess_loss = nullptr;   // session: per-sample losses (training, then test)
    int64_t sess_loss_n = 0;
    int32_t *sess_wrong = nullptr;  // 64 bytes: [0] wrong count (int32), float [8] reference loss
    float *stash = nullptr;       // large net, batch gradient: per-sample conv3 / FC1 operands
    int64_t stash_n = 0;          // samples the stash holds
    float *bpart = nullptr;       // their chunk partial sums: conv3 rows, then FC1 rows
    int64_t bpart_chunks = 0;
    int push_delay = 1;           // samples between a worker's pushes (atomic Hogwild)
    int n_replicas = 1;           // weight replicas read by the workers (atomic Hogwild)
    int refresh_every = 1;        // samples per replica between its refreshes
    float *replicas = nullptr;    // [n_replicas][device floats]
    int32_t *rep_counter = nullptr;  // [n_replicas]
    int delay_max_workers = 0;    // resident workers of the delayed-push kernel (0 = none)
};

// Partial-sum rows of chaos_forward_backward_noalloc: a fixed array on every
// device the library runs on, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in for
// the symbol): the device address comes from hipGetSymbolAddress, once per
// device, and is what the kernels receive.
constexpr int64_t kNoAllocFloats = (int64_t)32 << 18;  // 32 MiB
static __device__ __align__(256) float scratch[kNoAllocFloats];

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int ok() {
    g_last_error.clear();
    return CHAOS_OK;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(CHAOS_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                                     \
    do {                                                        \
        hipError_t e_ = (expr);                                 \
        if (e_ != hipSuccess) return hip_fail(e_, what);        \
    } while (0)

constexpr int64_t kIntLimit = (int64_t)1 << 30;  // every per-net size must fit int32

// Shape walk (Section II-A, Table I) and per-worker scratch layout.
int build_desc(int32_t in_h, int32_t in_w, const chaos_layer *layers, int32_t n_layers, Net &net) {
    if (!layers) return fail(CHAOS_EINVAL, "layers is NULL");
    if (n_layers < 1 || n_layers > chaos::kMaxLayers)
        return fail(CHAOS_EINVAL, "n_layers=%d outside [1,%d]", n_layers, chaos::kMaxLayers);
    if (in_h < 1 || in_w < 1) return fail(CHAOS_EINVAL, "input %dx%d", in_h, in_w);
    std::memset(&net, 0, sizeof(net));
    int64_t c = 1, h = in_h, w = in_w, off = 0, scr = 0, emax = (int64_t)in_h * in_w;
    for (int l = 0; l < n_layers; ++l) {
        const chaos_layer &src = layers[l];
        Layer &ly = net.L[l];
        ly.kind = src.kind;
        ly.k = src.kernel;
        ly.cin = (int)c; ly.hin = (int)h; ly.win = (int)w;
        int64_t nw = 0, nb = 0;
        if (src.kind == CHAOS_CONV) {
            if (src.maps < 1 || src.kernel < 1)
                return fail(CHAOS_EINVAL, "layer %d: conv maps=%d kernel=%d", l, src.maps, src.kernel);
            if (src.kernel > h || src.kernel > w)
                return fail(CHAOS_ESHAPE, "layer %d: kernel %d larger than the %lldx%lld map", l,
                            src.kernel, (long long)h, (long long)w);
            ly.cout = src.maps;
            ly.hout = (int)(h - src.kernel + 1);
            ly.wout = (int)(w - src.kernel + 1);
            nw = (int64_t)src.maps * c * src.kernel * src.kernel;
            nb = src.maps;
        } else if (src.kind == CHAOS_MAXPOOL) {
            if (src.kernel < 1) return fail(CHAOS_EINVAL, "layer %d: pool kernel %d", l, src.kernel);
            if (h % src.kernel || w % src.kernel)
                return fail(CHAOS_ESHAPE, "layer %d: pool %d does not divide the %lldx%lld map", l,
                            src.kernel, (long long)h, (long long)w);
            ly.cout = (int)c;
            ly.hout = (int)(h / src.kernel);
            ly.wout = (int)(w / src.kernel);
        } else if (src.kind == CHAOS_FC) {
            if (src.maps < 1) return fail(CHAOS_EINVAL, "layer %d: fc neurons=%d", l, src.maps);
            if (c * h * w > kIntLimit)
                return fail(CHAOS_EUNSUPPORTED, "layer %d: fc input beyond 2^30", l);
            ly.cin = (int)(c * h * w); ly.hin = 1; ly.win = 1;
            ly.cout = src.maps; ly.hout = 1; ly.wout = 1;
            nw = (int64_t)src.maps * c * h * w;
            nb = src.maps;
        } else {
            return fail(CHAOS_EINVAL, "layer %d: unknown kind %d", l, src.kind);
        }
        const int64_t nin = (int64_t)ly.cin * ly.hin * ly.win;
        const int64_t nout = (int64_t)ly.cout * ly.hout * ly.wout;
        if (nw + nb + off > kIntLimit || nin > kIntLimit || nout > kIntLimit)
            return fail(CHAOS_EUNSUPPORTED, "layer %d: sizes beyond 2^30", l);
        ly.nin = (int)nin;
        ly.nout = (int)nout;
        ly.w_off = (int)off;
        ly.b_off = (int)(off + nw);
        ly.nw = (int)nw;
        ly.nb = (int)nb;
        off += nw + nb;
        ly.y_off = (int)scr;
        scr += ly.nout;
        if (ly.kind == CHAOS_MAXPOOL) {
            ly.arg_off = (int)scr;  // int32 indices stored in the float scratch
            scr += ly.nout;
            ly.d_off = -1;
        } else {
            ly.d_off = (int)scr;
            scr += ly.nout;
            ly.arg_off = -1;
        }
        emax = std::max<int64_t>(emax, std::max(ly.nin, ly.nout));
        c = ly.cout; h = ly.hout; w = ly.wout;
    }
    net.n_layers = n_layers;
    net.in_size = in_h * in_w;
    net.n_out = (int)(c * h * w);
    net.n_params = (int)off;
    net.e_max = (int)emax;
    net.e_off0 = (int)scr;
    net.e_off1 = (int)(scr + emax);
    scr += 2 * emax;
    scr = (scr + 63) / 64 * 64;  // keep every worker's area 256-byte aligned
    if (scr > kIntLimit) return fail(CHAOS_EUNSUPPORTED, "per-worker scratch beyond 2^30 floats");
    net.scratch_floats = (int)scr;
    if (net.n_out > 256) return fail(CHAOS_EUNSUPPORTED, "more than 256 outputs");
    return CHAOS_OK;
}

int check_net(const chaos_net *net) {
    if (!net) return fail(CHAOS_EINVAL, "net is NULL");
    return CHAOS_OK;
}

int set_device(const chaos_net *net) {
    HIP_TRY(hipSetDevice(net->device), "hipSetDevice");
    return CHAOS_OK;
}

int check_io(const float *x, const int32_t *labels, int64_t n) {
    if (n < 0) return fail(CHAOS_EINVAL, "n=%lld < 0", (long long)n);
    if (n > 0 && (!x || !labels)) return fail(CHAOS_EINVAL, "x or labels is NULL");
    // the claim counter is int32 and may overshoot n by one claim per worker
    if (n > ((int64_t)1 << 31) - ((int64_t)1 << 24))
        return fail(CHAOS_EUNSUPPORTED, "n=%lld too large", (long long)n);
    return CHAOS_OK;
}

chaos::WorkArgs base_args(chaos_net *net, const float *x, const int32_t *labels, int64_t n) {
    chaos::WorkArgs a{};
    a.params = net->params;
    a.x = x;
    a.labels = labels;
    a.n = n;
    a.scratch = net->scratch;
    a.counter = net->counter;
    a.push_delay = 1;
    return a;
}

// Device address of `scratch` on `device` (which must be current), looked up
// on the first call for that device and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
float *g_scratch_ptr[kMaxDevices] = {};

int noalloc_scratch(int device, float **out) {
    if (device < 0 || device >= kMaxDevices)
        return fail(CHAOS_EUNSUPPORTED, "device %d beyond the %d the library tracks", device, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(CHAOS_EDEVICE, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[device] = static_cast<float *>(ptr);
    }
    *out = g_scratch_ptr[device];
    return CHAOS_OK;
}

hipError_t launch(chaos_net *net, int mode, const chaos::WorkArgs &a, int grid, hipStream_t s) {
    if (net->fused) return chaos::launch_fused_large(mode, a, grid, s);
    if (net->t1) return chaos::launch_fused_t1(mode, a, grid, s);
    if (net->cpcp) return chaos::launch_fused_cpcp(net->cpcp, mode, a, grid, s);
    return chaos::launch_worker(mode, net->desc, a, grid, net->block, s);
}

} // namespace

extern "C" {

const char *chaos_last_error(void) { return g_last_error.c_str(); }

int chaos_create_net(int32_t in_h, int32_t in_w, const chaos_layer *layers, int32_t n_layers,
                     const float *init_params_host, int64_t n_params, chaos_net **out) {
    if (!out) return fail(CHAOS_EINVAL, "out is NULL");
    *out = nullptr;
    Net desc;
    int rc = build_desc(in_h, in_w, layers, n_layers, desc);
    if (rc) return rc;
    if (n_params != desc.n_params)
        return fail(CHAOS_ESHAPE, "n_params=%lld but the architecture has %d weights",
                    (long long)n_params, desc.n_params);
    if (!init_params_host) return fail(CHAOS_EINVAL, "init_params_host is NULL");

    chaos_net *net = new (std::nothrow) chaos_net();
    if (!net) return fail(CHAOS_ENOMEM, "host allocation failed");
    net->desc = desc;
    net->n_params = n_params;
    hipError_t e = hipGetDevice(&net->device);
    int cus = 0;
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, net->device);
    if (e != hipSuccess) { delete net; return hip_fail(e, "device query"); }
    net->block = 256;
    net->fused = chaos::fused_large_matches(desc);
    net->t1 = !net->fused && chaos::fused_t1_matches(desc);
    net->cpcp = (net->fused || net->t1) ? 0 : chaos::fused_cpcp_variant(desc);
    int per_cu = net->fused ? chaos::fused_large_blocks_per_cu()
               : net->t1    ? chaos::fused_t1_blocks_per_cu()
               : net->cpcp  ? chaos::fused_cpcp_blocks_per_cu(net->cpcp)
                            : chaos::worker_blocks_per_cu(net->block);
    if (per_cu < 1) { delete net; return fail(CHAOS_EDEVICE, "occupancy query failed"); }
    net->max_workers = per_cu * cus;
    net->cus = cus;
    net->delay_max_workers = net->cpcp ? chaos::fused_cpcp_delay_blocks_per_cu(net->cpcp) * cus : 0;
    net->worker_limit = std::max(net->max_workers, chaos::worker_blocks_per_cu(64) * cus);
    // the fused kernels keep every per-sample value in LDS: no scratch
    size_t scratch_bytes = (net->fused || net->t1 || net->cpcp)
                               ? 0
                               : (size_t)net->max_workers * desc.scratch_floats * sizeof(float);
    if (net->fused) {
        chaos::fused_large_layout(net->layout);
        net->padded = true;
    } else if (net->t1) {
        chaos::fused_t1_layout(net->layout);
        net->padded = true;
    } else if (net->cpcp && chaos::fused_cpcp_layout(net->cpcp, net->layout)) {
        net->padded = true;
    } else {
        net->layout.n_seg = 1;
        net->layout.n_dev = (int)n_params;
        net->layout.seg[0] = chaos::ParamSegment{0, 0, 1, (int)n_params, (int)n_params};
    }
    // the initial weights in the device layout (padding zero)
    std::vector<float> dev;
    const float *init = init_params_host;
    if (net->padded) {
        dev.assign((size_t)net->layout.n_dev, 0.0f);
        for (int k = 0; k < net->layout.n_seg; ++k) {
            const chaos::ParamSegment &g = net->layout.seg[k];
            for (int r = 0; r < g.rows; ++r)
                std::memcpy(&dev[(size_t)g.dev_off + (size_t)r * g.dev_stride],
                            init_params_host + g.can_off + (size_t)r * g.len, (size_t)g.len * sizeof(float));
        }
        init = dev.data();
    }
    e = hipMalloc(&net->params, (size_t)net->layout.n_dev * sizeof(float));
    if (e == hipSuccess && scratch_bytes) e = hipMalloc(&net->scratch, scratch_bytes);
    if (e == hipSuccess) e = hipMalloc(&net->counter, 64);
    if (e == hipSuccess)
        e = hipMemcpy(net->params, init, (size_t)net->layout.n_dev * sizeof(float),
                      hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        chaos_destroy_net(net);
        return e == hipErrorOutOfMemory ? fail(CHAOS_ENOMEM, "device allocation failed")
                                        : hip_fail(e, "create");
    }
    *out = net;
    return ok();
}

int chaos_destroy_net(chaos_net *net) {
    if (!net) return ok();
    (void)hipSetDevice(net->device);
    (void)hipFree(net->params);
    (void)hipFree(net->canon);
    (void)hipFree(net->scratch);
    (void)hipFree(net->counter);
    (void)hipFree(net->grad_part);
    (void)hipFree(net->wide_scratch);
    (void)hipFree(net->sess_loss);
    (void)hipFree(net->sess_wrong);
    (void)hipFree(net->stash);
    (void)hipFree(net->bpart);
    (void)hipFree(net->replicas);
    (void)hipFree(net->rep_counter);
    delete net;
    return ok();
}

int64_t chaos_num_params(const chaos_net *net) {
    if (int rc = check_net(net)) return rc;
    return net->n_params;
}

int32_t chaos_num_outputs(const chaos_net *net) {
    if (int rc = check_net(net)) return rc;
    return net->desc.n_out;
}

int32_t chaos_max_workers(const chaos_net *net) {
    if (int rc = check_net(net)) return rc;
    return net->push_delay > 1 ? net->delay_max_workers : net->max_workers;
}

int32_t chaos_default_workers(const chaos_net *net) {
    if (int rc = check_net(net)) return rc;
    return std::min(chaos_max_workers(net), net->cus);
}

int chaos_set_push_delay(chaos_net *net, int32_t k) {
    if (int rc = check_net(net)) return rc;
    if (k < 1) return fail(CHAOS_EINVAL, "push delay %d < 1", k);
    if (k > 1 && net->delay_max_workers < 1)
        return fail(CHAOS_EUNSUPPORTED, "delayed pushes need a net whose weights fit in LDS");
    if (k > 1 && net->n_replicas > 1)
        return fail(CHAOS_EINVAL, "delayed pushes and weight replicas exclude each other");
    net->push_delay = k;
    return ok();
}

int chaos_set_replicas(chaos_net *net, int32_t r, int32_t m) {
    if (int rc = check_net(net)) return rc;
    if (r < 1 || r > 64) return fail(CHAOS_EINVAL, "replicas %d outside [1,64]", r);
    if (m < 1) return fail(CHAOS_EINVAL, "refresh interval %d < 1", m);
    if (r > 1 && !(net->cpcp && chaos::fused_cpcp_supports_replicas(net->cpcp)))
        return fail(CHAOS_EUNSUPPORTED, "weight replicas need a net whose weights fit in LDS");
    if (r > 1 && net->push_delay > 1)
        return fail(CHAOS_EINVAL, "delayed pushes and weight replicas exclude each other");
    if (int rc = set_device(net)) return rc;
    if (r > net->n_replicas || (r > 1 && !net->replicas)) {
        (void)hipFree(net->replicas);
        (void)hipFree(net->rep_counter);
        net->replicas = nullptr;
        net->rep_counter = nullptr;
        if (hipMalloc(&net->replicas, (size_t)r * net->layout.n_dev * sizeof(float)) != hipSuccess ||
            hipMalloc(&net->rep_counter, (size_t)r * sizeof(int32_t)) != hipSuccess) {
            (void)hipFree(net->replicas);
            net->replicas = nullptr;
            net->rep_counter = nullptr;
            net->n_replicas = 1;
            return fail(CHAOS_ENOMEM, "%d weight replicas", r);
        }
    }
    net->n_replicas = r;
    net->refresh_every = m;
    return ok();
}

int32_t chaos_worker_limit(const chaos_net *net) {
    if (int rc = check_net(net)) return rc;
    return net->worker_limit;
}

int chaos_get_params(const chaos_net *net, float *dst_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (!dst_dev) return fail(CHAOS_EINVAL, "dst_dev is NULL");
    if (int rc = set_device(net)) return rc;
    if (net->padded)
        HIP_TRY(chaos::launch_convert_params(net->params, dst_dev, net->layout, net->n_params, false,
                                             stream),
                "get_params");
    else
        HIP_TRY(hipMemcpyAsync(dst_dev, net->params, (size_t)net->n_params * sizeof(float),
                               hipMemcpyDeviceToDevice, stream),
                "get_params");
    return ok();
}

int chaos_set_params(chaos_net *net, const float *src_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (!src_dev) return fail(CHAOS_EINVAL, "src_dev is NULL");
    if (int rc = set_device(net)) return rc;
    if (net->padded)
        HIP_TRY(chaos::launch_convert_params(src_dev, net->params, net->layout, net->n_params, true,
                                             stream),
                "set_params");
    else
        HIP_TRY(hipMemcpyAsync(net->params, src_dev, (size_t)net->n_params * sizeof(float),
                               hipMemcpyDeviceToDevice, stream),
                "set_params");
    return ok();
}

int chaos_set_claim_counter(chaos_net *net, int32_t *claims_dev) {
    if (int rc = check_net(net)) return rc;
    net->claims = claims_dev;
    return ok();
}

int chaos_apply_update(chaos_net *net, const float *grad_dev, float lr, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (!grad_dev) return fail(CHAOS_EINVAL, "grad_dev is NULL");
    if (int rc = set_device(net)) return rc;
    if (net->padded)
        HIP_TRY(chaos::launch_axpy_mapped(net->params, grad_dev, -lr, net->layout, net->n_params, stream),
                "apply_update");
    else
        HIP_TRY(chaos::launch_axpy(net->params, grad_dev, -lr, net->n_params, stream), "apply_update");
    return ok();
}

int chaos_train_epoch(chaos_net *net, const float *x_dev, const int32_t *labels_dev, int64_t n,
                      float lr, int32_t mode, int32_t workers, float *loss_dev,
                      hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (int rc = check_io(x_dev, labels_dev, n)) return rc;
    if (mode != CHAOS_SEQUENTIAL && mode != CHAOS_HOGWILD_ATOMIC && mode != CHAOS_HOGWILD_RACY)
        return fail(CHAOS_EINVAL, "unknown mode %d", mode);
    if (workers < 0 || workers > net->worker_limit)
        return fail(CHAOS_EINVAL, "workers=%d outside [0,%d]", workers, net->worker_limit);
    if (int rc = set_device(net)) return rc;
    if (n == 0) return ok();
    if (mode == CHAOS_HOGWILD_ATOMIC && net->push_delay > 1) {
        // delayed pushes: the net's own kernel with a per-worker gradient sum
        if (workers > net->delay_max_workers)
            return fail(CHAOS_EINVAL, "workers=%d: delayed pushes run at most %d workers", workers,
                        net->delay_max_workers);
        chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
        a.lr = lr;
        a.loss = loss_dev;
        a.claims = net->claims;
        a.push_delay = net->push_delay;
        int grid = (int)std::min<int64_t>(workers == 0 ? chaos_default_workers(net) : workers, n);
        HIP_TRY(chaos::launch_fill_i32(net->counter, 0, 2, stream), "counter reset");
        HIP_TRY(launch(net, chaos::kTrainAtomic, a, grid, stream), "train launch");
        return ok();
    }
    if (mode != CHAOS_SEQUENTIAL && workers > net->max_workers) {
        // more workers than the net's kernel keeps resident: every worker is one
        // 64-thread wavefront of the generic kernel, with scratch in HBM
        if (!net->wide_scratch) {
            size_t bytes = (size_t)net->worker_limit * net->desc.scratch_floats * sizeof(float);
            if (hipMalloc(&net->wide_scratch, bytes) != hipSuccess) {
                net->wide_scratch = nullptr;
                return fail(CHAOS_ENOMEM, "scratch for %d workers", net->worker_limit);
            }
        }
        // the generic kernel reads the canonical layout: a padded net's
        // weights are copied to it and back around the launch
        if (net->padded && !net->canon) {
            if (hipMalloc(&net->canon, (size_t)net->n_params * sizeof(float)) != hipSuccess) {
                net->canon = nullptr;
                return fail(CHAOS_ENOMEM, "canonical weights for the generic kernel");
            }
        }
        chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
        a.scratch = net->wide_scratch;
        a.lr = lr;
        a.loss = loss_dev;
        a.claims = net->claims;
        if (net->padded) {
            a.params = net->canon;
            HIP_TRY(chaos::launch_convert_params(net->params, net->canon, net->layout, net->n_params,
                                                 false, stream),
                    "to canonical");
        }
        int kmode = mode == CHAOS_HOGWILD_RACY ? chaos::kTrainRacy : chaos::kTrainAtomic;
        int grid = (int)std::min<int64_t>(workers, n);
        HIP_TRY(chaos::launch_fill_i32(net->counter, 0, 2, stream), "counter reset");
        HIP_TRY(chaos::launch_worker(kmode, net->desc, a, grid, 64, stream), "train launch");
        if (net->padded)
            HIP_TRY(chaos::launch_convert_params(net->canon, net->params, net->layout, net->n_params,
                                                 true, stream),
                    "to device layout");
        return ok();
    }
    int grid = 1;
    int kmode = chaos::kTrainAtomic;
    if (mode != CHAOS_SEQUENTIAL) {
        grid = workers == 0 ? chaos_default_workers(net) : workers;
        if (mode == CHAOS_HOGWILD_RACY) kmode = chaos::kTrainRacy;
    }
    grid = (int)std::min<int64_t>(grid, n);
    chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
    a.lr = lr;
    a.loss = loss_dev;
    a.claims = net->claims;
    HIP_TRY(chaos::launch_fill_i32(net->counter, 0, 2, stream), "counter reset");
    if (kmode == chaos::kTrainAtomic && mode != CHAOS_SEQUENTIAL && net->n_replicas > 1) {
        // every replica starts the epoch equal to the shared weights
        a.replicas = net->replicas;
        a.rep_counter = net->rep_counter;
        a.n_replicas = net->n_replicas;
        a.refresh_every = net->refresh_every;
        HIP_TRY(chaos::launch_replicate(net->params, net->replicas, net->layout.n_dev, net->n_replicas,
                                        stream),
                "replica copy");
        HIP_TRY(chaos::launch_fill_i32(net->rep_counter, 0, net->n_replicas, stream), "replica counters");
    }
    HIP_TRY(launch(net, kmode, a, grid, stream), "train launch");
    return ok();
}

int chaos_forward_backward(chaos_net *net, const float *x_dev, const int32_t *labels_dev,
                           int64_t n, float *out_dev, float *loss_dev, float *grad_sum_dev,
                           float *grad_each_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (int rc = check_io(x_dev, labels_dev, n)) return rc;
    if (int rc = set_device(net)) return rc;
    if (n == 0) {
        if (grad_sum_dev)
            HIP_TRY(chaos::launch_fill_f32(grad_sum_dev, 0.0f, net->n_params, stream), "zero grad");
        return ok();
    }
    int grid = (int)std::min<int64_t>(net->max_workers, n);
    if (grad_sum_dev) {
        // fixed sample -> worker assignment (sample i goes to worker i mod grid,
        // in increasing i), partial sums per worker, then a fixed-order reduction
        int want = std::min(grid, 512);
        if (want > net->fb_workers) {
            (void)hipFree(net->grad_part);
            net->grad_part = nullptr;
            net->fb_workers = 0;
            hipError_t e = hipMalloc(&net->grad_part, (size_t)want * net->n_params * sizeof(float));
            if (e != hipSuccess) return fail(CHAOS_ENOMEM, "grad_part allocation failed");
            net->fb_workers = want;
        }
        grid = want;
    }
    // large net, gradient sum only: the conv3 and FC1 weight gradients are
    // contracted over the batch on the matrix cores from per-sample operands
    // the kernel leaves in HBM (47.6 KB per sample, allocated on first use)
    const bool batched = grad_sum_dev && !grad_each_dev && net->fused;
    constexpr int64_t kConv3W = 100 * 2160, kFc1W = 150 * 900;
    if (batched) {
        if (n > net->stash_n) {
            (void)hipFree(net->stash);
            net->stash = nullptr;
            net->stash_n = 0;
            if (hipMalloc(&net->stash, (size_t)n * chaos::kStashFloats * sizeof(float)) != hipSuccess) {
                net->stash = nullptr;
                return fail(CHAOS_ENOMEM, "batch gradient operands for %lld samples", (long long)n);
            }
            net->stash_n = n;
        }
        const int64_t nc = chaos::batch_grad_chunks(n);
        if (nc > net->bpart_chunks) {
            (void)hipFree(net->bpart);
            net->bpart = nullptr;
            net->bpart_chunks = 0;
            if (hipMalloc(&net->bpart, (size_t)nc * (kConv3W + kFc1W) * sizeof(float)) != hipSuccess) {
                net->bpart = nullptr;
                return fail(CHAOS_ENOMEM, "batch gradient partial sums");
            }
            net->bpart_chunks = nc;
        }
    }
    chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
    a.out = out_dev;
    a.loss = loss_dev;
    a.grad_each = grad_each_dev;
    a.grad_part = grad_sum_dev ? net->grad_part : nullptr;
    a.stash = batched ? net->stash : nullptr;
    if (grad_sum_dev)
        HIP_TRY(chaos::launch_fill_f32(net->grad_part, 0.0f, (int64_t)grid * net->n_params, stream),
                "zero partial sums");
    HIP_TRY(launch(net, chaos::kForwardBackward, a, grid, stream), "forward_backward launch");
    if (grad_sum_dev)
        HIP_TRY(chaos::launch_reduce_partials(net->grad_part, grid, net->n_params, grad_sum_dev,
                                              stream),
                "reduce");
    if (batched) {
        // the per-sample pass pushed nothing into these two weight blocks:
        // their sums replace the zeros the reduction left there
        const int64_t nc = chaos::batch_grad_chunks(n);
        float *part3 = net->bpart, *partf = net->bpart + nc * kConv3W;
        HIP_TRY(chaos::launch_batch_grad(net->stash, n, part3, partf, stream), "batch gradient");
        HIP_TRY(chaos::launch_reduce_partials(part3, nc, kConv3W, grad_sum_dev + net->desc.L[3].w_off,
                                              stream),
                "reduce conv3");
        HIP_TRY(chaos::launch_reduce_partials(partf, nc, kFc1W, grad_sum_dev + net->desc.L[5].w_off,
                                              stream),
                "reduce FC1");
    }
    return ok();
}

int chaos_train_session(chaos_net *net, const float *x_train_dev, const int32_t *labels_train_dev,
                        int64_t n_train, const float *x_test_dev, const int32_t *labels_test_dev,
                        int64_t n_test, int32_t epochs, float lr0, float decay, int32_t mode,
                        int32_t workers, float *stats_dev, float *ckpt_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (int rc = check_io(x_train_dev, labels_train_dev, n_train)) return rc;
    if (int rc = check_io(x_test_dev, labels_test_dev, n_test)) return rc;
    if (epochs < 0) return fail(CHAOS_EINVAL, "epochs=%d < 0", epochs);
    if (epochs > 0 && !stats_dev) return fail(CHAOS_EINVAL, "stats_dev is NULL");
    if (mode != CHAOS_SEQUENTIAL && mode != CHAOS_HOGWILD_ATOMIC && mode != CHAOS_HOGWILD_RACY)
        return fail(CHAOS_EINVAL, "unknown mode %d", mode);
    if (workers < 0 || workers > net->worker_limit)
        return fail(CHAOS_EINVAL, "workers=%d outside [0,%d]", workers, net->worker_limit);
    if (int rc = set_device(net)) return rc;
    const int64_t need = std::max<int64_t>(std::max(n_train, n_test), 1);
    if (need > net->sess_loss_n) {
        (void)hipFree(net->sess_loss);
        net->sess_loss = nullptr;
        net->sess_loss_n = 0;
        if (hipMalloc(&net->sess_loss, (size_t)need * sizeof(float)) != hipSuccess)
            return fail(CHAOS_ENOMEM, "session loss buffer");
        net->sess_loss_n = need;
    }
    if (!net->sess_wrong && hipMalloc(&net->sess_wrong, 64) != hipSuccess)
        return fail(CHAOS_ENOMEM, "session counter");
    // the divergence flag's reference: the mean loss at the starting weights
    // on the test set (the training set when there is no test set)
    float *ref = reinterpret_cast<float *>(net->sess_wrong) + 8;
    const bool ref_test = n_test > 0;
    if (epochs > 0) {
        const float *xr = ref_test ? x_test_dev : x_train_dev;
        const int32_t *yr = ref_test ? labels_test_dev : labels_train_dev;
        const int64_t nr = ref_test ? n_test : n_train;
        int rc = nr > 0 ? chaos_forward_backward(net, xr, yr, nr, nullptr, net->sess_loss, nullptr,
                                                 nullptr, stream)
                        : CHAOS_OK;
        if (rc) return rc;
        HIP_TRY(chaos::launch_mean(net->sess_loss, nr, ref, stream), "session reference loss");
    }
    for (int32_t e = 0; e < epochs; ++e) {
        float lr = (float)((double)lr0 * std::pow((double)decay, (double)e));
        float *st = stats_dev + 5 * (int64_t)e;
        int rc = chaos_train_epoch(net, x_train_dev, labels_train_dev, n_train, lr, mode, workers,
                                   n_train ? net->sess_loss : nullptr, stream);
        if (rc) return rc;
        if (ckpt_dev && (rc = chaos_get_params(net, ckpt_dev + (int64_t)e * net->n_params, stream)))
            return rc;
        HIP_TRY(chaos::launch_mean(net->sess_loss, n_train, st + 0, stream), "session mean");
        if ((rc = chaos_evaluate(net, x_train_dev, labels_train_dev, n_train, nullptr,
                                 net->sess_wrong, stream)))
            return rc;
        HIP_TRY(chaos::launch_count(net->sess_wrong, st + 1, stream), "session count");
        if ((rc = chaos_evaluate(net, x_test_dev, labels_test_dev, n_test, nullptr,
                                 net->sess_wrong, stream)))
            return rc;
        HIP_TRY(chaos::launch_count(net->sess_wrong, st + 2, stream), "session count");
        if (n_test > 0 &&
            (rc = chaos_forward_backward(net, x_test_dev, labels_test_dev, n_test, nullptr,
                                         net->sess_loss, nullptr, nullptr, stream)))
            return rc;
        HIP_TRY(chaos::launch_mean(net->sess_loss, n_test, st + 3, stream), "session mean");
        HIP_TRY(chaos::launch_above(ref_test ? st + 3 : st + 0, ref, st + 4, stream),
                "session divergence flag");
    }
    return ok();
}

int chaos_forward_backward_noalloc(chaos_net *net, const float *x_dev, const int32_t *labels_dev,
                                   int64_t n, float *out_dev, float *loss_dev, float *grad_sum_dev,
                                   float *grad_each_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (int rc = check_io(x_dev, labels_dev, n)) return rc;
    if (grad_sum_dev && net->n_params > kNoAllocFloats)
        return fail(CHAOS_EUNSUPPORTED,
                    "a gradient sum needs one partial-sum row of %lld floats; the fixed scratch "
                    "holds %lld",
                    (long long)net->n_params, (long long)kNoAllocFloats);
    if (int rc = set_device(net)) return rc;
    float *rows = nullptr;
    if (grad_sum_dev) {
        if (int rc = noalloc_scratch(net->device, &rows)) return rc;
    }
    if (n == 0) {
        if (grad_sum_dev)
            HIP_TRY(chaos::launch_fill_f32(grad_sum_dev, 0.0f, net->n_params, stream), "zero grad");
        return ok();
    }
    // as chaos_forward_backward: sample i goes to worker i mod grid, each
    // worker adds its samples' gradients into its own row in sample order,
    // then the rows are summed in a fixed order; here the grid is bounded by
    // the rows that fit in the fixed scratch (and the large net's conv3 / FC1
    // gradients are pushed per sample instead of contracted over the batch,
    // which would need per-sample operands in memory)
    int grid = (int)std::min<int64_t>(net->max_workers, n);
    if (grad_sum_dev) grid = (int)std::min<int64_t>({(int64_t)grid, 512, kNoAllocFloats / net->n_params});
    chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
    a.out = out_dev;
    a.loss = loss_dev;
    a.grad_each = grad_each_dev;
    a.grad_part = rows;
    if (grad_sum_dev)  // the rows hold the previous call's sums: clear them (a kernel, no memset node)
        HIP_TRY(chaos::launch_fill_f32(rows, 0.0f, (int64_t)grid * net->n_params, stream),
                "zero partial sums");
    HIP_TRY(launch(net, chaos::kForwardBackward, a, grid, stream), "forward_backward launch");
    if (grad_sum_dev)
        HIP_TRY(chaos::launch_reduce_partials(rows, grid, net->n_params, grad_sum_dev, stream),
                "reduce");
    return ok();
}

int chaos_evaluate(chaos_net *net, const float *x_dev, const int32_t *labels_dev, int64_t n,
                   float *out_dev, int32_t *n_wrong_dev, hipStream_t stream) {
    if (int rc = check_net(net)) return rc;
    if (int rc = check_io(x_dev, labels_dev, n)) return rc;
    if (!n_wrong_dev) return fail(CHAOS_EINVAL, "n_wrong_dev is NULL");
    if (int rc = set_device(net)) return rc;
    HIP_TRY(chaos::launch_fill_i32(n_wrong_dev, 0, 1, stream), "zero n_wrong");
    if (n == 0) return ok();
    int grid = (int)std::min<int64_t>(net->max_workers, n);
    chaos::WorkArgs a = base_args(net, x_dev, labels_dev, n);
    a.out = out_dev;
    a.n_wrong = n_wrong_dev;
    HIP_TRY(launch(net, chaos::kEvaluate, a, grid, stream), "evaluate launch");
    return ok();
}

} // extern "C"
