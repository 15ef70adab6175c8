// Exercises the host-side argument checks and the shape walk of the C ABI
// (the paths that return before any device work) under AddressSanitizer /
// UndefinedBehaviorSanitizer.  Built host-only against the library's host
// source; the kernel launchers it would call are stubs that fail, so no path
// here reaches a GPU.  Test infrastructure, run by tests/test_sanitizers.py.
#include "../../include/chaos.h"
#include "../../paper_1506_09067_amd/csrc/chaos_internal.h"

#include <cstdio>
#include <cstring>
#include <vector>

namespace chaos {
hipError_t launch_worker(int, const Net &, const WorkArgs &, int, int, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_fill_i32(int32_t *, int32_t, int64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_fill_f32(float *, float, int64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_reduce_partials(const float *, int64_t, int64_t, float *, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_axpy(float *, const float *, float, int64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_convert_params(const float *, float *, const ParamLayout &, int64_t, bool, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_axpy_mapped(float *, const float *, float, const ParamLayout &, int64_t, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_mean(const float *, int64_t, float *, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_count(const int32_t *, float *, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_above(const float *, const float *, float *, hipStream_t) { return hipErrorInvalidValue; }
hipError_t launch_replicate(const float *, float *, int64_t, int, hipStream_t) { return hipErrorInvalidValue; }
bool fused_cpcp_supports_replicas(int) { return false; }
int worker_blocks_per_cu(int) { return 0; }
bool fused_large_matches(const Net &) { return false; }
void fused_large_layout(ParamLayout &) {}
hipError_t launch_fused_large(int, const WorkArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
int fused_large_blocks_per_cu() { return 0; }
bool fused_t1_matches(const Net &) { return false; }
void fused_t1_layout(ParamLayout &) {}
hipError_t launch_fused_t1(int, const WorkArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
int fused_t1_blocks_per_cu() { return 0; }
int64_t batch_grad_chunks(int64_t n) { return n; }
hipError_t launch_batch_grad(const float *, int64_t, float *, float *, hipStream_t) { return hipErrorInvalidValue; }
int fused_cpcp_variant(const Net &) { return 0; }
bool fused_cpcp_layout(int, ParamLayout &) { return false; }
hipError_t launch_fused_cpcp(int, int, const WorkArgs &, int, hipStream_t) { return hipErrorInvalidValue; }
int fused_cpcp_blocks_per_cu(int) { return 0; }
int fused_cpcp_delay_blocks_per_cu(int) { return 0; }
}  // namespace chaos

static int fails = 0;
#define CHECK(c) do { if (!(c)) { std::fprintf(stderr, "check failed line %d: %s (%s)\n", __LINE__, #c, chaos_last_error()); ++fails; } } while (0)

int main() {
    chaos_net *net = reinterpret_cast<chaos_net *>(0x1);
    std::vector<float> p(1 << 20, 0.0f);
    const chaos_layer small[] = {{1, 5, 4}, {2, 0, 2}, {1, 10, 5}, {2, 0, 3}, {3, 50, 0}, {3, 10, 0}};
    // shape walk errors, each returned before any device call
    const chaos_layer big_kernel[] = {{1, 2, 30}};
    const chaos_layer bad_pool[] = {{1, 2, 4}, {2, 0, 3}};
    const chaos_layer bad_kind[] = {{9, 2, 4}};
    const chaos_layer zero_fc[] = {{3, 0, 0}};
    const chaos_layer neg_conv[] = {{1, -1, 3}};
    const chaos_layer wide_fc[] = {{3, 40000, 0}, {3, 40000, 0}};     // 1.6e9 weights: beyond 2^30
    const chaos_layer many_out[] = {{3, 300, 0}};                        // more than 256 outputs
    CHECK(chaos_create_net(29, 29, big_kernel, 1, p.data(), 2, &net) == CHAOS_ESHAPE && net == nullptr);
    CHECK(chaos_create_net(29, 29, bad_pool, 2, p.data(), 1, &net) == CHAOS_ESHAPE);
    CHECK(chaos_create_net(29, 29, bad_kind, 1, p.data(), 1, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, zero_fc, 1, p.data(), 1, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, neg_conv, 1, p.data(), 1, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, wide_fc, 2, p.data(), 1, &net) == CHAOS_EUNSUPPORTED);
    CHECK(chaos_create_net(29, 29, many_out, 1, p.data(), 300 * 842, &net) == CHAOS_EUNSUPPORTED);
    CHECK(chaos_create_net(29, 29, small, 6, p.data(), 6404, &net) == CHAOS_ESHAPE);  // weight count
    CHECK(chaos_create_net(29, 29, small, 6, nullptr, 6405, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, nullptr, 6, p.data(), 6405, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, small, 0, p.data(), 6405, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, small, 17, p.data(), 6405, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(0, 29, small, 6, p.data(), 6405, &net) == CHAOS_EINVAL);
    CHECK(chaos_create_net(29, 29, small, 6, p.data(), 6405, nullptr) == CHAOS_EINVAL);
    // a valid net: the shape walk succeeds, then the device query or the
    // occupancy stub fails cleanly (no GPU is used here)
    int rc = chaos_create_net(29, 29, small, 6, p.data(), 6405, &net);
    CHECK(rc == CHAOS_EDEVICE && net == nullptr);
    CHECK(std::strlen(chaos_last_error()) > 0);
    // NULL nets and arguments on every entry point
    float f = 0.0f;
    int32_t l = 0;
    CHECK(chaos_destroy_net(nullptr) == CHAOS_OK);
    CHECK(chaos_num_params(nullptr) == CHAOS_EINVAL);
    CHECK(chaos_num_outputs(nullptr) == CHAOS_EINVAL);
    CHECK(chaos_max_workers(nullptr) == CHAOS_EINVAL);
    CHECK(chaos_default_workers(nullptr) == CHAOS_EINVAL);
    CHECK(chaos_worker_limit(nullptr) == CHAOS_EINVAL);
    CHECK(chaos_get_params(nullptr, &f, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_set_params(nullptr, &f, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_apply_update(nullptr, &f, 1.0f, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_forward_backward(nullptr, &f, &l, 1, nullptr, nullptr, nullptr, nullptr, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_forward_backward_noalloc(nullptr, &f, &l, 1, nullptr, nullptr, nullptr, nullptr, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_train_epoch(nullptr, &f, &l, 1, 1e-3f, 0, 0, nullptr, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_evaluate(nullptr, &f, &l, 1, nullptr, &l, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_train_session(nullptr, &f, &l, 1, &f, &l, 1, 1, 1e-3f, 1.0f, 0, 0, &f, nullptr, nullptr) == CHAOS_EINVAL);
    CHECK(chaos_set_push_delay(nullptr, 2) == CHAOS_EINVAL);
    CHECK(chaos_set_replicas(nullptr, 8, 4) == CHAOS_EINVAL);
    CHECK(chaos_set_claim_counter(nullptr, nullptr) == CHAOS_EINVAL);
    if (fails) return 1;
    std::printf("host driver ok\n");
    return 0;
}
