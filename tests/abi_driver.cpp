// Host-side driver of the C ABI, linked with a test build of the library's
// host code (-DDERF_FAULT_INJECTION; for the CPU run also -fsanitize=address
// on the host side only -- device code is never instrumented):
//   * every argument check and early-failure path that needs no GPU, including
//     derf_create's clean-up of a handle whose device setup fails;
//   * allocation failures: each allocation of derf_create, derf_create_mixed,
//     the render workspace and derf_set_gate is made to fail in turn
//     (derf_debug_fail_alloc); each must return DERF_ERR_OOM, hand out no
//     handle, leave an existing handle working and release everything it had
//     taken (derf_debug_live_allocations back to its earlier count).  Without
//     a GPU only the handle's own allocation can be reached.
// Prints one line per failed expectation; exit status 0 when every call
// returned what the header promises.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include <hip/hip_runtime.h>

#include "derf.h"

// exported by fault-injection builds of the library only
extern "C" void derf_debug_fail_alloc(long n);
extern "C" long derf_debug_live_allocations(void);

static int failures = 0;

static void expect(bool ok, const char *what)
{
    if (!ok) {
        printf("FAILED: %s (last error: %s)\n", what, derf_last_error());
        ++failures;
    }
}

// Rays of a small pinhole frame looking at the origin from z = 4, heads of
// the 4x64 architecture with small deterministic weights.
struct Frame {
    int K = 64, R = 256, n = 32;
    std::vector<float> sites, weights, o, d;
    Frame()
    {
        const derf_head_arch a = {6, 4, 4, 64, -1, 0};
        const long long wc = derf_weights_count(&a);
        sites.resize(3 * K);
        for (int k = 0; k < K; ++k)
            for (int c = 0; c < 3; ++c)
                sites[3 * k + c] = (float)(((k * 37 + c * 11) % 97) / 48.5 - 1.0);
        weights.resize((size_t)wc * K);
        for (size_t i = 0; i < weights.size(); ++i)
            weights[i] = (float)(((i * 2654435761u) >> 8) % 2001) * 1e-4f - 0.1f;
        for (int r = 0; r < R; ++r) {
            const float px = (r % 16 - 7.5f) / 20.0f, py = (r / 16 - 7.5f) / 20.0f;
            o.insert(o.end(), {0.0f, 0.0f, 4.0f});
            d.insert(d.end(), {px, py, -1.0f});
        }
    }
};

static void fault_injection()
{
    int devices = 0;
    const bool gpu = hipGetDeviceCount(&devices) == hipSuccess && devices > 0;
    const derf_head_arch tiny = {6, 4, 4, 64, -1, 0};
    const derf_head_arch small = {10, 4, 6, 64, -1, 32};
    Frame f;
    const long base = derf_debug_live_allocations();
    // derf_create and derf_create_mixed: fail allocation n for n = 0, 1, ...
    // until a create succeeds (n past its last allocation)
    for (int mixed = 0; mixed < 2; ++mixed) {
        std::vector<derf_head_arch> archs(f.K, tiny);
        std::vector<float> w;
        if (mixed) {
            for (int k = 0; k < f.K; ++k) {
                archs[k] = k % 2 ? small : tiny;
                w.resize(w.size() + (size_t)derf_weights_count(&archs[k]), 0.01f);
            }
        }
        int failed_at = 0;
        for (long n = 0; n < 64; ++n) {
            derf_handle *h = reinterpret_cast<derf_handle *>(0x1);
            derf_debug_fail_alloc(n);
            const int rc = mixed ? derf_create_mixed(&h, f.K, f.sites.data(), archs.data(),
                                                     w.data(), DERF_PREC_BF16)
                                 : derf_create(&h, f.K, f.sites.data(), &tiny, f.weights.data(),
                                               DERF_PREC_FP32);
            derf_debug_fail_alloc(-1);
            if (rc == DERF_OK) {
                derf_destroy(h);
                break;
            }
            if (!gpu && n > 0)
                break;  // past the handle, a machine without a GPU fails in device setup
            expect(rc == DERF_ERR_OOM, "an injected allocation failure returns DERF_ERR_OOM");
            expect(h == nullptr, "no handle after a failed create");
            expect(derf_debug_live_allocations() == base, "a failed create releases everything");
            ++failed_at;
        }
        expect(derf_debug_live_allocations() == base, "destroy releases everything");
        if (gpu)
            expect(failed_at >= 4, "create's allocations were each made to fail");
        printf("fault injection: %s create failed cleanly at %d allocation(s)\n",
               mixed ? "mixed" : "plain", failed_at);
    }
    if (!gpu)
        return;
    // the render workspace and the gate on a live handle
    derf_handle *h = nullptr;
    expect(derf_create(&h, f.K, f.sites.data(), &tiny, f.weights.data(), DERF_PREC_FP32) ==
               DERF_OK,
           "create");
    if (!h)
        return;
    const size_t R = f.R;
    float *dev = nullptr;
    if (hipMalloc(reinterpret_cast<void **>(&dev), sizeof(float) * 14 * R) != hipSuccess) {
        expect(false, "test buffers");
        derf_destroy(h);
        return;
    }
    float *o = dev, *d = dev + 3 * R, *rgb = dev + 6 * R, *dep = dev + 9 * R, *op = dev + 10 * R;
    float *rgb2 = dev + 11 * R;
    (void)hipMemcpy(o, f.o.data(), sizeof(float) * 3 * R, hipMemcpyHostToDevice);
    (void)hipMemcpy(d, f.d.data(), sizeof(float) * 3 * R, hipMemcpyHostToDevice);
    const derf_sampling samp = {f.n, 0, 7, 1, 0};
    const long with_handle = derf_debug_live_allocations();
    derf_debug_fail_alloc(0);
    expect(derf_render(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb, dep, op, nullptr) == DERF_ERR_OOM,
           "a render whose workspace cannot be allocated returns DERF_ERR_OOM");
    derf_debug_fail_alloc(-1);
    expect(derf_debug_live_allocations() == with_handle, "the failed render holds no workspace");
    expect(derf_render(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb, dep, op, nullptr) == DERF_OK,
           "the handle renders after the failure");
    expect(derf_render(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb2, dep, op, nullptr) == DERF_OK,
           "and again");
    expect(hipDeviceSynchronize() == hipSuccess, "renders completed");
    std::vector<float> a(3 * R), b(3 * R);
    (void)hipMemcpy(a.data(), rgb, sizeof(float) * 3 * R, hipMemcpyDeviceToHost);
    (void)hipMemcpy(b.data(), rgb2, sizeof(float) * 3 * R, hipMemcpyDeviceToHost);
    expect(a == b, "renders after the failure agree");
    const long gw = derf_gate_weights_count(f.K, 6, 16);
    std::vector<float> gate((size_t)gw, 0.05f);
    const long with_ws = derf_debug_live_allocations();
    derf_debug_fail_alloc(0);
    expect(derf_set_gate(h, 6, 16, gate.data()) == DERF_ERR_OOM, "gate allocation failure");
    derf_debug_fail_alloc(-1);
    expect(derf_debug_live_allocations() == with_ws, "the failed gate holds nothing");
    expect(derf_render_gated(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb, dep, op, nullptr, nullptr) ==
               DERF_ERR_INVALID_ARG,
           "no gate was set");
    expect(derf_set_gate(h, 6, 16, gate.data()) == DERF_OK, "gate after the failure");
    expect(derf_render_gated(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb, dep, op, nullptr, nullptr) ==
               DERF_OK,
           "gated render");
    expect(hipDeviceSynchronize() == hipSuccess, "gated render completed");
    // the stored encoding: its larger workspace fails cleanly too (the old
    // one is released first), and its outputs are the fused form's
    expect(derf_set_encoding(h, DERF_ENCODING_STORED) == DERF_OK, "stored encoding");
    const long with_ws2 = derf_debug_live_allocations();
    derf_debug_fail_alloc(0);
    expect(derf_render(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb2, dep, op, nullptr) == DERF_ERR_OOM,
           "a stored-encoding render whose workspace cannot be allocated returns DERF_ERR_OOM");
    derf_debug_fail_alloc(-1);
    expect(derf_debug_live_allocations() == with_ws2 - 1, "the failed render holds no workspace");
    expect(derf_render(h, o, d, f.R, 2.0f, 6.0f, &samp, rgb2, dep, op, nullptr) == DERF_OK,
           "stored-encoding render after the failure");
    expect(hipDeviceSynchronize() == hipSuccess, "stored-encoding render completed");
    (void)hipMemcpy(b.data(), rgb2, sizeof(float) * 3 * R, hipMemcpyDeviceToHost);
    expect(a == b, "the stored encoding renders the fused form's pixels");
    expect(derf_set_encoding(h, 2) == DERF_ERR_INVALID_ARG, "unknown encoding mode");
    expect(derf_set_encoding(h, DERF_ENCODING_FUSED) == DERF_OK, "fused encoding");
    derf_destroy(h);
    (void)hipFree(dev);
    expect(derf_debug_live_allocations() == base, "everything released at the end");
    printf("fault injection: render workspace, gate and stored-encoding failures handled\n");
}

int main()
{
    const derf_head_arch tiny = {6, 4, 4, 64, -1, 0};
    const derf_head_arch bad_depth = {10, 4, 0, 128, -1, 0};
    const derf_head_arch no_kernel = {10, 4, 8, 96, 5, 64};
    const long long n = derf_weights_count(&tiny);
    expect(n > 0, "weights count of the 4x64 head");
    expect(derf_weights_count(&bad_depth) == -1, "weights count of depth 0");
    expect(derf_weights_count(nullptr) == -1, "weights count of NULL");

    const int K = 4;
    std::vector<float> sites(3 * 257, 0.0f), weights((size_t)n * K, 0.0f);
    derf_handle *h = reinterpret_cast<derf_handle *>(0x1);
    expect(derf_create(nullptr, K, sites.data(), &tiny, weights.data(), 0) == DERF_ERR_INVALID_ARG,
           "create without an output pointer");
    expect(derf_create(&h, 0, sites.data(), &tiny, weights.data(), 0) == DERF_ERR_INVALID_ARG &&
               h == nullptr,
           "create with no sites clears the handle");
    expect(derf_create(&h, 257, sites.data(), &tiny, weights.data(), 0) == DERF_ERR_INVALID_ARG,
           "create with 257 sites");
    expect(derf_create(&h, K, sites.data(), &tiny, weights.data(), 9) == DERF_ERR_INVALID_ARG,
           "create with an unknown precision");
    expect(derf_create(&h, K, sites.data(), nullptr, weights.data(), 0) == DERF_ERR_INVALID_ARG,
           "create without an architecture");
    expect(derf_create(&h, K, sites.data(), &no_kernel, weights.data(), 1) == DERF_ERR_UNSUPPORTED,
           "create with an architecture that has no kernel");
    sites[4] = NAN;
    expect(derf_create(&h, K, sites.data(), &tiny, weights.data(), 0) == DERF_ERR_INVALID_ARG,
           "create with a non-finite site");
    sites[4] = 0.0f;
    weights[(size_t)n * K - 1] = INFINITY;
    expect(derf_create(&h, K, sites.data(), &tiny, weights.data(), 0) == DERF_ERR_INVALID_ARG,
           "create with a non-finite weight");
    weights[(size_t)n * K - 1] = 0.0f;
    // valid arguments: on a machine without a GPU the device setup fails and
    // the partly built handle is destroyed; with one, a handle comes back
    h = reinterpret_cast<derf_handle *>(0x1);
    const int rc = derf_create(&h, K, sites.data(), &tiny, weights.data(), 0);
    expect((rc == DERF_OK) == (h != nullptr), "a handle exactly when create succeeds");
    expect(rc == DERF_OK || rc == DERF_ERR_HIP || rc == DERF_ERR_OOM, "create's status");
    derf_destroy(h);

    derf_head_arch mixed[3] = {tiny, tiny, no_kernel};
    h = reinterpret_cast<derf_handle *>(0x1);
    expect(derf_create_mixed(&h, 3, sites.data(), mixed, weights.data(), 1) ==
                   DERF_ERR_UNSUPPORTED &&
               h == nullptr,
           "mixed create with one unsupported head");
    expect(strstr(derf_last_error(), "head 2") != nullptr, "the error names the head");

    const derf_sampling samp = {32, 0, 1, 1, 0};
    float dummy[16] = {0};
    expect(derf_render(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, dummy, dummy, dummy,
                       nullptr) == DERF_ERR_INVALID_ARG,
           "render without a handle");
    expect(derf_render_noalloc(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, dummy, dummy, dummy,
                               nullptr) == DERF_ERR_INVALID_ARG,
           "no-allocation render without a handle");
    expect(derf_render_debug(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, dummy, dummy, dummy,
                             nullptr, nullptr) == DERF_ERR_INVALID_ARG,
           "debug render without a handle");
    expect(derf_render_soft(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, 1.0f, dummy, dummy, dummy,
                            nullptr, nullptr) == DERF_ERR_INVALID_ARG,
           "soft render without a handle");
    expect(derf_render_culled(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, 1e-3f, 4, 0, dummy,
                              dummy, dummy, nullptr, nullptr) == DERF_ERR_INVALID_ARG,
           "culled render without a handle");
    expect(derf_render_gated(nullptr, dummy, dummy, 1, 2.0f, 6.0f, &samp, dummy, dummy, dummy,
                             nullptr, nullptr) == DERF_ERR_INVALID_ARG,
           "gated render without a handle");
    expect(derf_set_gate(nullptr, 6, 16, dummy) == DERF_ERR_INVALID_ARG, "gate without a handle");
    expect(derf_gate_weights_count(4, 6, 16) == 16 * 39 + 16 + 4 * 16 + 4, "gate weights count");
    expect(derf_gate_weights_count(0, 6, 16) == -1, "gate weights count of no heads");
    expect(derf_set_empty_heads(nullptr, nullptr) == DERF_ERR_INVALID_ARG,
           "empty heads without a handle");
    expect(derf_set_timing(nullptr, 1) == DERF_ERR_INVALID_ARG, "timing without a handle");
    expect(derf_set_encoding(nullptr, DERF_ENCODING_STORED) == DERF_ERR_INVALID_ARG,
           "encoding without a handle");
    expect(derf_reset_stats(nullptr) == DERF_ERR_INVALID_ARG, "reset without a handle");
    derf_stats st;
    expect(derf_get_stats(nullptr, &st) == DERF_ERR_INVALID_ARG, "stats without a handle");
    derf_destroy(nullptr);
    expect(strcmp(derf_status_string(DERF_ERR_OOM), "out of memory") == 0, "status string");
    expect(strcmp(derf_status_string(-99), "unknown status") == 0, "unknown status string");
    // an architecture whose weight count is huge is refused before the
    // weights are read
    derf_head_arch weird = tiny;
    weird.width = 4096;
    expect(derf_create(&h, K, sites.data(), &weird, weights.data(), 1) == DERF_ERR_UNSUPPORTED,
           "create with a very wide head");
    expect(strlen(derf_last_error()) < 512, "error text fits its buffer");
    fault_injection();
    printf("abi driver: %d failure(s)\n", failures);
    return failures == 0 ? 0 : 1;
}
