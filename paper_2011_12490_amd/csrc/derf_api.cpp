// Host side of the C ABI declared in include/derf.h: argument checking,
// weight layout at creation, workspace management and the stream-ordered
// launch sequence of a render.
#include "derf.h"

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <new>
#include <vector>

#include "derf_internal.h"
#include "derf_cull.h"

using namespace derf;

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(DERF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                  \
    do {                                     \
        hipError_t e_ = (expr);              \
        if (e_ != hipSuccess)                \
            return hip_fail(e_, what);       \
    } while (0)

long long weights_count(const derf_head_arch *a)
{
    const long long P = 3 + 6LL * a->pos_freqs, Dd = 3 + 6LL * a->dir_freqs, W = a->width;
    long long n = 0;
    for (int l = 0; l < a->depth; ++l) {
        const long long in = l == 0 ? P : (l == a->skip_layer ? P + W : W);
        n += W * in + W;
    }
    n += W + 1;
    if (a->rgb_hidden > 0)
        n += (long long)a->rgb_hidden * (W + Dd) + a->rgb_hidden + 3LL * a->rgb_hidden + 3;
    else
        n += 3 * (W + Dd) + 3;
    return n;
}

bool arch_values_valid(const derf_head_arch *a)
{
    return a->pos_freqs >= 0 && a->pos_freqs <= 16 && a->dir_freqs >= 0 && a->dir_freqs <= 16 &&
           a->depth >= 1 && a->depth <= 64 && a->width >= 1 && a->width <= 4096 &&
           (a->skip_layer == -1 || (a->skip_layer >= 1 && a->skip_layer < a->depth)) &&
           a->rgb_hidden >= 0 && a->rgb_hidden <= 4096;
}

struct Workspace {
    void *mem = nullptr;
    size_t bytes = 0;
};

// Scratch memory of derf_render_noalloc: a fixed device array instead of the
// handle's workspace, so that a render allocates nothing.  Each device that
// loads the library holds its own copy until the process ends.  In host code
// `scratch` names a host-side stand-in, not the device array: its device
// address comes from hipGetSymbolAddress, once per device (scratch_on_device),
// and only that address is ever passed to a kernel.
constexpr size_t kScratchBytes = size_t(DERF_NOALLOC_SCRATCH_BYTES);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Allocation-failure injection, compiled only into test builds
// (-DDERF_FAULT_INJECTION): after derf_debug_fail_alloc(n), the allocation
// n allocations later -- device memory or the handle and its host staging --
// fails as if memory had run out, once.  The tests use it to show that every
// such failure returns DERF_ERR_OOM, hands out no handle and leaks nothing.
// Those builds also count the live allocations (device blocks and handles),
// so that a test can see every one released.
#ifdef DERF_FAULT_INJECTION
std::atomic<long> g_fail_in{-1};
std::atomic<long> g_live{0};
bool injected_failure()
{
    long c = g_fail_in.load();
    while (c >= 0 && !g_fail_in.compare_exchange_weak(c, c - 1)) {
    }
    return c == 0;
}
void count_live(long d) { g_live += d; }
#else
constexpr bool injected_failure() { return false; }
inline void count_live(long) {}
#endif

hipError_t dev_alloc(void **p, size_t bytes)
{
    if (injected_failure()) {
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    const hipError_t e = hipMalloc(p, bytes);
    if (e == hipSuccess)
        count_live(1);
    return e;
}

hipError_t dev_free(void *p)
{
    if (!p)
        return hipSuccess;
    count_live(-1);
    return hipFree(p);
}

constexpr int kPasses = 2;
constexpr int kEvents = 2 * kPasses * DERF_NUM_STAGES;
inline int ev_index(int pass, int stage, int end) { return 2 * (pass * DERF_NUM_STAGES + stage) + end; }

}  // namespace

struct derf_handle {
    int device = 0;
    int num_sites = 0;
    bool bf16 = false;
    int mlp_grid = 0;
    float4 *sites = nullptr;
    // heads grouped by architecture: one MLP variant and one launch per group;
    // a group's weights are laid out for every head index, its own filled
    struct HeadGroup {
        const MlpVariant *mlp = nullptr;
        unsigned char *streams = nullptr;
        float *blocks = nullptr;
        HeadMask members{};
    } groups[kMaxHeadGroups];
    int num_groups = 0;
    Workspace ws;
    hipStream_t last_stream = nullptr;
    bool timing = false;
    // one event pair per (pass, stage): pass 0 is the single or coarse pass,
    // pass 1 the fine pass of hierarchical sampling
    hipEvent_t ev[kEvents] = {};
    unsigned ev_mask = 0;      // event pairs recorded by the pending render
    bool ev_pending = false;
    derf_stats stats{};
    // 0-capacity heads (derf_set_empty_heads)
    HeadMask empty{};
    // per-head counts of the last render (device pointers into the workspace)
    unsigned *totals = nullptr;
    unsigned *totals_fine = nullptr;
    int totals_sets = 1;  // a culled render: one set of K totals per level
    // segment counts of the last render's cell walks (nullptr: no walk)
    const unsigned char *walk_nseg = nullptr;
    unsigned walk_rays = 0;
    // device address of this device's noalloc scratch array
    void *scratch = nullptr;
    // MLP gating (derf_set_gate): the gate laid out for its kernel on the
    // device (gate_pack), or none
    unsigned char *gate_w = nullptr;
    int gate_freqs = 0;
    int gate_hidden = 0;
    // derf_set_encoding: gamma(x) stored in a table by a separate pass
    // (bytes per sample of the table), or 0: encoded inside the MLP
    size_t gx_bytes = 0;
};

namespace {

// assignment blocks of S samples (S up to 2^32 - 1: the sum is taken in 64 bits)
inline unsigned blocks_of(unsigned S)
{
    return (unsigned)(((unsigned long long)S + kBucketBlock - 1) / kBucketBlock);
}
inline unsigned blocks_of_ll(unsigned long long n)
{
    return (unsigned)((n + kBucketBlock - 1) / kBucketBlock);
}

template <class T>
T *carve(char *&p, size_t count)
{
    T *r = reinterpret_cast<T *>(p);
    p += ((count * sizeof(T) + 255) / 256) * 256;
    return r;
}

// Workspace of one render.  S samples of the single (or coarse) pass and Sf
// of the fine pass (0 without hierarchical sampling); the bucket and the
// per-block counts are reused by the fine pass.
struct Buffers {
    float *t;
    uint8_t *cell;
    float4 *sr;
    float *t_fine;
    uint8_t *cell_fine;
    float4 *sr_fine;
    unsigned *bucket;
    void *dirbuf;
    unsigned *counts;
    unsigned *totals;
    unsigned *totals_fine;
    unsigned *mlp_queue;
    SegRec *walk_seg;            // [R][kMaxSeg] (heads >= kWalkSites)
    unsigned char *walk_nseg;    // [R]
    void *gxtab;                 // [max(S, Sf)] rows of gx_bytes (stored encoding), or null
};

size_t layout(char *base, unsigned S, unsigned Sf, unsigned R, unsigned nblk, int K, bool bf16,
              size_t gx_bytes, Buffers *b)
{
    char *p = base;
    Buffers x;
    x.t = carve<float>(p, S);
    x.cell = carve<uint8_t>(p, (size_t)S + 16);
    x.sr = carve<float4>(p, S);
    x.t_fine = carve<float>(p, Sf);
    x.cell_fine = carve<uint8_t>(p, Sf ? (size_t)Sf + 16 : 0);
    x.sr_fine = carve<float4>(p, Sf);
    x.bucket = carve<unsigned>(p, S > Sf ? S : Sf);
    x.dirbuf = carve<char>(p, (size_t)R * kDirPad * (bf16 ? 2 : 4));
    x.counts = carve<unsigned>(p, (size_t)nblk * K);
    x.totals = carve<unsigned>(p, K);
    x.totals_fine = carve<unsigned>(p, K);
    x.mlp_queue = carve<unsigned>(p, kMlpQueues * kMaxHeadGroups);
    const bool walk = K >= kWalkSites;
    x.walk_seg = walk ? carve<SegRec>(p, (size_t)R * kMaxSeg) : nullptr;
    x.walk_nseg = walk ? carve<unsigned char>(p, R) : nullptr;
    x.gxtab = gx_bytes ? carve<char>(p, (size_t)(S > Sf ? S : Sf) * gx_bytes) : nullptr;
    if (b)
        *b = x;
    return (size_t)(p - base);
}

}  // namespace

// The grouped-MLP variant of a head architecture, or nullptr if none is built.
const MlpVariant *derf::find_mlp_variant(const HeadArch &a, bool bf16)
{
    if (a.dir_freqs != 4)
        return nullptr;
    auto is = [&](int p, int d, int w, int sk, int rh) {
        return a.pos_freqs == p && a.depth == d && a.width == w && a.skip_layer == sk &&
               a.rgb_hidden == rh;
    };
    if (is(6, 4, 64, -1, 0))
        return mlp_variant_4x64(bf16);
    if (is(10, 8, 128, 5, 64))
        return mlp_variant_8x128(bf16);
    if (is(10, 6, 64, -1, 32))
        return mlp_variant_6x64(bf16);
    if (is(10, 8, 256, 5, 128))
        return mlp_variant_8x256(bf16);
    return nullptr;
}

namespace {

// The grouped MLP over every head: one launch per architecture group, each
// skipping the other groups' heads and the 0-capacity ones, with its own
// tile counters.  gxtab: the stored gamma(x) table of g's samples (the
// stored-encoding forms run), or null.
hipError_t launch_groups(const derf_handle *h, const unsigned *bucket, const unsigned *totals,
                         const RenderGeometry &g, const float *t, const void *dirbuf, float4 *sr,
                         unsigned *queue, bool soft, hipStream_t s,
                         const unsigned *offsets = nullptr, const void *gxtab = nullptr)
{
    for (int gi = 0; gi < h->num_groups; ++gi) {
        const derf_handle::HeadGroup &grp = h->groups[gi];
        const MlpVariant *v = gxtab ? grp.mlp->stored : grp.mlp;
        if (!v)
            return hipErrorInvalidValue;
        HeadMask skip;
        for (int w = 0; w < kMaxSites / 32; ++w)
            skip.w[w] = ~grp.members.w[w] | h->empty.w[w];
        const hipError_t e =
            v->launch(bucket, totals, offsets, h->num_sites, g, t, dirbuf, gxtab, grp.streams,
                      grp.blocks, sr, queue + kMlpQueues * gi, h->mlp_grid, soft, skip, s);
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

// The device address of the noalloc scratch array on device dev (the current
// device), looked up once per device and kept.
int scratch_on_device(int dev, void **out)
{
    if (dev < 0 || dev >= kMaxDevices)
        return fail(DERF_ERR_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DERF_OK;
}

// Grows the handle's workspace to at least need bytes.  Every device
// allocation of the library goes through dev_alloc.
int ensure_workspace(derf_handle *h, size_t need)
{
    if (need <= h->ws.bytes)
        return DERF_OK;
    // the old workspace may still be in use by work on the previous stream
    if (h->last_stream || h->ws.mem)
        HIP_TRY(hipStreamSynchronize(h->last_stream), "hipStreamSynchronize");
    if (h->ws.mem)
        HIP_TRY(dev_free(h->ws.mem), "hipFree");
    h->ws.mem = nullptr;
    h->ws.bytes = 0;
    const size_t grow = need + need / 8;
    if (dev_alloc(&h->ws.mem, grow) != hipSuccess) {
        (void)hipGetLastError();
        h->ws.mem = nullptr;
        return fail(DERF_ERR_OOM, "workspace of %zu bytes", grow);
    }
    h->ws.bytes = grow;
    return DERF_OK;
}

// Workspace of a soft render: S samples, every head's outputs for each.
struct SoftBuffers {
    float *t;
    uint8_t *cell;
    unsigned *bucket;
    void *dirbuf;
    unsigned *counts;
    unsigned *totals;
    unsigned *mlp_queue;
    float4 *sr;  // [K][S]
};

size_t layout_soft(char *base, unsigned S, unsigned R, unsigned nblk, int K, bool bf16,
                   SoftBuffers *b)
{
    char *p = base;
    SoftBuffers x;
    x.t = carve<float>(p, S);
    x.cell = carve<uint8_t>(p, (size_t)S + 16);
    x.bucket = carve<unsigned>(p, S);
    x.dirbuf = carve<char>(p, (size_t)R * kDirPad * (bf16 ? 2 : 4));
    x.counts = carve<unsigned>(p, (size_t)nblk * K);
    x.totals = carve<unsigned>(p, K);
    x.mlp_queue = carve<unsigned>(p, kMlpQueues * kMaxHeadGroups);
    x.sr = carve<float4>(p, (size_t)K * S);
    if (b)
        *b = x;
    return (size_t)(p - base);
}

// Adds the pending render's stage times: per stage, the sum over passes;
// stage_launches counts the renders that ran the stage.
void accumulate_timing(derf_handle *h)
{
    if (!h->ev_pending)
        return;
    for (int s = 0; s < DERF_NUM_STAGES; ++s) {
        bool ran = false;
        for (int pass = 0; pass < kPasses; ++pass) {
            const int k = pass * DERF_NUM_STAGES + s;
            float ms = 0.0f;
            if ((h->ev_mask >> k) & 1u &&
                hipEventElapsedTime(&ms, h->ev[ev_index(pass, s, 0)], h->ev[ev_index(pass, s, 1)]) ==
                    hipSuccess) {
                h->stats.stage_ms[s] += ms;
                ran = true;
            }
        }
        if (ran)
            h->stats.stage_launches[s] += 1;
    }
    h->ev_pending = false;
}

// the last event the pending render recorded
hipEvent_t last_event(const derf_handle *h)
{
    for (int k = kPasses * DERF_NUM_STAGES - 1; k >= 0; --k)
        if ((h->ev_mask >> k) & 1u)
            return h->ev[2 * k + 1];
    return nullptr;
}

// fixed_ws: a workspace of fixed_bytes to use instead of the handle's own
// (derf_render_noalloc: nothing is allocated, larger frames are refused).
int render_impl(derf_handle *h, const float *rays_o, const float *rays_d, long long num_rays,
                float near_t, float far_t, const derf_sampling *samp, float *out_rgb,
                float *out_depth, float *out_opacity, const derf_debug_out *dbg, void *stream,
                void *fixed_ws = nullptr, size_t fixed_bytes = 0)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (!samp)
        return fail(DERF_ERR_INVALID_ARG, "null sampling descriptor");
    if (num_rays < 0 || num_rays >= (1LL << 30))
        return fail(DERF_ERR_INVALID_ARG, "need 0 <= num_rays < 2^30");
    if (!(near_t < far_t) || !isfinite(near_t) || !isfinite(far_t))
        return fail(DERF_ERR_INVALID_ARG, "need finite near < far");
    if (samp->n_coarse < 1 || samp->n_fine < 0 || samp->n_coarse + samp->n_fine > 1024)
        return fail(DERF_ERR_INVALID_ARG, "need 1 <= n_coarse, 0 <= n_fine, total <= 1024");
    if (samp->n_fine > 0 && samp->n_coarse < 2)
        return fail(DERF_ERR_INVALID_ARG, "hierarchical sampling needs n_coarse >= 2");
    if (num_rays == 0)
        return DERF_OK;
    if (!rays_o || !rays_d || !out_rgb || !out_depth || !out_opacity)
        return fail(DERF_ERR_INVALID_ARG, "null ray or output pointer");
    const unsigned long long S64 =
        (unsigned long long)num_rays * (unsigned)(samp->n_coarse + samp->n_fine);
    if (S64 >= (1ull << 32))
        return fail(DERF_ERR_INVALID_ARG,
                    "num_rays * (n_coarse + n_fine) must be < 2^32 per call");

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
    const bool hier = samp->n_fine > 0;
    const unsigned R = (unsigned)num_rays, N = (unsigned)samp->n_coarse, NF = (unsigned)samp->n_fine;
    const unsigned S = R * N, Sf = R * NF;
    const unsigned nblk = blocks_of(S);
    const unsigned nblk_f = blocks_of(Sf);
    const unsigned nblk_max = nblk > nblk_f ? nblk : nblk_f;
    const size_t need =
        layout(nullptr, S, Sf, R, nblk_max, h->num_sites, h->bf16, h->gx_bytes, nullptr);
    int rc = DERF_OK;
    if (fixed_ws) {
        if (need > fixed_bytes)
            return fail(DERF_ERR_INVALID_ARG,
                        "frame needs %zu bytes of scratch, the no-allocation render has %zu "
                        "(render fewer rays per call)",
                        need, fixed_bytes);
    } else {
        rc = ensure_workspace(h, need);
        if (rc != DERF_OK)
            return rc;
    }
    if (h->timing && h->ev_pending) {
        HIP_TRY(hipEventSynchronize(last_event(h)), "hipEventSynchronize");
        accumulate_timing(h);
    }
    Buffers b;
    layout(reinterpret_cast<char *>(fixed_ws ? fixed_ws : h->ws.mem), S, Sf, R, nblk_max,
           h->num_sites, h->bf16, h->gx_bytes, &b);

    RenderGeometry g;
    g.rays_o = rays_o;
    g.rays_d = rays_d;
    g.num_rays = R;
    g.n = N;
    g.num_samples = S;
    g.inv_n = 1.0 / (double)N;
    g.near_t = near_t;
    g.far_t = far_t;
    g.step = (far_t - near_t) / (float)N;
    g.seed = samp->seed;
    g.ray_offset = samp->ray_offset;
    g.perturb = samp->perturb ? 1 : 0;

    h->ev_mask = 0;
    auto mark = [&](int pass, int stage, int end) -> hipError_t {
        if (!h->timing)
            return hipSuccess;
        h->ev_mask |= 1u << (pass * DERF_NUM_STAGES + stage);
        return hipEventRecord(h->ev[ev_index(pass, stage, end)], s);
    };
    // assignment counts -> bucket -> per-head MLP of one pass
    auto bucket_and_mlp = [&](int pass, const RenderGeometry &gp, const float *t,
                              const uint8_t *cell, unsigned nb, unsigned *totals,
                              float4 *sr) -> int {
        HIP_TRY(mark(pass, DERF_STAGE_BUCKET_SCAN, 0), "hipEventRecord");
        HIP_TRY(launch_bucket_scan(b.counts, nb, h->num_sites, totals, b.mlp_queue, s),
                "bucket_scan launch");
        HIP_TRY(mark(pass, DERF_STAGE_BUCKET_SCAN, 1), "hipEventRecord");
        HIP_TRY(mark(pass, DERF_STAGE_BUCKET_SCATTER, 0), "hipEventRecord");
        HIP_TRY(launch_bucket_scatter(cell, b.counts, totals, gp.num_samples, nb, h->num_sites,
                                      h->empty, b.bucket, sr, s),
                "bucket_scatter launch");
        HIP_TRY(mark(pass, DERF_STAGE_BUCKET_SCATTER, 1), "hipEventRecord");
        HIP_TRY(mark(pass, DERF_STAGE_MLP, 0), "hipEventRecord");
        HIP_TRY(launch_groups(h, b.bucket, totals, gp, t, b.dirbuf, sr, b.mlp_queue, false, s,
                              nullptr, b.gxtab),
                "mlp launch");
        HIP_TRY(mark(pass, DERF_STAGE_MLP, 1), "hipEventRecord");
        return DERF_OK;
    };

    // ---- single or coarse pass: stratified samples (Sec. 3.1)
    HIP_TRY(mark(0, DERF_STAGE_SAMPLE, 0), "hipEventRecord");
    HIP_TRY(launch_ray_encode(g, b.dirbuf, h->bf16, s), "ray_encode launch");
    const WalkTable walk{b.walk_seg, b.walk_nseg};
    if (walk.seg)
        HIP_TRY(launch_ray_walk(g, h->sites, h->num_sites, b.walk_seg, b.walk_nseg, s),
                "ray_walk launch");
    HIP_TRY(launch_sample_assign(g, h->sites, h->num_sites, walk, b.t, b.cell,
                                 b.counts, nblk, s),
            "sample_assign launch");
    if (b.gxtab)
        HIP_TRY(h->groups[0].mlp->stored->encode(g, b.t, b.gxtab, h->mlp_grid, s),
                "gx_encode launch");
    HIP_TRY(mark(0, DERF_STAGE_SAMPLE, 1), "hipEventRecord");
    rc = bucket_and_mlp(0, g, b.t, b.cell, nblk, b.totals, b.sr);
    if (rc != DERF_OK)
        return rc;
    const bool want_dbg = dbg && (dbg->cell || dbg->t || dbg->sigma || dbg->rgb);
    if (!hier) {
        HIP_TRY(mark(0, DERF_STAGE_COMPOSITE, 0), "hipEventRecord");
        HIP_TRY(launch_composite(g, b.t, b.cell, b.sr, out_rgb, out_depth, out_opacity, s),
                "composite launch");
        HIP_TRY(mark(0, DERF_STAGE_COMPOSITE, 1), "hipEventRecord");
        if (want_dbg)
            HIP_TRY(launch_debug_expand(S, b.t, b.cell, b.sr, dbg->cell, dbg->t, dbg->sigma,
                                        dbg->rgb, s),
                    "debug_expand launch");
    } else {
        // ---- fine pass: inverse-CDF depths from the coarse weights, their
        // cells and heads; the coarse outputs are reused in the composite
        HIP_TRY(mark(0, DERF_STAGE_FINE, 0), "hipEventRecord");
        HIP_TRY(launch_fine_sample(g, b.t, b.sr, NF, b.t_fine, s), "fine_sample launch");
        HIP_TRY(mark(0, DERF_STAGE_FINE, 1), "hipEventRecord");
        RenderGeometry gf = g;
        gf.n = NF;
        gf.num_samples = Sf;
        gf.inv_n = 1.0 / (double)NF;
        HIP_TRY(mark(1, DERF_STAGE_SAMPLE, 0), "hipEventRecord");
        HIP_TRY(launch_assign_given(gf, h->sites, h->num_sites, walk, b.t_fine,
                                    b.cell_fine, b.counts, nblk_f, s),
                "assign launch");
        if (b.gxtab)
            HIP_TRY(h->groups[0].mlp->stored->encode(gf, b.t_fine, b.gxtab, h->mlp_grid, s),
                    "gx_encode launch");
        HIP_TRY(mark(1, DERF_STAGE_SAMPLE, 1), "hipEventRecord");
        rc = bucket_and_mlp(1, gf, b.t_fine, b.cell_fine, nblk_f, b.totals_fine, b.sr_fine);
        if (rc != DERF_OK)
            return rc;
        HIP_TRY(mark(1, DERF_STAGE_COMPOSITE, 0), "hipEventRecord");
        HIP_TRY(launch_merge_composite(g, b.t, b.cell, b.sr, NF, b.t_fine, b.cell_fine, b.sr_fine,
                                       out_rgb, out_depth, out_opacity,
                                       want_dbg ? dbg->cell : nullptr, want_dbg ? dbg->t : nullptr,
                                       want_dbg ? dbg->sigma : nullptr,
                                       want_dbg ? dbg->rgb : nullptr, s),
                "merge_composite launch");
        HIP_TRY(mark(1, DERF_STAGE_COMPOSITE, 1), "hipEventRecord");
    }
    h->ev_pending = h->timing;
    h->last_stream = s;
    h->totals = b.totals;
    h->totals_fine = hier ? b.totals_fine : nullptr;
    h->totals_sets = 1;
    h->walk_nseg = b.walk_nseg;
    h->walk_rays = b.walk_nseg ? R : 0;
    h->stats.renders += 1;
    h->stats.samples += (long long)S + Sf;
    return DERF_OK;
}

// Soft decomposition (Sec. 3.2 Eq. 4-6 with Eq. 8): stratified samples,
// every head on every sample, blend + composite (+ contributions).
int render_soft_impl(derf_handle *h, const float *rays_o, const float *rays_d,
                     long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                     float beta, float *out_rgb, float *out_depth, float *out_opacity,
                     float *out_contrib, void *stream)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (!samp)
        return fail(DERF_ERR_INVALID_ARG, "null sampling descriptor");
    if (num_rays < 0 || num_rays >= (1LL << 30))
        return fail(DERF_ERR_INVALID_ARG, "need 0 <= num_rays < 2^30");
    if (!(near_t < far_t) || !isfinite(near_t) || !isfinite(far_t))
        return fail(DERF_ERR_INVALID_ARG, "need finite near < far");
    if (!(beta >= 0.0f) || !isfinite(beta))
        return fail(DERF_ERR_INVALID_ARG, "need a finite beta >= 0");
    if (samp->n_coarse < 1 || samp->n_coarse > 1024 || samp->n_fine < 0)
        return fail(DERF_ERR_INVALID_ARG, "need 1 <= n_coarse <= 1024, n_fine >= 0");
    if (samp->n_fine != 0)
        return fail(DERF_ERR_UNSUPPORTED, "the soft render has no hierarchical sampling");
    if (h->gx_bytes)
        return fail(DERF_ERR_UNSUPPORTED, "the soft render has no stored encoding");
    if (num_rays == 0)
        return DERF_OK;
    if (!rays_o || !rays_d || !out_rgb || !out_depth || !out_opacity)
        return fail(DERF_ERR_INVALID_ARG, "null ray or output pointer");
    const unsigned long long KS64 =
        (unsigned long long)num_rays * (unsigned)samp->n_coarse * (unsigned)h->num_sites;
    if (KS64 >= (1ull << 32))
        return fail(DERF_ERR_INVALID_ARG, "num_rays * n_coarse * K must be < 2^32 per call");

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
    const unsigned R = (unsigned)num_rays, N = (unsigned)samp->n_coarse, S = R * N;
    const unsigned nblk = blocks_of(S);
    int rc = ensure_workspace(h, layout_soft(nullptr, S, R, nblk, h->num_sites, h->bf16, nullptr));
    if (rc != DERF_OK)
        return rc;
    if (h->timing && h->ev_pending) {
        HIP_TRY(hipEventSynchronize(last_event(h)), "hipEventSynchronize");
        accumulate_timing(h);
    }
    SoftBuffers b;
    layout_soft(reinterpret_cast<char *>(h->ws.mem), S, R, nblk, h->num_sites, h->bf16, &b);

    RenderGeometry g;
    g.rays_o = rays_o;
    g.rays_d = rays_d;
    g.num_rays = R;
    g.n = N;
    g.num_samples = S;
    g.inv_n = 1.0 / (double)N;
    g.near_t = near_t;
    g.far_t = far_t;
    g.step = (far_t - near_t) / (float)N;
    g.seed = samp->seed;
    g.ray_offset = samp->ray_offset;
    g.perturb = samp->perturb ? 1 : 0;

    h->ev_mask = 0;
    auto mark = [&](int stage, int end) -> hipError_t {
        if (!h->timing)
            return hipSuccess;
        h->ev_mask |= 1u << stage;
        return hipEventRecord(h->ev[ev_index(0, stage, end)], s);
    };
    // stratified depths (the owning cells it also writes are not used)
    HIP_TRY(mark(DERF_STAGE_SAMPLE, 0), "hipEventRecord");
    HIP_TRY(launch_ray_encode(g, b.dirbuf, h->bf16, s), "ray_encode launch");
    HIP_TRY(launch_sample_assign(g, h->sites, h->num_sites, WalkTable{nullptr, nullptr},
                                 b.t, b.cell, b.counts, nblk, s),
            "sample_assign launch");
    HIP_TRY(launch_soft_setup(S, h->num_sites, b.bucket, b.totals, b.mlp_queue, s),
            "soft_setup launch");
    HIP_TRY(mark(DERF_STAGE_SAMPLE, 1), "hipEventRecord");
    HIP_TRY(mark(DERF_STAGE_MLP, 0), "hipEventRecord");
    HIP_TRY(launch_groups(h, b.bucket, b.totals, g, b.t, b.dirbuf, b.sr, b.mlp_queue, true, s),
            "mlp launch");
    HIP_TRY(mark(DERF_STAGE_MLP, 1), "hipEventRecord");
    HIP_TRY(mark(DERF_STAGE_COMPOSITE, 0), "hipEventRecord");
    HIP_TRY(launch_soft_composite(g, h->sites, h->num_sites, h->empty, beta, b.t, b.sr, out_rgb,
                                  out_depth, out_opacity, out_contrib, s),
            "soft_composite launch");
    HIP_TRY(mark(DERF_STAGE_COMPOSITE, 1), "hipEventRecord");
    h->ev_pending = h->timing;
    h->last_stream = s;
    h->totals = b.totals;
    h->totals_fine = nullptr;
    h->totals_sets = 1;
    h->walk_nseg = nullptr;
    h->walk_rays = 0;
    h->stats.renders += 1;
    h->stats.samples += (long long)S;
    return DERF_OK;
}

// Workspace of a culled render: the single-pass buffers, then the level
// bounds, the transmittance and one set of head totals per level.
struct CullBuffers {
    unsigned *lb;            // [R][levels + 1]
    uint8_t *lvl;            // [S]
    float *trans;            // [R]
    unsigned *level_totals;  // [levels][K] samples evaluated per level and head
    // the one-pass (level, head) bucketing (levels K <= 256, levels > 1)
    unsigned *order;         // [S]
    unsigned *key_counts;    // [levels K][nblk]
    unsigned *key_totals;    // [levels K]
    unsigned *key_offsets;   // [levels K]
};

// The culled render buckets every level at once when its levels are pieces
// (many short levels: the one pass costs about two per-level passes and
// saves one per level) and the (level, head) keys fit the bucketing
// kernels' 256.
inline bool one_pass_levels(unsigned levels, int K, unsigned piece)
{
    return piece > 0 && levels > 2 && levels * K <= kMaxSites;
}

size_t layout_culled(char *base, unsigned S, unsigned R, unsigned nblk, int K, bool bf16,
                     unsigned levels, unsigned piece, Buffers *b, CullBuffers *c)
{
    char *p = base + layout(base, S, 0, R, nblk, K, bf16, 0, b);
    CullBuffers x;
    x.lb = carve<unsigned>(p, (size_t)R * (levels + 1));
    x.lvl = carve<uint8_t>(p, S);
    x.trans = carve<float>(p, R);
    x.level_totals = carve<unsigned>(p, (size_t)levels * K);
    const bool one = one_pass_levels(levels, K, piece);
    x.order = carve<unsigned>(p, one ? S : 0);
    x.key_counts = carve<unsigned>(p, one ? (size_t)levels * K * nblk : 0);
    x.key_totals = carve<unsigned>(p, one ? (size_t)levels * K : 0);
    x.key_offsets = carve<unsigned>(p, one ? (size_t)levels * K : 0);
    if (c)
        *c = x;
    return (size_t)(p - base);
}

// Painter's-order render with transmittance culling (Sec. 3.3): sampling and
// assignment as the single pass, then per level: counts of the live samples,
// offsets, scatter, the grouped MLP and the level's integration.
int render_culled_impl(derf_handle *h, const float *rays_o, const float *rays_d,
                       long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                       float eps, int levels, int piece, float *out_rgb, float *out_depth,
                       float *out_opacity, unsigned *out_evaluated, void *stream,
                       bool gated = false, int *out_cell = nullptr)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (gated && !h->gate_w)
        return fail(DERF_ERR_INVALID_ARG, "no gating network set (derf_set_gate)");
    if (!samp)
        return fail(DERF_ERR_INVALID_ARG, "null sampling descriptor");
    if (num_rays < 0 || num_rays >= (1LL << 30))
        return fail(DERF_ERR_INVALID_ARG, "need 0 <= num_rays < 2^30");
    if (!(near_t < far_t) || !isfinite(near_t) || !isfinite(far_t))
        return fail(DERF_ERR_INVALID_ARG, "need finite near < far");
    if (!(eps >= 0.0f) || !isfinite(eps))
        return fail(DERF_ERR_INVALID_ARG, "need a finite eps >= 0");
    if (levels < 1 || levels > kMaxLevels)
        return fail(DERF_ERR_INVALID_ARG, "need 1 <= levels <= %d", kMaxLevels);
    if (piece < 0)
        return fail(DERF_ERR_INVALID_ARG, "need piece >= 0");
    if (samp->n_coarse < 1 || samp->n_coarse > 1024 || samp->n_fine < 0)
        return fail(DERF_ERR_INVALID_ARG, "need 1 <= n_coarse <= 1024, n_fine >= 0");
    if (samp->n_fine != 0)
        return fail(DERF_ERR_UNSUPPORTED, "the culled render has no hierarchical sampling");
    if (h->gx_bytes)
        return fail(DERF_ERR_UNSUPPORTED, "the culled and gated renders have no stored encoding");
    if (num_rays == 0)
        return DERF_OK;
    if (!rays_o || !rays_d || !out_rgb || !out_depth || !out_opacity)
        return fail(DERF_ERR_INVALID_ARG, "null ray or output pointer");
    if ((unsigned long long)num_rays * (unsigned)samp->n_coarse >= (1ull << 32))
        return fail(DERF_ERR_INVALID_ARG, "num_rays * n_coarse must be < 2^32 per call");

    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
    const unsigned R = (unsigned)num_rays, N = (unsigned)samp->n_coarse, S = R * N;
    const unsigned L = (unsigned)levels, nblk = blocks_of(S);
    if (!gated && (L == 1 || eps == 0.0f ||
                   (h->num_sites == 1 && (piece == 0 || (unsigned)piece >= N)))) {
        // Nothing can stop a ray (one level; eps = 0, which every
        // transmittance passes; or one head in whole segments, where level 0
        // is the whole ray): the single pass, derf_render's outputs bitwise,
        // every sample evaluated.
        const int rc = render_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, out_rgb,
                                   out_depth, out_opacity, nullptr, stream);
        if (rc != DERF_OK)
            return rc;
        if (out_evaluated)
            HIP_TRY(launch_fill_u32(out_evaluated, R, N, reinterpret_cast<hipStream_t>(stream)),
                    "fill launch");
        return DERF_OK;
    }
    // a piece no shorter than the ray cuts nothing: the whole-segment levels
    const unsigned P = (unsigned)piece < N ? (unsigned)piece : 0u;
    const int K = h->num_sites;
    int rc =
        ensure_workspace(h, layout_culled(nullptr, S, R, nblk, K, h->bf16, L, P, nullptr, nullptr));
    if (rc != DERF_OK)
        return rc;
    if (h->timing && h->ev_pending) {
        HIP_TRY(hipEventSynchronize(last_event(h)), "hipEventSynchronize");
        accumulate_timing(h);
    }
    Buffers b;
    CullBuffers c;
    layout_culled(reinterpret_cast<char *>(h->ws.mem), S, R, nblk, K, h->bf16, L, P, &b, &c);

    RenderGeometry g;
    g.rays_o = rays_o;
    g.rays_d = rays_d;
    g.num_rays = R;
    g.n = N;
    g.num_samples = S;
    g.inv_n = 1.0 / (double)N;
    g.near_t = near_t;
    g.far_t = far_t;
    g.step = (far_t - near_t) / (float)N;
    g.seed = samp->seed;
    g.ray_offset = samp->ray_offset;
    g.perturb = samp->perturb ? 1 : 0;

    h->ev_mask = 0;
    auto mark = [&](int stage, int end) -> hipError_t {
        if (!h->timing)
            return hipSuccess;
        h->ev_mask |= 1u << stage;
        return hipEventRecord(h->ev[ev_index(0, stage, end)], s);
    };
    HIP_TRY(mark(DERF_STAGE_SAMPLE, 0), "hipEventRecord");
    HIP_TRY(launch_ray_encode(g, b.dirbuf, h->bf16, s), "ray_encode launch");
    // the gated assignment draws the depths itself and needs no nearest site
    const WalkTable walk{gated ? nullptr : b.walk_seg, gated ? nullptr : b.walk_nseg};
    if (gated) {
        HIP_TRY(launch_gate(g, h->gate_w, h->gate_freqs, h->gate_hidden, K, b.t, b.cell, out_cell,
                            h->mlp_grid, s),
                "gate launch");
    } else {
        if (walk.seg)
            HIP_TRY(launch_ray_walk(g, h->sites, K, b.walk_seg, b.walk_nseg, s),
                    "ray_walk launch");
        HIP_TRY(launch_sample_assign(g, h->sites, K, walk, b.t, b.cell, b.counts,
                                     nblk, s),
                "sample_assign launch");
    }
    HIP_TRY(launch_level_bounds(b.cell, N, R, L, P, c.lb, c.lvl, s),
            "level_bounds launch");
    // Levels cut into pieces: bucket every sample by (level, head) once; each
    // level after the first then compacts only its own samples, dropping
    // those of closed rays.  Otherwise each level counts and scatters its
    // live samples.
    const bool one_pass = one_pass_levels(L, K, P);
    if (one_pass) {
        HIP_TRY(launch_level_head_order(g, L, K, c.lvl, b.cell, h->empty, c.key_counts,
                                        nblk, c.key_totals, c.order, c.key_offsets,
                                        c.level_totals, b.sr, b.mlp_queue, s),
                "level_head_order launch");
    }
    HIP_TRY(mark(DERF_STAGE_SAMPLE, 1), "hipEventRecord");
    HIP_TRY(mark(DERF_STAGE_MLP, 0), "hipEventRecord");
    for (unsigned l = 0; l < L; ++l) {
        const CullLevel lv{c.lb, c.lvl, c.trans, out_evaluated, L, l, eps};
        unsigned *tot = c.level_totals + (size_t)l * K;
        if (one_pass) {
            const unsigned *src = c.order;
            if (l > 0) {
                // a level that is one piece holds at most P samples of each ray
                const unsigned lblk =
                    P > 0 && l + 1 < L ? std::min(nblk, blocks_of_ll((unsigned long long)R * P))
                                       : nblk;
                HIP_TRY(launch_level_compact(g, l, L, K, c.order, c.key_offsets,
                                             c.key_totals, c.lvl, b.cell, lblk, tot, b.bucket,
                                             b.mlp_queue, s),
                        "level_compact launch");
                src = b.bucket;
            }
            HIP_TRY(launch_groups(h, src, tot, g, b.t, b.dirbuf, b.sr, b.mlp_queue, false, s,
                                  c.key_offsets + (size_t)l * K),
                    "mlp launch");
        } else if (l + 1 < L) {
            // one run of one cell per open ray: bucketed ray by ray
            HIP_TRY(launch_level_ray_bucket(g, b.cell, K, h->empty, lv, b.counts, nblk, tot,
                                            b.totals, b.bucket, b.sr, b.mlp_queue, s),
                    "level_ray_bucket launch");
            HIP_TRY(launch_groups(h, b.bucket, tot, g, b.t, b.dirbuf, b.sr, b.mlp_queue, false, s),
                    "mlp launch");
        } else {
            HIP_TRY(launch_level_count(g, b.cell, K, lv, b.counts, nblk, s),
                    "level_count launch");
            HIP_TRY(launch_bucket_scan(b.counts, nblk, K, tot, b.mlp_queue, s),
                    "bucket_scan launch");
            HIP_TRY(launch_level_scatter(g, b.cell, b.counts, tot, nblk, K, h->empty,
                                         lv, b.bucket, b.sr, s),
                    "level_scatter launch");
            HIP_TRY(launch_groups(h, b.bucket, tot, g, b.t, b.dirbuf, b.sr, b.mlp_queue, false, s),
                    "mlp launch");
        }
        // every level but the last is one piece of at most P samples
        HIP_TRY(launch_level_composite(g, b.t, b.cell, b.sr, lv, l + 1 < L ? P : 0u, out_rgb,
                                       out_depth, out_opacity, s),
                "level_composite launch");
    }
    HIP_TRY(mark(DERF_STAGE_MLP, 1), "hipEventRecord");
    h->ev_pending = h->timing;
    h->last_stream = s;
    h->totals = c.level_totals;
    h->totals_fine = nullptr;
    h->totals_sets = levels;
    h->walk_nseg = walk.nseg;
    h->walk_rays = walk.nseg ? R : 0;
    h->stats.renders += 1;
    h->stats.samples += (long long)S;
    return DERF_OK;
}

// derf_create / derf_create_mixed: per_head says whether arch holds one
// architecture per head (weights then concatenated head after head) or one
// for all.  *h_out holds the handle under construction, so that a host
// allocation failure anywhere can free it (create_impl).
int create_body(derf_handle **out, int num_sites, const float *sites_xyz,
                const derf_head_arch *arch, bool per_head, const float *weights, int precision,
                derf_handle **h_out)
{
    if (!out)
        return fail(DERF_ERR_INVALID_ARG, "null output handle pointer");
    *out = nullptr;
    if (!sites_xyz || !arch || !weights)
        return fail(DERF_ERR_INVALID_ARG, "null sites, arch or weights");
    if (num_sites < 1 || num_sites > kMaxSites)
        return fail(DERF_ERR_INVALID_ARG, "num_sites must be in [1, 256]");
    if (precision != DERF_PREC_FP32 && precision != DERF_PREC_BF16)
        return fail(DERF_ERR_INVALID_ARG, "unknown precision %d", precision);
    for (int i = 0; i < 3 * num_sites; ++i)
        if (!isfinite(sites_xyz[i]))
            return fail(DERF_ERR_INVALID_ARG, "non-finite site coordinate");
    const bool bf16 = precision == DERF_PREC_BF16;
    // each head's kernel variant; heads sharing one form a group
    std::vector<const MlpVariant *> head_v(num_sites);
    std::vector<long long> woff(num_sites + 1, 0);
    for (int k = 0; k < num_sites; ++k) {
        const derf_head_arch *a = per_head ? arch + k : arch;
        if (!arch_values_valid(a))
            return fail(DERF_ERR_INVALID_ARG, "head %d: architecture values out of range", k);
        HeadArch ha{a->pos_freqs, a->dir_freqs, a->depth, a->width, a->skip_layer, a->rgb_hidden};
        head_v[k] = find_mlp_variant(ha, bf16);
        if (!head_v[k])
            return fail(DERF_ERR_UNSUPPORTED, "head %d: no %s kernel for arch (%d,%d,%d,%d,%d,%d)",
                        k, bf16 ? "bf16" : "fp32", a->pos_freqs, a->dir_freqs, a->depth, a->width,
                        a->skip_layer, a->rgb_hidden);
        woff[k + 1] = woff[k] + weights_count(a);
    }
    for (long long i = 0; i < woff[num_sites]; ++i)
        if (!isfinite(weights[i]))
            return fail(DERF_ERR_INVALID_ARG, "non-finite weight");

    derf_handle *h = injected_failure() ? nullptr : new (std::nothrow) derf_handle();
    if (!h)
        return fail(DERF_ERR_OOM, "handle");
    count_live(1);
    *h_out = h;
    auto cleanup = [&](int status) {
        derf_destroy(h);
        *h_out = nullptr;
        return status;
    };
    hipError_t e = hipGetDevice(&h->device);
    if (e != hipSuccess)
        return cleanup(hip_fail(e, "hipGetDevice"));
    int cus = 0;
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device);
    if (e != hipSuccess)
        return cleanup(hip_fail(e, "hipDeviceGetAttribute"));
    {
        const int rc = scratch_on_device(h->device, &h->scratch);
        if (rc != DERF_OK)
            return cleanup(rc);
    }
    h->num_sites = num_sites;
    h->bf16 = bf16;
    h->mlp_grid = cus;
    std::vector<int> head_group(num_sites);
    for (int k = 0; k < num_sites; ++k) {
        int gi = 0;
        while (gi < h->num_groups && h->groups[gi].mlp != head_v[k])
            ++gi;
        if (gi == h->num_groups) {
            if (h->num_groups == kMaxHeadGroups)
                return cleanup(fail(DERF_ERR_UNSUPPORTED, "more than %d head architectures",
                                    kMaxHeadGroups));
            h->groups[h->num_groups++].mlp = head_v[k];
        }
        head_group[k] = gi;
        h->groups[gi].members.w[k >> 5] |= 1u << (k & 31);
    }

    // sites as float4 (xyz, 0)
    std::vector<float4> sites(num_sites);
    for (int k = 0; k < num_sites; ++k)
        sites[k] = make_float4(sites_xyz[3 * k], sites_xyz[3 * k + 1], sites_xyz[3 * k + 2], 0.f);
    if (dev_alloc(reinterpret_cast<void **>(&h->sites), sizeof(float4) * num_sites) !=
        hipSuccess) {
        (void)hipGetLastError();
        return cleanup(fail(DERF_ERR_OOM, "device sites"));
    }
    e = hipMemcpy(h->sites, sites.data(), sizeof(float4) * num_sites, hipMemcpyHostToDevice);
    if (e != hipSuccess)
        return cleanup(hip_fail(e, "hipMemcpy"));
    // per group, the kernel layout of its heads (indexed by head; others zero)
    for (int gi = 0; gi < h->num_groups; ++gi) {
        derf_handle::HeadGroup &grp = h->groups[gi];
        const MlpVariant *v = grp.mlp;
        std::vector<unsigned char> streams;
        std::vector<float> blocks;
        try {
            if (injected_failure())
                throw std::bad_alloc();
            streams.assign(v->stream_bytes * num_sites, 0);
            blocks.assign(v->block_bytes / 4 * num_sites, 0.0f);
        } catch (...) {
            return cleanup(fail(DERF_ERR_OOM, "host staging"));
        }
        for (int k = 0; k < num_sites; ++k)
            if (head_group[k] == gi)
                v->pack(weights + woff[k], streams.data() + v->stream_bytes * k,
                        blocks.data() + v->block_bytes / 4 * k);
        if (dev_alloc(reinterpret_cast<void **>(&grp.streams), streams.size()) != hipSuccess ||
            dev_alloc(reinterpret_cast<void **>(&grp.blocks), blocks.size() * 4) != hipSuccess) {
            (void)hipGetLastError();
            return cleanup(fail(DERF_ERR_OOM, "device weights"));
        }
        e = hipMemcpy(grp.streams, streams.data(), streams.size(), hipMemcpyHostToDevice);
        if (e == hipSuccess)
            e = hipMemcpy(grp.blocks, blocks.data(), blocks.size() * 4, hipMemcpyHostToDevice);
        if (e != hipSuccess)
            return cleanup(hip_fail(e, "hipMemcpy"));
    }
    for (int i = 0; i < kEvents; ++i) {
        e = hipEventCreate(&h->ev[i]);
        if (e != hipSuccess)
            return cleanup(hip_fail(e, "hipEventCreate"));
    }
    e = hipDeviceSynchronize();
    if (e != hipSuccess)
        return cleanup(hip_fail(e, "hipDeviceSynchronize"));
    *out = h;
    *h_out = nullptr;
    return DERF_OK;
}

int create_impl(derf_handle **out, int num_sites, const float *sites_xyz,
                const derf_head_arch *arch, bool per_head, const float *weights, int precision)
{
    derf_handle *h = nullptr;
    try {
        return create_body(out, num_sites, sites_xyz, arch, per_head, weights, precision, &h);
    } catch (const std::bad_alloc &) {
        derf_destroy(h);
        if (out)
            *out = nullptr;
        return fail(DERF_ERR_OOM, "host memory");
    }
}

}  // namespace

extern "C" {

long long derf_weights_count(const derf_head_arch *arch)
{
    if (!arch || !arch_values_valid(arch))
        return -1;
    return weights_count(arch);
}

int derf_create(derf_handle **out, int num_sites, const float *sites_xyz,
                const derf_head_arch *arch, const float *weights, int precision)
{
    return create_impl(out, num_sites, sites_xyz, arch, false, weights, precision);
}

int derf_create_mixed(derf_handle **out, int num_sites, const float *sites_xyz,
                      const derf_head_arch *archs, const float *weights, int precision)
{
    return create_impl(out, num_sites, sites_xyz, archs, true, weights, precision);
}

int derf_render(derf_handle *h, const float *rays_o, const float *rays_d, long long num_rays,
                float near_t, float far_t, const derf_sampling *samp, float *out_rgb,
                float *out_depth, float *out_opacity, void *hip_stream)
{
    return render_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, out_rgb, out_depth,
                       out_opacity, nullptr, hip_stream);
}

int derf_render_debug(derf_handle *h, const float *rays_o, const float *rays_d,
                      long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                      float *out_rgb, float *out_depth, float *out_opacity,
                      const derf_debug_out *dbg, void *hip_stream)
{
    return render_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, out_rgb, out_depth,
                       out_opacity, dbg, hip_stream);
}

int derf_render_noalloc(derf_handle *h, const float *rays_o, const float *rays_d,
                        long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                        float *out_rgb, float *out_depth, float *out_opacity, void *hip_stream)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    return render_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, out_rgb, out_depth,
                       out_opacity, nullptr, hip_stream, h->scratch, kScratchBytes);
}

int derf_render_soft(derf_handle *h, const float *rays_o, const float *rays_d, long long num_rays,
                     float near_t, float far_t, const derf_sampling *samp, float beta,
                     float *out_rgb, float *out_depth, float *out_opacity, float *out_contrib,
                     void *hip_stream)
{
    return render_soft_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, beta, out_rgb,
                            out_depth, out_opacity, out_contrib, hip_stream);
}

int derf_render_culled(derf_handle *h, const float *rays_o, const float *rays_d,
                       long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                       float eps, int levels, int piece, float *out_rgb, float *out_depth,
                       float *out_opacity, unsigned *out_evaluated, void *hip_stream)
{
    return render_culled_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, eps, levels,
                              piece, out_rgb, out_depth, out_opacity, out_evaluated, hip_stream);
}

int derf_set_gate(derf_handle *h, int pos_freqs, int hidden, const float *weights)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (hidden == 0) {
        if (h->gate_w) {
            HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
            if (h->last_stream)
                HIP_TRY(hipStreamSynchronize(h->last_stream), "hipStreamSynchronize");
            HIP_TRY(dev_free(h->gate_w), "hipFree");
        }
        h->gate_w = nullptr;
        h->gate_freqs = h->gate_hidden = 0;
        return DERF_OK;
    }
    if (!weights)
        return fail(DERF_ERR_INVALID_ARG, "null gating weights");
    if (!derf::gate_shape_supported(pos_freqs, hidden))
        return fail(DERF_ERR_UNSUPPORTED, "no gating kernel for L = %d, %d hidden units",
                    pos_freqs, hidden);
    const long long count = derf_gate_weights_count(h->num_sites, pos_freqs, hidden);
    for (long long i = 0; i < count; ++i)
        if (!isfinite(weights[i]))
            return fail(DERF_ERR_INVALID_ARG, "non-finite gating weight");
    HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
    const size_t bytes = gate_packed_bytes(pos_freqs, hidden, h->num_sites);
    std::vector<unsigned char> host;
    try {
        if (injected_failure())
            throw std::bad_alloc();
        host.resize(bytes);
    } catch (const std::bad_alloc &) {
        return fail(DERF_ERR_OOM, "host staging of the gate");
    }
    gate_pack(pos_freqs, hidden, h->num_sites, weights, host.data());
    unsigned char *dev = nullptr;
    if (dev_alloc(reinterpret_cast<void **>(&dev), bytes) != hipSuccess) {
        (void)hipGetLastError();
        return fail(DERF_ERR_OOM, "gating weights");
    }
    hipError_t e = hipMemcpy(dev, host.data(), bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)dev_free(dev);
        HIP_TRY(e, "hipMemcpy");
    }
    if (h->gate_w) {
        if (h->last_stream)
            HIP_TRY(hipStreamSynchronize(h->last_stream), "hipStreamSynchronize");
        HIP_TRY(dev_free(h->gate_w), "hipFree");
    }
    h->gate_w = dev;
    h->gate_freqs = pos_freqs;
    h->gate_hidden = hidden;
    return DERF_OK;
}

long long derf_gate_weights_count(int num_sites, int pos_freqs, int hidden)
{
    if (num_sites < 1 || pos_freqs < 0 || hidden < 1)
        return -1;
    const long long P = 3 + 6LL * pos_freqs;
    return hidden * P + hidden + (long long)num_sites * hidden + num_sites;
}

int derf_render_gated(derf_handle *h, const float *rays_o, const float *rays_d,
                      long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                      float *out_rgb, float *out_depth, float *out_opacity, int *out_cell,
                      void *hip_stream)
{
    return render_culled_impl(h, rays_o, rays_d, num_rays, near_t, far_t, samp, 0.0f, 1, 0,
                              out_rgb, out_depth, out_opacity, nullptr, hip_stream, true,
                              out_cell);
}

int derf_set_empty_heads(derf_handle *h, const int *flags)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    HeadMask m{};
    if (flags)
        for (int k = 0; k < h->num_sites; ++k)
            if (flags[k])
                m.w[k >> 5] |= 1u << (k & 31);
    h->empty = m;
    return DERF_OK;
}

int derf_set_encoding(derf_handle *h, int mode)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (mode == DERF_ENCODING_FUSED) {
        h->gx_bytes = 0;
        return DERF_OK;
    }
    if (mode != DERF_ENCODING_STORED)
        return fail(DERF_ERR_INVALID_ARG, "unknown encoding mode %d", mode);
    // every group needs a stored form, and all of them one table layout
    const MlpVariant *first = nullptr;
    for (int gi = 0; gi < h->num_groups; ++gi) {
        const MlpVariant *v = h->groups[gi].mlp->stored;
        if (!v)
            return fail(DERF_ERR_UNSUPPORTED,
                        "stored encoding: no stored form for a head architecture with a skip "
                        "layer");
        if (first && (v->gx_bytes != first->gx_bytes || v->pos_freqs != first->pos_freqs))
            return fail(DERF_ERR_UNSUPPORTED,
                        "stored encoding: the heads' position encodings differ");
        if (!first)
            first = v;
    }
    if (!first)
        return fail(DERF_ERR_UNSUPPORTED, "stored encoding: no heads");
    h->gx_bytes = first->gx_bytes;
    return DERF_OK;
}

int derf_set_timing(derf_handle *h, int on)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    h->timing = on != 0;
    return DERF_OK;
}

int get_stats_impl(derf_handle *h, derf_stats *out);

int derf_get_stats(derf_handle *h, derf_stats *out)
{
    try {
        return get_stats_impl(h, out);
    } catch (const std::bad_alloc &) {
        return fail(DERF_ERR_OOM, "host memory for the head counts");
    }
}

int get_stats_impl(derf_handle *h, derf_stats *out)
{
    if (!h || !out)
        return fail(DERF_ERR_INVALID_ARG, "null handle or output");
    if (h->last_stream || h->totals) {
        HIP_TRY(hipSetDevice(h->device), "hipSetDevice");
        HIP_TRY(hipStreamSynchronize(h->last_stream), "hipStreamSynchronize");
    }
    accumulate_timing(h);
    memset(h->stats.head_samples, 0, sizeof(h->stats.head_samples));
    if (h->totals) {
        std::vector<unsigned> tot((size_t)h->num_sites * h->totals_sets);
        HIP_TRY(hipMemcpy(tot.data(), h->totals, sizeof(unsigned) * tot.size(),
                          hipMemcpyDeviceToHost),
                "hipMemcpy");
        for (size_t j = 0; j < tot.size(); ++j)
            h->stats.head_samples[j % h->num_sites] += tot[j];
        if (h->totals_fine) {
            HIP_TRY(hipMemcpy(tot.data(), h->totals_fine, sizeof(unsigned) * h->num_sites,
                              hipMemcpyDeviceToHost),
                    "hipMemcpy");
            for (int k = 0; k < h->num_sites; ++k)
                h->stats.head_samples[k] += tot[k];
        }
    }
    h->stats.walk_rays = h->walk_rays;
    h->stats.walk_fallback_rays = 0;
    if (h->walk_nseg && h->walk_rays) {
        std::vector<unsigned char> ns(h->walk_rays);
        HIP_TRY(hipMemcpy(ns.data(), h->walk_nseg, ns.size(), hipMemcpyDeviceToHost), "hipMemcpy");
        for (unsigned char v : ns)
            h->stats.walk_fallback_rays += v == 0;
    }
    *out = h->stats;
    return DERF_OK;
}

int derf_reset_stats(derf_handle *h)
{
    if (!h)
        return fail(DERF_ERR_INVALID_ARG, "null handle");
    if (h->ev_pending) {
        HIP_TRY(hipEventSynchronize(last_event(h)), "hipEventSynchronize");
        h->ev_pending = false;
    }
    memset(&h->stats, 0, sizeof(h->stats));
    return DERF_OK;
}

void derf_destroy(derf_handle *h)
{
    if (!h)
        return;
    (void)hipSetDevice(h->device);
    if (h->last_stream || h->ws.mem)
        (void)hipStreamSynchronize(h->last_stream);
    if (h->ws.mem)
        (void)dev_free(h->ws.mem);
    if (h->sites)
        (void)dev_free(h->sites);
    if (h->gate_w)
        (void)dev_free(h->gate_w);
    for (int gi = 0; gi < h->num_groups; ++gi) {
        if (h->groups[gi].streams)
            (void)dev_free(h->groups[gi].streams);
        if (h->groups[gi].blocks)
            (void)dev_free(h->groups[gi].blocks);
    }
    for (int i = 0; i < kEvents; ++i)
        if (h->ev[i])
            (void)hipEventDestroy(h->ev[i]);
    count_live(-1);
    delete h;
}

const char *derf_status_string(int status)
{
    switch (status) {
    case DERF_OK: return "ok";
    case DERF_ERR_INVALID_ARG: return "invalid argument";
    case DERF_ERR_UNSUPPORTED: return "unsupported";
    case DERF_ERR_OOM: return "out of memory";
    case DERF_ERR_HIP: return "HIP error";
    default: return "unknown status";
    }
}

const char *derf_last_error(void) { return g_last_error; }

#ifdef DERF_FAULT_INJECTION
// test builds only (not in derf.h): fail the allocation n allocations from
// now (0: the next one); n < 0 disarms
void derf_debug_fail_alloc(long n) { g_fail_in.store(n < 0 ? -1 : n); }
// device blocks and handles allocated and not yet released
long derf_debug_live_allocations(void) { return g_live.load(); }
#endif

}  // extern "C"
