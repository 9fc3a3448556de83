// The soft decomposition on gfx950 (Sec. 3.2 Eq. 4-6 with the soft Voronoi
// weights of Sec. 3.3 Eq. 8): every head evaluates every sample (the grouped
// MLP with one all-samples bucket per head), then each sample's outputs are
// blended by
//   w_k(x) = exp(-beta |x - phi_k|) / sum_j exp(-beta |x - phi_j|)
// and the ray is composited front to back.  The per-ray head contributions
// of Eq. 6 come out of the same pass.
//
// Sample positions use the same explicit fused multiply-adds as the
// nearest-site path (no other contraction).
#pragma clang fp contract(off)

#include "derf_device.h"
#include "derf_internal.h"

namespace derf {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

// bucket[i] = i for every sample, totals[k] = S for every head, and the MLP's
// tile counters cleared: every head's rows are all the samples.
__global__ __launch_bounds__(kThreads) void soft_setup_kernel(unsigned S, int num_sites,
                                                              unsigned *__restrict__ bucket,
                                                              unsigned *__restrict__ totals,
                                                              unsigned *__restrict__ queue)
{
    const unsigned i0 = blockIdx.x * kThreads + threadIdx.x;
    if (i0 < (unsigned)num_sites)
        totals[i0] = S;
    if (i0 < (unsigned)(kMlpQueues * kMaxHeadGroups))
        queue[i0] = 0;
    for (unsigned i = i0; i < S; i += gridDim.x * kThreads)
        bucket[i] = i;
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
        v += __shfl_xor(v, o);
    return v;
}

// product of v over lanes 0 .. lane
__device__ __forceinline__ float wave_inclusive_product(float v, int lane)
{
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const float u = __shfl_up(v, o);
        if (lane >= o)
            v *= u;
    }
    return v;
}

__device__ __forceinline__ float site_distance(const float4 &p, float x, float y, float z)
{
    const float ex = x - p.x, ey = y - p.y, ez = z - p.z;
    return sqrtf(fmaf(ez, ez, fmaf(ey, ey, ex * ex)));
}

// One wave per ray, 64 samples at a time (one per lane).  sr holds head k's
// (sigma, r, g, b) of sample s at k * S + s.  The blend is normalised by its
// own sum, and the weights are shifted by the nearest site's distance so that
// the largest is exp(0) = 1 and none overflows.  Compositing uses the
// midpoint intervals of the nearest-site path; the running transmittance
// passes from chunk to chunk.  CONTRIB: after each chunk the samples'
// positions, nearest distances and rendering weight / normaliser go through
// LDS, and lane k accumulates head k's share (heads k, k + 64, ...).
template <bool CONTRIB>
__global__ __launch_bounds__(kThreads) void soft_composite_kernel(
    RenderGeometry g, const float4 *__restrict__ sites, int num_sites, HeadMask empty, float beta,
    const float *__restrict__ t, const float4 *__restrict__ sr, float *__restrict__ rgb,
    float *__restrict__ depth, float *__restrict__ opacity, float *__restrict__ contrib)
{
    __shared__ float4 s_sites[kMaxSites];
    __shared__ float4 s_x[CONTRIB ? kWaves : 1][64];     // position, nearest distance
    __shared__ float s_coef[CONTRIB ? kWaves : 1][64];   // rendering weight / normaliser
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        s_sites[k] = sites[k];
    __syncthreads();
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const unsigned r = blockIdx.x * kWaves + wv;
    if (r >= g.num_rays)
        return;
    const unsigned n = g.n;
    const size_t S = g.num_samples;
    const float ox = g.rays_o[3 * r], oy = g.rays_o[3 * r + 1], oz = g.rays_o[3 * r + 2];
    const float dx = g.rays_d[3 * r], dy = g.rays_d[3 * r + 1], dz = g.rays_d[3 * r + 2];

    float C0 = 0.0f, C1 = 0.0f, C2 = 0.0f, D = 0.0f, T = 1.0f;
    float W[CONTRIB ? kMaxSites / 64 : 1] = {};
    for (unsigned c0 = 0; c0 < n; c0 += 64) {
        const unsigned i = c0 + lane;
        const bool ok = i < n;
        const size_t si = (size_t)r * n + (ok ? i : 0);
        float ti = 0.0f, x = 0.0f, y = 0.0f, z = 0.0f, dmin = INFINITY, Z = 1.0f;
        float sig = 0.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f, delta = 0.0f;
        if (ok) {
            ti = t[si];
            x = fmaf(ti, dx, ox);
            y = fmaf(ti, dy, oy);
            z = fmaf(ti, dz, oz);
            for (int k = 0; k < num_sites; ++k)
                dmin = fminf(dmin, site_distance(s_sites[k], x, y, z));
            Z = 0.0f;
            for (int k = 0; k < num_sites; ++k) {
                const float wk = __expf(-beta * (site_distance(s_sites[k], x, y, z) - dmin));
                // a 0-capacity head contributes no density and no colour
                const float4 v = empty.test(k) ? make_float4(0.0f, 0.0f, 0.0f, 0.0f)
                                               : sr[(size_t)k * S + si];
                Z += wk;
                sig = fmaf(wk, v.x, sig);
                cr = fmaf(wk, v.y, cr);
                cg = fmaf(wk, v.z, cg);
                cb = fmaf(wk, v.w, cb);
            }
            const float iz = 1.0f / Z;
            sig *= iz;
            cr *= iz;
            cg *= iz;
            cb *= iz;
            // midpoint interval of sample i (Sec. 3.1 Eq. 1-2)
            const float lo = i == 0 ? g.near_t : 0.5f * (t[si - 1] + ti);
            const float hi = i + 1 == n ? g.far_t : 0.5f * (ti + t[si + 1]);
            delta = hi - lo;
        }
        const float tau = ok ? __expf(-sig * delta) : 1.0f;
        const float alpha = 1.0f - tau;
        const float incl = wave_inclusive_product(tau, lane);
        float excl = __shfl_up(incl, 1);
        if (lane == 0)
            excl = 1.0f;
        const float w = T * excl * alpha;  // rendering weight T_i alpha_i
        C0 += wave_sum(w * cr);
        C1 += wave_sum(w * cg);
        C2 += wave_sum(w * cb);
        D += wave_sum(w * ti);
        T *= __shfl(incl, 63);
        if constexpr (CONTRIB) {
            s_x[wv][lane] = make_float4(x, y, z, dmin);
            s_coef[wv][lane] = ok ? w / Z : 0.0f;
            const unsigned cnt = n - c0 < 64u ? n - c0 : 64u;
            for (unsigned j = 0; j < cnt; ++j) {
                const float4 q = s_x[wv][j];
                const float cf = s_coef[wv][j];
#pragma unroll
                for (int m = 0; m < kMaxSites / 64; ++m) {
                    const int k = lane + 64 * m;
                    if (k < num_sites)
                        W[m] = fmaf(cf, __expf(-beta * (site_distance(s_sites[k], q.x, q.y, q.z) - q.w)),
                                    W[m]);
                }
            }
        }
    }
    if (lane == 0) {
        rgb[3 * r] = C0;
        rgb[3 * r + 1] = C1;
        rgb[3 * r + 2] = C2;
        depth[r] = D;
        opacity[r] = 1.0f - T;
    }
    if constexpr (CONTRIB) {
#pragma unroll
        for (int m = 0; m < kMaxSites / 64; ++m) {
            const int k = lane + 64 * m;
            if (k < num_sites)
                contrib[(size_t)r * num_sites + k] = W[m];
        }
    }
}

}  // namespace

hipError_t launch_soft_setup(unsigned S, int num_sites, unsigned *bucket, unsigned *totals,
                             unsigned *queue, hipStream_t s)
{
    const unsigned blocks = (S + kThreads - 1) / kThreads;
    soft_setup_kernel<<<blocks < 4096u ? (blocks ? blocks : 1u) : 4096u, kThreads, 0, s>>>(
        S, num_sites, bucket, totals, queue);
    return hipGetLastError();
}

hipError_t launch_soft_composite(const RenderGeometry &g, const float4 *sites, int num_sites,
                                 const HeadMask &empty, float beta, const float *t,
                                 const float4 *sr, float *rgb, float *depth, float *opacity,
                                 float *contrib, hipStream_t s)
{
    const unsigned blocks = (g.num_rays + kWaves - 1) / kWaves;
    if (contrib)
        soft_composite_kernel<true><<<blocks, kThreads, 0, s>>>(
            g, sites, num_sites, empty, beta, t, sr, rgb, depth, opacity, contrib);
    else
        soft_composite_kernel<false><<<blocks, kThreads, 0, s>>>(
            g, sites, num_sites, empty, beta, t, sr, rgb, depth, opacity, nullptr);
    return hipGetLastError();
}

}  // namespace derf
