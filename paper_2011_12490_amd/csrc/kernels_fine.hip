// Hierarchical sampling for gfx950: inverse-CDF fine depths drawn from the
// coarse pass's quadrature weights, and the compositing of the coarse and
// fine samples merged in depth order.  The hierarchical scheme is NeRF's,
// which the paper adopts unchanged for its heads (Sec. 4 implementation
// details); the coarse heads' outputs are reused in the fine composite.
#pragma clang fp contract(off)

#include "derf_device.h"
#include "derf_internal.h"

namespace derf {
namespace {

constexpr int kWaves = 4;  // rays (one wave each) per workgroup

// ---------------------------------------------------------------------------
// Fine depths of one ray per wave.
//
// The coarse samples' quadrature weights w_i = T_i alpha_i (T_i the
// transmittance in front of sample i, alpha_i = 1 - exp(-sigma_i delta_i)
// on the midpoint interval [b_i, b_{i+1}) of sample i) plus a floor of 1e-5
// give a piecewise-constant density over [near, far].  Fine draw j is
// u_j = (j + xi_j) / n_fine with xi_j from generator stream 1, mapped
// through the inverse of that density's CDF.  Everything from the densities
// on is float64: the draws land inside intervals whose CDF span can be as
// small as the floor, where float32 would leave only a few significant
// bits.  The depths come out sorted (the inverse CDF is monotone and each
// draw is clamped to its interval).
//
// LDS per wave: F [nc + 1] doubles (the CDF), then tc [nc] floats.  Every
// wave runs every barrier; waves past the last ray compute ray 0 and store
// nothing.
__global__ __launch_bounds__(kWaves * 64) void fine_sample_kernel(
    const float *__restrict__ tc, const float4 *__restrict__ src, unsigned nc, unsigned nf,
    unsigned num_rays, float near_t, float far_t, uint2 key, uint64_t ray_offset, int perturb,
    float *__restrict__ tf)
{
    extern __shared__ double smem[];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const unsigned ray = blockIdx.x * kWaves + wv;
    const bool live = ray < num_rays;
    const unsigned r = live ? ray : 0u;
    double *F = smem + wv * (nc + 1);
    float *T = reinterpret_cast<float *>(smem + kWaves * (nc + 1)) + wv * nc;
    const size_t base = (size_t)r * nc;

    for (unsigned i = lane; i < nc; i += 64)
        T[i] = tc[base + i];
    __syncthreads();

    // lane chunk [i0, i1)
    const unsigned c = (nc + 63) / 64;
    const unsigned i0 = min(lane * c, nc), i1 = min(i0 + c, nc);
    auto bound = [&](unsigned i) -> double {  // b_i, i in [0, nc]
        return i == 0 ? (double)near_t : i == nc ? (double)far_t : 0.5 * ((double)T[i - 1] + (double)T[i]);
    };

    // transmittance through this lane's chunk, then exclusive product over lanes
    double prod = 1.0;
    for (unsigned i = i0; i < i1; ++i)
        prod *= exp(-(double)src[base + i].x * (bound(i + 1) - bound(i)));
    double incl = prod;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const double y = __shfl_up(incl, off);
        if (lane >= off)
            incl *= y;
    }
    double Tin = __shfl_up(incl, 1);
    if (lane == 0)
        Tin = 1.0;

    // pdf masses w_i + 1e-5 (kept in F[i + 1]) and their lane sum
    double sum = 0.0;
    for (unsigned i = i0; i < i1; ++i) {
        const double x = (double)src[base + i].x * (bound(i + 1) - bound(i));
        const double p = Tin * -expm1(-x) + 1e-5;
        Tin *= exp(-x);
        F[i + 1] = p;
        sum += p;
    }
    double run = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const double y = __shfl_up(run, off);
        if (lane >= off)
            run += y;
    }
    const double total = __shfl(run, 63);
    run -= sum;  // exclusive
    for (unsigned i = i0; i < i1; ++i) {
        run += F[i + 1];
        F[i + 1] = run / total;
    }
    if (lane == 0)
        F[0] = 0.0;
    __syncthreads();
    if (lane == 0)
        F[nc] = 1.0;
    __syncthreads();

    for (unsigned j = lane; j < nf; j += 64) {
        const double xi = perturb ? (double)jitter(key, ray_offset + r, j, 1u) : 0.5;
        const double u = ((double)j + xi) / (double)nf;
        // interval i = largest index in [0, nc - 1] with F[i] <= u: the first
        // k in [1, nc - 1] with F[k] > u (nc if none), minus one
        unsigned lo = 1, hi = nc;
        while (lo < hi) {
            const unsigned mid = (lo + hi) >> 1;
            if (F[mid] <= u)
                lo = mid + 1;
            else
                hi = mid;
        }
        const unsigned i = lo - 1;
        const double b0 = bound(i), b1 = bound(i + 1);
        const double span = F[i + 1] - F[i];
        double frac = span > 0.0 ? (u - F[i]) / span : 0.0;
        frac = frac < 0.0 ? 0.0 : (frac > 1.0 ? 1.0 : frac);
        if (live)
            tf[(size_t)r * nf + j] = (float)(b0 + frac * (b1 - b0));
    }
}

// ---------------------------------------------------------------------------
// Composite of the merged coarse + fine samples of one ray per wave.
//
// Both lists are sorted; the merged order is the stable merge with coarse
// samples first on equal depths: coarse i lands at i + #{fine depths < tc_i},
// fine j at j + #{coarse depths <= tf_j}.  The merged (t, cell, sigma, rgb)
// are scattered into LDS, integrated per segment and merged front to back as
// in the single-pass composite, and optionally written out (debug).
//
// LDS per wave (N = nc + nf): sr [N] float4, t [N] float, pos [N] u16,
// cell [N] u8.  Every wave runs every barrier; waves past the last ray
// compute ray 0 and store nothing.
struct MergedLds {
    float4 *sr;
    float *t;
    unsigned short *pos;
    uint8_t *cell;
};

__host__ __device__ constexpr size_t pos_offset(unsigned N) { return (size_t)N * 20; }
__host__ __device__ constexpr size_t cell_offset(unsigned N)
{
    return pos_offset(N) + ((size_t)N * 2 + 3) / 4 * 4;
}
// one wave's share, a multiple of 16 bytes so every wave's float4s stay aligned
__host__ __device__ constexpr size_t merged_lds_bytes_per_wave(unsigned N)
{
    return (cell_offset(N) + N + 15) / 16 * 16;
}
constexpr size_t kLdsBudget = 65536;

__global__ __launch_bounds__(kWaves * 64) void merge_composite_kernel(
    const float *__restrict__ tc, const uint8_t *__restrict__ cc, const float4 *__restrict__ sc,
    unsigned nc, const float *__restrict__ tf, const uint8_t *__restrict__ cf,
    const float4 *__restrict__ sf, unsigned nf, unsigned num_rays, float near_t, float far_t,
    float *__restrict__ out_rgb, float *__restrict__ out_depth, float *__restrict__ out_opacity,
    int *dcell, float *dt, float *dsigma, float *drgb)
{
    extern __shared__ float4 smem4[];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const unsigned ray = blockIdx.x * (blockDim.x >> 6) + wv;
    const bool live = ray < num_rays;
    const unsigned r = live ? ray : 0u;
    const unsigned N = nc + nf;
    unsigned char *mine = reinterpret_cast<unsigned char *>(smem4) + wv * merged_lds_bytes_per_wave(N);
    MergedLds L;
    L.sr = reinterpret_cast<float4 *>(mine);
    L.t = reinterpret_cast<float *>(mine + (size_t)N * 16);
    L.pos = reinterpret_cast<unsigned short *>(mine + pos_offset(N));
    L.cell = reinterpret_cast<uint8_t *>(mine + cell_offset(N));
    const size_t bc = (size_t)r * nc, bf = (size_t)r * nf;

    // the two sorted depth lists, side by side in L.t
    for (unsigned k = lane; k < N; k += 64)
        L.t[k] = k < nc ? tc[bc + k] : tf[bf + (k - nc)];
    __syncthreads();
    // merged position of every sample
    for (unsigned k = lane; k < N; k += 64) {
        const float v = L.t[k];
        const bool coarse = k < nc;
        // coarse: count fine depths < v; fine: count coarse depths <= v
        const float *other = coarse ? L.t + nc : L.t;
        unsigned lo = 0, hi = coarse ? nf : nc;
        while (lo < hi) {
            const unsigned mid = (lo + hi) >> 1;
            const float o = other[mid];
            if (coarse ? (o < v) : (o <= v))
                lo = mid + 1;
            else
                hi = mid;
        }
        L.pos[k] = (unsigned short)((coarse ? k : k - nc) + lo);
    }
    __syncthreads();
    for (unsigned k = lane; k < N; k += 64) {
        const unsigned p = L.pos[k];
        if (k < nc) {
            L.t[p] = tc[bc + k];
            L.cell[p] = cc[bc + k];
            L.sr[p] = sc[bc + k];
        } else {
            L.t[p] = tf[bf + (k - nc)];
            L.cell[p] = cf[bf + (k - nc)];
            L.sr[p] = sf[bf + (k - nc)];
        }
    }
    __syncthreads();

    const unsigned c = (N + 63) / 64;
    const unsigned i0 = min(lane * c, N), i1 = min(i0 + c, N);
    Over acc = integrate_runs(
        i0, i1, N, near_t, far_t, [&](unsigned i) { return L.t[i]; },
        [&](unsigned i) { return (unsigned)L.cell[i]; }, [&](unsigned i) { return L.sr[i]; });
    acc = wave_over(acc, lane);
    if (live && lane == 0) {
        out_rgb[3 * ray] = acc.r;
        out_rgb[3 * ray + 1] = acc.g;
        out_rgb[3 * ray + 2] = acc.b;
        out_depth[ray] = acc.d;
        out_opacity[ray] = 1.0f - acc.t;
    }
    if (live && (dcell || dt || dsigma || drgb)) {
        const size_t bm = (size_t)ray * N;
        for (unsigned k = lane; k < N; k += 64) {
            if (dcell)
                dcell[bm + k] = L.cell[k];
            if (dt)
                dt[bm + k] = L.t[k];
            if (dsigma)
                dsigma[bm + k] = L.sr[k].x;
            if (drgb) {
                drgb[3 * (bm + k)] = L.sr[k].y;
                drgb[3 * (bm + k) + 1] = L.sr[k].z;
                drgb[3 * (bm + k) + 2] = L.sr[k].w;
            }
        }
    }
}

inline unsigned blocks_for(size_t items, unsigned per) { return (unsigned)((items + per - 1) / per); }

}  // namespace

size_t fine_sample_lds_bytes(unsigned nc)
{
    return (size_t)kWaves * (nc + 1) * sizeof(double) + (size_t)kWaves * nc * sizeof(float);
}

// rays per workgroup of the merged composite: as many as fit the LDS budget
static unsigned merge_waves(unsigned n_total)
{
    const size_t w = kLdsBudget / merged_lds_bytes_per_wave(n_total);
    return w >= (size_t)kWaves ? kWaves : (unsigned)w;
}

hipError_t launch_fine_sample(const RenderGeometry &g, const float *tc, const float4 *src,
                              unsigned n_fine, float *tf, hipStream_t s)
{
    const uint2 key = make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32));
    fine_sample_kernel<<<blocks_for(g.num_rays, kWaves), kWaves * 64, fine_sample_lds_bytes(g.n), s>>>(
        tc, src, g.n, n_fine, g.num_rays, g.near_t, g.far_t, key, g.ray_offset, g.perturb, tf);
    return hipGetLastError();
}

hipError_t launch_merge_composite(const RenderGeometry &g, const float *tc, const uint8_t *cc,
                                  const float4 *sc, unsigned n_fine, const float *tf,
                                  const uint8_t *cf, const float4 *sf, float *rgb, float *depth,
                                  float *opacity, int *dcell, float *dt, float *dsigma,
                                  float *drgb, hipStream_t s)
{
    const unsigned N = g.n + n_fine, waves = merge_waves(N);
    if (waves < 1)
        return hipErrorInvalidValue;
    merge_composite_kernel<<<blocks_for(g.num_rays, waves), waves * 64,
                             waves * merged_lds_bytes_per_wave(N), s>>>(
        tc, cc, sc, g.n, tf, cf, sf, n_fine, g.num_rays, g.near_t, g.far_t, rgb, depth, opacity,
        dcell, dt, dsigma, drgb);
    return hipGetLastError();
}

}  // namespace derf
