// Ray sampling, nearest-site assignment, per-head bucketing and segment
// compositing for gfx950.
//
// The sample depths and positions decide which Voronoi cell owns a sample,
// so they are computed with explicit fused multiply-adds and no other
// contraction (the pragma below), giving the same float32 values on every
// run and in every reference.
#pragma clang fp contract(off)

#include <type_traits>

#include "derf_device.h"
#include "derf_internal.h"
#include "derf_cull.h"

namespace derf {
namespace {

constexpr int kThreads = 256;

// sample index s -> (ray, index within the ray); s < 2^32, n <= 1024.  The
// float64 quotient is at most one below the true one (at exact multiples).
__device__ __forceinline__ void split_sample(unsigned s, unsigned n, double inv_n, unsigned &r,
                                             unsigned &i)
{
    r = (unsigned)((double)s * inv_n);
    i = s - r * n;
    if (i >= n) {
        ++r;
        i -= n;
    }
}

// sin(pi y) and cos(pi y) for y = 2^l p: v_sin/v_cos take revolutions, so the
// argument is 2^(l-1) p, reduced exactly to [0, 1) first.
__device__ __forceinline__ void sincos_pi_pow2(float p, int l, float &s, float &c)
{
    const float u = __builtin_amdgcn_fractf(ldexpf(p, l - 1));
    s = __builtin_amdgcn_sinf(u);
    c = __builtin_amdgcn_cosf(u);
}

// ---------------------------------------------------------------------------
// Per-ray direction features: f = [gamma_4(d / |d|) (27 values), 0 x 5],
// stored as bf16 (round to nearest even) or float.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void ray_encode_kernel(const float *__restrict__ rays_d,
                                                              unsigned num_rays, void *dirbuf)
{
    const unsigned r = blockIdx.x * kThreads + threadIdx.x;
    if (r >= num_rays)
        return;
    const float dx = rays_d[3 * r], dy = rays_d[3 * r + 1], dz = rays_d[3 * r + 2];
    const float inv = 1.0f / sqrtf(dx * dx + dy * dy + dz * dz);
    const float p[3] = {dx * inv, dy * inv, dz * inv};
    float f[kDirPad];
#pragma unroll
    for (int j = 0; j < kDirPad; ++j)
        f[j] = 0.0f;
    f[0] = p[0];
    f[1] = p[1];
    f[2] = p[2];
#pragma unroll
    for (int l = 0; l < 4; ++l) {
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            float s, co;
            sincos_pi_pow2(p[c], l, s, co);
            f[3 + 6 * l + c] = s;
            f[3 + 6 * l + 3 + c] = co;
        }
    }
    if constexpr (BF16) {
        typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
        bf16x8 *out = reinterpret_cast<bf16x8 *>(dirbuf) + (size_t)r * (kDirPad / 8);
#pragma unroll
        for (int q = 0; q < kDirPad / 8; ++q) {
            bf16x8 v;
#pragma unroll
            for (int j = 0; j < 8; ++j)
                v[j] = (__bf16)f[8 * q + j];
            out[q] = v;
        }
    } else {
        float4 *out = reinterpret_cast<float4 *>(dirbuf) + (size_t)r * (kDirPad / 4);
#pragma unroll
        for (int q = 0; q < kDirPad / 4; ++q)
            out[q] = make_float4(f[4 * q], f[4 * q + 1], f[4 * q + 2], f[4 * q + 3]);
    }
}

// ---------------------------------------------------------------------------
// Runs of equal keys among the lanes of a wave: a run is a maximal stretch of
// consecutive lanes, all in `valid`, holding one key.  Along a ray the keys
// (heads, levels) change rarely, so a 64-lane step holds a few runs, and the
// run leaders -- not one ballot per key bit -- do the step's bookkeeping.
// Two runs of one key in a step (two rays, or a key coming back) are two
// runs: each leader adds or reserves its own count.
struct LaneRuns {
    uint64_t starts;  // lanes that start a run
    unsigned len;     // the run's length (meaningful in its start lane)
    int first;        // the lane that starts this lane's run (valid lanes)
};
__device__ __forceinline__ LaneRuns lane_runs(unsigned key, bool ok, uint64_t valid)
{
    const int lane = (int)(threadIdx.x & 63);
    // the key of lane - 1 (DPP wave shift right by one)
    const unsigned prev = (unsigned)__builtin_amdgcn_update_dpp(0, (int)key, 0x138, 0xF, 0xF, false);
    const bool prev_ok = lane > 0 && ((valid >> (lane - 1)) & 1ull);
    LaneRuns r;
    r.starts = __ballot(ok && (!prev_ok || prev != key));
    // the next start or invalid lane above this one ends the run
    const uint64_t above = ~((2ull << lane) - 1ull);  // lanes lane + 1 .. 63
    const uint64_t brk = (r.starts | ~valid) & above;
    r.len = (unsigned)((brk ? __builtin_ctzll(brk) : 64) - lane);
    const uint64_t upto = ~0ull >> (63 - lane);
    const uint64_t mine = r.starts & upto;
    r.first = mine ? 63 - __builtin_clzll(mine) : lane;
    return r;
}

// out[step] = p[wbase + 64 step + lane], or 0 from index n on: a wave's
// 64 STEPS consecutive bytes, read as dwords four to a lane (a quarter of
// the load instructions of one byte per lane, which kept the texture-data
// path busy) and handed to their lanes by lane permutes.  p + wbase must be
// 4-byte aligned, and a dword that starts below n must lie in p's
// allocation (byte buffers are allocated in whole 256-byte units).
template <int STEPS>
__device__ __forceinline__ void wave_bytes(const uint8_t *__restrict__ p, unsigned wbase,
                                           unsigned n, unsigned (&out)[STEPS])
{
    static_assert(STEPS % 4 == 0, "whole dwords per lane");
    const int lane = (int)(threadIdx.x & 63);
    unsigned word[STEPS / 4];
#pragma unroll
    for (int q = 0; q < STEPS / 4; ++q) {
        const unsigned first = wbase + 256 * q + 4 * lane;
        word[q] = first < n ? *reinterpret_cast<const unsigned *>(p + first) : 0u;
    }
#pragma unroll
    for (int q = 0; q < STEPS / 4; ++q)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            // byte 256 q + 64 j + lane lies in the dword of lane 16 j + lane / 4
            const unsigned v = (unsigned)__shfl((int)word[q], 16 * j + (lane >> 2));
            const unsigned idx = wbase + 256 * q + 64 * j + lane;
            out[4 * q + j] = idx < n ? (v >> (8 * (lane & 3))) & 0xFFu : 0u;
        }
}

// ---------------------------------------------------------------------------
// Cross-lane helpers over the aligned group of L lanes (L = 1, 2, 4, 8, 16)
// holding this lane: DPP quad permutes (lane ^ 1, lane ^ 2) and the 8- and
// 16-lane mirrors, each pairing the halves of the next larger group, so
// every lane of the group ends with the group's result.
template <int CTRL>
__device__ __forceinline__ unsigned dpp_u32(unsigned x)
{
    return (unsigned)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

template <int L, class Step>
__device__ __forceinline__ void group_steps(Step step)
{
    if constexpr (L >= 2)
        step(std::integral_constant<int, 0xB1>{});
    if constexpr (L >= 4)
        step(std::integral_constant<int, 0x4E>{});
    if constexpr (L >= 8)
        step(std::integral_constant<int, 0x141>{});
    if constexpr (L >= 16)
        step(std::integral_constant<int, 0x140>{});
}

// lexicographic minimum of (v, j)
template <int L>
__device__ __forceinline__ void group_argmin(double &v, int &j)
{
    group_steps<L>([&](auto ctrl) {
        constexpr int C = decltype(ctrl)::value;
        const unsigned long long b = (unsigned long long)__double_as_longlong(v);
        const unsigned lo = dpp_u32<C>((unsigned)b), hi = dpp_u32<C>((unsigned)(b >> 32));
        const int jo = (int)dpp_u32<C>((unsigned)j);
        const double vo = __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
        if (vo < v || (vo == v && jo < j)) {
            v = vo;
            j = jo;
        }
    });
}

template <int L>
__device__ __forceinline__ unsigned group_sum(unsigned x)
{
    group_steps<L>([&](auto ctrl) { x += dpp_u32<decltype(ctrl)::value>(x); });
    return x;
}

template <int L>
__device__ __forceinline__ unsigned long long group_or(unsigned long long x)
{
    group_steps<L>([&](auto ctrl) {
        constexpr int C = decltype(ctrl)::value;
        x |= ((unsigned long long)dpp_u32<C>((unsigned)(x >> 32)) << 32) | dpp_u32<C>((unsigned)x);
    });
    return x;
}

// sum of x over the lanes of the group below this one (gl: lane in group)
template <int L>
__device__ __forceinline__ unsigned group_exclusive_sum(unsigned x, int gl)
{
    unsigned inc = x;
    auto up = [&](auto ctrl, int n) {  // row_shr:n (within the 16-lane row)
        const unsigned y = dpp_u32<decltype(ctrl)::value>(inc);
        if (gl >= n)
            inc += y;
    };
    if constexpr (L >= 2)
        up(std::integral_constant<int, 0x111>{}, 1);
    if constexpr (L >= 4)
        up(std::integral_constant<int, 0x112>{}, 2);
    if constexpr (L >= 8)
        up(std::integral_constant<int, 0x114>{}, 4);
    if constexpr (L >= 16)
        up(std::integral_constant<int, 0x118>{}, 8);
    return inc - x;
}

// Cells along each ray, in float64, by a group of L lanes per ray (lane l
// holds the sites [l m, (l + 1) m), m = ceil(K / L)).  From t0 = near, c is
// the nearest site; moving along the ray, site j overtakes c where
// f_j(t) = |x(t) - phi_j|^2 - |x(t) - phi_c|^2, a linear function of t with
// slope 2 d.(phi_c - phi_j), reaches 0 from above; the segment of c ends at
// the first such crossing (or at far), and the ray enters the crossing
// site's cell.  Each move strictly increases d.phi of the current site, so a
// ray takes at most K segments and never returns to a cell.
//
// Each segment keeps, in ascending order, c and every site j with
// min(f_j(t0), f_j(t1)) <= tau at its ends t0, t1 (tau = 1e-4 (1 + the
// squared distances to c there)).  f_j is linear, so a site left out is
// farther than c by more than tau on the whole segment -- far above the
// float32 rounding of the squared distances (a few ulp) -- and can neither
// be the float32 nearest site of a sample in the segment nor tie with it:
// the float32 argmin over the segment's candidates is the float32 argmin over
// all sites, whatever crossing ends the segment.  A ray with more than
// kMaxSeg segments, or a segment with more than kMaxCand candidates, is
// marked (nseg = 0) for the search over all sites.
//
// One lane per ray (the largest frames) asks for 8 waves per SIMD: 64
// registers without spills, against 96 and 5 waves by default, to cover the
// lanes' differing walk lengths.  The grouped forms would spill at 64.
template <int L>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(L == 1 ? 8 : 1)))
void ray_walk_kernel(RenderGeometry g, const float4 *__restrict__ sites, int num_sites,
                     SegRec *__restrict__ seg, unsigned char *__restrict__ nseg)
{
    static_assert(L == 1 || L == 2 || L == 4 || L == 8 || L == 16, "group size");
    // the sites in float64 with their squared norms: |x - phi|^2 = |x|^2 +
    // q(x, phi), q = |phi|^2 - 2 x.phi, so differences of squared distances
    // at one x are differences of q (three fused multiply-adds per site)
    __shared__ double4 s_sites[kMaxSites];
    for (int k = threadIdx.x; k < num_sites; k += kThreads) {
        const float4 p = sites[k];
        const double px = p.x, py = p.y, pz = p.z;
        s_sites[k] = make_double4(px, py, pz, px * px + py * py + pz * pz);
    }
    __syncthreads();
    const size_t r = ((size_t)blockIdx.x * kThreads + threadIdx.x) / L;
    if (r >= g.num_rays)
        return;
    const int gl = threadIdx.x & (L - 1);
    const int per = (num_sites + L - 1) / L;
    const int j0 = min(gl * per, num_sites), j1 = min(j0 + per, num_sites);
    const double ox = g.rays_o[3 * r], oy = g.rays_o[3 * r + 1], oz = g.rays_o[3 * r + 2];
    const double dx = g.rays_d[3 * r], dy = g.rays_d[3 * r + 1], dz = g.rays_d[3 * r + 2];
    auto q = [&](double x, double y, double z, int k) {
        const double4 p = s_sites[k];
        return fma(-2.0, fma(x, p.x, fma(y, p.y, z * p.z)), p.w);
    };
    auto dproj = [&](int k) {  // d.phi_k
        const double4 p = s_sites[k];
        return fma(dx, p.x, fma(dy, p.y, dz * p.z));
    };
    double t0 = g.near_t;
    double x0 = ox + t0 * dx, y0 = oy + t0 * dy, z0 = oz + t0 * dz;
    int c = 0x7FFFFFFF;
    {
        double best = INFINITY;
        for (int k = j0; k < j1; ++k) {
            const double v = q(x0, y0, z0, k);
            if (v < best) {
                best = v;
                c = k;
            }
        }
        group_argmin<L>(best, c);
    }
    SegRec *out = seg + (size_t)r * kMaxSeg;
    int ns = 0;
    bool ok = true;
    for (;;) {
        const double qc0 = q(x0, y0, z0, c), bc = dproj(c);
        // the first crossing: smallest f_j(t0) / (-slope_j) over slope_j < 0,
        // f_j = q_j - q_c, slope_j = 2 d.(phi_c - phi_j)
        double bf = 0.0, bb = 0.0;
        int nextc = 0x7FFFFFFF;
        for (int j = j0; j < j1; ++j) {
            if (j == c)
                continue;
            const double b = 2.0 * (bc - dproj(j));
            if (b < 0.0) {
                const double f0 = fmax(q(x0, y0, z0, j) - qc0, 0.0);
                if (nextc == 0x7FFFFFFF || f0 * -bb < bf * -b) {
                    bf = f0;
                    bb = b;
                    nextc = j;
                }
            }
        }
        double tq = nextc == 0x7FFFFFFF ? INFINITY : bf / -bb;
        group_argmin<L>(tq, nextc);
        double t1 = g.far_t;
        if (nextc != 0x7FFFFFFF && t0 + tq < t1)
            t1 = t0 + tq;
        else
            nextc = -1;
        const double x1 = ox + t1 * dx, y1 = oy + t1 * dy, z1 = oz + t1 * dz;
        const double qc1 = q(x1, y1, z1, c);
        const double dc0 = fma(x0, x0, fma(y0, y0, z0 * z0)) + qc0;
        const double dc1 = fma(x1, x1, fma(y1, y1, z1 * z1)) + qc1;
        const double tau = 1e-4 * (1.0 + fmax(dc0, dc1));
        // this lane's candidates, ascending, as a byte string (at most 12 kept)
        unsigned long long lo = 0, hi = 0;
        unsigned cl = 0;
        for (int j = j0; j < j1; ++j) {
            bool take = j == c;
            if (!take)
                take = fmin(q(x0, y0, z0, j) - qc0, q(x1, y1, z1, j) - qc1) <= tau;
            if (take) {
                if (cl < 8)
                    lo |= (unsigned long long)j << (8 * cl);
                else if (cl < 12)
                    hi |= (unsigned long long)j << (8 * (cl - 8));
                cl = min(cl + 1, 12u);
            }
        }
        const unsigned nc = group_sum<L>(cl);
        if (nc > (unsigned)kMaxCand || ns == kMaxSeg) {
            ok = false;
            break;
        }
        // the group's list in lane order (ascending sites), after the count byte
        const int k = 8 * (int)(group_exclusive_sum<L>(cl, gl) + 1);
        if (k >= 64) {
            hi = lo << (k - 64);
            lo = 0;
        } else {
            hi = (hi << k) | (lo >> (64 - k));
            lo <<= k;
        }
        lo = group_or<L>(lo);
        hi = group_or<L>(hi);
        if (gl == 0) {
            const float te = nextc < 0 ? INFINITY : (float)t1;
            *reinterpret_cast<uint4 *>(out + ns) = make_uint4(
                __float_as_uint(te), (unsigned)lo | nc, (unsigned)(lo >> 32), (unsigned)hi);
        }
        ++ns;
        if (nextc < 0)
            break;
        t0 = t1;
        x0 = x1;
        y0 = y1;
        z0 = z1;
        c = nextc;
    }
    if (gl == 0)
        nseg[r] = ok ? (unsigned char)ns : 0;
}

// Owning cell of a sample at x (depth t): through its ray's walk table tab
// of ns segments (the float32 nearest among the segment's candidates,
// ascending), or, with ns == 0, over all sites.
__device__ __forceinline__ unsigned nearest_site(const float4 *s_sites, int num_sites,
                                                 const SegRec *tab, unsigned ns, float t,
                                                 float x, float y, float z)
{
    float best = INFINITY;
    unsigned bk = 0;
    auto consider = [&](unsigned k) {
        const float4 p = s_sites[k];
        const float ex = x - p.x, ey = y - p.y, ez = z - p.z;
        const float d2 = fmaf(ez, ez, fmaf(ey, ey, ex * ex));
        if (d2 < best) {
            best = d2;
            bk = k;
        }
    };
    if (ns == 0) {
        for (int k = 0; k < num_sites; ++k)
            consider(k);
        return bk;
    }
    // the first segment whose end is >= t (the last one's end is +inf)
    unsigned lo = 0, hi = ns - 1;
    while (lo < hi) {
        const unsigned mid = (lo + hi) >> 1;
        if (tab[mid].t_end >= t)
            hi = mid;
        else
            lo = mid + 1;
    }
    const uint4 rec = *reinterpret_cast<const uint4 *>(tab + lo);
    const unsigned nc = rec.y & 0xFFu;
    const unsigned words[3] = {rec.y, rec.z, rec.w};
#pragma unroll
    for (unsigned q = 0; q < (unsigned)kMaxCand; ++q)
        if (q < nc)
            consider((words[(q + 1) >> 2] >> (8 * ((q + 1) & 3))) & 0xFFu);
    return bk;
}

// Stratified depths t, owning cell (nearest site, ties to the lowest index)
// and per-block head histograms.  Block b covers samples
// [b * kBucketBlock, (b + 1) * kBucketBlock); each thread takes 4 consecutive
// samples per round, so one Philox block serves 4 samples of a ray.  With
// FROM_T the depths are given (t is read, not written): the assignment of
// the inverse-CDF samples of hierarchical sampling.  WALK: the owning cell
// comes from the ray's walk table (nearest_site), which gives the same cell
// as the search over all sites.  The lookup waits on its table reads, so
// WALK asks for 8 waves per SIMD (at most 64 registers, no spills; the
// staging below keeps 8 blocks within the CU's LDS).
template <bool FROM_T, bool WALK>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(WALK ? 8 : 1)))
void sample_assign_kernel(
    RenderGeometry g, const float4 *__restrict__ sites, int num_sites,
    WalkTable walk, float *__restrict__ t_out, uint8_t *__restrict__ cell_out,
    unsigned *__restrict__ counts, unsigned num_blocks)
{
    __shared__ float4 s_sites[kMaxSites];
    __shared__ unsigned s_hist[kMaxSites];
    // walk tables of the block's rays, when they are few enough (n >= ~152):
    // 14 KB, so that 8 blocks fit in 160 KB of LDS with the sites
    constexpr int kStageRays = 28;
    __shared__ SegRec s_seg[WALK ? kStageRays * kMaxSeg : 1];
    __shared__ unsigned char s_nseg[WALK ? kStageRays : 1];
    for (int k = threadIdx.x; k < num_sites; k += kThreads) {
        s_sites[k] = sites[k];
        s_hist[k] = 0;
    }
    const unsigned block_base = blockIdx.x * (unsigned)kBucketBlock;
    unsigned r_first = 0;
    bool staged = false;
    if constexpr (WALK) {
        unsigned i_;
        unsigned r_last;
        split_sample(block_base, g.n, g.inv_n, r_first, i_);
        split_sample((unsigned)(min((unsigned long long)block_base + kBucketBlock,
                                    (unsigned long long)g.num_samples) - 1),
                     g.n, g.inv_n, r_last, i_);
        staged = r_last - r_first < (unsigned)kStageRays;
        if (staged) {
            const unsigned nr = r_last - r_first + 1;
            for (unsigned q = threadIdx.x; q < nr; q += kThreads)
                s_nseg[q] = walk.nseg[r_first + q];
            __syncthreads();
            // the rays' written records only
            const uint4 *src = reinterpret_cast<const uint4 *>(walk.seg + (size_t)r_first * kMaxSeg);
            for (unsigned q = threadIdx.x; q < nr * kMaxSeg; q += kThreads)
                if (q % kMaxSeg < s_nseg[q / kMaxSeg])
                    reinterpret_cast<uint4 *>(s_seg)[q] = src[q];
        }
    }
    __syncthreads();
    // owning cell of a sample of ray r: through its walk table (segment count
    // 0: search all sites).  The staged and the global table are separate
    // calls so that each keeps its address space: a pointer that may be
    // either would turn the table reads into generic loads, which go through
    // the texture path even when they hit LDS.
    auto cell_of = [&](unsigned r, float t, float x, float y, float z) -> unsigned {
        if constexpr (WALK) {
            if (staged)
                return nearest_site(s_sites, num_sites, s_seg + (r - r_first) * kMaxSeg,
                                    s_nseg[r - r_first], t, x, y, z);
            return nearest_site(s_sites, num_sites, walk.seg + (size_t)r * kMaxSeg,
                                walk.nseg[r], t, x, y, z);
        } else {
            return nearest_site(s_sites, num_sites, nullptr, 0u, t, x, y, z);
        }
    };

    const uint2 key = make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32));
    const uint64_t lane_bit = 1ull << (threadIdx.x & 63);
    for (int round = 0; round < kBucketBlock / (4 * kThreads); ++round) {
        const unsigned s0 = block_base + round * (4 * kThreads) + 4 * threadIdx.x;
        unsigned r, i;
        split_sample(s0 < g.num_samples ? s0 : 0, g.n, g.inv_n, r, i);
        float tv[4];
        unsigned cv[4];
        uint4 blk = make_uint4(0, 0, 0, 0);
        if constexpr (FROM_T) {
            if (s0 + 3 < g.num_samples) {
                const float4 q = *reinterpret_cast<const float4 *>(t_out + s0);
                tv[0] = q.x;
                tv[1] = q.y;
                tv[2] = q.z;
                tv[3] = q.w;
            } else {
                for (int v = 0; v < 4; ++v)
                    tv[v] = s0 + v < g.num_samples ? t_out[s0 + v] : 0.0f;
            }
        }
        float ox = 0, oy = 0, oz = 0, dx = 0, dy = 0, dz = 0;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const unsigned s = s0 + v;
            cv[v] = 0xFFFFFFFFu;
            if constexpr (!FROM_T)
                tv[v] = 0.0f;
            if (s < g.num_samples) {
                if (v == 0 || i == 0) {
                    ox = g.rays_o[3 * r];
                    oy = g.rays_o[3 * r + 1];
                    oz = g.rays_o[3 * r + 2];
                    dx = g.rays_d[3 * r];
                    dy = g.rays_d[3 * r + 1];
                    dz = g.rays_d[3 * r + 2];
                }
                float t;
                if constexpr (FROM_T) {
                    t = tv[v];
                } else {
                    if (v == 0 || (i & 3u) == 0) {
                        const uint64_t rg = g.ray_offset + r;
                        blk = philox4x32_10(make_uint4(i >> 2, (unsigned)rg, (unsigned)(rg >> 32), 0u), key);
                    }
                    const float xi =
                        g.perturb ? (float)(philox_word(blk, i & 3u) >> 8) * 0x1.0p-24f : 0.5f;
                    t = fmaf(g.step, (float)i + xi, g.near_t);
                }
                const float x = fmaf(t, dx, ox), y = fmaf(t, dy, oy), z = fmaf(t, dz, oz);
                tv[v] = t;
                cv[v] = cell_of(r, t, x, y, z);
            }
            // next sample of the same thread
            if (++i == g.n) {
                i = 0;
                ++r;
            }
        }
        if (s0 + 3 < g.num_samples) {
            if constexpr (!FROM_T)
                *reinterpret_cast<float4 *>(t_out + s0) = make_float4(tv[0], tv[1], tv[2], tv[3]);
            *reinterpret_cast<unsigned *>(cell_out + s0) =
                cv[0] | (cv[1] << 8) | (cv[2] << 16) | (cv[3] << 24);
        } else {
            for (int v = 0; v < 4; ++v)
                if (s0 + v < g.num_samples) {
                    if constexpr (!FROM_T)
                        t_out[s0 + v] = tv[v];
                    cell_out[s0 + v] = (uint8_t)cv[v];
                }
        }
        // histogram: the first lane of each run of equal cells adds the run's length
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const bool ok = s0 + v < g.num_samples;
            const LaneRuns r = lane_runs(cv[v], ok, __ballot(ok));
            if ((r.starts & lane_bit) != 0)
                atomicAdd(&s_hist[cv[v]], r.len);
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        counts[(size_t)k * num_blocks + blockIdx.x] = s_hist[k];
}

// ---------------------------------------------------------------------------
// Exclusive prefix over blocks of each head's counts (one block per head),
// in place; the head's total goes to totals[head].  Block 0 also clears the
// tile counters of the MLP launch that follows on the stream.  The column
// goes through LDS 8192 counts at a time (coalesced loads and stores, the
// next chunk's loads in flight during the current chunk's scan); each thread
// scans 8 consecutive counts, and the block scans the threads' sums.
// (One count per thread and round took 64 rounds of four barriers for a
// column of 65,536 blocks.)  LDS rows are padded by one word per 32 so that
// the threads' strided reads hit distinct banks.
__global__ __launch_bounds__(1024) void bucket_scan_kernel(unsigned *__restrict__ counts,
                                                           unsigned num_blocks,
                                                           unsigned *__restrict__ totals,
                                                           unsigned *__restrict__ mlp_queue)
{
    constexpr unsigned kItems = 8, kChunk = 1024 * kItems;
    if (blockIdx.x == 0 && threadIdx.x < (unsigned)(kMlpQueues * kMaxHeadGroups))
        mlp_queue[threadIdx.x] = 0;
    __shared__ unsigned s_v[kChunk + kChunk / 32];
    __shared__ unsigned s_wave[16];
    __shared__ unsigned s_carry;
    auto at = [](unsigned i) { return i + (i >> 5); };
    unsigned *col = counts + (size_t)blockIdx.x * num_blocks;
    const unsigned tid = threadIdx.x;
    const int lane = tid & 63, w = tid >> 6;
    if (tid == 0)
        s_carry = 0;
    // the next chunk's counts, loaded while the current one is scanned
    unsigned nxt[kItems];
    auto load = [&](unsigned b0) {
#pragma unroll
        for (unsigned j = 0; j < kItems; ++j) {
            const unsigned i = b0 + j * 1024 + tid;
            nxt[j] = i < num_blocks ? col[i] : 0u;
        }
    };
    load(0);
    for (unsigned base = 0; base < num_blocks; base += kChunk) {
        const unsigned len = min(kChunk, num_blocks - base);
#pragma unroll
        for (unsigned j = 0; j < kItems; ++j)
            s_v[at(j * 1024 + tid)] = nxt[j];
        if (base + kChunk < num_blocks)
            load(base + kChunk);  // counts not yet overwritten: the stores below are this chunk's
        __syncthreads();
        unsigned loc[kItems], sum = 0;
#pragma unroll
        for (unsigned j = 0; j < kItems; ++j) {
            loc[j] = s_v[at(kItems * tid + j)];
            sum += loc[j];
        }
        // inclusive scan of the threads' sums within the wave
        unsigned x = sum;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const unsigned y = __shfl_up(x, off);
            if (lane >= off)
                x += y;
        }
        if (lane == 63)
            s_wave[w] = x;
        __syncthreads();
        if (w == 0) {
            unsigned ws = lane < 16 ? s_wave[lane] : 0u;
#pragma unroll
            for (int off = 1; off < 16; off <<= 1) {
                const unsigned y = __shfl_up(ws, off);
                if (lane >= off)
                    ws += y;
            }
            if (lane < 16)
                s_wave[lane] = ws;  // inclusive over waves
        }
        __syncthreads();
        const unsigned carry = s_carry;
        unsigned run = carry + (w > 0 ? s_wave[w - 1] : 0u) + x - sum;  // before this thread
#pragma unroll
        for (unsigned j = 0; j < kItems; ++j) {
            s_v[at(kItems * tid + j)] = run;
            run += loc[j];
        }
        __syncthreads();
#pragma unroll
        for (unsigned j = 0; j < kItems; ++j) {
            const unsigned i = j * 1024 + tid;
            if (i < len)
                col[base + i] = s_v[at(i)];
        }
        if (tid == 0)
            s_carry = carry + s_wave[15];
        __syncthreads();
    }
    if (threadIdx.x == 0)
        totals[blockIdx.x] = s_carry;
}

// First bucket position of each head's part in block b: the heads below k
// take sum_{j<k} totals_j entries, and within head k the blocks before b
// take prefix[k][b] (exclusive scan over blocks).  Computed by wave 0, 4
// heads per lane (K <= 256), all loads in flight at once.
__device__ __forceinline__ void head_block_base(const unsigned *__restrict__ prefix,
                                                const unsigned *__restrict__ totals,
                                                unsigned num_blocks, int num_sites,
                                                unsigned *s_base)
{
    if (threadIdx.x >= 64)
        return;
    const int lane = threadIdx.x;
    unsigned tot[4], pre[4], sum = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int k = 4 * lane + j;
        tot[j] = k < num_sites ? totals[k] : 0u;
        pre[j] = k < num_sites ? prefix[(size_t)k * num_blocks + blockIdx.x] : 0u;
        sum += tot[j];
    }
    unsigned incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const unsigned y = __shfl_up(incl, off);
        if (lane >= off)
            incl += y;
    }
    unsigned acc = incl - sum;  // heads below this lane's first
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int k = 4 * lane + j;
        if (k < num_sites)
            s_base[k] = acc + pre[j];
        acc += tot[j];
    }
}

// ---------------------------------------------------------------------------
// Painter's-order culling (Sec. 3.3).  The Painter's order visits a ray's
// segments front to back, so the transmittance in front of a segment is
// known before its head runs.  Level l of a ray is its segment of ordinal l
// (the last level: every later segment); lb[r * (levels + 1) + l] is the
// first sample of level l (lb[.. + 0] = 0, lb[.. + levels] = n; a level the
// ray does not reach starts at n).  Each level is bucketed, evaluated and
// integrated in turn; a ray whose transmittance has fallen below eps takes
// no part in later levels.

// Sample s is live at the level: lvl[s] holds its level, or kDeadLevel once
// its ray has closed (the level composite that closes a ray marks the ray's
// later samples), so the same test serves every level.
constexpr uint8_t kDeadLevel = 0xFF;
struct LevelLive {
    const uint8_t *lvl;
    unsigned level;
    unsigned heads;  // K, for the (level, head) keys
    __device__ __forceinline__ bool operator()(unsigned s) const { return lvl[s] == level; }
};

// The key a bucketing pass sorts by.  kCellKey: the sample's head (every
// sample); kCellAtLevel: the head, of the samples live at one level;
// kLevelCell: level K + head (every sample), for the one-pass bucketing of
// all levels at once.
constexpr int kCellKey = 0, kCellAtLevel = 1, kLevelCell = 2;

// Level bounds, one wave per ray, 64 samples per step.  A sample opens a
// segment when its cell differs from the previous sample's.  With piece > 0 a
// sample also opens a piece when it lies a multiple of piece samples past the
// start of its segment (its last change at or before it, carried across
// steps), so a segment is cut from its start into parts of at most piece
// samples.  A sample's ordinal is the number of openings up to it; its level,
// min(ordinal, levels - 1), goes to lvl, and lane j (1 <= j < levels) records
// where the j-th opening is (the start of piece j), taking the (j - seen)-th
// set bit of the step's opening ballot.
//
// WORDS (n a multiple of 4, both byte arrays 4-byte aligned): the wave moves
// its ray's cells and level bytes through LDS 256 at a time, as one dword per
// lane each way.  One byte per lane and step, as the other form does, keeps
// the texture path busy four times as long for the same bytes.
template <bool WORDS>
__global__ __launch_bounds__(kThreads) void level_bounds_kernel(const uint8_t *__restrict__ cell,
                                                               unsigned n, unsigned num_rays,
                                                               unsigned levels, unsigned piece,
                                                               unsigned *__restrict__ lb,
                                                               uint8_t *__restrict__ lvl)
{
    __shared__ uint32_t s_in[WORDS ? kThreads : 1], s_out[WORDS ? kThreads : 1];
    const unsigned lane = threadIdx.x & 63;
    const unsigned ray = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (ray >= num_rays)
        return;  // a whole wave: the LDS rows are per wave, with no block barrier
    const size_t base = (size_t)ray * n;
    const uint64_t upto = ~0ull >> (63 - lane);  // lanes 0 .. lane
    unsigned mine = n;  // start of level `lane`
    unsigned seen = 0;  // openings before this step (wave-uniform)
    unsigned seg0 = 0;  // start of the segment open at the step's first sample (wave-uniform)
    // the step of samples c0 .. c0 + 63: cur and prv are the cells of sample
    // i = c0 + lane and of i - 1 (read when 0 < i < n); returns i's level
    auto step = [&](unsigned c0, unsigned cur, unsigned prv) -> unsigned {
        const unsigned i = c0 + lane;
        const bool change = i > 0 && i < n && cur != prv;
        uint64_t m = __ballot(change);
        if (piece > 0) {
            const uint64_t before = m & upto;
            const unsigned start = before ? c0 + 63u - (unsigned)__builtin_clzll(before) : seg0;
            if (m)
                seg0 = c0 + 63u - (unsigned)__builtin_clzll(m);
            // a change is at its own segment start, so it opens a piece too
            m = __ballot(i > 0 && i < n && (i - start) % piece == 0);
        }
        const unsigned cnt = (unsigned)__popcll(m);
        if (lane < levels && lane > seen && lane <= seen + cnt) {
            uint64_t mm = m;
            for (unsigned q = lane - seen; q > 1; --q)
                mm &= mm - 1;
            mine = c0 + (unsigned)__builtin_ctzll(mm);
        }
        const unsigned v = min(seen + (unsigned)__popcll(m & upto), levels - 1);
        seen += cnt;
        return v;
    };
    if constexpr (!WORDS) {
        for (unsigned c0 = 0; c0 < n; c0 += 64) {
            const unsigned i = c0 + lane;
            const unsigned cur = i < n ? cell[base + i] : 0u;
            const unsigned prv = i > 0 && i < n ? cell[base + i - 1] : 0u;
            const unsigned v = step(c0, cur, prv);
            if (i < n)
                lvl[base + i] = (uint8_t)v;
        }
    } else {
        // LDS written by some lanes of the wave and read by others
        auto wave_sync = [] {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        };
        uint32_t *const w_in = s_in + (threadIdx.x & ~63u);
        uint32_t *const w_out = s_out + (threadIdx.x & ~63u);
        const uint8_t *const b_in = reinterpret_cast<const uint8_t *>(w_in);
        uint8_t *const b_out = reinterpret_cast<uint8_t *>(w_out);
        unsigned last = 0;  // cell of the sample before the chunk
        for (unsigned a = 0; a < n; a += 256) {
            const unsigned len = min(256u, n - a);  // a multiple of 4
            if (4 * lane < len)
                w_in[lane] = *reinterpret_cast<const uint32_t *>(cell + base + a + 4 * lane);
            wave_sync();
            for (unsigned q = 0; q < len; q += 64) {
                const unsigned k = q + lane;  // within the chunk
                const unsigned cur = k < len ? b_in[k] : 0u;
                const unsigned prv = k == 0 ? last : k < len ? b_in[k - 1] : 0u;
                const unsigned v = step(a + q, cur, prv);
                if (k < len)
                    b_out[k] = (uint8_t)v;
            }
            last = b_in[len - 1];
            wave_sync();
            if (4 * lane < len)
                *reinterpret_cast<uint32_t *>(lvl + base + a + 4 * lane) = w_out[lane];
            wave_sync();  // the next chunk's writes come after these reads
        }
    }
    if (lane <= levels)
        lb[(size_t)ray * (levels + 1) + lane] = lane == 0 ? 0u : mine;
}

// Per-block key histograms (the layout of the assignment's counts:
// counts[key * num_blocks + b]; num_keys keys), MODE
// kCellAtLevel or kLevelCell.  Thread t takes samples t + 256 q of the block
// (q < 16); all 16 level bytes and cells are loaded up front, so the loads
// are in flight together.
template <int MODE>
__global__ __launch_bounds__(kThreads) void level_count_kernel(const uint8_t *__restrict__ cell,
                                                              unsigned num_samples, int num_keys,
                                                              LevelLive live,
                                                              unsigned *__restrict__ counts,
                                                              unsigned num_blocks)
{
    constexpr int kSteps = kBucketBlock / kThreads;
    __shared__ unsigned s_hist[kMaxSites];
    for (int k = threadIdx.x; k < num_keys; k += kThreads)
        s_hist[k] = 0;
    const unsigned long long base = (unsigned long long)blockIdx.x * kBucketBlock + threadIdx.x;
    uint8_t lv[kSteps], cs[kSteps];
#pragma unroll
    for (int q = 0; q < kSteps; ++q) {
        const unsigned long long s64 = base + (unsigned)q * kThreads;
        const bool in = s64 < num_samples;
        lv[q] = in ? live.lvl[s64] : kDeadLevel;
        cs[q] = in ? cell[s64] : (uint8_t)0;
    }
    __syncthreads();
    const uint64_t lane_bit = 1ull << (threadIdx.x & 63);
#pragma unroll
    for (int q = 0; q < kSteps; ++q) {
        const bool ok = MODE == kLevelCell ? lv[q] != kDeadLevel : lv[q] == live.level;
        const unsigned key = MODE == kLevelCell ? lv[q] * live.heads + cs[q] : cs[q];
        const uint64_t any = __ballot(ok);
        if (any == 0)
            continue;  // no live sample in this wave's step
        const LaneRuns r = lane_runs(key, ok, any);
        if ((r.starts & lane_bit) != 0)
            atomicAdd(&s_hist[key], r.len);
    }
    __syncthreads();
    for (int k = threadIdx.x; k < num_keys; k += kThreads)
        counts[(size_t)k * num_blocks + blockIdx.x] = s_hist[k];
}

// Bucketing of a level below the last, ray by ray.  Such a level is one
// piece of each ray (between two consecutive openings), so a ray's samples
// there form one run of one cell.  A ray takes part while it is open: level
// 0, or its transmittance after the previous level at least eps (exactly the
// rays whose level bytes the earlier level composites left live).  The
// order of the runs within a head's bucket is not fixed (each sample's MLP
// outputs do not depend on it), so positions are reserved by atomics,
// aggregated over the lanes of a wave that share a cell.
struct RayRun {
    bool on;
    unsigned k, len;
    unsigned long long s0;  // first sample of the run
};
__device__ __forceinline__ RayRun level_ray_run(const uint8_t *__restrict__ cell,
                                                const unsigned *__restrict__ lb,
                                                const float *__restrict__ trans, unsigned n,
                                                unsigned num_rays, unsigned level,
                                                unsigned levels, float eps)
{
    RayRun r{false, 0u, 0u, 0ull};
    const unsigned ray = blockIdx.x * kThreads + threadIdx.x;
    if (ray >= num_rays)
        return r;
    const unsigned *r_lb = lb + (size_t)ray * (levels + 1) + level;
    const unsigned a = r_lb[0], b = r_lb[1];
    if (a >= b || (level > 0 && !(trans[ray] >= eps)))
        return r;
    r.on = true;
    r.s0 = (unsigned long long)ray * n + a;
    r.len = b - a;
    r.k = cell[r.s0];
    return r;
}

// counts[k * num_blocks + b] += the samples of each open ray's run in block
// b (zero on entry; the layout of the per-sample counts, so bucket_scan
// turns them into per-block prefixes).  A run is shorter than a block, so it
// touches at most two.  One thread per ray.
__global__ __launch_bounds__(kThreads) void level_ray_count_kernel(
    const uint8_t *__restrict__ cell, const unsigned *__restrict__ lb,
    const float *__restrict__ trans, unsigned n, unsigned num_rays, unsigned level,
    unsigned levels, float eps, unsigned *__restrict__ counts, unsigned num_blocks)
{
    const RayRun r = level_ray_run(cell, lb, trans, n, num_rays, level, levels, eps);
    if (!r.on)
        return;
    const unsigned long long s1 = r.s0 + r.len;
    const unsigned long long b0 = r.s0 / kBucketBlock, split = (b0 + 1) * kBucketBlock;
    unsigned *row = counts + (size_t)r.k * num_blocks;
    atomicAdd(row + b0, (unsigned)((s1 < split ? s1 : split) - r.s0));
    if (s1 > split)
        atomicAdd(row + b0 + 1, (unsigned)(s1 - split));
}

// head_off[k] = sum of totals below k (where head k's stretch starts).  One
// block, K <= 256.
__global__ __launch_bounds__(kThreads) void head_offsets_kernel(const unsigned *__restrict__ totals,
                                                                int num_sites,
                                                                unsigned *__restrict__ head_off)
{
    __shared__ unsigned s_v[kThreads];
    const int t = threadIdx.x;
    const unsigned v = t < num_sites ? totals[t] : 0u;
    s_v[t] = v;
    __syncthreads();
    for (int o = 1; o < kThreads; o <<= 1) {
        const unsigned y = t >= o ? s_v[t - o] : 0u;
        __syncthreads();
        s_v[t] += y;
        __syncthreads();
    }
    if (t < num_sites)
        head_off[t] = s_v[t] - v;
}

// Each open ray's run (in at most two block pieces) goes to head k's
// stretch at head_off[k] plus a position reserved from the block's prefix
// prefix[k * num_blocks + b] (the scanned counts: rays of one block and
// head share a counter, so reservations rarely contend).  The wave then
// writes its pieces one after another with all its lanes (coalesced).
// Samples of 0-capacity heads get zero density and colour in sr, as in the
// per-sample scatter.
__global__ __launch_bounds__(kThreads) void level_ray_scatter_kernel(
    const uint8_t *__restrict__ cell, const unsigned *__restrict__ lb,
    const float *__restrict__ trans, unsigned n, unsigned num_rays, unsigned num_samples,
    unsigned level, unsigned levels, float eps, HeadMask empty,
    const unsigned *__restrict__ head_off, unsigned *__restrict__ prefix, unsigned num_blocks,
    unsigned *__restrict__ bucket, float4 *__restrict__ sr)
{
    const RayRun r = level_ray_run(cell, lb, trans, n, num_rays, level, levels, eps);
    const int lane = (int)(threadIdx.x & 63);
    unsigned pos[2] = {0u, 0u}, len[2] = {0u, 0u};
    if (r.on) {
        const unsigned long long s1 = r.s0 + r.len;
        const unsigned long long b0 = r.s0 / kBucketBlock, split = (b0 + 1) * kBucketBlock;
        unsigned *row = prefix + (size_t)r.k * num_blocks;
        const unsigned base = head_off[r.k];
        len[0] = (unsigned)((s1 < split ? s1 : split) - r.s0);
        pos[0] = base + atomicAdd(row + b0, len[0]);
        if (s1 > split) {
            len[1] = (unsigned)(s1 - split);
            pos[1] = base + atomicAdd(row + b0 + 1, len[1]);
        }
    }
#pragma unroll
    for (int part = 0; part < 2; ++part) {
        uint64_t todo = __ballot(len[part] > 0);
        while (todo) {
            const int q = __builtin_ctzll(todo);
            todo &= todo - 1;
            const unsigned qpos = (unsigned)__shfl((int)pos[part], q);
            const unsigned qlen = (unsigned)__shfl((int)len[part], q);
            const unsigned qk = (unsigned)__shfl((int)r.k, q);
            const unsigned long long s_first = r.s0 + (part ? len[0] : 0u);
            const unsigned lo = (unsigned)__shfl((int)(unsigned)s_first, q);
            const unsigned hi = (unsigned)__shfl((int)(unsigned)(s_first >> 32), q);
            const unsigned long long qs = ((unsigned long long)hi << 32) | lo;
            const bool zero = empty.test((int)qk);
            for (unsigned j = lane; j < qlen; j += 64) {
                // within the bucket whenever the counts are consistent
                if (qpos + j < num_samples)
                    bucket[qpos + j] = (unsigned)(qs + j);
                if (zero)
                    sr[qs + j] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
        }
    }
}

// Stable scatter of sample ids into per-head buckets.  Bucket k occupies
// [offset_k, offset_k + total_k) with offset_k = sum of totals below k;
// within it samples keep increasing sample-id order, so each ray's run
// through cell k stays contiguous.  Block b's samples are its 4096 of the
// counting pass; wave w takes the 1024 consecutive ones from 1024 w, in 16
// steps of 64 (all 16 cells loaded up front, four to a lane: wave_bytes).
// Pass 1 counts each wave's samples per head (equal-cell runs, wave-private
// counters); after one
// barrier every wave knows its first position per head (the block's base
// plus the earlier waves' counts); pass 2 ranks each step's samples of one
// head by ballot and advances the wave's own counters.  A sample owned by a
// 0-capacity head keeps its bucket slot (the offsets are the same) but gets
// zero density and colour in sr: the MLP does not evaluate that head.
// MODE: the key (kCellKey, kCellAtLevel, kLevelCell); num_sites counts the
// keys.
template <int MODE>
__global__ __launch_bounds__(kThreads) void bucket_scatter_kernel(
    const uint8_t *__restrict__ cell, const unsigned *__restrict__ prefix,
    const unsigned *__restrict__ totals, unsigned num_samples, unsigned num_blocks,
    int num_sites, HeadMask empty, LevelLive live, unsigned *__restrict__ bucket,
    float4 *__restrict__ sr)
{
    constexpr bool LEVEL = MODE == kCellAtLevel;
    constexpr int kWavesPerBlock = kThreads / 64;
    constexpr int kSteps = kBucketBlock / kThreads;  // 64-sample steps per wave
    __shared__ unsigned s_base[kMaxSites];
    __shared__ unsigned s_pos[kWavesPerBlock][kMaxSites];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    head_block_base(prefix, totals, num_blocks, num_sites, s_base);
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        for (int v = 0; v < kWavesPerBlock; ++v)
            s_pos[v][k] = 0;
    const unsigned wbase = blockIdx.x * (unsigned)kBucketBlock + w * (kSteps * 64);
    unsigned cs[kSteps];
    bool in[kSteps];  // the sample exists (LEVEL: and is live at this level)
    wave_bytes(cell, wbase, num_samples, cs);
    unsigned lv[MODE == kCellKey ? 1 : kSteps];
    if constexpr (MODE != kCellKey)
        wave_bytes(live.lvl, wbase, num_samples, lv);
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        in[step] = wbase + step * 64 + lane < num_samples;
        if constexpr (LEVEL)
            in[step] = in[step] && lv[step] == live.level;
        if constexpr (MODE == kLevelCell)
            cs[step] += in[step] ? lv[step] * live.heads : 0u;
    }
    __syncthreads();
    // pass 1: this wave's count per head (run leaders)
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const bool ok = in[step];
        const uint64_t any = __ballot(ok);
        if (LEVEL && any == 0)
            continue;
        const LaneRuns r = lane_runs(cs[step], ok, any);
        if ((r.starts >> lane) & 1ull)
            atomicAdd(&s_pos[w][cs[step]], r.len);
    }
    __syncthreads();
    // counts -> each wave's first position per head
    for (int k = threadIdx.x; k < num_sites; k += kThreads) {
        unsigned acc = s_base[k];
        for (int v = 0; v < kWavesPerBlock; ++v) {
            const unsigned cnt = s_pos[v][k];
            s_pos[v][k] = acc;
            acc += cnt;
        }
    }
    __syncthreads();
    // pass 2: scatter, advancing the wave's positions
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const unsigned s = wbase + step * 64 + lane;
        const bool ok = in[step];
        const uint64_t any = __ballot(ok);
        if (LEVEL && any == 0)
            continue;
        const unsigned c = cs[step];
        // each run's leader reserves the run's positions; its lanes follow it
        const LaneRuns r = lane_runs(c, ok, any);
        unsigned start = 0;
        if ((r.starts >> lane) & 1ull)
            start = atomicAdd(&s_pos[w][c], r.len);
        start = __shfl(start, r.first);
        if (ok) {
            const unsigned pos = start + (unsigned)(lane - r.first);
            if (pos < num_samples)  // always true when the counts are consistent
                bucket[pos] = s;
            if (empty.test(MODE == kLevelCell ? c % live.heads : c))
                sr[s] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
    }
}

// After the one-pass (level, head) bucketing: offsets[key] = where key
// (level l, head k at l K + k) starts in the level-major order, an exclusive
// scan of totals over the L K <= 256 keys; live[l][k], the entries the MLP
// will evaluate, starts as every sample for level 0 (no ray has closed) and
// 0 for the levels the compaction fills.  One block of 256 threads; also
// clears the MLP's tile counters.
__global__ __launch_bounds__(kThreads) void level_head_init_kernel(
    const unsigned *__restrict__ totals, int num_keys, int heads, unsigned *__restrict__ offsets,
    unsigned *__restrict__ live, unsigned *__restrict__ mlp_queue)
{
    __shared__ unsigned s_wave[kThreads / 64];
    const int k = threadIdx.x, lane = k & 63, w = k >> 6;
    if (k < kMlpQueues * kMaxHeadGroups)
        mlp_queue[k] = 0;
    const unsigned v = k < num_keys ? totals[k] : 0u;
    unsigned x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const unsigned y = __shfl_up(x, off);
        if (lane >= off)
            x += y;
    }
    if (lane == 63)
        s_wave[w] = x;
    __syncthreads();
    unsigned before = x - v;
    for (int j = 0; j < w; ++j)
        before += s_wave[j];
    if (k < num_keys) {
        offsets[k] = before;
        live[k] = k < heads ? v : 0u;
    }
}

// Per-level compaction (levels 1 ..): the level's entries of the (level,
// head) order, [offsets[l K], offsets[l K] + the level's total), go to the
// same positions of bucket, each head's live ones (their ray still open)
// packed at the front of the head's stretch; live[k] counts them.  Wave w of
// block b takes 1024 consecutive entries in 16 steps of 64: pass 1 counts
// them per head (equal-head ballots), one atomic per head and wave reserves
// their positions, pass 2 ranks and writes.  The order of the waves' pieces
// within a head is not fixed; each sample's outputs do not depend on it.
// Block 0 clears the MLP's tile counters.
__global__ __launch_bounds__(kThreads) void level_compact_kernel(
    const unsigned *__restrict__ order, const unsigned *__restrict__ offsets,
    const unsigned *__restrict__ totals, const uint8_t *__restrict__ lvl,
    const uint8_t *__restrict__ cell, unsigned level, unsigned levels, int heads,
    unsigned num_samples, unsigned *__restrict__ live, unsigned *__restrict__ bucket,
    unsigned *__restrict__ mlp_queue)
{
    constexpr int kWavesPerBlock = kThreads / 64;
    constexpr int kSteps = kBucketBlock / kThreads;
    __shared__ unsigned s_pos[kWavesPerBlock][kMaxSites];
    if (blockIdx.x == 0 && threadIdx.x < (unsigned)(kMlpQueues * kMaxHeadGroups))
        mlp_queue[threadIdx.x] = 0;
    const unsigned begin = offsets[level * heads];
    const unsigned end = level + 1 < levels ? offsets[(level + 1) * heads] : num_samples;
    if ((unsigned long long)blockIdx.x * kBucketBlock >= end - begin)
        return;  // (block-uniform) past the level's entries
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int k = lane; k < heads; k += 64)
        s_pos[w][k] = 0;
    const unsigned wbase = begin + blockIdx.x * (unsigned)kBucketBlock + w * (kSteps * 64);
    unsigned sid[kSteps], cs[kSteps];
    bool ok[kSteps];
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const unsigned j = wbase + step * 64 + lane;
        const bool in = j < end;
        sid[step] = in ? order[j] : 0u;
    }
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const unsigned j = wbase + step * 64 + lane;
        const bool in = j < end;
        cs[step] = in ? cell[sid[step]] : 0u;
        ok[step] = in && lvl[sid[step]] == level;
    }
    __syncthreads();
    // pass 1: this wave's live entries per head (run leaders)
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const uint64_t any = __ballot(ok[step]);
        if (any == 0)
            continue;
        const LaneRuns r = lane_runs(cs[step], ok[step], any);
        if ((r.starts >> lane) & 1ull)
            atomicAdd(&s_pos[w][cs[step]], r.len);
    }
    __syncthreads();
    // reserve each head's positions
    for (int k = lane; k < heads; k += 64) {
        const unsigned cnt = s_pos[w][k];
        s_pos[w][k] = cnt ? atomicAdd(live + k, cnt) : 0u;
    }
    __syncthreads();
    // pass 2: ranks and writes
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const uint64_t any = __ballot(ok[step]);
        if (any == 0)
            continue;
        const unsigned c = cs[step];
        const LaneRuns r = lane_runs(c, ok[step], any);
        unsigned start = 0;
        if ((r.starts >> lane) & 1ull)
            start = atomicAdd(&s_pos[w][c], r.len);
        start = __shfl(start, r.first);
        if (ok[step]) {
            const unsigned rank = start + (unsigned)(lane - r.first);
            const unsigned pos = offsets[level * heads + c] + rank;
            // within the head's stretch whenever the totals are consistent
            if (rank < totals[level * heads + c] && pos < num_samples)
                bucket[pos] = sid[step];
        }
    }
}

// ---------------------------------------------------------------------------
// Segment integration and Painter's merge, one wave per ray.  The ray's
// samples are staged through LDS in chunks of kChunk with coalesced loads
// (lane l loads samples l + 64 v); within a chunk lane j takes the
// contiguous samples [j c, j c + c), c = ceil(chunk / 64), integrates its
// runs (integrate_runs), and the 64 lane results are merged in lane order;
// the chunk results are merged in chunk order.  A segment cut by a lane or
// chunk boundary is integrated in pieces merged by "over", which is exact.
constexpr int kChunk = 256;

__global__ __launch_bounds__(kThreads) void composite_kernel(
    const float *__restrict__ t, const uint8_t *__restrict__ cell, const float4 *__restrict__ sr,
    unsigned n, unsigned num_rays, float near_t, float far_t, float *__restrict__ out_rgb,
    float *__restrict__ out_depth, float *__restrict__ out_opacity)
{
    __shared__ float4 s_sr[kThreads / 64][kChunk];
    __shared__ float s_t[kThreads / 64][kChunk + 2];  // [0]: sample before the chunk, [len + 1]: after
    __shared__ uint8_t s_c[kThreads / 64][kChunk];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const unsigned ray = blockIdx.x * (kThreads / 64) + wv;
    // every wave runs every barrier; waves past the last ray stage ray 0 and store nothing
    const bool live = ray < num_rays;
    const size_t base = (size_t)(live ? ray : 0u) * n;
    Over acc{0.f, 0.f, 0.f, 0.f, 1.f};
    for (unsigned c0 = 0; c0 < n; c0 += kChunk) {
        const unsigned len = min((unsigned)kChunk, n - c0);
        for (unsigned k = lane; k < len; k += 64) {
            s_sr[wv][k] = sr[base + c0 + k];
            s_t[wv][k + 1] = t[base + c0 + k];
            s_c[wv][k] = cell[base + c0 + k];
        }
        if (lane == 0)
            s_t[wv][0] = c0 > 0 ? t[base + c0 - 1] : 0.0f;
        if (lane == 1)
            s_t[wv][len + 1] = c0 + len < n ? t[base + c0 + len] : 0.0f;
        __syncthreads();
        const unsigned cl = (len + 63) / 64;
        const unsigned i0 = min(lane * cl, len), i1 = min(i0 + cl, len);
        Over part = integrate_runs(
            c0 + i0, c0 + i1, n, near_t, far_t, [&](unsigned i) { return s_t[wv][i - c0 + 1]; },
            [&](unsigned i) { return (unsigned)s_c[wv][i - c0]; },
            [&](unsigned i) { return s_sr[wv][i - c0]; });
        part = wave_over(part, lane);
        acc = over(acc, part);  // meaningful in lane 0
        __syncthreads();
    }
    if (live && lane == 0) {
        out_rgb[3 * ray] = acc.r;
        out_rgb[3 * ray + 1] = acc.g;
        out_rgb[3 * ray + 2] = acc.b;
        out_depth[ray] = acc.d;
        out_opacity[ray] = 1.0f - acc.t;
    }
}

// The state the levels of a culled render carry from one to the next.
struct LevelState {
    const unsigned *lb;
    uint8_t *lvl;          // [S] sample levels; a closing ray's later samples become dead
    float *trans;          // [R]
    unsigned *evaluated;   // [R] samples integrated so far, or null
    unsigned levels, level;
    float eps;
};

// Integration of one culling level: only the ray's samples of the level,
// [lb[l], lb[l + 1]), are integrated, and the result is merged behind the
// ray's state from the earlier levels (rgb, depth and the transmittance
// trans); a ray whose transmittance is below eps is left as it is, and the
// level that takes a ray below eps marks its later samples dead.
//
// G lanes per ray, 64 / G rays per wave, each wave on its own LDS rows (no
// block barrier: the waves of a block run different numbers of chunks).  A
// ray's range goes in chunks of 4 G samples, staged with consecutive lanes
// on consecutive samples (one load instruction covers 16 G contiguous bytes
// of colours per ray; lanes each reading a stretch of their own from memory
// touched a cache line per lane, and 4x the L2 requests); lane gl then
// integrates the chunk's samples [4 gl, 4 gl + 4) from LDS, the group merges
// its lanes in order (the first log2 G steps of the wave merge), and the
// chunks are merged front to back.
template <int G>
__global__ __launch_bounds__(kThreads) void level_composite_kernel(
    const float *__restrict__ t, const uint8_t *__restrict__ cell, const float4 *__restrict__ sr,
    unsigned n, unsigned num_rays, float near_t, float far_t, LevelState lv,
    float *__restrict__ out_rgb, float *__restrict__ out_depth, float *__restrict__ out_opacity)
{
    constexpr int CH = 4 * G, RPW = 64 / G;  // samples per chunk, rays per wave
    __shared__ float4 s_sr[kThreads / 64][RPW][CH];
    __shared__ float s_t[kThreads / 64][RPW][CH + 2];  // [0]: before the chunk, [len + 1]: after
    __shared__ uint8_t s_c[kThreads / 64][RPW][CH];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, gl = lane & (G - 1), gr = lane / G;
    const unsigned ray = (blockIdx.x * kThreads + threadIdx.x) / G;
    // groups past the last ray stage nothing and store nothing
    const bool live = ray < num_rays;
    const size_t base = (size_t)(live ? ray : 0u) * n;
    Over acc{0.f, 0.f, 0.f, 0.f, 1.f};  // meaningful in the group's first lane
    unsigned a = 0, b = 0;
    bool go = live;
    if (live) {
        const unsigned *r_lb = lv.lb + (size_t)ray * (lv.levels + 1) + lv.level;
        a = r_lb[0];
        b = r_lb[1];
        if (lv.level > 0) {
            acc = Over{out_rgb[3 * ray], out_rgb[3 * ray + 1], out_rgb[3 * ray + 2], out_depth[ray],
                       lv.trans[ray]};
            go = acc.t >= lv.eps;
        }
    }
    if (!go)
        a = b = 0;
    float4 *const gsr = s_sr[wv][gr];
    float *const gt = s_t[wv][gr];
    uint8_t *const gc = s_c[wv][gr];
    // LDS written by some lanes of the wave and read by others
    auto wave_sync = [] {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    // (wave-uniform) until every group of the wave has passed its range's end
    for (unsigned c0 = a; __ballot(c0 < b) != 0; c0 += CH) {
        const unsigned len = c0 < b ? min((unsigned)CH, b - c0) : 0u;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const unsigned j = gl + G * k;
            if (j < len) {
                gsr[j] = sr[base + c0 + j];
                gc[j] = cell[base + c0 + j];
                gt[j + 1] = t[base + c0 + j];
            }
        }
        if (len > 0 && gl == 0)
            gt[0] = c0 > 0 ? t[base + c0 - 1] : 0.0f;
        if (len > 0 && gl == 1)
            gt[len + 1] = c0 + len < n ? t[base + c0 + len] : 0.0f;
        wave_sync();
        const unsigned i0 = min(4u * gl, len), i1 = min(i0 + 4u, len);
        Over part = integrate_runs(
            c0 + i0, c0 + i1, n, near_t, far_t, [&](unsigned i) { return gt[i - c0 + 1]; },
            [&](unsigned i) { return (unsigned)gc[i - c0]; }, [&](unsigned i) { return gsr[i - c0]; });
        part = group_over<G>(part, gl);
        acc = over(acc, part);
        wave_sync();  // the rows are rewritten by the next chunk
    }
    if (go && gl == 0) {
        out_rgb[3 * ray] = acc.r;
        out_rgb[3 * ray + 1] = acc.g;
        out_rgb[3 * ray + 2] = acc.b;
        out_depth[ray] = acc.d;
        out_opacity[ray] = 1.0f - acc.t;
        lv.trans[ray] = acc.t;
        if (lv.evaluated)
            lv.evaluated[ray] = (lv.level > 0 ? lv.evaluated[ray] : 0u) + (b - a);
    }
    // a ray that closes here takes no part in later levels
    const float tr = __shfl(acc.t, lane & ~(G - 1));
    if (go && tr < lv.eps && lv.level + 1 < lv.levels)
        for (unsigned i = b + gl; i < n; i += G)
            lv.lvl[base + i] = kDeadLevel;
}

__global__ __launch_bounds__(kThreads) void debug_expand_kernel(
    unsigned num_samples, const float *__restrict__ t, const uint8_t *__restrict__ cell,
    const float4 *__restrict__ sr, int *dcell, float *dt, float *dsigma, float *drgb)
{
    const unsigned s = blockIdx.x * kThreads + threadIdx.x;
    if (s >= num_samples)
        return;
    if (dcell)
        dcell[s] = cell[s];
    if (dt)
        dt[s] = t[s];
    if (dsigma || drgb) {
        const float4 v = sr[s];
        if (dsigma)
            dsigma[s] = v.x;
        if (drgb) {
            drgb[3 * (size_t)s] = v.y;
            drgb[3 * (size_t)s + 1] = v.z;
            drgb[3 * (size_t)s + 2] = v.w;
        }
    }
}

__global__ __launch_bounds__(kThreads) void fill_u32_kernel(unsigned *__restrict__ p, unsigned count,
                                                          unsigned v)
{
    const unsigned i = blockIdx.x * kThreads + threadIdx.x;
    if (i < count)
        p[i] = v;
}

inline unsigned blocks_for(size_t items, unsigned per) { return (unsigned)((items + per - 1) / per); }

}  // namespace

hipError_t launch_fill_u32(unsigned *p, unsigned count, unsigned v, hipStream_t s)
{
    if (count == 0)
        return hipSuccess;
    fill_u32_kernel<<<blocks_for(count, kThreads), kThreads, 0, s>>>(p, count, v);
    return hipGetLastError();
}

hipError_t launch_ray_encode(const RenderGeometry &g, void *dirbuf, bool bf16, hipStream_t s)
{
    const unsigned grid = blocks_for(g.num_rays, kThreads);
    if (bf16)
        ray_encode_kernel<true><<<grid, kThreads, 0, s>>>(g.rays_d, g.num_rays, dirbuf);
    else
        ray_encode_kernel<false><<<grid, kThreads, 0, s>>>(g.rays_d, g.num_rays, dirbuf);
    return hipGetLastError();
}

hipError_t launch_ray_walk(const RenderGeometry &g, const float4 *sites, int num_sites,
                           SegRec *seg, unsigned char *nseg, hipStream_t s)
{
    // 1, 2 or 4 lanes per ray: enough waves in flight to hide the float64
    // latency of short frames, no more reductions than needed for long ones
    if (g.num_rays >= (1u << 19))
        ray_walk_kernel<1><<<blocks_for(g.num_rays, kThreads), kThreads, 0, s>>>(g, sites, num_sites,
                                                                                 seg, nseg);
    else if (g.num_rays >= (1u << 18))
        ray_walk_kernel<2><<<blocks_for((size_t)g.num_rays * 2, kThreads), kThreads, 0, s>>>(
            g, sites, num_sites, seg, nseg);
    else
        ray_walk_kernel<4><<<blocks_for((size_t)g.num_rays * 4, kThreads), kThreads, 0, s>>>(
            g, sites, num_sites, seg, nseg);
    return hipGetLastError();
}

hipError_t launch_sample_assign(const RenderGeometry &g, const float4 *sites, int num_sites,
                                const WalkTable &walk, float *t, uint8_t *cell,
                                unsigned *counts, unsigned num_blocks, hipStream_t s)
{
    if (walk.seg)
        sample_assign_kernel<false, true><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, walk, t, cell, counts, num_blocks);
    else
        sample_assign_kernel<false, false><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, walk, t, cell, counts, num_blocks);
    return hipGetLastError();
}

hipError_t launch_assign_given(const RenderGeometry &g, const float4 *sites, int num_sites,
                               const WalkTable &walk, const float *t,
                               uint8_t *cell, unsigned *counts, unsigned num_blocks,
                               hipStream_t s)
{
    // t is only read in these instantiations
    if (walk.seg)
        sample_assign_kernel<true, true><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, walk, const_cast<float *>(t), cell, counts, num_blocks);
    else
        sample_assign_kernel<true, false><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, walk, const_cast<float *>(t), cell, counts, num_blocks);
    return hipGetLastError();
}

hipError_t launch_bucket_scan(unsigned *counts, unsigned num_blocks, int num_sites,
                              unsigned *totals, unsigned *mlp_queue, hipStream_t s)
{
    bucket_scan_kernel<<<num_sites, 1024, 0, s>>>(counts, num_blocks, totals, mlp_queue);
    return hipGetLastError();
}

hipError_t launch_bucket_scatter(const uint8_t *cell, const unsigned *counts,
                                 const unsigned *totals, unsigned num_samples,
                                 unsigned num_blocks, int num_sites,
                                 const HeadMask &empty, unsigned *bucket, float4 *sr,
                                 hipStream_t s)
{
    bucket_scatter_kernel<kCellKey><<<num_blocks, kThreads, 0, s>>>(
        cell, counts, totals, num_samples, num_blocks, num_sites, empty, LevelLive{},
        bucket, sr);
    return hipGetLastError();
}

hipError_t launch_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                            const float4 *sr, float *rgb, float *depth, float *opacity,
                            hipStream_t s)
{
    const unsigned grid = blocks_for(g.num_rays, kThreads / 64);
    composite_kernel<<<grid, kThreads, 0, s>>>(t, cell, sr, g.n, g.num_rays, g.near_t, g.far_t, rgb,
                                               depth, opacity);
    return hipGetLastError();
}

hipError_t launch_level_bounds(const uint8_t *cell, unsigned n, unsigned num_rays,
                               unsigned levels, unsigned piece, unsigned *lb, uint8_t *lvl,
                               hipStream_t s)
{
    const unsigned grid = blocks_for(num_rays, kThreads / 64);
    if (n % 4 == 0 && ((uintptr_t)cell | (uintptr_t)lvl) % 4 == 0)
        level_bounds_kernel<true><<<grid, kThreads, 0, s>>>(cell, n, num_rays, levels, piece, lb,
                                                            lvl);
    else
        level_bounds_kernel<false><<<grid, kThreads, 0, s>>>(cell, n, num_rays, levels, piece, lb,
                                                             lvl);
    return hipGetLastError();
}

static LevelLive level_live(const CullLevel &lv) { return LevelLive{lv.lvl, lv.level, 0u}; }

hipError_t launch_level_ray_bucket(const RenderGeometry &g, const uint8_t *cell, int num_sites,
                                   const HeadMask &empty, const CullLevel &lv, unsigned *counts,
                                   unsigned num_blocks, unsigned *totals, unsigned *head_off,
                                   unsigned *bucket, float4 *sr, unsigned *mlp_queue,
                                   hipStream_t s)
{
    if (lv.level + 1 >= lv.levels || num_sites < 1 || num_sites > kMaxSites)
        return hipErrorInvalidValue;
    hipError_t e = launch_fill_u32(counts, (unsigned)num_sites * num_blocks, 0u, s);
    if (e != hipSuccess)
        return e;
    const unsigned grid = blocks_for(g.num_rays, kThreads);
    if (grid > 0) {
        level_ray_count_kernel<<<grid, kThreads, 0, s>>>(cell, lv.lb, lv.trans, g.n, g.num_rays,
                                                         lv.level, lv.levels, lv.eps, counts,
                                                         num_blocks);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    if ((e = launch_bucket_scan(counts, num_blocks, num_sites, totals, mlp_queue, s)) !=
        hipSuccess)
        return e;
    head_offsets_kernel<<<1, kThreads, 0, s>>>(totals, num_sites, head_off);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (grid > 0)
        level_ray_scatter_kernel<<<grid, kThreads, 0, s>>>(
            cell, lv.lb, lv.trans, g.n, g.num_rays, g.num_samples, lv.level, lv.levels, lv.eps,
            empty, head_off, counts, num_blocks, bucket, sr);
    return hipGetLastError();
}

hipError_t launch_level_count(const RenderGeometry &g, const uint8_t *cell, int num_sites,
                              const CullLevel &lv, unsigned *counts,
                              unsigned num_blocks, hipStream_t s)
{
    level_count_kernel<kCellAtLevel><<<num_blocks, kThreads, 0, s>>>(
        cell, g.num_samples, num_sites, level_live(lv), counts, num_blocks);
    return hipGetLastError();
}

hipError_t launch_level_head_order(const RenderGeometry &g, unsigned levels, int heads,
                                   const uint8_t *lvl, const uint8_t *cell,
                                   const HeadMask &empty, unsigned *counts, unsigned num_blocks,
                                   unsigned *totals, unsigned *order, unsigned *offsets,
                                   unsigned *live, float4 *sr, unsigned *mlp_queue, hipStream_t s)
{
    const int keys = (int)levels * heads;
    const LevelLive lk{lvl, 0u, (unsigned)heads};
    level_count_kernel<kLevelCell><<<num_blocks, kThreads, 0, s>>>(cell, g.num_samples, keys,
                                                                   lk, counts, num_blocks);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    e = launch_bucket_scan(counts, num_blocks, keys, totals, mlp_queue, s);
    if (e != hipSuccess)
        return e;
    bucket_scatter_kernel<kLevelCell><<<num_blocks, kThreads, 0, s>>>(
        cell, counts, totals, g.num_samples, num_blocks, keys, empty, lk, order, sr);
    e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    level_head_init_kernel<<<1, kThreads, 0, s>>>(totals, keys, heads, offsets, live, mlp_queue);
    return hipGetLastError();
}

hipError_t launch_level_compact(const RenderGeometry &g, unsigned level, unsigned levels,
                                int heads, const unsigned *order,
                                const unsigned *offsets, const unsigned *totals,
                                const uint8_t *lvl, const uint8_t *cell, unsigned num_blocks,
                                unsigned *live, unsigned *bucket, unsigned *mlp_queue,
                                hipStream_t s)
{
    level_compact_kernel<<<num_blocks, kThreads, 0, s>>>(order, offsets, totals, lvl, cell, level,
                                                         levels, heads, g.num_samples,
                                                         live, bucket, mlp_queue);
    return hipGetLastError();
}

hipError_t launch_level_scatter(const RenderGeometry &g, const uint8_t *cell,
                                const unsigned *counts, const unsigned *totals,
                                unsigned num_blocks, int num_sites,
                                const HeadMask &empty, const CullLevel &lv, unsigned *bucket,
                                float4 *sr, hipStream_t s)
{
    bucket_scatter_kernel<kCellAtLevel><<<num_blocks, kThreads, 0, s>>>(
        cell, counts, totals, g.num_samples, num_blocks, num_sites, empty,
        level_live(lv), bucket, sr);
    return hipGetLastError();
}

hipError_t launch_level_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                                  const float4 *sr, const CullLevel &lv, unsigned max_len,
                                  float *rgb, float *depth, float *opacity, hipStream_t s)
{
    const LevelState st{lv.lb, lv.lvl, lv.trans, lv.evaluated, lv.levels, lv.level, lv.eps};
    // pieces of at most 32 samples: one chunk of 8 lanes per ray; otherwise
    // 16 lanes, in as many chunks of 64 as the range needs
    if (max_len > 0 && max_len <= 32)
        level_composite_kernel<8><<<blocks_for((size_t)g.num_rays * 8, kThreads), kThreads, 0, s>>>(
            t, cell, sr, g.n, g.num_rays, g.near_t, g.far_t, st, rgb, depth, opacity);
    else
        level_composite_kernel<16><<<blocks_for((size_t)g.num_rays * 16, kThreads), kThreads, 0,
                                     s>>>(t, cell, sr, g.n, g.num_rays, g.near_t, g.far_t, st, rgb,
                                          depth, opacity);
    return hipGetLastError();
}

hipError_t launch_debug_expand(unsigned num_samples, const float *t, const uint8_t *cell,
                               const float4 *sr, int *dcell, float *dt, float *dsigma,
                               float *drgb, hipStream_t s)
{
    debug_expand_kernel<<<blocks_for(num_samples, kThreads), kThreads, 0, s>>>(
        num_samples, t, cell, sr, dcell, dt, dsigma, drgb);
    return hipGetLastError();
}

}  // namespace derf
