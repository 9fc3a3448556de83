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
// Lanes of this wave whose value equals mine, among the lanes in `valid`:
// one ballot per bit of the value.
__device__ __forceinline__ uint64_t match_peers(unsigned v, int bits, uint64_t valid)
{
    uint64_t peers = valid;
    for (int b = 0; b < bits; ++b) {
        const bool bit = (v >> b) & 1u;
        const uint64_t m = __ballot(bit);
        peers &= bit ? m : ~m;
    }
    return peers;
}

// Stratified depths t, owning cell (nearest site, ties to the lowest index)
// and per-block head histograms.  Block b covers samples
// [b * kBucketBlock, (b + 1) * kBucketBlock); each thread takes 4 consecutive
// samples per round, so one Philox block serves 4 samples of a ray.  With
// FROM_T the depths are given (t is read, not written): the assignment of
// the inverse-CDF samples of hierarchical sampling.
template <bool FROM_T>
__global__ __launch_bounds__(kThreads) void sample_assign_kernel(
    RenderGeometry g, const float4 *__restrict__ sites, int num_sites, int site_bits,
    float *__restrict__ t_out, uint8_t *__restrict__ cell_out, unsigned *__restrict__ counts,
    unsigned num_blocks)
{
    __shared__ float4 s_sites[kMaxSites];
    __shared__ unsigned s_hist[kMaxSites];
    for (int k = threadIdx.x; k < num_sites; k += kThreads) {
        s_sites[k] = sites[k];
        s_hist[k] = 0;
    }
    __syncthreads();

    const uint2 key = make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32));
    const unsigned block_base = blockIdx.x * (unsigned)kBucketBlock;
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
                float best = INFINITY;
                unsigned bk = 0;
                for (int k = 0; k < num_sites; ++k) {
                    const float4 p = s_sites[k];
                    const float ex = x - p.x, ey = y - p.y, ez = z - p.z;
                    const float d2 = fmaf(ez, ez, fmaf(ey, ey, ex * ex));
                    if (d2 < best) {
                        best = d2;
                        bk = k;
                    }
                }
                tv[v] = t;
                cv[v] = bk;
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
        // histogram: the lowest lane of each group of equal cells adds the group size
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const bool ok = s0 + v < g.num_samples;
            const uint64_t valid = __ballot(ok);
            const uint64_t peers = match_peers(cv[v], site_bits, valid);
            if (ok && (peers & (lane_bit - 1)) == 0)
                atomicAdd(&s_hist[cv[v]], (unsigned)__popcll(peers));
        }
    }
    __syncthreads();
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        counts[(size_t)k * num_blocks + blockIdx.x] = s_hist[k];
}

// Wave-wide minimum / maximum, result in every lane, without LDS: DPP
// within each 16-lane row (quad swaps, half-row and row mirrors), then the
// row-pair and half swaps.
template <bool MAX>
__device__ __forceinline__ float wave_reduce(float v)
{
    auto op = [](float a, float b) { return MAX ? fmaxf(a, b) : fminf(a, b); };
    auto dpp = [](float x, auto ctrl) {
        return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), decltype(ctrl)::value, 0xF, 0xF, false));
    };
    v = op(v, dpp(v, std::integral_constant<int, 0xB1>{}));   // quad_perm [1,0,3,2]
    v = op(v, dpp(v, std::integral_constant<int, 0x4E>{}));   // quad_perm [2,3,0,1]
    v = op(v, dpp(v, std::integral_constant<int, 0x141>{}));  // row_half_mirror
    v = op(v, dpp(v, std::integral_constant<int, 0x140>{}));  // row_mirror
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return op(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float wave_min(float v) { return wave_reduce<false>(v); }
__device__ __forceinline__ float wave_max(float v) { return wave_reduce<true>(v); }

// Heads at or above this count use site pruning in the assignment (below it
// the brute force over all sites costs less than the per-slice bounds).
constexpr int kPruneSites = 48;

// The same, for many heads: in a round wave w takes 256 consecutive
// samples, lane l the samples l + 64 v (v = 0..3), so each v is a slice of
// 64 consecutive samples -- a short piece of one or two rays.  Per slice the
// wave takes the bounding box of its sample points and
// keeps only the sites whose smallest squared distance to the box is within
// a factor 1 + 1e-4 of the smallest largest squared distance of any site to
// the box.  For every point of the box a dropped site is farther, by more
// than that relative margin, than the site attaining that bound, and the
// float32 distances are accurate to a few ulp, so a dropped site can neither
// win nor tie: the argmin over the kept sites (in ascending index order,
// same arithmetic) is the argmin over all sites.
template <bool FROM_T>
__global__ __launch_bounds__(kThreads) void sample_assign_pruned_kernel(
    RenderGeometry g, const float4 *__restrict__ sites, int num_sites, int site_bits,
    float *__restrict__ t_out, uint8_t *__restrict__ cell_out, unsigned *__restrict__ counts,
    unsigned num_blocks)
{
    __shared__ float4 s_sites[kMaxSites];
    __shared__ unsigned s_hist[kMaxSites];
    for (int k = threadIdx.x; k < num_sites; k += kThreads) {
        s_sites[k] = sites[k];
        s_hist[k] = 0;
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const uint64_t lane_bit = 1ull << lane;
    const uint2 key = make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32));
    const unsigned block_base = blockIdx.x * (unsigned)kBucketBlock;
    // with n % 4 == 0 the 4 samples sharing a generator block sit in 4
    // neighbouring lanes: each lane computes one block and they trade words
    const bool quad = (g.n & 3u) == 0;
    for (int round = 0; round < kBucketBlock / (4 * kThreads); ++round) {
        const unsigned wbase = block_base + round * (4 * kThreads) + wv * 256;
        uint4 qb = make_uint4(0, 0, 0, 0);
        if constexpr (!FROM_T) {
            if (g.perturb && quad) {
                // lane L: block of samples wbase + 64 (L / 16) + 4 (L % 16) + 0..3
                const unsigned sq = wbase + 64 * (lane >> 4) + 4 * (lane & 15);
                unsigned rq, iq;
                split_sample(sq < g.num_samples ? sq : 0, g.n, g.inv_n, rq, iq);
                const uint64_t rg = g.ray_offset + rq;
                qb = philox4x32_10(make_uint4(iq >> 2, (unsigned)rg, (unsigned)(rg >> 32), 0u), key);
            }
        }
        float tv[4];
        unsigned cv[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const unsigned s = wbase + 64 * v + lane;
            const bool ok = s < g.num_samples;
            unsigned r, i;
            split_sample(ok ? s : 0, g.n, g.inv_n, r, i);
            float t;
            if constexpr (FROM_T) {
                t = ok ? t_out[s] : 0.0f;
            } else {
                float xi = 0.5f;
                if (g.perturb) {
                    unsigned w;
                    if (quad) {
                        const int src = 16 * v + (lane >> 2);
                        const unsigned w0 = __shfl(qb.x, src), w1 = __shfl(qb.y, src);
                        const unsigned w2 = __shfl(qb.z, src), w3 = __shfl(qb.w, src);
                        const unsigned q = lane & 3;
                        w = q == 0 ? w0 : q == 1 ? w1 : q == 2 ? w2 : w3;
                    } else {
                        const uint64_t rg = g.ray_offset + r;
                        w = philox_word(philox4x32_10(make_uint4(i >> 2, (unsigned)rg, (unsigned)(rg >> 32), 0u), key),
                                        i & 3u);
                    }
                    xi = (float)(w >> 8) * 0x1.0p-24f;
                }
                t = fmaf(g.step, (float)i + xi, g.near_t);
            }
            const float x = fmaf(t, g.rays_d[3 * r], g.rays_o[3 * r]);
            const float y = fmaf(t, g.rays_d[3 * r + 1], g.rays_o[3 * r + 1]);
            const float z = fmaf(t, g.rays_d[3 * r + 2], g.rays_o[3 * r + 2]);

            float best = INFINITY;
            unsigned bk = 0;
            const float lx = wave_min(ok ? x : INFINITY), hx = wave_max(ok ? x : -INFINITY);
            const float ly = wave_min(ok ? y : INFINITY), hy = wave_max(ok ? y : -INFINITY);
            const float lz = wave_min(ok ? z : INFINITY), hz = wave_max(ok ? z : -INFINITY);
            // smallest over sites of the largest squared distance to the box
            float thr = INFINITY;
            for (int k = lane; k < num_sites; k += 64) {
                const float4 p = s_sites[k];
                const float ax = fmaxf(p.x - lx, hx - p.x), ay = fmaxf(p.y - ly, hy - p.y);
                const float az = fmaxf(p.z - lz, hz - p.z);
                thr = fminf(thr, fmaf(az, az, fmaf(ay, ay, ax * ax)));
            }
            thr = wave_min(thr) * (1.0f + 1e-4f);
            for (int m = 0; 64 * m < num_sites; ++m) {
                const int kl = 64 * m + lane;
                bool keep = false;
                if (kl < num_sites) {
                    const float4 p = s_sites[kl];
                    const float bx = fmaxf(fmaxf(lx - p.x, p.x - hx), 0.0f);
                    const float by = fmaxf(fmaxf(ly - p.y, p.y - hy), 0.0f);
                    const float bz = fmaxf(fmaxf(lz - p.z, p.z - hz), 0.0f);
                    keep = fmaf(bz, bz, fmaf(by, by, bx * bx)) <= thr;
                }
                uint64_t mk = __ballot(keep);
                while (mk) {
                    const int k = 64 * m + __builtin_ctzll(mk);
                    mk &= mk - 1;
                    const float4 p = s_sites[k];
                    const float ex = x - p.x, ey = y - p.y, ez = z - p.z;
                    const float d2 = fmaf(ez, ez, fmaf(ey, ey, ex * ex));
                    if (d2 < best) {
                        best = d2;
                        bk = k;
                    }
                }
            }
            tv[v] = t;
            cv[v] = ok ? bk : 0xFFFFFFFFu;
            if (ok) {
                if constexpr (!FROM_T)
                    t_out[s] = t;
                cell_out[s] = (uint8_t)bk;
            }
        }
        // histogram: the lowest lane of each group of equal cells adds the group size
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const bool ok = wbase + 64 * v + lane < g.num_samples;
            const uint64_t valid = __ballot(ok);
            const uint64_t peers = match_peers(cv[v], site_bits, valid);
            if (ok && (peers & (lane_bit - 1)) == 0)
                atomicAdd(&s_hist[cv[v]], (unsigned)__popcll(peers));
        }
        (void)tv;
    }
    __syncthreads();
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        counts[(size_t)k * num_blocks + blockIdx.x] = s_hist[k];
}

// ---------------------------------------------------------------------------
// Exclusive prefix over blocks of each head's counts (one block per head),
// in place; the head's total goes to totals[head].  Block 0 also clears the
// tile counters of the MLP launch that follows on the stream.
__global__ __launch_bounds__(1024) void bucket_scan_kernel(unsigned *__restrict__ counts,
                                                           unsigned num_blocks,
                                                           unsigned *__restrict__ totals,
                                                           unsigned *__restrict__ mlp_queue)
{
    if (blockIdx.x == 0 && threadIdx.x < (unsigned)kMlpQueues)
        mlp_queue[threadIdx.x] = 0;
    __shared__ unsigned s_wave[16];
    __shared__ unsigned s_carry;
    unsigned *col = counts + (size_t)blockIdx.x * num_blocks;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (threadIdx.x == 0)
        s_carry = 0;
    __syncthreads();
    for (unsigned base = 0; base < num_blocks; base += 1024) {
        const unsigned idx = base + threadIdx.x;
        const unsigned v = idx < num_blocks ? col[idx] : 0u;
        // inclusive scan within the wave
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
        const unsigned before = (w > 0 ? s_wave[w - 1] : 0u) + x - v;
        if (idx < num_blocks)
            col[idx] = carry + before;
        __syncthreads();
        if (threadIdx.x == 0)
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

// Stable scatter of sample ids into per-head buckets.  Bucket k occupies
// [offset_k, offset_k + total_k) with offset_k = sum of totals below k;
// within it samples keep increasing sample-id order, so each ray's run
// through cell k stays contiguous.  Block b's samples are its 4096 of the
// counting pass; wave w takes the 1024 consecutive ones from 1024 w, in 16
// steps of 64 (all 16 cells loaded up front).  Pass 1 counts each wave's
// samples per head (equal-cell ballots, wave-private counters); after one
// barrier every wave knows its first position per head (the block's base
// plus the earlier waves' counts); pass 2 ranks each step's samples of one
// head by ballot and advances the wave's own counters.
__global__ __launch_bounds__(kThreads) void bucket_scatter_kernel(
    const uint8_t *__restrict__ cell, const unsigned *__restrict__ prefix,
    const unsigned *__restrict__ totals, unsigned num_samples, unsigned num_blocks,
    int num_sites, int site_bits, unsigned *__restrict__ bucket)
{
    constexpr int kWavesPerBlock = kThreads / 64;
    constexpr int kSteps = kBucketBlock / kThreads;  // 64-sample steps per wave
    __shared__ unsigned s_base[kMaxSites];
    __shared__ unsigned s_pos[kWavesPerBlock][kMaxSites];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t below = (1ull << lane) - 1;
    head_block_base(prefix, totals, num_blocks, num_sites, s_base);
    for (int k = threadIdx.x; k < num_sites; k += kThreads)
        for (int v = 0; v < kWavesPerBlock; ++v)
            s_pos[v][k] = 0;
    const unsigned wbase = blockIdx.x * (unsigned)kBucketBlock + w * (kSteps * 64);
    unsigned cs[kSteps];
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const unsigned s = wbase + step * 64 + lane;
        cs[step] = s < num_samples ? cell[s] : 0u;
    }
    __syncthreads();
    // pass 1: this wave's count per head
#pragma unroll
    for (int step = 0; step < kSteps; ++step) {
        const bool ok = wbase + step * 64 + lane < num_samples;
        const uint64_t peers = match_peers(cs[step], site_bits, __ballot(ok));
        if (ok && (peers & below) == 0)
            s_pos[w][cs[step]] += (unsigned)__popcll(peers);
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
        const bool ok = s < num_samples;
        const unsigned c = cs[step];
        const uint64_t peers = match_peers(c, site_bits, __ballot(ok));
        const unsigned start = ok ? s_pos[w][c] : 0u;
        if (ok) {
            const unsigned pos = start + (unsigned)__popcll(peers & below);
            if (pos < num_samples)  // always true when the counts are consistent
                bucket[pos] = s;
            if ((peers & below) == 0)
                s_pos[w][c] = start + (unsigned)__popcll(peers);
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

inline unsigned blocks_for(unsigned items, unsigned per) { return (items + per - 1) / per; }

}  // namespace

hipError_t launch_ray_encode(const RenderGeometry &g, void *dirbuf, bool bf16, hipStream_t s)
{
    const unsigned grid = blocks_for(g.num_rays, kThreads);
    if (bf16)
        ray_encode_kernel<true><<<grid, kThreads, 0, s>>>(g.rays_d, g.num_rays, dirbuf);
    else
        ray_encode_kernel<false><<<grid, kThreads, 0, s>>>(g.rays_d, g.num_rays, dirbuf);
    return hipGetLastError();
}

hipError_t launch_sample_assign(const RenderGeometry &g, const float4 *sites, int num_sites,
                                int site_bits, float *t, uint8_t *cell, unsigned *counts,
                                unsigned num_blocks, hipStream_t s)
{
    if (num_sites >= kPruneSites)
        sample_assign_pruned_kernel<false><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, site_bits, t, cell, counts, num_blocks);
    else
        sample_assign_kernel<false><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, site_bits, t, cell, counts, num_blocks);
    return hipGetLastError();
}

hipError_t launch_assign_given(const RenderGeometry &g, const float4 *sites, int num_sites,
                               int site_bits, const float *t, uint8_t *cell, unsigned *counts,
                               unsigned num_blocks, hipStream_t s)
{
    // t is only read in this instantiation
    if (num_sites >= kPruneSites)
        sample_assign_pruned_kernel<true><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, site_bits, const_cast<float *>(t), cell, counts, num_blocks);
    else
        sample_assign_kernel<true><<<num_blocks, kThreads, 0, s>>>(
            g, sites, num_sites, site_bits, const_cast<float *>(t), cell, counts, num_blocks);
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
                                 unsigned num_blocks, int num_sites, int site_bits,
                                 unsigned *bucket, hipStream_t s)
{
    bucket_scatter_kernel<<<num_blocks, kThreads, 0, s>>>(cell, counts, totals, num_samples,
                                                          num_blocks, num_sites, site_bits, bucket);
    return hipGetLastError();
}

hipError_t launch_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                            const float4 *sr, float *rgb, float *depth, float *opacity,
                            hipStream_t s)
{
    const unsigned grid = blocks_for(g.num_rays, kThreads / 64);
    composite_kernel<<<grid, kThreads, 0, s>>>(t, cell, sr, g.n, g.num_rays, g.near_t, g.far_t,
                                               rgb, depth, opacity);
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
