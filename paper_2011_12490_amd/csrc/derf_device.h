// Device helpers shared by the sampling, compositing and hierarchical
// kernels: the counter-based generator of the sample jitter, the "over"
// operator of the Painter's merge and the per-lane segment integration.
//
// Include after `#pragma clang fp contract(off)`: the sample depths decide
// which Voronoi cell owns a sample, so every fused multiply-add here is
// written out and nothing else may be contracted.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace derf {

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 32x32->64-bit products, Weyl-sequence key schedule between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint2 k)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k.x += 0x9E3779B9u;
            k.y += 0xBB67AE85u;
        }
        const unsigned lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
        const unsigned lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
        c = make_uint4(hi1 ^ c.y ^ k.x, lo1, hi0 ^ c.w ^ k.y, lo0);
    }
    return c;
}

__device__ __forceinline__ unsigned philox_word(uint4 v, unsigned i)
{
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Uniform in [0, 1) on the 2^-24 grid for draw i of frame ray rg in a stream
// (0: stratum jitter, 1: inverse-CDF draws): word i % 4 of the block at
// counter (i / 4, ray low word, ray high word, stream).
__device__ __forceinline__ float jitter(uint2 key, uint64_t rg, unsigned i, unsigned stream)
{
    const uint4 b = philox4x32_10(make_uint4(i >> 2, (unsigned)rg, (unsigned)(rg >> 32), stream), key);
    return (float)(philox_word(b, i & 3u) >> 8) * 0x1.0p-24f;
}

// Painter's merge state of a stretch of a ray: colour, depth and the
// transmittance through it.  "over" is associative: (C, D, T) then
// (C', D', T') gives (C + T C', D + T D', T T').
struct Over {
    float r, g, b, d, t;
};

__device__ __forceinline__ Over over(const Over &a, const Over &b)
{
    return Over{fmaf(a.t, b.r, a.r), fmaf(a.t, b.g, a.g), fmaf(a.t, b.b, a.b),
                fmaf(a.t, b.d, a.d), a.t * b.t};
}

// Integrate samples [i0, i1) of a ray of n samples on [near, far] (Sec. 3.1
// Eq. 1-2 with midpoint intervals).  Each maximal run of one cell is
// integrated with its own local transmittance (Sec. 3.3), and the runs are
// merged front to back.  t_at(i), cell_at(i), sr_at(i) fetch sample i's
// depth, cell and (sigma, r, g, b).
template <class TAt, class CAt, class SAt>
__device__ __forceinline__ Over integrate_runs(unsigned i0, unsigned i1, unsigned n, float near_t,
                                               float far_t, TAt t_at, CAt cell_at, SAt sr_at)
{
    Over acc{0.f, 0.f, 0.f, 0.f, 1.f};  // merged runs
    Over seg{0.f, 0.f, 0.f, 0.f, 1.f};  // current run, local transmittance
    unsigned cur = 0xFFFFFFFFu;
    float t_prev = (i0 > 0 && i0 < n) ? t_at(i0 - 1) : 0.0f;
    float t_cur = i0 < n ? t_at(i0) : 0.0f;
    for (unsigned i = i0; i < i1; ++i) {
        const float t_next = (i + 1 < n) ? t_at(i + 1) : 0.0f;
        const float lo = (i == 0) ? near_t : 0.5f * (t_prev + t_cur);
        const float hi = (i + 1 == n) ? far_t : 0.5f * (t_cur + t_next);
        const unsigned ci = cell_at(i);
        const float4 v = sr_at(i);
        const float tau = __expf(-v.x * (hi - lo));
        const float alpha = 1.0f - tau;
        if (ci != cur) {
            acc = over(acc, seg);
            seg = Over{0.f, 0.f, 0.f, 0.f, 1.f};
            cur = ci;
        }
        const float w = seg.t * alpha;
        seg.r = fmaf(w, v.y, seg.r);
        seg.g = fmaf(w, v.z, seg.g);
        seg.b = fmaf(w, v.w, seg.b);
        seg.d = fmaf(w, t_cur, seg.d);
        seg.t *= tau;
        t_prev = t_cur;
        t_cur = t_next;
    }
    return over(acc, seg);
}

// Value of lane + OFF (OFF = 1, 2, 4, 8; within the 16-lane row) by DPP
// row shift; other lanes' results are unused by the merge below.
template <int OFF>
__device__ __forceinline__ float from_lane_above(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x100 + OFF, 0xF, 0xF, false));
}
// Value of lane + 16 for lanes 0 and 32 (row-pair swap), of lane + 32 for
// lane 0 (half swap).
__device__ __forceinline__ float from_row_above(float x)
{
    return __uint_as_float(__builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false)[1]);
}
__device__ __forceinline__ float from_half_above(float x)
{
    return __uint_as_float(__builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false)[1]);
}

// Ordered merge of the 64 lane results of a wave (lane j's stretch precedes
// lane j + 1's): at step k lane j (j a multiple of 2^(k+1)) absorbs lane
// j + 2^k.  The lane exchanges are DPP row shifts and row/half swaps (no
// LDS).  The result is valid in lane 0.
__device__ __forceinline__ Over wave_over(Over acc, int lane)
{
    auto step = [&](auto fetch, int off) {
        const Over o{fetch(acc.r), fetch(acc.g), fetch(acc.b), fetch(acc.d), fetch(acc.t)};
        if ((lane & (2 * off - 1)) == 0)
            acc = over(acc, o);
    };
    step([](float x) { return from_lane_above<1>(x); }, 1);
    step([](float x) { return from_lane_above<2>(x); }, 2);
    step([](float x) { return from_lane_above<4>(x); }, 4);
    step([](float x) { return from_lane_above<8>(x); }, 8);
    step([](float x) { return from_row_above(x); }, 16);
    step([](float x) { return from_half_above(x); }, 32);
    return acc;
}

// The same ordered merge within each aligned group of G lanes (G = 2, 4,
// 8, 16; gl: lane within the group): valid in the group's first lane.
template <int G>
__device__ __forceinline__ Over group_over(Over acc, int gl)
{
    auto step = [&](auto fetch, int off) {
        const Over o{fetch(acc.r), fetch(acc.g), fetch(acc.b), fetch(acc.d), fetch(acc.t)};
        if ((gl & (2 * off - 1)) == 0)
            acc = over(acc, o);
    };
    if constexpr (G >= 2)
        step([](float x) { return from_lane_above<1>(x); }, 1);
    if constexpr (G >= 4)
        step([](float x) { return from_lane_above<2>(x); }, 2);
    if constexpr (G >= 8)
        step([](float x) { return from_lane_above<4>(x); }, 4);
    if constexpr (G >= 16)
        step([](float x) { return from_lane_above<8>(x); }, 8);
    return acc;
}

}  // namespace derf
