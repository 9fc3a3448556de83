// Grouped per-head MLP on gfx950 matrix cores.
//
// Every ray sample is evaluated by the single head that owns it (Sec. 3.2:
// the decomposition weights are one-hot, so only that head contributes).
// After bucketing, the samples of head k are one contiguous range, so the
// head network becomes a chain of dense products with M = (samples of k):
// one workgroup takes a tile of a head's samples and runs it through every
// layer with the activations held in registers, while the head's weights
// stream through LDS, one stage (two 32-row output tiles of one layer) at a
// time, double-buffered with direct global->LDS loads.
//
// Operand layout (v_mfma_f32_32x32x16_bf16 / v_mfma_f32_32x32x2_f32):
// weights are the A operand (32 output rows x k), samples the B operand
// (k x 32 samples), so a wave owns NB x 32 samples.  Lane l = n + 32 g holds
// sample n; a 32x32 result leaves in lane l the 16 rows
// 8 (i / 4) + 4 g + (i % 4), i = 0..15.  The next layer consumes those
// registers directly as its B operand; the k-order this implies is folded
// into the weight layout at creation time, so no data moves between layers.
#include <type_traits>
#include <vector>

#include "derf_internal.h"

namespace derf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

template <int N>
using ic = std::integral_constant<int, N>;

template <int B, int E, class F>
__host__ __device__ __forceinline__ void static_for(F &&f)
{
    if constexpr (B < E) {
        f(ic<B>{});
        static_for<B + 1, E>(f);
    }
}

// Row of a 32-row output tile held by lane group g in accumulator register i.
__host__ __device__ constexpr int c_row(int g, int i) { return 8 * (i / 4) + 4 * g + (i % 4); }

// ---------------------------------------------------------------------------
// Compile-time description of one head architecture / precision.
template <bool BF16_, int W_, int D_, int SKIP_, int RH_, int LP_>
struct Cfg {
    static constexpr bool BF16 = BF16_;
    static constexpr int W = W_, D = D_, SKIP = SKIP_, RH = RH_, LP = LP_;
    static constexpr int E = BF16 ? 8 : 1;     // k-entries per lane per MFMA
    static constexpr int CPU = BF16 ? 1 : 4;   // MFMA k-chunks per 1 KB LDS unit
    static constexpr int NB = BF16 ? 2 : 1;    // 32-sample column blocks per wave
    static constexpr int WAVES = (W >= 256) ? 4 : 8;
    static constexpr int THREADS = WAVES * 64;
    static constexpr int TILE = WAVES * NB * 32;
    static constexpr int P = 3 + 6 * LP;       // gamma(x) length
    static constexpr int DD = 27;              // gamma(d) length (4 frequencies)
    static constexpr int P0 = 3 * LP / 2;      // sin/cos pairs held by lane group 0
    static constexpr int EX = ((2 + 2 * P0) + 7) / 8 * 8;  // gamma(x) entries per lane
    static constexpr int EH = W / 2;           // hidden entries per lane
    static constexpr int ED = 16;              // direction entries per lane
    static constexpr int MT = W / 32;          // output tiles per hidden layer
    static constexpr int MTR = (RH + 31) / 32; // output tiles of the colour hidden layer
    static constexpr int ERH = MTR * 16;
    static constexpr int TPS = 2;              // output tiles per stage
    static constexpr int SPL = (MT + TPS - 1) / TPS;
    static constexpr int SPR = (MTR + TPS - 1) / TPS;
    static constexpr int NS = D * SPL + SPR;   // stages per tile
    static_assert(LP % 2 == 0, "pos_freqs must be even");
    static_assert(W % 64 == 0 || W == 32, "width");

    // stage s: kind (0 hidden, 1 colour hidden), layer, first tile, tiles, input entries
    static constexpr int st_kind(int s) { return s < D * SPL ? 0 : 1; }
    static constexpr int st_layer(int s) { return s < D * SPL ? s / SPL : D; }
    static constexpr int st_tile0(int s) { return s < D * SPL ? (s % SPL) * TPS : (s - D * SPL) * TPS; }
    static constexpr int st_ntiles(int s)
    {
        return st_kind(s) == 0 ? (MT - st_tile0(s) < TPS ? MT - st_tile0(s) : TPS)
                               : (MTR - st_tile0(s) < TPS ? MTR - st_tile0(s) : TPS);
    }
    static constexpr int st_entries(int s)
    {
        return st_kind(s) == 1 ? EH + ED
               : st_layer(s) == 0 ? EX
               : st_layer(s) == SKIP ? EX + EH
                                     : EH;
    }
    static constexpr int st_chunks(int s) { return st_entries(s) / E; }
    static constexpr int st_units(int s) { return st_ntiles(s) * st_chunks(s) / CPU; }
    static constexpr int st_offset(int s)  // in units
    {
        int o = 0;
        for (int q = 0; q < s; ++q)
            o += st_units(q);
        return o;
    }
    static constexpr int max_units()
    {
        int m = 0;
        for (int q = 0; q < NS; ++q)
            m = st_units(q) > m ? st_units(q) : m;
        return m;
    }
    static constexpr int STREAM_UNITS = st_offset(NS);
    static constexpr int SMAX = max_units();

    // resident per-head block (floats): biases in accumulator layout, the
    // density row and the colour output rows in lane-entry order
    static constexpr int B_HID = 0;                           // [D][MT][2][16]
    static constexpr int B_RGBH = B_HID + D * MT * 32;        // [MTR][2][16]
    static constexpr int B_WSIG = B_RGBH + MTR * 32;          // [2][EH]
    static constexpr int B_BSIG = B_WSIG + 2 * EH;            // [4]
    static constexpr int B_WC = B_BSIG + 4;                   // [3][2][ERH] or [3][2][EH]
    static constexpr int B_WCD = B_WC + 3 * 2 * (RH > 0 ? ERH : EH);  // [3][2][ED]
    static constexpr int B_BC = B_WCD + (RH > 0 ? 0 : 3 * 2 * ED);    // [4]
    static constexpr int BLOCK_FLOATS = (B_BC + 4 + 255) / 256 * 256;
    static constexpr int BLOCK_UNITS = BLOCK_FLOATS / 256;
    // bf16 path: gamma(x) and gamma(d) chunks wait in LDS, not registers
    static constexpr bool XLDS = BF16;
    static constexpr int GX_UNITS = NB * EX / 8;
    static constexpr int GD_UNITS = NB * 2;
    static constexpr int G_WAVE_BYTES = XLDS ? (GX_UNITS + GD_UNITS) * 1024 : 0;
    static constexpr int G_OFF = 2 * SMAX * 1024 + BLOCK_FLOATS * 4;
    static constexpr int LDS_BYTES = G_OFF + WAVES * G_WAVE_BYTES;
    static_assert(LDS_BYTES + 4 * 1024 <= 160 * 1024, "LDS budget");
};

// Input column (in the packed layer's input order) of lane-entry e of lane
// group g, or -1 for a zero pad.  Layer inputs per lane group are lists:
// gamma(x): entry 0 = x | z, entry 1 = y | pad, then sin/cos pairs
// p = q + g P0 (level p / 3, coordinate p % 3) at entries 2 + 2q, 3 + 2q;
// hidden: entry e = 16 mt + i is row 32 mt + c_row(g, i) of the previous
// layer; direction: entries 0..7 are f[8 g + j], 8..15 are f[16 + 8 g + j].
template <class C>
constexpr int x_col(int g, int e)
{
    if (e == 0)
        return g ? 2 : 0;
    if (e == 1)
        return g ? -1 : 1;
    const int q = (e - 2) / 2;
    if (q >= C::P0)
        return -1;
    const int p = q + g * C::P0;
    const int l = p / 3, c = p % 3;
    return 3 + 6 * l + ((e - 2) % 2 ? 3 : 0) + c;
}
constexpr int h_col(int g, int e) { return 32 * (e / 16) + c_row(g, e % 16); }
constexpr int d_col(int g, int e) { return e < 8 ? 8 * g + e : 16 + 8 * g + (e - 8); }

// ---------------------------------------------------------------------------
// Host-side packing of one head (fp32 packed order of derf.h -> kernel layout).
template <class C>
struct Packer {
    struct View {
        const float *W;
        const float *b;
        int out, in;
    };

    static void views(const float *w, std::vector<View> &v)
    {
        const float *p = w;
        for (int l = 0; l < C::D; ++l) {
            const int in = l == 0 ? C::P : (l == C::SKIP ? C::P + C::W : C::W);
            v.push_back(View{p, p + C::W * in, C::W, in});
            p += C::W * in + C::W;
        }
        v.push_back(View{p, p + C::W, 1, C::W});  // density
        p += C::W + 1;
        if (C::RH > 0) {
            v.push_back(View{p, p + C::RH * (C::W + C::DD), C::RH, C::W + C::DD});
            p += C::RH * (C::W + C::DD) + C::RH;
            v.push_back(View{p, p + 3 * C::RH, 3, C::RH});
        } else {
            v.push_back(View{p, p + 3 * (C::W + C::DD), 3, C::W + C::DD});
        }
    }

    // input column of entry e (lane group g) for stage s, or -1
    static int in_col(int s, int g, int e)
    {
        if (C::st_kind(s) == 1)
            return e < C::EH ? h_col(g, e) : (d_col(g, e - C::EH) < C::DD ? C::W + d_col(g, e - C::EH) : -1);
        const int l = C::st_layer(s);
        if (l == 0)
            return x_col<C>(g, e);
        if (l == C::SKIP) {
            if (e < C::EX) {
                const int c = x_col<C>(g, e);
                return c;
            }
            return C::P + h_col(g, e - C::EX);
        }
        return h_col(g, e);
    }

    static void pack(const float *w, unsigned char *stream, float *block)
    {
        std::vector<View> v;
        views(w, v);
        for (int s = 0; s < C::NS; ++s) {
            const View &L = C::st_kind(s) == 0 ? v[C::st_layer(s)] : v[C::D + 1];
            unsigned char *base = stream + (size_t)C::st_offset(s) * 1024;
            const int chunks = C::st_chunks(s);
            for (int t = 0; t < C::st_ntiles(s); ++t) {
                const int mt = C::st_tile0(s) + t;
                for (int u = 0; u < chunks / C::CPU; ++u) {
                    unsigned char *unit = base + (size_t)(t * (chunks / C::CPU) + u) * 1024;
                    for (int lane = 0; lane < 64; ++lane) {
                        const int m = 32 * mt + lane % 32, g = lane / 32;
                        for (int j = 0; j < 8 / (C::BF16 ? 1 : 2); ++j) {
                            // bf16: 8 k-entries of chunk u; fp32: chunks 4u + j, entry g
                            const int e = C::BF16 ? 8 * u + j : 4 * u + j;
                            const int col = in_col(s, g, e);
                            const float val = (m < L.out && col >= 0) ? L.W[(size_t)m * L.in + col] : 0.0f;
                            if (C::BF16) {
                                const __bf16 bv = (__bf16)val;
                                __builtin_memcpy(unit + lane * 16 + 2 * j, &bv, 2);
                            } else {
                                __builtin_memcpy(unit + lane * 16 + 4 * j, &val, 4);
                            }
                        }
                    }
                }
            }
        }
        for (int i = 0; i < C::BLOCK_FLOATS; ++i)
            block[i] = 0.0f;
        for (int l = 0; l < C::D; ++l)
            for (int mt = 0; mt < C::MT; ++mt)
                for (int g = 0; g < 2; ++g)
                    for (int i = 0; i < 16; ++i)
                        block[C::B_HID + ((l * C::MT + mt) * 2 + g) * 16 + i] = v[l].b[32 * mt + c_row(g, i)];
        if (C::RH > 0) {
            const View &R = v[C::D + 1];
            for (int mt = 0; mt < C::MTR; ++mt)
                for (int g = 0; g < 2; ++g)
                    for (int i = 0; i < 16; ++i) {
                        const int row = 32 * mt + c_row(g, i);
                        block[C::B_RGBH + (mt * 2 + g) * 16 + i] = row < C::RH ? R.b[row] : 0.0f;
                    }
        }
        const View &S = v[C::D];
        for (int g = 0; g < 2; ++g)
            for (int e = 0; e < C::EH; ++e)
                block[C::B_WSIG + g * C::EH + e] = S.W[h_col(g, e)];
        block[C::B_BSIG] = S.b[0];
        const View &O = v.back();
        for (int c = 0; c < 3; ++c) {
            for (int g = 0; g < 2; ++g) {
                if (C::RH > 0) {
                    for (int e = 0; e < C::ERH; ++e) {
                        const int row = h_col(g, e);
                        block[C::B_WC + (c * 2 + g) * C::ERH + e] = row < C::RH ? O.W[c * O.in + row] : 0.0f;
                    }
                } else {
                    for (int e = 0; e < C::EH; ++e)
                        block[C::B_WC + (c * 2 + g) * C::EH + e] = O.W[c * O.in + h_col(g, e)];
                    for (int e = 0; e < C::ED; ++e) {
                        const int f = d_col(g, e);
                        block[C::B_WCD + (c * 2 + g) * C::ED + e] = f < C::DD ? O.W[c * O.in + C::W + f] : 0.0f;
                    }
                }
            }
            block[C::B_BC + c] = O.b[c];
        }
    }
};

// ---------------------------------------------------------------------------
// Device helpers
__device__ __forceinline__ f32x16 mfma(const bf16x8 &a, const bf16x8 &b, const f32x16 &c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma(float a, float b, const f32x16 &c)
{
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

// One wave copies 64 x 16 bytes global -> LDS: lane l reads src_lane and the
// data lands at lds_base + 16 l (lds_base must be the same for the wave).
__device__ __forceinline__ void load_lds16(const void *src_lane, unsigned char *lds_base)
{
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void *)src_lane,
                                     (__attribute__((address_space(3))) void *)lds_base, 16, 0, 0);
}
__device__ __forceinline__ void load_unit_async(const unsigned char *src, unsigned char *lds_unit, int lane)
{
    load_lds16(src + lane * 16, lds_unit);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Round 8 floats to bf16 (nearest even) into one B chunk.
__device__ __forceinline__ bf16x8 to_bf16x8(const float *f)
{
    unsigned w[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
        w[j] = __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{f[2 * j], f[2 * j + 1]}, bf16x2));
    return __builtin_bit_cast(bf16x8, w);
}

// ReLU then round to bf16: accumulator registers 8h .. 8h+7 -> one B chunk.
// A negative bf16 is a negative int16, so the ReLU is a packed int16 max with 0.
__device__ __forceinline__ bf16x8 relu_bf16(const f32x16 &a, int h)
{
    i16x2 p[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const bf16x2 v = __builtin_convertvector(f32x2{a[8 * h + 2 * j], a[8 * h + 2 * j + 1]}, bf16x2);
        p[j] = __builtin_elementwise_max(__builtin_bit_cast(i16x2, v), i16x2{0, 0});
    }
    return __builtin_bit_cast(bf16x8, p);
}

__device__ __forceinline__ float sigmoid(float x) { return __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

// sin(pi 2^l p), cos(pi 2^l p): v_sin/v_cos take revolutions; 2^(l-1) p is
// exact and its fractional part is an exact reduction.
__device__ __forceinline__ void sincos_pi_pow2(float p, int l, float &s, float &c)
{
    const float u = __builtin_amdgcn_fractf(ldexpf(p, l - 1));
    s = __builtin_amdgcn_sinf(u);
    c = __builtin_amdgcn_cosf(u);
}

template <class C>
using Chunk = std::conditional_t<C::BF16, bf16x8, float>;

// Number of A-fragment reads kept in flight ahead of the MFMA that uses them.
constexpr int kPrefetch = 3;

template <class C>
__global__ __launch_bounds__(C::THREADS, 1) void mlp_kernel(
    const unsigned *__restrict__ bucket, const unsigned *__restrict__ totals, int num_sites,
    RenderGeometry geo, const float *__restrict__ tbuf, const void *__restrict__ dirbuf,
    const unsigned char *__restrict__ streams, const float *__restrict__ blocks,
    float4 *__restrict__ sr)
{
    using CT = Chunk<C>;
    constexpr int NB = C::NB, E = C::E;
    constexpr int EXC = C::EX / E, EHC = C::EH / E, EDC = C::ED / E;  // chunks
    extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
    unsigned char *buf0 = lds;
    unsigned char *buf1 = lds + C::SMAX * 1024;
    float *hb = reinterpret_cast<float *>(lds + 2 * C::SMAX * 1024);
    __shared__ unsigned s_off[kMaxSites + 1];   // bucket offset of each head
    __shared__ unsigned s_tile[kMaxSites + 1];  // first tile of each head

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = lane & 31, g = lane >> 5;
    // this wave's staging of gamma(x) and gamma(d) (bf16 path): chunk c of
    // column block nb at ((nb * chunks + c) * 64 + lane) * 16
    unsigned char *gxl = lds + C::G_OFF + wave * C::G_WAVE_BYTES;
    unsigned char *gdl = gxl + C::GX_UNITS * 1024;

    if (tid == 0) {
        unsigned off = 0, tl = 0;
        for (int k = 0; k < num_sites; ++k) {
            s_off[k] = off;
            s_tile[k] = tl;
            off += totals[k];
            tl += (totals[k] + C::TILE - 1) / C::TILE;
        }
        s_off[num_sites] = off;
        s_tile[num_sites] = tl;
    }
    __syncthreads();
    const unsigned total_tiles = s_tile[num_sites];
    // contiguous tile ranges per workgroup; workgroups are dealt round-robin
    // to the 8 XCDs, so map block b to range (b % 8) * G/8 + b / 8 and each
    // XCD (with its own L2) walks one contiguous stretch of heads
    const unsigned G = gridDim.x;
    const unsigned lb = (G % 8 == 0) ? (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8 : blockIdx.x;
    const unsigned t_begin = (unsigned)(((unsigned long long)total_tiles * lb) / G);
    const unsigned t_end = (unsigned)(((unsigned long long)total_tiles * (lb + 1)) / G);

    int head = 0, loaded_head = -1;
    for (unsigned tile = t_begin; tile < t_end; ++tile) {
        while (s_tile[head + 1] <= tile)
            ++head;
        // tile bookkeeping is uniform across the workgroup: keep it scalar
        head = __builtin_amdgcn_readfirstlane(head);
        const unsigned row0 = __builtin_amdgcn_readfirstlane(s_off[head] + (tile - s_tile[head]) * C::TILE);
        // rows never pass the sample count when the bucket counts are
        // consistent; the clamps keep every access in bounds regardless
        const unsigned row_end = __builtin_amdgcn_readfirstlane(min(s_off[head + 1], geo.num_samples));
        if (row0 >= row_end)
            continue;
        const unsigned char *stream = streams + (size_t)head * C::STREAM_UNITS * 1024;

        __syncthreads();  // previous tile is done with the buffers, the head block and staging
        if (head != loaded_head) {
            const unsigned char *src = reinterpret_cast<const unsigned char *>(blocks + (size_t)head * C::BLOCK_FLOATS);
            for (int u = wave; u < C::BLOCK_UNITS; u += C::WAVES)
                load_unit_async(src + u * 1024, reinterpret_cast<unsigned char *>(hb) + u * 1024, lane);
            loaded_head = head;
        }
        for (int u = wave; u < C::st_units(0); u += C::WAVES)
            load_unit_async(stream + (size_t)(C::st_offset(0) + u) * 1024, buf0 + u * 1024, lane);

        // ---- gather the wave's samples and encode them ----------------------
        CT gx[C::XLDS ? 1 : NB][EXC];
        CT gd[C::XLDS ? 1 : NB][EDC];
        unsigned sid[NB];
        bool valid[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const unsigned row = row0 + (wave * NB + nb) * 32 + n;
            valid[nb] = row < row_end;
            sid[nb] = min(bucket[valid[nb] ? row : row0], geo.num_samples - 1);
            unsigned r = (unsigned)((double)sid[nb] * geo.inv_n);
            if (sid[nb] - r * geo.n >= geo.n)
                ++r;
            const float t = tbuf[sid[nb]];
            float x[3];
#pragma unroll
            for (int c = 0; c < 3; ++c)
                x[c] = fmaf(t, geo.rays_d[3 * r + c], geo.rays_o[3 * r + c]);
            float f[C::EX];
            f[0] = g ? x[2] : x[0];
            f[1] = g ? 0.0f : x[1];
#pragma unroll
            for (int q = 0; q < C::P0; ++q) {
                const int l = q / 3 + g * (C::P0 / 3);
                sincos_pi_pow2(x[q % 3], l, f[2 + 2 * q], f[3 + 2 * q]);
            }
#pragma unroll
            for (int e = 2 + 2 * C::P0; e < C::EX; ++e)
                f[e] = 0.0f;
            if constexpr (C::XLDS) {
#pragma unroll
                for (int ch = 0; ch < EXC; ++ch)
                    *reinterpret_cast<bf16x8 *>(gxl + ((nb * EXC + ch) * 64 + lane) * 16) = to_bf16x8(f + 8 * ch);
                // gamma(d) chunks f[8g..8g+7] and f[16+8g..16+8g+7] straight to LDS
                const unsigned char *dp = reinterpret_cast<const unsigned char *>(dirbuf) + (size_t)r * (kDirPad * 2);
                load_lds16(dp + g * 16, gdl + (nb * 2 + 0) * 1024);
                load_lds16(dp + 32 + g * 16, gdl + (nb * 2 + 1) * 1024);
            } else {
#pragma unroll
                for (int e = 0; e < C::EX; ++e)
                    gx[nb][e] = f[e];
                const float4 *dp = reinterpret_cast<const float4 *>(dirbuf) + (size_t)r * (kDirPad / 4);
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const float4 a = dp[4 * h + 2 * g], b = dp[4 * h + 2 * g + 1];
                    gd[nb][8 * h + 0] = a.x; gd[nb][8 * h + 1] = a.y;
                    gd[nb][8 * h + 2] = a.z; gd[nb][8 * h + 3] = a.w;
                    gd[nb][8 * h + 4] = b.x; gd[nb][8 * h + 5] = b.y;
                    gd[nb][8 * h + 6] = b.z; gd[nb][8 * h + 7] = b.w;
                }
            }
        }

        CT act[NB][EHC];
        CT nact[NB][EHC];
        float sig[NB], rgb[3][NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            sig[nb] = 0.0f;
            rgb[0][nb] = rgb[1][nb] = rgb[2][nb] = 0.0f;
        }

        // ---- stages -----------------------------------------------------------
        static_for<0, C::NS>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            constexpr int kind = C::st_kind(s), layer = C::st_layer(s);
            constexpr int tile0 = C::st_tile0(s), ntiles = C::st_ntiles(s);
            constexpr int chunks = C::st_chunks(s);
            constexpr int UPT = chunks / C::CPU;   // LDS units per output tile
            constexpr int NF = ntiles * UPT;       // fragment reads of this stage
            // chunks of this stage's input that come from gamma(x) / gamma(d)
            constexpr bool uses_gx = kind == 0 && (layer == 0 || layer == C::SKIP);
            constexpr bool uses_gd = kind == 1;
            unsigned char *cur = (s % 2 == 0) ? buf0 : buf1;
            unsigned char *nxt = (s % 2 == 0) ? buf1 : buf0;

            __builtin_amdgcn_s_waitcnt(0);  // this wave's loads of stage s landed
            __syncthreads();                // ... and everyone else's; stage s-1 is done
            if constexpr (s + 1 < C::NS) {
                for (int u = wave; u < C::st_units(s + 1); u += C::WAVES)
                    load_unit_async(stream + (size_t)(C::st_offset(s + 1) + u) * 1024, nxt + u * 1024, lane);
            }

            // A fragments of this stage, read kPrefetch ahead of their use
            using AT = std::conditional_t<C::BF16, bf16x8, f32x4>;
            auto frag = [&](int j) -> AT {
                const int t = j % ntiles, u = j / ntiles;
                return *reinterpret_cast<const AT *>(cur + ((t * UPT + u) * 64 + lane) * 16);
            };
            AT fr[kPrefetch];
            static_for<0, (kPrefetch < NF ? kPrefetch : NF)>([&](auto ic0) {
                constexpr int i = decltype(ic0)::value;
                fr[i] = frag(i);
            });

            // staged encodings needed by this stage (bf16 path)
            CT xin[NB][(C::XLDS && uses_gx) ? EXC : 1];
            CT din[NB][(C::XLDS && uses_gd) ? 2 : 1];
            if constexpr (C::XLDS && uses_gx) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int ch = 0; ch < EXC; ++ch)
                        xin[nb][ch] = *reinterpret_cast<const bf16x8 *>(gxl + ((nb * EXC + ch) * 64 + lane) * 16);
            }
            if constexpr (C::XLDS && uses_gd) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int ch = 0; ch < 2; ++ch)
                        din[nb][ch] = *reinterpret_cast<const bf16x8 *>(gdl + ((nb * 2 + ch) * 64 + lane) * 16);
            }

            // B operand chunk c of this stage's input for column block nb
            auto in_chunk = [&](auto cc, int nb) -> CT {
                constexpr int c = decltype(cc)::value;
                if constexpr (kind == 1) {
                    if constexpr (c < EHC) return act[nb][c];
                    else if constexpr (C::XLDS) return din[nb][c - EHC];
                    else return gd[nb][c - EHC];
                } else if constexpr (layer == 0) {
                    if constexpr (C::XLDS) return xin[nb][c];
                    else return gx[nb][c];
                } else if constexpr (layer == C::SKIP) {
                    if constexpr (c < EXC) {
                        if constexpr (C::XLDS) return xin[nb][c];
                        else return gx[nb][c];
                    } else {
                        return act[nb][c - EXC];
                    }
                } else {
                    return act[nb][c];
                }
            };

            f32x16 acc[C::TPS][NB];
#pragma unroll
            for (int t = 0; t < ntiles; ++t) {
                const float *bsrc = (kind == 0)
                    ? hb + C::B_HID + ((layer * C::MT + tile0 + t) * 2 + g) * 16
                    : hb + C::B_RGBH + ((tile0 + t) * 2 + g) * 16;
                f32x16 b;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const f32x4 v = *reinterpret_cast<const f32x4 *>(bsrc + 4 * j);
                    b[4 * j] = v[0]; b[4 * j + 1] = v[1]; b[4 * j + 2] = v[2]; b[4 * j + 3] = v[3];
                }
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    acc[t][nb] = b;
            }

            static_for<0, NF>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                constexpr int t = j % ntiles, u = j / ntiles;
                const AT a = fr[j % kPrefetch];
                if constexpr (j + kPrefetch < NF)
                    fr[j % kPrefetch] = frag(j + kPrefetch);
                if constexpr (C::BF16) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[t][nb] = mfma(a, in_chunk(ic<u>{}, nb), acc[t][nb]);
                } else {
                    static_for<0, 4>([&](auto jj) {
                        constexpr int q = decltype(jj)::value;
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
                            acc[t][nb] = mfma(a[q], in_chunk(ic<4 * u + q>{}, nb), acc[t][nb]);
                    });
                }
            });

            // ---- epilogue -------------------------------------------------------
#pragma unroll
            for (int t = 0; t < ntiles; ++t) {
                const int mt = tile0 + t;
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    if constexpr (kind == 0) {
                        if constexpr (C::BF16) {
                            nact[nb][2 * mt] = relu_bf16(acc[t][nb], 0);
                            nact[nb][2 * mt + 1] = relu_bf16(acc[t][nb], 1);
                        } else {
#pragma unroll
                            for (int i = 0; i < 16; ++i)
                                nact[nb][16 * mt + i] = fmaxf(acc[t][nb][i], 0.0f);
                        }
                        if constexpr (layer == C::D - 1) {
                            const float *ws = hb + C::B_WSIG + g * C::EH + 16 * mt;
#pragma unroll
                            for (int i = 0; i < 16; ++i)
                                sig[nb] = fmaf(ws[i], fmaxf(acc[t][nb][i], 0.0f), sig[nb]);
                            if constexpr (C::RH == 0) {
#pragma unroll
                                for (int c3 = 0; c3 < 3; ++c3) {
                                    const float *wc = hb + C::B_WC + (c3 * 2 + g) * C::EH + 16 * mt;
#pragma unroll
                                    for (int i = 0; i < 16; ++i)
                                        rgb[c3][nb] = fmaf(wc[i], fmaxf(acc[t][nb][i], 0.0f), rgb[c3][nb]);
                                }
                            }
                        }
                    } else {
#pragma unroll
                        for (int c3 = 0; c3 < 3; ++c3) {
                            const float *wc = hb + C::B_WC + (c3 * 2 + g) * C::ERH + 16 * mt;
#pragma unroll
                            for (int i = 0; i < 16; ++i)
                                rgb[c3][nb] = fmaf(wc[i], fmaxf(acc[t][nb][i], 0.0f), rgb[c3][nb]);
                        }
                    }
                }
            }
            if constexpr (kind == 0 && tile0 + ntiles == C::MT) {
                // layer complete: its output becomes the next input
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                    for (int c = 0; c < EHC; ++c)
                        act[nb][c] = nact[nb][c];
            }
        });

        // ---- heads' outputs ----------------------------------------------------
        if constexpr (C::RH == 0) {
            // colour logits also read gamma(d) directly
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int c3 = 0; c3 < 3; ++c3) {
                    const float *wd = hb + C::B_WCD + (c3 * 2 + g) * C::ED;
#pragma unroll
                    for (int e = 0; e < C::ED; ++e) {
                        float dv;
                        if constexpr (C::XLDS)
                            dv = (float)reinterpret_cast<const __bf16 *>(gdl + ((nb * 2 + e / 8) * 64 + lane) * 16)[e % 8];
                        else
                            dv = gd[nb][e];
                        rgb[c3][nb] = fmaf(wd[e], dv, rgb[c3][nb]);
                    }
                }
        }
        const float bsig = hb[C::B_BSIG];
        const float bc0 = hb[C::B_BC], bc1 = hb[C::B_BC + 1], bc2 = hb[C::B_BC + 2];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const float s_all = sig[nb] + __shfl_xor(sig[nb], 32) + bsig;
            const float r0 = rgb[0][nb] + __shfl_xor(rgb[0][nb], 32) + bc0;
            const float r1 = rgb[1][nb] + __shfl_xor(rgb[1][nb], 32) + bc1;
            const float r2 = rgb[2][nb] + __shfl_xor(rgb[2][nb], 32) + bc2;
            if (g == 0 && valid[nb])
                sr[sid[nb]] = make_float4(s_all > 0.0f ? s_all : 0.0f, sigmoid(r0), sigmoid(r1), sigmoid(r2));
        }
    }
}

template <class C>
hipError_t launch_mlp(const unsigned *bucket, const unsigned *totals, int num_sites,
                      const RenderGeometry &g, const float *t, const void *dirbuf,
                      const unsigned char *streams, const float *blocks, float4 *sr, int grid,
                      hipStream_t s)
{
    static bool configured = false;
    if (!configured) {
        // raises the dynamic LDS limit where the runtime keeps one; a runtime
        // without the limit may refuse the call, and the launch below reports
        // any real problem
        if (hipFuncSetAttribute((const void *)mlp_kernel<C>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES) != hipSuccess)
            (void)hipGetLastError();
        configured = true;
    }
    mlp_kernel<C><<<grid, C::THREADS, C::LDS_BYTES, s>>>(bucket, totals, num_sites, g, t, dirbuf,
                                                        streams, blocks, sr);
    return hipGetLastError();
}

template <class C>
const MlpVariant *variant()
{
    static const MlpVariant v = {(size_t)C::STREAM_UNITS * 1024, (size_t)C::BLOCK_FLOATS * 4,
                                 C::TILE, &Packer<C>::pack, &launch_mlp<C>};
    return &v;
}

const MlpVariant *find_mlp_variant(const HeadArch &a, bool bf16)
{
    if (a.dir_freqs != 4)
        return nullptr;
    auto is = [&](int p, int d, int w, int sk, int rh) {
        return a.pos_freqs == p && a.depth == d && a.width == w && a.skip_layer == sk && a.rgb_hidden == rh;
    };
    if (is(6, 4, 64, -1, 0))
        return bf16 ? variant<Cfg<true, 64, 4, -1, 0, 6>>() : variant<Cfg<false, 64, 4, -1, 0, 6>>();
    if (is(10, 8, 128, 5, 64))
        return bf16 ? variant<Cfg<true, 128, 8, 5, 64, 10>>() : variant<Cfg<false, 128, 8, 5, 64, 10>>();
    if (is(10, 6, 64, -1, 32))
        return bf16 ? variant<Cfg<true, 64, 6, -1, 32, 10>>() : variant<Cfg<false, 64, 6, -1, 32, 10>>();
    if (is(10, 8, 256, 5, 128))
        return bf16 ? variant<Cfg<true, 256, 8, 5, 128, 10>>() : nullptr;
    return nullptr;
}

}  // namespace derf
