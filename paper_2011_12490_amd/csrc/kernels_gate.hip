// MLP-gating decomposition (Sec. 4, "Decompositions with MLPs"): a small
// network with a softmax output gives each point its head weights; at
// inference the sample goes to the head of largest weight.  The softmax is
// monotone, so that head is the argmax of the logits:
//   h = ReLU(W1 gamma_L(x) + b1),  logits = W2 h + b2,  cell = argmax logits
// (ties to the lowest index).  Unlike a Voronoi cell, a gated cell need not
// be convex, so a ray may enter one cell several times; the integration
// merges runs of one cell front to back, which is exact for any partition.
//
// Both products run on the bf16 matrix cores (v_mfma_f32_32x32x16_bf16,
// float32 accumulate) with every float32 operand carried as two bf16 values,
// a = a_hi + a_lo, and every product as a_hi b_hi + a_hi b_lo + a_lo b_hi --
// three MFMAs per step, each term exact, about 16 significant bits per
// operand kept (the dropped parts are below 2^-18 |a b| each).  The decision
// is taken in that precision, as the oracle's is.  A vector-ALU version in
// float32 was bound by its fused multiply-adds (2,528 per sample for L = 10,
// H = 32, K = 16); here they go to the matrix cores and the vector ALUs keep
// the encoding and the operand splits.
//
// Work split.  The network runs on 32 samples at a time, one per lane pair:
// lanes n and n + 32 both hold sample n and each encodes half of gamma(x) --
// the k-split of the MFMA B operand -- so the 32x32 tiles are
//   layer 1: A = W1 (32 hidden units x 16 inputs), B = gamma (16 x 32 samples)
//   layer 2: A = W2 (32 heads x 16 hidden), B = h (16 x 32 samples),
// and a layer-1 result, which leaves hidden unit 8 (i / 4) + 4 g + i % 4 in
// register i of lane group g, is the layer-2 B operand as it stands (the
// k-order this implies is folded into the packed W2).  Weights and biases
// are packed once by derf_set_gate into 1 KB fragments -- one wave's A
// operand registers of one 16-wide k-chunk -- and copied to LDS when a
// workgroup starts; the workgroups are persistent.  The kernel also draws
// each sample's stratified depth, so the gated render needs neither the cell
// walk nor the nearest-site search.
#pragma clang fp contract(off)

#include <string.h>

#include "derf_device.h"
#include "derf_internal.h"

namespace derf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kGateThreads = 256;
constexpr int kGateWaves = kGateThreads / 64;

// Row of a 32-row MFMA result held by lane group g in accumulator register i.
__host__ __device__ constexpr int acc_row(int g, int i) { return 8 * (i / 4) + 4 * g + (i % 4); }

// Shape of a gate: L frequencies, H hidden units.
struct GateShape {
    int L, H;
    int P;    // gamma length 3 + 6 L
    int P0;   // sin/cos pairs per lane group (half of 3 L)
    int LV;   // levels per lane group
    int EX;   // gamma entries per lane group (padded to whole chunks)
    int NC;   // layer-1 k-chunks (16 inputs each: 8 per lane group)
    int MT1;  // layer-1 output tiles (32 hidden units each)
    int NC2;  // layer-2 k-chunks (16 hidden units each)
    __host__ __device__ constexpr GateShape(int L_, int H_)
        : L(L_), H(H_), P(3 + 6 * L_), P0(3 * L_ / 2), LV(L_ / 2),
          EX((2 + 3 * L_ + 7) / 8 * 8), NC((2 + 3 * L_ + 7) / 8), MT1((H_ + 31) / 32),
          NC2(2 * ((H_ + 31) / 32))
    {
    }
};

// Input column of gamma held at entry e by lane group g, or -1 for padding.
// Entries 0 and 1: x | z and y | pad; then the sin/cos pairs p = q + g P0
// (level p / 3, coordinate p % 3) at entries 2 + 2q and 3 + 2q: each lane
// group holds consecutive levels, which the encoder fills by double angles.
__host__ __device__ constexpr int gamma_col(const GateShape &s, int g, int e)
{
    if (e == 0)
        return g ? 2 : 0;
    if (e == 1)
        return g ? -1 : 1;
    const int q = (e - 2) / 2;
    if (q >= s.P0)
        return -1;
    const int p = q + g * s.P0;
    return 3 + 6 * (p / 3) + ((e - 2) % 2 ? 3 : 0) + p % 3;
}
// Hidden unit held at layer-2 entry e (16 per layer-1 tile) by lane group g.
__host__ __device__ constexpr int hidden_col(int g, int e) { return 32 * (e / 16) + acc_row(g, e % 16); }

// Packed layout (bytes): W1 fragments [MT1][NC][2] (hi, lo), W2 fragments
// [MT2][NC2][2], b1 tiles [MT1][2][16], b2 tiles [MT2][2][16] (floats, lane
// group g's 16 rows).  A fragment: lane l = m + 32 g holds 8 bf16 of row m
// of the tile, columns of chunk entries 8 c .. 8 c + 7 of lane group g.
struct GateLayout {
    size_t w1, w2, b1, b2, bytes;
    int MT2;
    __host__ __device__ GateLayout(const GateShape &s, int K)
    {
        MT2 = (K + 31) / 32;
        w1 = 0;
        w2 = w1 + (size_t)s.MT1 * s.NC * 2 * 1024;
        b1 = w2 + (size_t)MT2 * s.NC2 * 2 * 1024;
        b2 = b1 + (size_t)s.MT1 * 32 * 4;
        bytes = b2 + (size_t)MT2 * 32 * 4;
    }
};

uint16_t bf16_bits(float v)
{
    uint32_t u;
    memcpy(&u, &v, 4);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);  // nearest even; v finite
}
float bf16_value(uint16_t b)
{
    const uint32_t u = (uint32_t)b << 16;
    float v;
    memcpy(&v, &u, 4);
    return v;
}

// v as hi + lo (two bf16 of nearest-even rounding), packed 8 at a time.
__device__ __forceinline__ void split8(const float *v, bf16x8 &hi, bf16x8 &lo)
{
    unsigned h[4], l[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const bf16x2 p = __builtin_convertvector(f32x2{v[2 * j], v[2 * j + 1]}, bf16x2);
        const unsigned u = __builtin_bit_cast(unsigned, p);
        const float h0 = __uint_as_float(u << 16), h1 = __uint_as_float(u & 0xFFFF0000u);
        const bf16x2 q = __builtin_convertvector(f32x2{v[2 * j] - h0, v[2 * j + 1] - h1}, bf16x2);
        h[j] = u;
        l[j] = __builtin_bit_cast(unsigned, q);
    }
    hi = __builtin_bit_cast(bf16x8, h);
    lo = __builtin_bit_cast(bf16x8, l);
}

__device__ __forceinline__ f32x16 mfma(const bf16x8 &a, const bf16x8 &b, const f32x16 &c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// This lane group's gamma entries at x (see gamma_col): the group's first
// level from the hardware sine and cosine of exactly reduced revolutions,
// each further level by sin 2a = 2 sin a cos a, cos 2a = 1 - 2 sin^2 a.
template <int L>
__device__ __forceinline__ void encode(const float x[3], int g, float *f)
{
    constexpr GateShape S(L, 32);
    f[0] = g ? x[2] : x[0];
    f[1] = g ? 0.0f : x[1];
    float sn[3], cs[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const float u = __builtin_amdgcn_fractf(ldexpf(x[k], g * S.LV - 1));
        sn[k] = __builtin_amdgcn_sinf(u);
        cs[k] = __builtin_amdgcn_cosf(u);
    }
#pragma unroll
    for (int lv = 0; lv < S.LV; ++lv)
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            f[2 + 2 * (3 * lv + k)] = sn[k];
            f[3 + 2 * (3 * lv + k)] = cs[k];
            if (lv + 1 < S.LV) {
                const float t = sn[k] * cs[k];
                cs[k] = fmaf(-(sn[k] + sn[k]), sn[k], 1.0f);
                sn[k] = t + t;
            }
        }
#pragma unroll
    for (int e = 2 + 2 * S.P0; e < S.EX; ++e)
        f[e] = 0.0f;
}

// Persistent workgroups; wave w of workgroup b takes the 256-sample
// stretches b kGateWaves + w + j gridDim.x kGateWaves, in blocks of 64.  Each
// lane computes the depth of one sample of a block; the network then runs
// twice, on the block's first and second 32 samples, with the positions
// exchanged between the lane halves.  packed: the layout above,
// staged in LDS.  Writes each sample's depth to t and its gated head to cell
// (and to out_cell, int32, when given).
template <int L, int H>
__global__ __launch_bounds__(kGateThreads) void gate_kernel(RenderGeometry g,
                                                            const unsigned char *__restrict__ packed,
                                                            unsigned bytes, int num_sites,
                                                            float *__restrict__ t,
                                                            uint8_t *__restrict__ cell,
                                                            int *__restrict__ out_cell)
{
    constexpr GateShape S(L, H);
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const GateLayout lay(S, num_sites);
    for (unsigned o = threadIdx.x * 16; o < bytes; o += kGateThreads * 16)
        *reinterpret_cast<uint4 *>(lds + o) = *reinterpret_cast<const uint4 *>(packed + o);
    __syncthreads();

    const int lane = threadIdx.x & 63, lg = lane >> 5;
    const unsigned wave = threadIdx.x >> 6;
    const uint2 key = make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32));
    auto frag = [&](size_t off) { return *reinterpret_cast<const bf16x8 *>(lds + off + lane * 16); };
    auto bias = [&](size_t off) {
        const float *b = reinterpret_cast<const float *>(lds + off) + lg * 16;
        f32x16 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4 q = *reinterpret_cast<const f32x4 *>(b + 4 * j);
            v[4 * j] = q[0];
            v[4 * j + 1] = q[1];
            v[4 * j + 2] = q[2];
            v[4 * j + 3] = q[3];
        }
        return v;
    };
    // The gated head of the sample at x, for 32 samples: lanes n and n + 32
    // hold the same sample n and return the same head.
    auto decide = [&](const float x[3]) {
        // layer 1: gamma split into hi and lo chunks, three MFMAs per chunk
        bf16x8 xh[S.NC], xl[S.NC];
        {
            float f[S.EX];
            encode<L>(x, lg, f);
#pragma unroll
            for (int c = 0; c < S.NC; ++c)
                split8(f + 8 * c, xh[c], xl[c]);
        }
        bf16x8 hh[S.NC2], hl[S.NC2];
#pragma unroll
        for (int mt = 0; mt < S.MT1; ++mt) {
            f32x16 acc = bias(lay.b1 + (size_t)mt * 128);
#pragma unroll
            for (int c = 0; c < S.NC; ++c) {
                const size_t o = lay.w1 + ((size_t)(mt * S.NC + c) * 2) * 1024;
                const bf16x8 ah = frag(o), al = frag(o + 1024);
                acc = mfma(al, xh[c], acc);
                acc = mfma(ah, xl[c], acc);
                acc = mfma(ah, xh[c], acc);
            }
            // ReLU on the bit pattern: a float with the sign bit set is
            // negative (or -0) as an integer too
            float hv[16];
#pragma unroll
            for (int r = 0; r < 16; ++r)
                hv[r] = __int_as_float(max(__float_as_int(acc[r]), 0));
            split8(hv, hh[2 * mt], hl[2 * mt]);
            split8(hv + 8, hh[2 * mt + 1], hl[2 * mt + 1]);
        }

        // layer 2, tile by tile, and the running argmax (rows ascending:
        // strictly larger keeps the lowest head on ties; the rows past the
        // last head have bias -inf and zero weights, so they never win)
        float best = -INFINITY;
        int bk = 0;
        for (int mt2 = 0; mt2 < lay.MT2; ++mt2) {
            f32x16 acc = bias(lay.b2 + (size_t)mt2 * 128);
#pragma unroll
            for (int c = 0; c < S.NC2; ++c) {
                const size_t o = lay.w2 + ((size_t)(mt2 * S.NC2 + c) * 2) * 1024;
                const bf16x8 ah = frag(o), al = frag(o + 1024);
                acc = mfma(al, hh[c], acc);
                acc = mfma(ah, hl[c], acc);
                acc = mfma(ah, hh[c], acc);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const bool take = acc[r] > best;
                best = take ? acc[r] : best;
                bk = take ? 32 * mt2 + acc_row(lg, r) : bk;
            }
        }
        // the other lane group holds the other rows of the same sample
        const float ob = __shfl_xor(best, 32);
        const int ok = __shfl_xor(bk, 32);
        if (ob > best || (ob == best && ok < bk))
            bk = ok;
        return bk < num_sites ? bk : num_sites - 1;
    };

    // A wave takes 256 samples at a time, in four blocks of 64.  The jitter
    // of samples 4 j .. 4 j + 3 of a ray is one Philox block (its four
    // words); when the sample count per ray is a multiple of 4, those
    // quadruples never straddle two rays, so lane l draws the block of the
    // quadruple 4 l .. 4 l + 3 of the 256 once, and each sample reads its
    // word from that lane.  Otherwise every lane draws its own sample's.
    const bool quads = g.perturb && g.n % 4u == 0;
    const unsigned long long NS = g.num_samples;
    const unsigned supers = (unsigned)((NS + 255) / 256);
    for (unsigned sb = blockIdx.x * kGateWaves + wave; sb < supers;
         sb += gridDim.x * kGateWaves) {
        uint4 blk4 = make_uint4(0u, 0u, 0u, 0u);
        if (quads) {
            const unsigned long long s4 = (unsigned long long)sb * 256 + 4 * lane;
            const unsigned sc = s4 < NS ? (unsigned)s4 : 0u;
            unsigned ray = (unsigned)((double)sc * g.inv_n), i = sc - ray * g.n;
            if (i >= g.n) {
                ++ray;
                i -= g.n;
            }
            const uint64_t rg = g.ray_offset + ray;
            blk4 = philox4x32_10(make_uint4(i >> 2, (unsigned)rg, (unsigned)(rg >> 32), 0u), key);
        }
#pragma unroll 1
        for (int w = 0; w < 4; ++w) {
            const unsigned long long s64 = (unsigned long long)sb * 256 + 64 * w + lane;
            const bool valid = s64 < NS;
            const unsigned s = (unsigned)s64;
            // s -> (ray, index within the ray); the float64 quotient is at
            // most one below the true one
            const unsigned sc = valid ? s : 0u;
            unsigned ray = (unsigned)((double)sc * g.inv_n), i = sc - ray * g.n;
            if (i >= g.n) {
                ++ray;
                i -= g.n;
            }
            float xi = 0.5f;
            if (quads) {
                // word i % 4 (= lane % 4) of the block drawn by lane 16 w + lane / 4
                const int src = 16 * w + (lane >> 2);
                const unsigned w0 = __shfl(blk4.x, src), w1 = __shfl(blk4.y, src);
                const unsigned w2 = __shfl(blk4.z, src), w3 = __shfl(blk4.w, src);
                const int e = lane & 3;
                const unsigned word = e == 0 ? w0 : e == 1 ? w1 : e == 2 ? w2 : w3;
                xi = (float)(word >> 8) * 0x1.0p-24f;
            } else if (g.perturb) {
                xi = jitter(key, g.ray_offset + ray, i, 0u);
            }
            const float ts = fmaf(g.step, (float)i + xi, g.near_t);
            float x[3], xa[3], xb[3];
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                x[c] = fmaf(ts, g.rays_d[3 * (size_t)ray + c], g.rays_o[3 * (size_t)ray + c]);
                // lane n holds sample n of the block, lane n + 32 sample n +
                // 32: the first pass takes samples 0..31 on both halves, the
                // second samples 32..63
                const float other = __shfl_xor(x[c], 32);
                xa[c] = lg ? other : x[c];
                xb[c] = lg ? x[c] : other;
            }
            if (valid)
                t[s] = ts;
            const int ka = decide(xa);
            const int kb = decide(xb);
            if (valid) {
                const int k = lg ? kb : ka;
                cell[s] = (uint8_t)k;
                if (out_cell)
                    out_cell[s] = k;
            }
        }
    }
}

template <int L, int H>
hipError_t launch_gate_lh(const RenderGeometry &g, const unsigned char *packed, int num_sites,
                          float *t, uint8_t *cell, int *out_cell, int cus, hipStream_t s)
{
    const GateLayout lay(GateShape(L, H), num_sites);
    const size_t lds = (lay.bytes + 15) / 16 * 16;
    // the largest gates (64 hidden units, 256 heads) need 81 KB of LDS: raise
    // the kernel's dynamic limit to the CU's 160 KB once (a runtime that
    // refuses leaves the launch below to report a real problem)
    static const bool raised = [] {
        if (hipFuncSetAttribute((const void *)gate_kernel<L, H>,
                                hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) !=
            hipSuccess) {
            (void)hipGetLastError();
            return false;
        }
        return true;
    }();
    (void)raised;
    // as many resident workgroups per CU as the LDS allows, at most 4
    const unsigned fit = (unsigned)(160u * 1024u / (lds + 1024));
    const unsigned per_cu = fit < 1 ? 1 : (fit > 4 ? 4 : fit);
    const unsigned supers = (unsigned)(((unsigned long long)g.num_samples + 255) / 256);
    const unsigned want = (supers + kGateWaves - 1) / kGateWaves;
    const unsigned cap = (unsigned)cus * per_cu;
    const unsigned grid = want < cap ? want : cap;
    gate_kernel<L, H><<<grid, kGateThreads, lds, s>>>(g, packed, (unsigned)lay.bytes, num_sites, t,
                                                      cell, out_cell);
    return hipGetLastError();
}

template <int L>
hipError_t launch_gate_l(const RenderGeometry &g, const unsigned char *packed, int hidden,
                         int num_sites, float *t, uint8_t *cell, int *out_cell, int cus,
                         hipStream_t s)
{
    switch (hidden) {
    case 16:
        return launch_gate_lh<L, 16>(g, packed, num_sites, t, cell, out_cell, cus, s);
    case 32:
        return launch_gate_lh<L, 32>(g, packed, num_sites, t, cell, out_cell, cus, s);
    case 64:
        return launch_gate_lh<L, 64>(g, packed, num_sites, t, cell, out_cell, cus, s);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace

bool gate_shape_supported(int pos_freqs, int hidden)
{
    return (pos_freqs == 6 || pos_freqs == 10) && (hidden == 16 || hidden == 32 || hidden == 64);
}

size_t gate_packed_bytes(int pos_freqs, int hidden, int num_sites)
{
    return GateLayout(GateShape(pos_freqs, hidden), num_sites).bytes;
}

void gate_pack(int pos_freqs, int hidden, int num_sites, const float *w, unsigned char *out)
{
    const GateShape S(pos_freqs, hidden);
    const GateLayout lay(S, num_sites);
    const int K = num_sites, H = hidden, P = S.P;
    const float *W1 = w, *b1 = W1 + (size_t)H * P, *W2 = b1 + H, *b2 = W2 + (size_t)K * H;
    memset(out, 0, lay.bytes);
    // one fragment pair (hi, lo) of chunk `chunk`: value(m, g, e) for row m
    // of the tile, lane group g, entry e
    auto put = [&](size_t off, int chunk, auto value) {
        for (int part = 0; part < 2; ++part)
            for (int lane = 0; lane < 64; ++lane) {
                const int m = lane % 32, gg = lane / 32;
                for (int j = 0; j < 8; ++j) {
                    const float v = value(m, gg, 8 * chunk + j);
                    const uint16_t hi = bf16_bits(v);
                    const uint16_t b = part == 0 ? hi : bf16_bits(v - bf16_value(hi));
                    memcpy(out + off + (size_t)part * 1024 + lane * 16 + 2 * j, &b, 2);
                }
            }
    };
    for (int mt = 0; mt < S.MT1; ++mt)
        for (int c = 0; c < S.NC; ++c)
            put(lay.w1 + (size_t)(mt * S.NC + c) * 2 * 1024, c, [&](int m, int gg, int e) {
                const int row = 32 * mt + m, col = gamma_col(S, gg, e);
                return row < H && col >= 0 ? W1[(size_t)row * P + col] : 0.0f;
            });
    for (int mt2 = 0; mt2 < lay.MT2; ++mt2)
        for (int c = 0; c < S.NC2; ++c)
            put(lay.w2 + (size_t)(mt2 * S.NC2 + c) * 2 * 1024, c, [&](int m, int gg, int e) {
                const int row = 32 * mt2 + m, col = hidden_col(gg, e);
                return row < K && col < H ? W2[(size_t)row * H + col] : 0.0f;
            });
    for (int mt = 0; mt < S.MT1; ++mt)
        for (int gg = 0; gg < 2; ++gg)
            for (int i = 0; i < 16; ++i) {
                const int row = 32 * mt + acc_row(gg, i);
                const float v = row < H ? b1[row] : 0.0f;
                memcpy(out + lay.b1 + ((size_t)mt * 32 + gg * 16 + i) * 4, &v, 4);
            }
    for (int mt2 = 0; mt2 < lay.MT2; ++mt2)
        for (int gg = 0; gg < 2; ++gg)
            for (int i = 0; i < 16; ++i) {
                const int row = 32 * mt2 + acc_row(gg, i);
                const float v = row < K ? b2[row] : -INFINITY;
                memcpy(out + lay.b2 + ((size_t)mt2 * 32 + gg * 16 + i) * 4, &v, 4);
            }
}

hipError_t launch_gate(const RenderGeometry &g, const unsigned char *packed, int pos_freqs,
                       int hidden, int num_sites, float *t, uint8_t *cell, int *out_cell, int cus,
                       hipStream_t s)
{
    if (g.num_samples == 0)
        return hipSuccess;
    if (pos_freqs == 6)
        return launch_gate_l<6>(g, packed, hidden, num_sites, t, cell, out_cell, cus, s);
    if (pos_freqs == 10)
        return launch_gate_l<10>(g, packed, hidden, num_sites, t, cell, out_cell, cus, s);
    return hipErrorInvalidValue;
}

}  // namespace derf
