// Grouped per-head MLP on gfx950 matrix cores: the kernel template and its
// host-side launch and weight packing.  Included by one translation unit
// per head architecture (mlp_*.hip), which instantiates its variants.
//
// Every ray sample is evaluated by the single head that owns it (Sec. 3.2:
// the decomposition weights are one-hot, so only that head contributes).
// After bucketing, the samples of head k are one contiguous range, so the
// head network becomes a chain of dense products with M = (samples of k).
//
// Work split.  A workgroup of 4 waves (one per SIMD) takes a tile of one
// head's samples, NB x 32 per wave, and runs it through the whole network
// with the activations held in registers.  Two workgroups share a CU (one for
// width 256, three for bf16 width 64); they do not synchronise with each
// other, so one's barriers and gathers are covered by another's matrix work.
// Workgroups are persistent and take tiles from per-XCD queues, each over a
// contiguous stretch of tiles (so an XCD's L2 sees few heads), stealing from
// the other stretches when their own runs out.
//
// Operand layout (v_mfma_f32_32x32x16_bf16 / v_mfma_f32_32x32x2_f32):
// weights are the A operand (32 output rows x k), samples the B operand
// (k x 32 samples).  Lane l = n + 32 g holds sample n; a 32x32 result leaves
// in lane l the 16 rows 8 (i / 4) + 4 g + (i % 4), i = 0..15, and the next
// layer consumes those registers directly as its B operand.  The k-order this
// implies is folded into the weight layout at creation time, so layers chain
// with no data movement.
//
// Weight streaming.  A head's weights are cut into stages -- one 32-row
// output tile and at most UMAX KB of its input chunks -- laid out as 1 KB units
// that are exactly one wave's A-operand registers.  Stages stream
// global -> LDS (global_load_lds_dwordx4, issued as asm so the compiler's
// LDS wait bookkeeping stays exact) through an 8-slot ring, six stages ahead
// (across tile boundaries too).  Stages are consumed in groups of two: before
// a group, each wave waits with a counted vmcnt for exactly the loads that
// group needs (the count is simulated at compile time from the issue order)
// and one fence-free barrier makes every wave's loads visible and orders
// slot reuse.  The per-step schedule is explicit: A fragments are read from
// LDS a few steps ahead (a window continuous across stages), and a tile's
// bias, ReLU and bf16 rounding are spread over the next tile's MFMAs.
// Density and colour come out of one extra 32-row output tile (row 0
// density, rows 1-3 colour logits), so the network tail needs no cross-lane
// reduction.
#pragma once
#include <type_traits>
#include <vector>

#include "derf_internal.h"

namespace derf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
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
//
// Output tiles, in order: hidden layer l, tile mt (l * MT + mt); the colour
// hidden layer's tiles; the output tile.  Each tile's input is cut into
// stages of at most UMAX units.
enum { K_HID = 0, K_RGBH = 1, K_OUT = 2 };

// A-fragment reads kept in flight ahead of the MFMA that uses them: during
// step F (the F-th fragment of a tile) the wave reads fragment F + kPrefetch.
constexpr int kPrefetch = 3;

// GX_: the stored-encoding form, which reads each sample's gamma(x) entries
// from a table in HBM (gx_encode_kernel) instead of encoding them in the
// tile prologue; kept to measure what the fusion saves.
template <bool BF16_, int W_, int D_, int SKIP_, int RH_, int LP_, bool GX_ = false>
struct Cfg {
    static constexpr bool BF16 = BF16_;
    static constexpr int W = W_, D = D_, SKIP = SKIP_, RH = RH_, LP = LP_;
    static constexpr bool GX = GX_;
    static constexpr int E = BF16 ? 8 : 1;     // k-entries per lane per MFMA
    static constexpr int CPU = BF16 ? 1 : 4;   // MFMA k-chunks per 1 KB unit
    static constexpr int NB = BF16 ? 2 : 1;    // 32-sample column blocks per wave
    static constexpr int WAVES = 4;
    static constexpr int THREADS = WAVES * 64;
    // 64-wide bf16 heads: three workgroups per CU (4 KB ring slots, at most
    // 168 VGPRs), so that more waves hide the per-tile gathers and encoding
    static constexpr int WG_PER_CU = W >= 256 ? 1 : (BF16 && W == 64 ? 3 : 2);
    static constexpr int TILE = WAVES * NB * 32;
    static constexpr int P = 3 + 6 * LP;       // gamma(x) length
    static constexpr int DD = 27;              // gamma(d) length (4 frequencies)
    static constexpr int P0 = 3 * LP / 2;      // sin/cos pairs held by lane group 0
    static constexpr int EX = ((2 + 2 * P0) + 7) / 8 * 8;  // gamma(x) entries per lane
    static constexpr int EH = W / 2;           // hidden entries per lane
    static constexpr int ED = 16;              // direction entries per lane
    static constexpr int MT = W / 32;          // output tiles per hidden layer
    static constexpr int MTR = (RH + 31) / 32; // output tiles of the colour hidden layer
    static constexpr int ERH = MTR * 16;       // colour-hidden entries per lane
    static constexpr int EXC = EX / E, EHC = EH / E, EDC = ED / E, ERHC = ERH / E;
    static constexpr int UMAX = BF16 && W == 64 ? 4 : 8;  // units per stage
    static constexpr int CMAX = UMAX * CPU;    // chunks per stage
    static constexpr int NBUF = 8;             // LDS ring slots (power of two)
    static constexpr int G = 2;                // stages per barrier
    static constexpr int LA = 6;               // weight loads issued this many stages ahead
    static constexpr int NT = D * MT + MTR + 1;
    static_assert(LP % 2 == 0, "pos_freqs must be even");
    static_assert(!GX || SKIP < 0, "the stored encoding has no skip-layer re-encode");
    static_assert(W % 64 == 0, "width");

    static constexpr int t_kind(int T) { return T < D * MT ? K_HID : (T < D * MT + MTR ? K_RGBH : K_OUT); }
    static constexpr int t_layer(int T) { return T < D * MT ? T / MT : -1; }
    static constexpr int t_mt(int T) { return T < D * MT ? T % MT : (T < D * MT + MTR ? T - D * MT : 0); }
    static constexpr int t_entries(int T)
    {
        return t_kind(T) == K_RGBH ? EH + ED
               : t_kind(T) == K_OUT ? EH + (RH > 0 ? ERH : ED)
               : t_layer(T) == 0    ? EX
               : t_layer(T) == SKIP ? EX + EH
                                    : EH;
    }
    static constexpr int t_chunks(int T) { return t_entries(T) / E; }
    static constexpr int t_splits(int T) { return (t_chunks(T) + CMAX - 1) / CMAX; }

    static constexpr int count_stages()
    {
        int n = 0;
        for (int T = 0; T < NT; ++T)
            n += t_splits(T);
        return n;
    }
    static constexpr int NS = count_stages();

    // per-stage table, built once at compile time
    struct StageTab {
        int tile[NS], split[NS], c0[NS], c1[NS], units[NS], lpw[NS], off[NS + 1], foff[NS + 1];
    };
    static constexpr StageTab make_tab()
    {
        StageTab t{};
        int s = 0;
        for (int T = 0; T < NT; ++T)
            for (int k = 0; k < t_splits(T); ++k, ++s) {
                t.tile[s] = T;
                t.split[s] = k;
                t.c0[s] = k * CMAX;
                t.c1[s] = (k + 1) * CMAX < t_chunks(T) ? (k + 1) * CMAX : t_chunks(T);
                t.units[s] = (t.c1[s] - t.c0[s]) / CPU;
                t.lpw[s] = (t.units[s] + WAVES - 1) / WAVES;
            }
        t.off[0] = 0;
        t.foff[0] = 0;
        for (int q = 0; q < NS; ++q) {
            t.off[q + 1] = t.off[q] + t.lpw[q] * WAVES;
            t.foff[q + 1] = t.foff[q] + t.units[q];
        }
        return t;
    }
    static constexpr StageTab TAB = make_tab();

    static constexpr int st_tile(int s) { return TAB.tile[s]; }
    static constexpr int st_split(int s) { return TAB.split[s]; }
    static constexpr int st_c0(int s) { return TAB.c0[s]; }
    static constexpr int st_c1(int s) { return TAB.c1[s]; }
    static constexpr bool st_first(int s) { return TAB.split[s] == 0; }
    static constexpr int st_units(int s) { return TAB.units[s]; }
    static constexpr int st_lpw(int s) { return TAB.lpw[s]; }  // loads per wave
    static constexpr int st_units_pad(int s) { return TAB.lpw[s] * WAVES; }
    static constexpr int st_offset(int s) { return TAB.off[s]; }  // in units
    static constexpr int STREAM_UNITS = TAB.off[NS];

    // A fragments of a tile's stages, numbered consecutively: stage s's
    // fragment j is number foff(s) + j.  The register window holds fragment
    // F in slot F % kPrefetch.
    static constexpr int foff(int s) { return TAB.foff[s]; }
    static constexpr int FTOTAL = TAB.foff[NS];
    static constexpr int f_stage(int F)
    {
        int q = 0;
        while (q + 1 < NS && TAB.foff[q + 1] <= F)
            ++q;
        return q;
    }
    static constexpr int f_index(int F) { return F - TAB.foff[f_stage(F)]; }

    static constexpr int first_stage_of_tile(int T)
    {
        int s = 0;
        for (int q = 0; q < T; ++q)
            s += t_splits(q);
        return s;
    }
    // first stage of the skip layer (gamma(x) is re-encoded one stage
    // earlier), first stage reading gamma(d), stage issuing the gamma(d) loads
    static constexpr int S_SKIP = SKIP >= 0 ? first_stage_of_tile(SKIP * MT) : -1;
    static constexpr int S_GDUSE = first_stage_of_tile(RH > 0 ? D * MT : D * MT + MTR);
    static constexpr int S_GD = S_GDUSE >= 4 ? (S_GDUSE - 4) / G * G : 0;  // a group start
    static constexpr int NGD = NB * (BF16 ? 2 : 4);  // gamma(d) load instructions per wave
    // The next tile's sample records are prefetched into LDS during this one:
    // its bucket ids at group start S_PA (NPA loads per wave), then, once the
    // group wait of S_PB has covered those, its depths and ray origins and
    // directions (NPB loads per wave; none in the stored-encoding form, whose
    // gamma(x) rows are read at the tile start).  The last tile re-reads its
    // own, so that the wait counts do not depend on whether a next tile exists.
    static constexpr int S_PA = 0, S_PB = LA;
    static constexpr int NPA = 1, NPB = GX ? 0 : 7;

    // Barrier groups: stages [a, a + G) of a tile share one barrier.  At a
    // group start a the wave issues the weight loads of stages a + LA ..
    // (the next tile's stages past the end), then the gamma(d) loads if a ==
    // S_GD.  Before the barrier of group a, the units of stage need(a) -- the
    // last stage the group's fragment reads reach: kPrefetch fragments past
    // its last step, which is beyond the next stage when that one is shorter
    // (the 2-unit stages of the 8x256 colour layer) -- must have landed;
    // vm_allowed(a) counts this wave's memory operations issued
    // after those loads (every operation before them has landed too: they
    // complete in issue order).  -1: nothing to wait for (the tile prologue
    // drained everything issued before stage LA's loads).
    static_assert(NS >= LA + G, "pipeline deeper than the stage list");
    static_assert(NBUF >= LA + G, "ring too small for the lookahead");
    static constexpr int grp_end(int a) { return a + G - 1 < NS ? a + G - 1 : NS - 1; }
    static constexpr int need(int a)
    {
        const int next = grp_end(a) + 1 < NS ? grp_end(a) + 1 : grp_end(a);
        const int fe = TAB.foff[grp_end(a) + 1] - 1 + kPrefetch;  // furthest fragment read
        const int reach = f_stage(fe < FTOTAL ? fe : FTOTAL - 1);
        return reach > next ? reach : next;
    }
    // every fragment a group reads lies in a stage its wait covers
    static constexpr bool waits_cover_reads()
    {
        for (int a = 0; a < NS; a += G) {
            const int fe = TAB.foff[grp_end(a) + 1] - 1 + kPrefetch;
            if ((fe < FTOTAL ? fe : FTOTAL - 1) >= TAB.foff[need(a) + 1])
                return false;
        }
        return true;
    }
    // the loads of need(a) were issued before group a (or drained by the tile
    // prologue), so the wait before its barrier can cover them
    static constexpr bool needs_issued_earlier()
    {
        for (int a = 0; a < NS; a += G)
            if (need(a) >= LA && (need(a) - LA) / G * G >= a)
                return false;
        return true;
    }
    static constexpr int vm_allowed(int a, bool has_next)
    {
        const int xn = need(a);
        if (xn < LA)
            return -1;
        const int gn = (xn - LA) / G * G;
        int cnt = 0;
        for (int g = gn; g < a; g += G) {
            for (int x = g + LA; x <= grp_end(g) + LA; ++x) {
                if (g == gn && x <= xn)
                    continue;
                if (x < NS)
                    cnt += st_lpw(x);
                else if (has_next)
                    cnt += st_lpw(x - NS);
            }
            if (g == S_GD)
                cnt += NGD;
            if (g == S_PA)
                cnt += NPA;
            if (g == S_PB)
                cnt += NPB;
        }
        return cnt;
    }
    // loads this wave issues after the S_PB prefetch until the next tile
    // starts (it has one: its records were prefetched)
    static constexpr int loads_after_pb()
    {
        int cnt = 0;
        for (int g = S_PB + G; g < NS; g += G)
            for (int x = g + LA; x <= grp_end(g) + LA; ++x)
                cnt += x < NS ? st_lpw(x) : st_lpw(x - NS);
        return cnt + (S_GD > S_PB ? NGD : 0);
    }
    static_assert(waits_cover_reads(), "a fragment read runs ahead of the group wait");
    static_assert(needs_issued_earlier(), "a group waits for weight loads issued after it");
    static_assert(S_PA % G == 0 && S_PB % G == 0 && S_PB < NS, "prefetch at group starts");
    // the group wait at S_PB covers the S_PA loads: the loads it waits for
    // were issued at a later group start
    static_assert((need(S_PB) - LA) / G * G > S_PA, "prefetch phases too close");

    // per-head resident block: bias of every output tile in accumulator layout
    static constexpr int BLOCK_FLOATS = (NT * 32 + 255) / 256 * 256;
    static constexpr int BLOCK_UNITS = BLOCK_FLOATS / 256;

    // LDS: ring | head block | per wave: the next tile's sample records
    // (bucket id, depth, origin xyz, direction xyz; 64 dwords each)
    static constexpr int SLOT_BYTES = UMAX * 1024;
    static constexpr int HB_OFF = NBUF * SLOT_BYTES;
    static constexpr int PF_OFF = HB_OFF + BLOCK_FLOATS * 4;
    static constexpr int PF_WAVE = 8 * 64 * 4;
    static constexpr int LDS_BYTES = PF_OFF + WAVES * PF_WAVE;
    static_assert(WG_PER_CU * (LDS_BYTES + 3 * 1024) <= 160 * 1024, "LDS budget");
    // a stage's loads cover its units padded to a multiple of WAVES
    static constexpr int max_units_pad()
    {
        int m = 0;
        for (int q = 0; q < NS; ++q)
            m = TAB.lpw[q] * WAVES > m ? TAB.lpw[q] * WAVES : m;
        return m;
    }
    static_assert(max_units_pad() * 1024 <= SLOT_BYTES, "a stage overflows its ring slot");
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

    // weight of output tile T, row m (0..31 within the tile), lane group g, entry e
    static float wval(const std::vector<View> &v, int T, int m, int g, int e)
    {
        const int kind = C::t_kind(T);
        if (kind == K_HID) {
            const int l = C::t_layer(T);
            const View &L = v[l];
            const int row = 32 * C::t_mt(T) + m;
            int col;
            if (l == 0)
                col = x_col<C>(g, e);
            else if (l == C::SKIP)
                col = e < C::EX ? x_col<C>(g, e) : C::P + h_col(g, e - C::EX);
            else
                col = h_col(g, e);
            return col >= 0 ? L.W[(size_t)row * L.in + col] : 0.0f;
        }
        if (kind == K_RGBH) {
            const View &L = v[C::D + 1];
            const int row = 32 * C::t_mt(T) + m;
            if (row >= C::RH)
                return 0.0f;
            int col;
            if (e < C::EH)
                col = h_col(g, e);
            else
                col = d_col(g, e - C::EH) < C::DD ? C::W + d_col(g, e - C::EH) : -1;
            return col >= 0 ? L.W[(size_t)row * L.in + col] : 0.0f;
        }
        // output tile: row 0 density (reads h), rows 1..3 colour logits
        if (m == 0) {
            const View &S = v[C::D];
            return e < C::EH ? S.W[h_col(g, e)] : 0.0f;
        }
        if (m > 3)
            return 0.0f;
        const View &O = v.back();
        const int c3 = m - 1;
        if (C::RH > 0) {
            if (e < C::EH)
                return 0.0f;
            const int row = h_col(g, e - C::EH);
            return row < C::RH ? O.W[(size_t)c3 * O.in + row] : 0.0f;
        }
        if (e < C::EH)
            return O.W[(size_t)c3 * O.in + h_col(g, e)];
        const int f = d_col(g, e - C::EH);
        return f < C::DD ? O.W[(size_t)c3 * O.in + C::W + f] : 0.0f;
    }

    static float bval(const std::vector<View> &v, int T, int row)
    {
        const int kind = C::t_kind(T);
        if (kind == K_HID)
            return v[C::t_layer(T)].b[32 * C::t_mt(T) + row];
        if (kind == K_RGBH) {
            const int r = 32 * C::t_mt(T) + row;
            return r < C::RH ? v[C::D + 1].b[r] : 0.0f;
        }
        if (row == 0)
            return v[C::D].b[0];
        return row <= 3 ? v.back().b[row - 1] : 0.0f;
    }

    static void pack(const float *w, unsigned char *stream, float *block)
    {
        std::vector<View> v;
        views(w, v);
        for (int s = 0; s < C::NS; ++s) {
            const int T = C::st_tile(s), c0 = C::st_c0(s);
            unsigned char *base = stream + (size_t)C::st_offset(s) * 1024;
            for (int u = 0; u < C::st_units_pad(s); ++u) {
                unsigned char *unit = base + (size_t)u * 1024;
                for (int lane = 0; lane < 64; ++lane) {
                    const int m = lane % 32, g = lane / 32;
                    for (int j = 0; j < (C::BF16 ? 8 : 4); ++j) {
                        // bf16: 8 k-entries of chunk c0 + u; fp32: chunk c0 + 4u + j, one entry
                        const int e = C::BF16 ? 8 * (c0 + u) + j : c0 + 4 * u + j;
                        const float val = u < C::st_units(s) ? wval(v, T, m, g, e) : 0.0f;
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
        for (int i = 0; i < C::BLOCK_FLOATS; ++i)
            block[i] = 0.0f;
        for (int T = 0; T < C::NT; ++T)
            for (int g = 0; g < 2; ++g)
                for (int i = 0; i < 16; ++i)
                    block[(T * 2 + g) * 16 + i] = bval(v, T, c_row(g, i));
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

// One wave copies 64 x 16 bytes global -> LDS: lane l reads base + voff and
// the data lands at lds_base + 16 l (base and lds_base are wave-uniform).
// Issued as asm so that the compiler does not track it: its completion is
// awaited explicitly with vmcnt (where it is counted), and the compiler's own
// LDS wait bookkeeping stays exact for the ds_reads around it (it would
// otherwise wait for every outstanding LDS read whenever one of these is in
// flight).  M0 carries the LDS address; nothing else in these kernels uses M0.
__device__ __forceinline__ void load_lds16(const unsigned char *base, unsigned voff,
                                           unsigned char *lds_base)
{
    const unsigned l = (unsigned)(unsigned long)(__attribute__((address_space(3))) unsigned char *)lds_base;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(__builtin_amdgcn_readfirstlane(l)), "v"(voff), "s"(base)
                 : "memory");
}

// One wave gathers 64 dwords global -> LDS: lane l reads *p and the dword
// lands at lds_base + 4 l (lds_base wave-uniform).  Asm for the same reasons
// as load_lds16.
__device__ __forceinline__ void load_lds4(const void *p, unsigned char *lds_base)
{
    const unsigned l = (unsigned)(unsigned long)(__attribute__((address_space(3))) unsigned char *)lds_base;
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off"
                 :: "s"(__builtin_amdgcn_readfirstlane(l)), "v"(p)
                 : "memory");
}

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

// This lane group's gamma(x) entries (see x_col): the lowest level of the
// group is evaluated directly, each higher level by the double-angle
// identities sin 2a = 2 sin a cos a, cos 2a = 1 - 2 sin^2 a.  The rounding
// error at most doubles per level (about 2^-19 after four doublings), far
// below the tolerance of either precision.
template <class C>
__device__ __forceinline__ void encode_x(const float x[3], int g, float *f)
{
    constexpr int LV = C::P0 / 3;  // levels per lane group
    f[0] = g ? x[2] : x[0];
    f[1] = g ? 0.0f : x[1];
    float s[3], c[3];
#pragma unroll
    for (int k = 0; k < 3; ++k)
        sincos_pi_pow2(x[k], g * LV, s[k], c[k]);
#pragma unroll
    for (int lv = 0; lv < LV; ++lv) {
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            f[2 + 2 * (3 * lv + k)] = s[k];
            f[3 + 2 * (3 * lv + k)] = c[k];
            if (lv + 1 < LV) {
                const float t = s[k] * c[k];
                c[k] = fmaf(-(s[k] + s[k]), s[k], 1.0f);
                s[k] = t + t;
            }
        }
    }
#pragma unroll
    for (int e = 2 + 2 * C::P0; e < C::EX; ++e)
        f[e] = 0.0f;
}

// Wait until at most N vector-memory operations of this wave are in flight.
// Written as asm with a memory clobber so that the compiler cannot move a
// memory access across it (the count relies on the issue order).
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_all() { asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory"); }

// Workgroup barrier without the memory fences of __syncthreads(): the waits
// that make LDS data visible are explicit, so in-flight weight loads for
// later stages are not drained at every stage.  The memory clobber keeps the
// compiler from moving LDS accesses across it.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <class C>
using Chunk = std::conditional_t<C::BF16, bf16x8, float>;

// "no tile left" from the work queues
constexpr unsigned kNoTile = 0xFFFFFFFFu;

// SOFT: every head takes every sample (see MlpVariant::launch).  OFFS: each
// head's entries start at offsets[k] (not SOFT).
// gxtab (stored-encoding form only): gamma(x) rows of gx_encode_kernel.
template <class C, bool SOFT, bool OFFS>
__global__ __launch_bounds__(C::THREADS, C::WG_PER_CU) void mlp_kernel(
    const unsigned *__restrict__ bucket, const unsigned *__restrict__ totals,
    const unsigned *__restrict__ offsets, int num_sites, RenderGeometry geo,
    const float *__restrict__ tbuf, const void *__restrict__ dirbuf,
    const Chunk<C> *__restrict__ gxtab,
    const unsigned char *__restrict__ streams, const float *__restrict__ blocks,
    float4 *__restrict__ sr, unsigned *__restrict__ queue, HeadMask empty)
{
    constexpr bool soft = SOFT;
    using CT = Chunk<C>;
    using AT = std::conditional_t<C::BF16, bf16x8, f32x4>;  // one LDS unit per lane
    constexpr int NB = C::NB, NS = C::NS;
    extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
    float *hb = reinterpret_cast<float *>(lds + C::HB_OFF);
    __shared__ unsigned s_off[kMaxSites + 1];   // bucket offset of each head
    __shared__ unsigned s_tile[kMaxSites + 1];  // first tile of each head
    __shared__ unsigned s_q[2];                 // tile indices handed out by the queues

    const int tid = threadIdx.x, lane = tid & 63;
    // wave-uniform by construction; saying so keeps LDS-destination pointers scalar
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane & 31, g = lane >> 5;

    // bucket offset and first tile of each head: exclusive scans of the
    // totals (or the given offsets, where the heads' entries need not be
    // adjacent) and of their tile counts, by wave 0 with 4 heads per lane
    if (tid < 64) {
        unsigned tot[4], nt[4], so = 0, st = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = 4 * tid + j;
            tot[j] = k < num_sites ? totals[k] : 0u;
            // a 0-capacity head keeps its rows but gets no tiles
            nt[j] = k < num_sites && empty.test(k) ? 0u : tot[j] / C::TILE + (tot[j] % C::TILE != 0);
            so += tot[j];
            st += nt[j];
        }
        unsigned io = so, it = st;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const unsigned yo = __shfl_up(io, o), yt = __shfl_up(it, o);
            if (tid >= o) {
                io += yo;
                it += yt;
            }
        }
        unsigned off = io - so, tl = it - st;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int k = 4 * tid + j;
            if (k < num_sites) {
                s_off[k] = OFFS ? offsets[k] : off;
                s_tile[k] = tl;
            }
            off += tot[j];
            tl += nt[j];
        }
        if (tid == 63) {
            s_off[num_sites] = off;
            s_tile[num_sites] = tl;
        }
    }
    __syncthreads();
    const unsigned total_tiles = s_tile[num_sites];

    // Tiles are handed out dynamically.  The tile range is cut into 8
    // contiguous stretches, one per XCD (each XCD has its own L2, and a
    // stretch covers few heads); queue[x] counts the tiles taken from
    // stretch x.  A workgroup takes from its own XCD's stretch, then from the
    // others.  The two workgroups sharing a CU do not get equal shares of its
    // matrix pipe, so static ranges would leave one finishing long after the
    // other.  The counters are zero at launch (the bucket scan clears them).
    const unsigned xcc = (unsigned)__builtin_amdgcn_s_getreg(20 | (31 << 11)) & 7u;  // XCC_ID
    auto q_base = [&](unsigned x) { return (unsigned)(((unsigned long long)total_tiles * x) / 8); };
    // finish a take whose first attempt on the own stretch returned t
    auto take_rest = [&](unsigned t) -> unsigned {
        if (t < q_base(xcc + 1) - q_base(xcc))
            return q_base(xcc) + t;
        for (unsigned k = 1; k < 8; ++k) {
            const unsigned x = (xcc + k) & 7u;
            const unsigned u = atomicAdd(queue + x, 1u);
            if (u < q_base(x + 1) - q_base(x))
                return q_base(x) + u;
        }
        return kNoTile;
    };
    if (tid == 0) {
        s_q[0] = take_rest(atomicAdd(queue + xcc, 1u));
        s_q[1] = take_rest(atomicAdd(queue + xcc, 1u));
    }
    __syncthreads();
    unsigned tile = __builtin_amdgcn_readfirstlane(s_q[0]);
    unsigned next = __builtin_amdgcn_readfirstlane(s_q[1]);
    if (tile == kNoTile)
        return;

    // head owning a tile: the last h with s_tile[h] <= tile (empty heads
    // have s_tile[h] == s_tile[h + 1] and are skipped)
    auto head_of = [&](unsigned t) {
        int lo = 0, hi = num_sites;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (s_tile[mid] <= t)
                lo = mid;
            else
                hi = mid;
        }
        return __builtin_amdgcn_readfirstlane(lo);
    };
    // This wave's first unit of head h's stream.  The base is made opaque so
    // that each unit's address is formed from it with a compile-time offset,
    // instead of the compiler hoisting one wave-dependent offset per unit out
    // of the tile loop (more scalar registers than there are).
    auto stream_of = [&](int h) {
        const unsigned char *p = streams + ((size_t)h * C::STREAM_UNITS + wave) * 1024;
        asm volatile("" : "+s"(p));
        return p;
    };
    auto slot = [&](unsigned k) { return lds + (k & (C::NBUF - 1)) * C::SLOT_BYTES; };
    unsigned char *const lds_wave = lds + wave * 1024;
    // this wave's records of the next tile: [0] bucket id, [1] depth,
    // [2..4] origin, [5..7] direction, slot q = sample nb * 32 + n
    unsigned char *const pf_wave = lds + C::PF_OFF + wave * C::PF_WAVE;
    const unsigned *const pf = reinterpret_cast<const unsigned *>(pf_wave);
    // issue this wave's share of stage s's units into ring slot k
    auto issue = [&](auto sc, const unsigned char *src, unsigned k) {
        constexpr int s = decltype(sc)::value;
        constexpr int lpw = C::st_lpw(s), off = C::st_offset(s);
        unsigned char *dst = lds_wave + (k & (C::NBUF - 1)) * C::SLOT_BYTES;
#pragma unroll
        for (int q = 0; q < lpw; ++q)
            load_lds16(src + (size_t)(off + q * C::WAVES) * 1024, lane * 16, dst + q * C::WAVES * 1024);
        // keep the issue order the wait counts assume
        asm volatile("" ::: "memory");
    };

    // rows end at the sample count; with soft, each head's rows are all the
    // samples again (head k's at k S, read through bucket[row - k S])
    const unsigned row_cap = soft ? s_off[num_sites] : geo.num_samples;
    // end of head h's entries (with offsets, from memory: scalar loads)
    auto head_end = [&](int h) -> unsigned {
        if constexpr (OFFS)
            return offsets[h] + totals[h];
        else
            return s_off[h + 1];
    };
    // the two prefetch phases for the tile whose rows are [r0, r_end) and
    // whose bucket entries start at row base
    auto prefetch_ids = [&](unsigned r0, unsigned r_end, unsigned base) {
        // bucket ids (rows past the head's end read row 0's); offsets from r0,
        // so that a tile padded past 2^32 - 1 does not wrap into range
        const unsigned off = wave * (NB * 32) + lane % (NB * 32);
        const unsigned row = off < r_end - r0 ? r0 + off : r0;
        load_lds4(bucket + min(row - base, geo.num_samples - 1), pf_wave);
    };
    auto prefetch_rays = [&]() {
        if constexpr (C::GX)
            return;
        // depths, ray origins and directions of the ids in LDS
        const unsigned sn = min(pf[lane], geo.num_samples - 1);
        unsigned r = (unsigned)((double)sn * geo.inv_n);
        if (sn - r * geo.n >= geo.n)
            ++r;
        load_lds4(tbuf + sn, pf_wave + 256);
        const float *o = geo.rays_o + 3 * (size_t)r, *d = geo.rays_d + 3 * (size_t)r;
#pragma unroll
        for (int c = 0; c < 3; ++c)
            load_lds4(o + c, pf_wave + 256 * (2 + c));
#pragma unroll
        for (int c = 0; c < 3; ++c)
            load_lds4(d + c, pf_wave + 256 * (5 + c));
    };

    int head = head_of(tile);
    const unsigned char *stream = stream_of(head);
    // the first tile's records, waited for in full
    prefetch_ids(__builtin_amdgcn_readfirstlane(s_off[head] + (tile - s_tile[head]) * C::TILE),
                 __builtin_amdgcn_readfirstlane(min(head_end(head), row_cap)),
                 soft ? s_off[head] : 0u);
    wait_vmcnt<0>();
    prefetch_rays();
    wait_vmcnt<0>();
    unsigned ring = 0;  // ring slot of stage 0 of the current tile (mod NBUF)
    static_for<0, C::LA>([&](auto sc) { issue(sc, stream, ring + decltype(sc)::value); });
    int loaded_head = -1;

    while (tile != kNoTile) {
        const bool has_next = next != kNoTile;
        const int nhead = has_next ? head_of(next) : head;
        const unsigned char *nstream = stream_of(nhead);
        const unsigned row0 = __builtin_amdgcn_readfirstlane(s_off[head] + (tile - s_tile[head]) * C::TILE);
        // rows never pass the sample count when the bucket counts are
        // consistent; the clamps keep every access in bounds regardless
        const unsigned row_end = __builtin_amdgcn_readfirstlane(min(head_end(head), row_cap));
        // rows of the tile whose records are prefetched (this one's if last)
        const unsigned pf_tile = has_next ? next : tile;
        const unsigned nrow0 = __builtin_amdgcn_readfirstlane(s_off[nhead] + (pf_tile - s_tile[nhead]) * C::TILE);
        const unsigned nrow_end = __builtin_amdgcn_readfirstlane(min(head_end(nhead), row_cap));

        wg_barrier();  // previous tile is done with the head block and the staging
        // this tile's records have landed (at most that many loads were issued
        // after them)
        wait_vmcnt<(C::loads_after_pb() < 63 ? C::loads_after_pb() : 63)>();
        // take the tile after next: the attempt on the own stretch is issued
        // here and completes under the prologue's full wait below, so it
        // never disturbs the counted waits of the weight stream
        unsigned q_first = 0;
        if (tid == 0)
            q_first = atomicAdd(queue + xcc, 1u);
        if (head != loaded_head) {
            const unsigned char *src = reinterpret_cast<const unsigned char *>(blocks + (size_t)head * C::BLOCK_FLOATS);
            for (int u = wave; u < C::BLOCK_UNITS; u += C::WAVES)
                load_lds16(src + u * 1024, lane * 16, reinterpret_cast<unsigned char *>(hb) + u * 1024);
            loaded_head = head;
        }

        // ---- gather the wave's samples and encode them ------------------------
        CT gx[NB][C::EXC];
        float xs[NB][3];  // sample positions, kept to re-encode for the skip layer
        unsigned sid[NB], ray[NB];
        bool valid[NB];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            valid[nb] = (wave * NB + nb) * 32 + n < row_end - row0;
            const unsigned q = nb * 32 + n;
            sid[nb] = min(pf[q], geo.num_samples - 1);
            unsigned r = (unsigned)((double)sid[nb] * geo.inv_n);
            if (sid[nb] - r * geo.n >= geo.n)
                ++r;
            ray[nb] = r;
            if constexpr (C::GX) {
                // this lane group's entries of the sample's row, as stored
                const Chunk<C> *src = gxtab + ((size_t)sid[nb] * 2 + g) * C::EXC;
                if constexpr (C::BF16) {
#pragma unroll
                    for (int ch = 0; ch < C::EXC; ++ch)
                        gx[nb][ch] = src[ch];
                } else {
#pragma unroll
                    for (int e = 0; e < C::EX; e += 4) {
                        const f32x4 v = *reinterpret_cast<const f32x4 *>(src + e);
                        gx[nb][e] = v[0]; gx[nb][e + 1] = v[1]; gx[nb][e + 2] = v[2]; gx[nb][e + 3] = v[3];
                    }
                }
                continue;
            }
            const float t = __uint_as_float(pf[64 + q]);
            float x[3];
#pragma unroll
            for (int c = 0; c < 3; ++c)
                x[c] = fmaf(t, __uint_as_float(pf[64 * (5 + c) + q]), __uint_as_float(pf[64 * (2 + c) + q]));
            xs[nb][0] = x[0];
            xs[nb][1] = x[1];
            xs[nb][2] = x[2];
            float f[C::EX];
            encode_x<C>(x, g, f);
            if constexpr (C::BF16) {
#pragma unroll
                for (int ch = 0; ch < C::EXC; ++ch)
                    gx[nb][ch] = to_bf16x8(f + 8 * ch);
            } else {
#pragma unroll
                for (int e = 0; e < C::EX; ++e)
                    gx[nb][e] = f[e];
            }
        }
        wait_all();  // weight stages 0..2 and the head block have landed
        if (tid == 0)
            s_q[0] = take_rest(q_first);
        asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");  // the store above
        wg_barrier();

        CT hbuf[2][NB][C::EHC];                    // hidden outputs, by layer parity
        CT gbuf[NB][C::ERHC > 0 ? C::ERHC : 1];    // colour hidden outputs
        CT gxs[NB][C::EXC];                        // gamma(x) again, for the skip layer
        CT gd[NB][C::EDC];                         // gamma(d)
        f32x16 acc[2][NB];                         // by output-tile parity
        AT fr[kPrefetch];

        auto frag = [&](auto sc, int j) -> AT {
            constexpr int s = decltype(sc)::value;
            return *reinterpret_cast<const AT *>(slot(ring + s) + (j * 64 + lane) * 16);
        };
        auto load_bias = [&](auto tc) {
            constexpr int T = decltype(tc)::value;
            const float *b = hb + (T * 2 + g) * 16;
            f32x16 v;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const f32x4 q = *reinterpret_cast<const f32x4 *>(b + 4 * j);
                v[4 * j] = q[0]; v[4 * j + 1] = q[1]; v[4 * j + 2] = q[2]; v[4 * j + 3] = q[3];
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                acc[T % 2][nb] = v;
        };
        // ReLU + conversion of output tile T into the next layer's input chunks,
        // in pieces so that it can be spread over the next tile's MFMAs:
        // bf16 piece p converts half p / NB of column block p % NB, fp32 piece
        // p a quarter of it
        auto epilogue_piece = [&](auto tc, auto pc) {
            constexpr int T = decltype(tc)::value, p = decltype(pc)::value;
            constexpr int kind = C::t_kind(T), mt = C::t_mt(T), par = C::t_layer(T) % 2;
            constexpr int nb = p % NB, h = p / NB;
            const f32x16 &a = acc[T % 2][nb];
            if constexpr (kind != K_OUT) {
                if constexpr (C::BF16) {
                    if constexpr (kind == K_HID)
                        hbuf[par][nb][2 * mt + h] = relu_bf16(a, h);
                    else
                        gbuf[nb][2 * mt + h] = relu_bf16(a, h);
                } else {
#pragma unroll
                    for (int i = 4 * h; i < 4 * h + 4; ++i) {
                        if constexpr (kind == K_HID)
                            hbuf[par][nb][16 * mt + i] = fmaxf(a[i], 0.0f);
                        else
                            gbuf[nb][16 * mt + i] = fmaxf(a[i], 0.0f);
                    }
                }
            }
        };
        constexpr int NPIECE = C::BF16 ? 2 * NB : 4 * NB;

        // stage 0's bias and the first fragments of the window
        load_bias(ic<0>{});
        static_for<0, (kPrefetch < C::FTOTAL ? kPrefetch : C::FTOTAL)>([&](auto fc) {
            constexpr int F = decltype(fc)::value;
            constexpr int fs = C::f_stage(F), fi = C::f_index(F);
            fr[F % kPrefetch] = frag(ic<fs>{}, fi);
        });

        // ---- stages ------------------------------------------------------------
        static_for<0, NS>([&](auto sc) {
            constexpr int s = decltype(sc)::value;
            constexpr int T = C::st_tile(s), kind = C::t_kind(T), layer = C::t_layer(T);
            constexpr int c0 = C::st_c0(s), NF = C::st_units(s);
            constexpr bool first = C::st_first(s);
            constexpr bool next_first = s + 1 < NS ? C::st_first(s + 1) : false;
            constexpr int next_tile = s + 1 < NS ? C::st_tile(s + 1) : 0;

            if constexpr (s % C::G == 0) {
                // group start: wait for the units the group needs, then one barrier
                constexpr int wa = C::vm_allowed(s, true), wb = C::vm_allowed(s, false);
                if constexpr (s > 0) {
                    if constexpr (wa >= 0 && wa == wb) {
                        wait_vmcnt<wa>();
                    } else if constexpr (wa >= 0) {
                        if (has_next)
                            wait_vmcnt<wa>();
                        else
                            wait_vmcnt<(wb >= 0 ? wb : 0)>();
                    }
                    wg_barrier();
                }
                // weights LA stages ahead (the next tile's past the end)
                static_for<s + C::LA, C::grp_end(s) + C::LA + 1>([&](auto xc) {
                    constexpr int x = decltype(xc)::value;
                    if constexpr (x < NS)
                        issue(ic<x>{}, stream, ring + x);
                    else if (has_next)
                        issue(ic<x - NS>{}, nstream, ring + x);
                });
            }
            if constexpr (s == C::S_GD) {
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    const unsigned char *dp = reinterpret_cast<const unsigned char *>(dirbuf) +
                                              (size_t)ray[nb] * (kDirPad * (C::BF16 ? 2 : 4));
                    if constexpr (C::BF16) {
                        gd[nb][0] = *reinterpret_cast<const bf16x8 *>(dp + g * 16);
                        gd[nb][1] = *reinterpret_cast<const bf16x8 *>(dp + 32 + g * 16);
                    } else {
                        const f32x4 a0 = *reinterpret_cast<const f32x4 *>(dp + g * 32);
                        const f32x4 a1 = *reinterpret_cast<const f32x4 *>(dp + g * 32 + 16);
                        const f32x4 b0 = *reinterpret_cast<const f32x4 *>(dp + 64 + g * 32);
                        const f32x4 b1 = *reinterpret_cast<const f32x4 *>(dp + 64 + g * 32 + 16);
                        static_for<0, 4>([&](auto kc) {
                            constexpr int k = decltype(kc)::value;
                            gd[nb][k] = a0[k];
                            gd[nb][4 + k] = a1[k];
                            gd[nb][8 + k] = b0[k];
                            gd[nb][12 + k] = b1[k];
                        });
                    }
                }
            }
            if constexpr (s == C::S_PA)
                prefetch_ids(nrow0, nrow_end, soft ? s_off[nhead] : 0u);
            if constexpr (s == C::S_PB)
                prefetch_rays();  // the group wait above covered the ids
            if constexpr (s + 1 == C::S_SKIP) {
                // gamma(x) again for the skip layer, overlapping this stage's MFMAs
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) {
                    float f[C::EX];
                    encode_x<C>(xs[nb], g, f);
                    if constexpr (C::BF16) {
#pragma unroll
                        for (int ch = 0; ch < C::EXC; ++ch)
                            gxs[nb][ch] = to_bf16x8(f + 8 * ch);
                    } else {
#pragma unroll
                        for (int e = 0; e < C::EX; ++e)
                            gxs[nb][e] = f[e];
                    }
                }
            }

            // B operand chunk c of this tile's input for column block nb
            auto in_chunk = [&](auto cc, int nb) -> CT {
                constexpr int c = decltype(cc)::value;
                if constexpr (kind == K_HID) {
                    if constexpr (layer == 0) {
                        return gx[nb][c];
                    } else if constexpr (layer == C::SKIP) {
                        if constexpr (c < C::EXC) return gxs[nb][c];
                        else return hbuf[(layer - 1) % 2][nb][c - C::EXC];
                    } else {
                        return hbuf[(layer - 1) % 2][nb][c];
                    }
                } else if constexpr (kind == K_RGBH) {
                    if constexpr (c < C::EHC) return hbuf[(C::D - 1) % 2][nb][c];
                    else return gd[nb][c - C::EHC];
                } else {
                    if constexpr (c < C::EHC) return hbuf[(C::D - 1) % 2][nb][c];
                    else if constexpr (C::RH > 0) return gbuf[nb][c - C::EHC];
                    else return gd[nb][c - C::EHC];
                }
            };

            // Schedule of one step j: a piece of the previous tile's epilogue
            // (first stage of a tile), the read of the fragment kPrefetch
            // ahead (possibly the next stage's), the next tile's bias (late in
            // its last stage), then this step's MFMAs; sched_barrier keeps the
            // order, so LDS latency hides behind the MFMAs in between.
            constexpr bool EPI = first && T > 0;
            constexpr int ESTEPS = EPI ? (NF < NPIECE ? NF : NPIECE) : 0;
            constexpr int JB0 = NF >= 2 ? NF - 2 : 0;
            constexpr int JB = next_first ? (JB0 > ESTEPS ? JB0 : ESTEPS) : NF;  // bias step
            static_for<0, NF>([&](auto jc) {
                constexpr int j = decltype(jc)::value;
                constexpr int F = C::foff(s) + j;
                if constexpr (EPI && j < ESTEPS) {
                    // pieces p with p * ESTEPS / NPIECE == j
                    static_for<0, NPIECE>([&](auto pc) {
                        constexpr int pp = decltype(pc)::value;
                        if constexpr (pp * ESTEPS / NPIECE == j)
                            epilogue_piece(ic<T - 1>{}, pc);
                    });
                }
                const AT a = fr[F % kPrefetch];
                if constexpr (F + kPrefetch < C::FTOTAL) {
                    constexpr int fs = C::f_stage(F + kPrefetch), fi = C::f_index(F + kPrefetch);
                    fr[F % kPrefetch] = frag(ic<fs>{}, fi);
                }
                if constexpr (j == JB && next_first)
                    load_bias(ic<next_tile>{});
                if constexpr (C::BF16) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[T % 2][nb] = mfma(a, in_chunk(ic<c0 + j>{}, nb), acc[T % 2][nb]);
                } else {
                    static_for<0, 4>([&](auto qc) {
                        constexpr int q = decltype(qc)::value;
#pragma unroll
                        for (int nb = 0; nb < NB; ++nb)
                            acc[T % 2][nb] = mfma(a[q], in_chunk(ic<c0 + 4 * j + q>{}, nb), acc[T % 2][nb]);
                    });
                }
                __builtin_amdgcn_sched_barrier(0);
            });
            if constexpr (JB >= NF && next_first)
                load_bias(ic<next_tile>{});
        });

        // ---- density and colour: rows 0..3 of the output tile, lanes g = 0 ----
        constexpr int TO = C::NT - 1;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const f32x16 &a = acc[TO % 2][nb];
            if (g == 0 && valid[nb])
                sr[soft ? row0 + (wave * NB + nb) * 32 + n : sid[nb]] =
                    make_float4(fmaxf(a[0], 0.0f), sigmoid(a[1]), sigmoid(a[2]), sigmoid(a[3]));
        }
        ring += NS;
        head = nhead;
        stream = nstream;
        tile = next;
        next = __builtin_amdgcn_readfirstlane(s_q[0]);
    }
    // the last tile's prefetch re-read its own records: no LDS write may be
    // in flight when the workgroup's LDS is released
    wait_vmcnt<0>();
}

// gamma(x) of every sample into the table the stored-encoding form reads:
// row s holds lane group 0's EX entries, then lane group 1's, exactly as the
// tile prologue would hold them (the same encode_x and rounding), so both
// forms give the same outputs bit for bit.  One lane per (sample, group)
// encodes its entries into LDS; the block then writes its 256 rows out as
// one contiguous stretch, each store 16 contiguous bytes per lane.
template <class C>
__global__ __launch_bounds__(256) void gx_encode_kernel(RenderGeometry geo,
                                                        const float *__restrict__ tbuf,
                                                        Chunk<C> *__restrict__ out)
{
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    constexpr int U = C::EX * (C::BF16 ? 2 : 4) / 16;  // 16-byte units per row
    __shared__ u32x4 stage[256 * U];
    const unsigned long long rows = 2ull * geo.num_samples;
    u32x4 *const dst_all = reinterpret_cast<u32x4 *>(out);
    for (unsigned long long base = (unsigned long long)blockIdx.x * 256; base < rows;
         base += (unsigned long long)gridDim.x * 256) {
        const unsigned long long i = base + threadIdx.x;
        if (i < rows) {
            const unsigned sn = (unsigned)(i >> 1);
            const int g = (int)(i & 1);
            unsigned r = (unsigned)((double)sn * geo.inv_n);
            if (sn - r * geo.n >= geo.n)
                ++r;
            const float t = tbuf[sn];
            float x[3];
#pragma unroll
            for (int c = 0; c < 3; ++c)
                x[c] = fmaf(t, geo.rays_d[3 * (size_t)r + c], geo.rays_o[3 * (size_t)r + c]);
            float f[C::EX];
            encode_x<C>(x, g, f);
            u32x4 *mine = stage + threadIdx.x * U;
            if constexpr (C::BF16) {
#pragma unroll
                for (int ch = 0; ch < C::EXC; ++ch)
                    mine[ch] = __builtin_bit_cast(u32x4, to_bf16x8(f + 8 * ch));
            } else {
#pragma unroll
                for (int u = 0; u < U; ++u)
                    mine[u] = u32x4{__float_as_uint(f[4 * u]), __float_as_uint(f[4 * u + 1]),
                                    __float_as_uint(f[4 * u + 2]), __float_as_uint(f[4 * u + 3])};
            }
        }
        __syncthreads();
        const unsigned long long left = rows - base;
        const unsigned units = (unsigned)(left < 256 ? left : 256) * U;
        u32x4 *dst = dst_all + base * U;
#pragma unroll
        for (int k = 0; k < U; ++k) {
            const unsigned idx = k * 256 + threadIdx.x;
            if (idx < units)
                dst[idx] = stage[idx];
        }
        __syncthreads();  // the stage is rewritten by the next stretch
    }
}

template <class C>
hipError_t launch_gx_encode(const RenderGeometry &g, const float *t, void *gxtab, int cus,
                            hipStream_t s)
{
    if (g.num_samples == 0)
        return hipSuccess;
    const unsigned long long lanes = 2ull * g.num_samples;
    const unsigned long long want = (lanes + 255) / 256, cap = (unsigned long long)cus * 64;
    gx_encode_kernel<C><<<(unsigned)(want < cap ? want : cap), 256, 0, s>>>(
        g, t, reinterpret_cast<Chunk<C> *>(gxtab));
    return hipGetLastError();
}

template <class C>
hipError_t launch_mlp(const unsigned *bucket, const unsigned *totals, const unsigned *offsets,
                      int num_sites,
                      const RenderGeometry &g, const float *t, const void *dirbuf,
                      const void *gxtab, const unsigned char *streams, const float *blocks,
                      float4 *sr, unsigned *queue, int cus, bool soft, const HeadMask &empty,
                      hipStream_t s)
{
    if (C::GX ? (soft || !gxtab) : gxtab != nullptr)
        return hipErrorInvalidValue;
    // raises the dynamic LDS limit where the runtime keeps one, once per
    // variant (thread-safe); a runtime without the limit may refuse the
    // call, and the launch below reports any real problem
    static const bool raised = [] {
        for (const void *k : {(const void *)mlp_kernel<C, false, false>,
                              (const void *)mlp_kernel<C, !C::GX, false>,
                              (const void *)mlp_kernel<C, false, true>})
            if (hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS_BYTES) !=
                hipSuccess)
                (void)hipGetLastError();
        return true;
    }();
    (void)raised;
    const Chunk<C> *gx = reinterpret_cast<const Chunk<C> *>(gxtab);
    const dim3 grid(cus * C::WG_PER_CU), block(C::THREADS);
    if constexpr (!C::GX) {
        if (soft) {
            mlp_kernel<C, true, false><<<grid, block, C::LDS_BYTES, s>>>(
                bucket, totals, nullptr, num_sites, g, t, dirbuf, gx, streams, blocks, sr, queue,
                empty);
            return hipGetLastError();
        }
    }
    if (offsets)
        mlp_kernel<C, false, true><<<grid, block, C::LDS_BYTES, s>>>(
            bucket, totals, offsets, num_sites, g, t, dirbuf, gx, streams, blocks, sr, queue, empty);
    else
        mlp_kernel<C, false, false><<<grid, block, C::LDS_BYTES, s>>>(
            bucket, totals, nullptr, num_sites, g, t, dirbuf, gx, streams, blocks, sr, queue, empty);
    return hipGetLastError();
}

// The stored-encoding form of an architecture without a skip layer.
template <class C>
using StoredForm = Cfg<C::BF16, C::W, C::D, C::SKIP, C::RH, C::LP, true>;

template <class C>
const MlpVariant *variant()
{
    const MlpVariant *stored = nullptr;
    if constexpr (C::SKIP < 0 && !C::GX) {
        static_assert(StoredForm<C>::STREAM_UNITS == C::STREAM_UNITS &&
                          StoredForm<C>::BLOCK_FLOATS == C::BLOCK_FLOATS,
                      "both forms take the same packed weights");
        stored = variant<StoredForm<C>>();
    }
    static const MlpVariant v = {(size_t)C::STREAM_UNITS * 1024,
                                 (size_t)C::BLOCK_FLOATS * 4,
                                 C::TILE,
                                 &Packer<C>::pack,
                                 &launch_mlp<C>,
                                 stored,
                                 C::GX ? (size_t)2 * C::EX * (C::BF16 ? 2 : 4) : 0,
                                 C::LP,
                                 C::GX ? &launch_gx_encode<C> : nullptr};
    return &v;
}

}  // namespace derf
