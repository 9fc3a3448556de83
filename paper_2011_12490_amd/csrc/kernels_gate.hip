// MLP-gating decomposition (Sec. 4, "Decompositions with MLPs"): a small
// network with a softmax output gives each point its head weights; at
// inference the sample goes to the head of largest weight.  The softmax is
// monotone, so that head is the argmax of the logits:
//   h = ReLU(W1 gamma_L(x) + b1),  logits = W2 h + b2,  cell = argmax logits
// (ties to the lowest index).  Unlike a Voronoi cell, a gated cell need not
// be convex, so a ray may enter one cell several times; the integration
// merges runs of one cell front to back, which is exact for any partition.
//
// One thread per sample, fp32 with fused multiply-adds in index order.  The
// weights (at most 64 (3 + 6 L) + 65 K floats) are read with wave-uniform
// addresses, so they come through the scalar cache; the encoded input and
// the hidden layer stay in registers.  The kernel also draws each sample's
// stratified depth, so the gated render needs neither the cell walk nor the
// nearest-site search.  Measured, it is bound by its fp32 FMAs on the vector
// ALUs (about 96 % of their issue rate, the FMAs alone about 86 % of the
// cycles).
#pragma clang fp contract(off)

#include "derf_device.h"
#include "derf_internal.h"

namespace derf {
namespace {

constexpr int kGateThreads = 256;

// gamma_L(p): p, then sin(pi 2^l p) and cos(pi 2^l p) per level l.  The
// hardware sine and cosine take revolutions: sin(pi y) = sin(2 pi frac(y / 2)),
// where y / 2 = 2^(l-1) p is exact and so is its fractional part, so each
// pair costs a scale, a fract and the two transcendental instructions.
template <int L>
__device__ __forceinline__ void gate_encode(const float x[3], float f[3 + 6 * L])
{
#pragma unroll
    for (int c = 0; c < 3; ++c)
        f[c] = x[c];
#pragma unroll
    for (int l = 0; l < L; ++l)
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            const float u = __builtin_amdgcn_fractf(ldexpf(x[c], l - 1));
            f[3 + 6 * l + c] = __builtin_amdgcn_sinf(u);
            f[6 + 6 * l + c] = __builtin_amdgcn_cosf(u);
        }
}

// w: W1 [H][P], b1 [H], W2 [K][H], b2 [K] (P = 3 + 6 L).  Draws the sample's
// stratified depth (Sec. 3.1, the generator of the single pass) and writes
// it to t, then its gated head to cell and to out_cell (int32 [S]) when given.
template <int L, int H>
__global__ __launch_bounds__(kGateThreads) void gate_kernel(RenderGeometry g,
                                                            const float *__restrict__ w,
                                                            int num_sites, float *__restrict__ t,
                                                            uint8_t *__restrict__ cell,
                                                            int *__restrict__ out_cell)
{
    constexpr int P = 3 + 6 * L;
    const unsigned s = blockIdx.x * kGateThreads + threadIdx.x;
    if (s >= g.num_samples)
        return;
    // s -> (ray, index within the ray); the float64 quotient is at most one
    // below the true one
    unsigned ray = (unsigned)((double)s * g.inv_n), i = s - ray * g.n;
    if (i >= g.n) {
        ++ray;
        i -= g.n;
    }
    const float xi = g.perturb ? jitter(make_uint2((unsigned)g.seed, (unsigned)(g.seed >> 32)),
                                        g.ray_offset + ray, i, 0u)
                               : 0.5f;
    const float ts = fmaf(g.step, (float)i + xi, g.near_t);
    t[s] = ts;
    float x[3];
#pragma unroll
    for (int c = 0; c < 3; ++c)
        x[c] = fmaf(ts, g.rays_d[3 * (size_t)ray + c], g.rays_o[3 * (size_t)ray + c]);
    float f[P];
    gate_encode<L>(x, f);
    const float *b1 = w + H * P, *w2 = b1 + H, *b2 = w2 + (size_t)num_sites * H;
    float h[H];
#pragma unroll
    for (int j = 0; j < H; ++j) {
        float acc = b1[j];
#pragma unroll
        for (int c = 0; c < P; ++c)
            acc = fmaf(w[j * P + c], f[c], acc);
        h[j] = fmaxf(acc, 0.0f);
    }
    // logits two at a time, so that both rows' weight loads are in flight
    // together; each logit and the order of the comparisons are unchanged
    int best = 0;
    float top = -INFINITY;
    int k = 0;
    for (; k + 1 < num_sites; k += 2) {
        float a0 = b2[k], a1 = b2[k + 1];
#pragma unroll
        for (int j = 0; j < H; ++j) {
            a0 = fmaf(w2[k * H + j], h[j], a0);
            a1 = fmaf(w2[(k + 1) * H + j], h[j], a1);
        }
        if (a0 > top) {  // strictly larger: ties keep the lower index
            top = a0;
            best = k;
        }
        if (a1 > top) {
            top = a1;
            best = k + 1;
        }
    }
    if (k < num_sites) {
        float acc = b2[k];
#pragma unroll
        for (int j = 0; j < H; ++j)
            acc = fmaf(w2[k * H + j], h[j], acc);
        if (acc > top) {
            top = acc;
            best = k;
        }
    }
    cell[s] = (uint8_t)best;
    if (out_cell)
        out_cell[s] = best;
}

template <int L>
hipError_t launch_gate_l(const RenderGeometry &g, const float *w, int hidden, int num_sites,
                         float *t, uint8_t *cell, int *out_cell, hipStream_t s)
{
    const unsigned grid = (unsigned)(((size_t)g.num_samples + kGateThreads - 1) / kGateThreads);
    switch (hidden) {
    case 16:
        gate_kernel<L, 16><<<grid, kGateThreads, 0, s>>>(g, w, num_sites, t, cell, out_cell);
        break;
    case 32:
        gate_kernel<L, 32><<<grid, kGateThreads, 0, s>>>(g, w, num_sites, t, cell, out_cell);
        break;
    case 64:
        gate_kernel<L, 64><<<grid, kGateThreads, 0, s>>>(g, w, num_sites, t, cell, out_cell);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

bool gate_shape_supported(int pos_freqs, int hidden)
{
    return (pos_freqs == 6 || pos_freqs == 10) && (hidden == 16 || hidden == 32 || hidden == 64);
}

hipError_t launch_gate(const RenderGeometry &g, const float *w, int pos_freqs, int hidden,
                       int num_sites, float *t, uint8_t *cell, int *out_cell, hipStream_t s)
{
    if (g.num_samples == 0)
        return hipSuccess;
    if (pos_freqs == 6)
        return launch_gate_l<6>(g, w, hidden, num_sites, t, cell, out_cell, s);
    if (pos_freqs == 10)
        return launch_gate_l<10>(g, w, hidden, num_sites, t, cell, out_cell, s);
    return hipErrorInvalidValue;
}

}  // namespace derf
