/*
 * DeRF reference oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-file CPU implementation of the inference path of
 * "DeRF: Decomposed Radiance Fields" (Rebain, Jiang, Yazdani, Li, Yi,
 * Tagliasacchi): render rays through a radiance field split into Voronoi
 * cells, each cell owned by its own small NeRF head.
 *
 * Only the test-suite, the smoke check and the benchmark's CPU baseline may
 * load this library.  It shares no code with the GPU library.
 *
 * Precision.  The paper does not fix one, so everything that produces a
 * real-valued result (positional encoding, the head networks, quadrature and
 * compositing) is computed in double.  The values that decide an integer --
 * the sample depths t and positions x, which decide the owning Voronoi cell
 * -- are computed in float32, with explicit fused multiply-adds, because the
 * GPU path takes the same decisions in float32: both sides must reach the
 * same cell for the same sample.
 *
 * Steps (the paper's order):
 *   Sec. 3.1, Eq. 1-2   stratified samples on [near, far], quadrature of the
 *                       volume-rendering integral (midpoint tiling of the
 *                       interval so that the quadrature weights cover it);
 *   Sec. 3.2            one head per point: the decomposition weights are
 *                       one-hot, so only the owning head is evaluated;
 *   Sec. 3.3, Eq. 8     the owning head is the nearest site (the limit of
 *                       the soft Voronoi weights as the temperature grows);
 *   Sec. 3.3 Painter's  each cell's contiguous ray segment is integrated on
 *                       its own, then the segments are composited in order
 *                       along the ray (front to back; "over" is associative,
 *                       so this equals the back-to-front Painter's order).
 *
 * Self-test helpers (not on the method's path): a plain single-network NeRF
 * render, a soft-Voronoi render at finite temperature (Eq. 4-5 with Eq. 8),
 * direct (unsegmented) and back-to-front compositing.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------ RNG --
 * Philox4x32-10 counter-based generator, written from its definition in
 * Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3"
 * (SC 2011): ten rounds of two 32x32->64 multiplies, with a Weyl sequence on
 * the 2-word key between rounds.
 */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_W0;
            k1 += PHILOX_W1;
        }
        uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* Jitter xi in [0, 1) for sample i of ray r.  Counter (i / 4, ray low word,
 * ray high word, stream), key = seed words; word i % 4 of the block; the top
 * 24 bits scaled by 2^-24 (exact in float32).  Stream 0 jitters the coarse
 * strata, stream 1 the inverse-CDF draws of hierarchical sampling. */
float oracle_jitter(uint64_t seed, uint64_t ray, uint32_t i, uint32_t stream)
{
    uint32_t ctr[4] = { i >> 2, (uint32_t)ray, (uint32_t)(ray >> 32), stream };
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    return (float)(out[i & 3u] >> 8) * 0x1.0p-24f;
}

/* ------------------------------------------------------------- sampling --
 * Stratified sampling of [near, far] into n equal strata (Eq. 1 bounds):
 * t_i = near + (i + xi_i) * (far - near) / n, in float32 with one fma.
 * perturb == 0 puts every sample at its stratum midpoint (xi = 1/2). */
void oracle_sample_depths(uint64_t seed, uint64_t ray, float near_t, float far_t, int n,
                          int perturb, float *t)
{
    float step = (far_t - near_t) / (float)n;
    for (int i = 0; i < n; ++i) {
        float xi = perturb ? oracle_jitter(seed, ray, (uint32_t)i, 0u) : 0.5f;
        t[i] = fmaf(step, (float)i + xi, near_t);
    }
}

/* x = o + t d per component, float32, one fma each. */
static void sample_point(const float o[3], const float d[3], float t, float x[3])
{
    x[0] = fmaf(t, d[0], o[0]);
    x[1] = fmaf(t, d[1], o[1]);
    x[2] = fmaf(t, d[2], o[2]);
}

/* ----------------------------------------------------------- assignment --
 * The owning head of x is its nearest Voronoi site (Sec. 3.3: the soft
 * Voronoi weights of Eq. 8 become a partition as the temperature grows).
 * Squared distance in float32: one rounding per coordinate difference, then
 * ((e_x*e_x) + e_y^2) + e_z^2 with fmas.  Exact ties go to the lowest index. */
int oracle_nearest_site(int K, const float *sites, const float x[3])
{
    int best_k = 0;
    float best = INFINITY;
    for (int k = 0; k < K; ++k) {
        float ex = x[0] - sites[3 * k + 0];
        float ey = x[1] - sites[3 * k + 1];
        float ez = x[2] - sites[3 * k + 2];
        float d2 = fmaf(ez, ez, fmaf(ey, ey, ex * ex));
        if (d2 < best) {
            best = d2;
            best_k = k;
        }
    }
    return best_k;
}

/* Distance (double) from x to the boundary of the cell of site a: the cell is
 * the intersection of the half-spaces closer to a than to each b, so the
 * distance is the smallest signed distance to a bisector plane. */
double oracle_bisector_margin(int K, const float *sites, const float x[3], int a)
{
    double m = INFINITY;
    double xa = x[0], ya = x[1], za = x[2];
    for (int b = 0; b < K; ++b) {
        if (b == a)
            continue;
        double pax = sites[3 * a], pay = sites[3 * a + 1], paz = sites[3 * a + 2];
        double pbx = sites[3 * b], pby = sites[3 * b + 1], pbz = sites[3 * b + 2];
        double da = (xa - pax) * (xa - pax) + (ya - pay) * (ya - pay) + (za - paz) * (za - paz);
        double db = (xa - pbx) * (xa - pbx) + (ya - pby) * (ya - pby) + (za - pbz) * (za - pbz);
        double sep = sqrt((pax - pbx) * (pax - pbx) + (pay - pby) * (pay - pby) +
                          (paz - pbz) * (paz - pbz));
        double dist = sep > 0.0 ? (db - da) / (2.0 * sep) : INFINITY;
        if (dist < m)
            m = dist;
    }
    return m;
}

/* ------------------------------------------------------------- encoding --
 * Positional encoding of NeRF, used by every head (Sec. 4.1 keeps NeRF's
 * settings): gamma_L(p) = (p, sin(pi 2^0 p), cos(pi 2^0 p), ...,
 * sin(pi 2^{L-1} p), cos(pi 2^{L-1} p)), where p is a 3-vector and each
 * sin/cos block lists x, y, z.  3 + 6L entries.
 * sin(pi y) is evaluated after the exact reduction r = y - 2 rint(y / 2),
 * so large 2^l p lose no accuracy. */
static double sinpi_d(double y)
{
    double r = y - 2.0 * rint(0.5 * y);
    return sin(M_PI * r);
}

static double cospi_d(double y)
{
    double r = y - 2.0 * rint(0.5 * y);
    return cos(M_PI * r);
}

void oracle_posenc(int L, const double p[3], double *out)
{
    out[0] = p[0];
    out[1] = p[1];
    out[2] = p[2];
    for (int l = 0; l < L; ++l) {
        double s = ldexp(1.0, l);
        for (int c = 0; c < 3; ++c) {
            out[3 + 6 * l + c] = sinpi_d(s * p[c]);
            out[3 + 6 * l + 3 + c] = cospi_d(s * p[c]);
        }
    }
}

/* ---------------------------------------------------------- head network --
 * One head is a NeRF MLP (Sec. 4.1, settings of NeRF): `depth` ReLU layers
 * of `width` units on gamma(x), the skip layer taking [gamma(x); h]; a ReLU
 * density output from h; a colour branch on [h; gamma(d)] (an optional ReLU
 * hidden layer) ending in a sigmoid.
 *
 * Packed weights of one head, float32, in this order: for each hidden layer
 * W [width][in] row-major then b [width]; w_sigma [width], b_sigma [1];
 * then either W_v [rgb_hidden][width + dir_dim], b_v, W_c [3][rgb_hidden],
 * b_c [3], or (rgb_hidden == 0) W_c [3][width + dir_dim], b_c [3]. */
typedef struct {
    int pos_freqs;
    int dir_freqs;
    int depth;
    int width;
    int skip_layer;
    int rgb_hidden;
} oracle_arch;

static int pos_dim(const oracle_arch *a) { return 3 + 6 * a->pos_freqs; }
static int dir_dim(const oracle_arch *a) { return 3 + 6 * a->dir_freqs; }

static int layer_in(const oracle_arch *a, int l)
{
    if (l == 0)
        return pos_dim(a);
    if (l == a->skip_layer)
        return pos_dim(a) + a->width;
    return a->width;
}

long long oracle_weights_count(const oracle_arch *a)
{
    long long n = 0;
    for (int l = 0; l < a->depth; ++l)
        n += (long long)a->width * layer_in(a, l) + a->width;
    n += a->width + 1;
    if (a->rgb_hidden > 0) {
        n += (long long)a->rgb_hidden * (a->width + dir_dim(a)) + a->rgb_hidden;
        n += 3LL * a->rgb_hidden + 3;
    } else {
        n += 3LL * (a->width + dir_dim(a)) + 3;
    }
    return n;
}

/* y[o] = sum_i W[o][i] in[i] + b[o], summed in index order. */
static void dense(const float *W, const float *b, int n_out, int n_in, const double *in, double *y)
{
    for (int o = 0; o < n_out; ++o) {
        double acc = 0.0;
        const float *row = W + (size_t)o * n_in;
        for (int i = 0; i < n_in; ++i)
            acc += (double)row[i] * in[i];
        y[o] = acc + (double)b[o];
    }
}

static double relu(double v) { return v > 0.0 ? v : 0.0; }

/* Evaluate one head at encoded position gx (pos_dim) and encoded direction gd
 * (dir_dim).  scratch must hold 4 * (pos_dim + width + dir_dim + rgb_hidden). */
void oracle_head_eval(const oracle_arch *a, const float *w, const double *gx, const double *gd,
                      double *sigma, double rgb[3], double *scratch)
{
    int W = a->width, P = pos_dim(a), Dd = dir_dim(a);
    double *h = scratch;                 /* width            */
    double *in = h + W;                  /* P + W + Dd       */
    double *g = in + P + W + Dd;         /* rgb_hidden       */
    const float *p = w;
    for (int l = 0; l < a->depth; ++l) {
        int n_in = layer_in(a, l);
        if (l == 0) {
            memcpy(in, gx, sizeof(double) * P);
        } else if (l == a->skip_layer) {
            memcpy(in, gx, sizeof(double) * P);
            memcpy(in + P, h, sizeof(double) * W);
        } else {
            memcpy(in, h, sizeof(double) * W);
        }
        dense(p, p + (size_t)W * n_in, W, n_in, in, h);
        for (int o = 0; o < W; ++o)
            h[o] = relu(h[o]);
        p += (size_t)W * n_in + W;
    }
    double s;
    dense(p, p + W, 1, W, h, &s);
    *sigma = relu(s);
    p += W + 1;
    memcpy(in, h, sizeof(double) * W);
    memcpy(in + W, gd, sizeof(double) * Dd);
    double logit[3];
    if (a->rgb_hidden > 0) {
        int Hc = a->rgb_hidden;
        dense(p, p + (size_t)Hc * (W + Dd), Hc, W + Dd, in, g);
        for (int o = 0; o < Hc; ++o)
            g[o] = relu(g[o]);
        p += (size_t)Hc * (W + Dd) + Hc;
        dense(p, p + 3 * Hc, 3, Hc, g, logit);
    } else {
        dense(p, p + 3 * (W + Dd), 3, W + Dd, in, logit);
    }
    for (int c = 0; c < 3; ++c)
        rgb[c] = 1.0 / (1.0 + exp(-logit[c]));
}

/* --------------------------------------------------------- quadrature -----
 * The integral of Eq. 1 is discretised on intervals that tile [near, far]:
 * boundaries b_0 = near, b_i = (t_{i-1} + t_i) / 2, b_n = far; sample i
 * stands for [b_i, b_{i+1}) of length delta_i.  Per sample the opacity is
 * alpha = 1 - exp(-sigma delta) and the transmittance factor tau = exp(-sigma
 * delta) (Eq. 2 on one interval). */
static void intervals(const float *t, int n, float near_t, float far_t, double *delta)
{
    double prev = near_t;
    for (int i = 0; i < n; ++i) {
        double next = (i + 1 < n) ? 0.5 * ((double)t[i] + (double)t[i + 1]) : (double)far_t;
        delta[i] = next - prev;
        prev = next;
    }
}

/* Per-segment integration and Painter's merge (Sec. 3.3).  A segment is a
 * maximal run of samples with the same cell; by the convexity of Voronoi
 * cells each cell contributes at most one run per ray.  Within a segment the
 * local transmittance starts at 1 and the segment yields (C_s, D_s, T_s); the
 * segments are then composited front to back: C += T C_s, D += T D_s,
 * T *= T_s.  Returns rgb = C, depth = D, opacity = 1 - T.
 * If w_out is given it receives the per-sample compositing weights T_i alpha_i
 * with T_i the transmittance accumulated over all earlier samples. */
static void composite_segments(int n, const int *cell, const float *t, const double *sigma,
                               const double *rgb, const double *delta, double out_rgb[3],
                               double *out_depth, double *out_opacity, double *w_out)
{
    double C[3] = {0.0, 0.0, 0.0}, D = 0.0, T = 1.0;
    int i = 0;
    while (i < n) {
        int j = i;
        double Cs[3] = {0.0, 0.0, 0.0}, Ds = 0.0, Tloc = 1.0;
        while (j < n && cell[j] == cell[i]) {
            double x = sigma[j] * delta[j];
            double alpha = -expm1(-x);
            double tau = exp(-x);
            double w = Tloc * alpha;
            if (w_out)
                w_out[j] = T * w;
            Cs[0] += w * rgb[3 * j + 0];
            Cs[1] += w * rgb[3 * j + 1];
            Cs[2] += w * rgb[3 * j + 2];
            Ds += w * (double)t[j];
            Tloc *= tau;
            ++j;
        }
        C[0] += T * Cs[0];
        C[1] += T * Cs[1];
        C[2] += T * Cs[2];
        D += T * Ds;
        T *= Tloc;
        i = j;
    }
    out_rgb[0] = C[0];
    out_rgb[1] = C[1];
    out_rgb[2] = C[2];
    *out_depth = D;
    *out_opacity = 1.0 - T;
}

/* Direct front-to-back compositing of all samples, ignoring cells.  w_out
 * (optional) receives each sample's rendering weight T_j alpha_j. */
static void composite_direct(int n, const float *t, const double *sigma, const double *rgb,
                             const double *delta, double out_rgb[3], double *out_depth,
                             double *out_opacity, double *w_out)
{
    double C[3] = {0.0, 0.0, 0.0}, D = 0.0, T = 1.0;
    for (int j = 0; j < n; ++j) {
        double x = sigma[j] * delta[j];
        double w = T * -expm1(-x);
        if (w_out)
            w_out[j] = w;
        C[0] += w * rgb[3 * j + 0];
        C[1] += w * rgb[3 * j + 1];
        C[2] += w * rgb[3 * j + 2];
        D += w * (double)t[j];
        T *= exp(-x);
    }
    out_rgb[0] = C[0];
    out_rgb[1] = C[1];
    out_rgb[2] = C[2];
    *out_depth = D;
    *out_opacity = 1.0 - T;
}

/* Back-to-front compositing (the Painter's Algorithm as the paper states it):
 * walking from the far end, C = C_i alpha_i + (1 - alpha_i) C; the depth and
 * the transmittance use the same recurrence. */
static void composite_back_to_front(int n, const float *t, const double *sigma,
                                    const double *rgb, const double *delta, double out_rgb[3],
                                    double *out_depth, double *out_opacity)
{
    double C[3] = {0.0, 0.0, 0.0}, D = 0.0, T = 1.0;
    for (int j = n - 1; j >= 0; --j) {
        double x = sigma[j] * delta[j];
        double alpha = -expm1(-x);
        double tau = exp(-x);
        C[0] = alpha * rgb[3 * j + 0] + tau * C[0];
        C[1] = alpha * rgb[3 * j + 1] + tau * C[1];
        C[2] = alpha * rgb[3 * j + 2] + tau * C[2];
        D = alpha * (double)t[j] + tau * D;
        T = tau * T;
    }
    out_rgb[0] = C[0];
    out_rgb[1] = C[1];
    out_rgb[2] = C[2];
    *out_depth = D;
    *out_opacity = 1.0 - T;
}

/* ------------------------------------------------- hierarchical sampling --
 * NeRF's coarse-to-fine sampling (the paper keeps NeRF's settings): the
 * coarse compositing weights w_i define a piecewise-constant density over
 * the coarse intervals [b_i, b_{i+1}), with a floor of 1e-5 per interval;
 * n_fine draws u_j = (j + xi_j) / n_fine (stream 1) are mapped through its
 * inverse CDF.  The fine depths are rounded to float32 (they decide cells)
 * and merged with the coarse ones in sorted order (coarse first on ties). */
static void fine_depths(uint64_t seed, uint64_t ray, int perturb, int nc, int nf, const float *tc,
                        float near_t, float far_t, const double *w, double *cdf, float *tf)
{
    double total = 0.0;
    cdf[0] = 0.0;
    for (int i = 0; i < nc; ++i) {
        total += w[i] + 1e-5;
        cdf[i + 1] = total;
    }
    for (int i = 0; i <= nc; ++i)
        cdf[i] /= total;
    cdf[nc] = 1.0;
    for (int j = 0; j < nf; ++j) {
        double xi = perturb ? (double)oracle_jitter(seed, ray, (uint32_t)j, 1u) : 0.5;
        double u = ((double)j + xi) / (double)nf;
        /* largest i with cdf[i] <= u, i in [0, nc-1] */
        int i = 0;
        while (i + 1 < nc && cdf[i + 1] <= u)
            ++i;
        double b0 = (i == 0) ? (double)near_t : 0.5 * ((double)tc[i - 1] + (double)tc[i]);
        double b1 = (i + 1 == nc) ? (double)far_t : 0.5 * ((double)tc[i] + (double)tc[i + 1]);
        double span = cdf[i + 1] - cdf[i];
        double frac = span > 0.0 ? (u - cdf[i]) / span : 0.0;
        if (frac < 0.0)
            frac = 0.0;
        if (frac > 1.0)
            frac = 1.0;
        tf[j] = (float)(b0 + frac * (b1 - b0));
    }
}

static void merge_sorted(const float *a, int na, const float *b, int nb, float *out)
{
    int i = 0, j = 0, k = 0;
    while (i < na || j < nb) {
        if (j >= nb || (i < na && a[i] <= b[j]))
            out[k++] = a[i++];
        else
            out[k++] = b[j++];
    }
}

/* ------------------------------------------------------------ MLP gating --
 * The alternative decomposition of Sec. 4 ("decompositions with MLPs"): a
 * small network with a softmax output gives every point its head weights,
 * and at inference a point belongs to the head of largest weight.  The
 * softmax is monotone, so that head is the first largest logit.  The paper
 * fixes neither the network's size nor its input; the reading here is one
 * ReLU hidden layer of H units on the heads' positional encoding
 * gamma_L(x):
 *   h = max(0, W1 gamma_L(x) + b1),  z = W2 h + b2   (K logits)
 * Packed float32 weights: W1 [H][3 + 6L] row-major, b1 [H], W2 [K][H], b2 [K].
 * The decision is an integer, so both sides take it in the precision of the
 * kernel, which runs the two products on bf16 matrix cores: every float32
 * operand a is carried as two bfloat16 values, a_hi = bf16(a) and
 * a_lo = bf16(a - a_hi) (round to nearest even each), and every product a b
 * of a weight and an activation as a_hi b_hi + a_hi b_lo + a_lo b_hi (each
 * exact; the dropped a_lo b_lo and the rounding of a_lo are below
 * 2^-18 |a b| each).  The encoding is rounded to float32 first, each dot
 * product is the bias plus those terms (summed here in double), and the
 * hidden layer is rounded to float32 after the ReLU, as the kernel's float32
 * accumulators hold it.  The split keeps about 16 significant bits per
 * operand, so these logits stay within about 1e-5 relative of the plain
 * float32 network. */
long long oracle_gate_weights_count(int K, int L, int H)
{
    if (K < 1 || L < 0 || H < 1)
        return -1;
    return (long long)H * (3 + 6 * L) + H + (long long)K * H + K;
}

/* v rounded to bfloat16 (8 significant bits), nearest even; v finite. */
static float bf16_rne(float v)
{
    uint32_t u;
    memcpy(&u, &v, sizeof(u));
    u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
    float r;
    memcpy(&r, &u, sizeof(r));
    return r;
}

/* a b in the gate's arithmetic: a = a_hi + a_lo, b = b_hi + b_lo as two
 * bfloat16 values each (a - a_hi is exact in float32), and the three
 * products that keep 16 significant bits of each operand. */
static double gate_mul(float a, float b)
{
    const float ah = bf16_rne(a), al = bf16_rne(a - ah);
    const float bh = bf16_rne(b), bl = bf16_rne(b - bh);
    return (double)ah * bh + (double)ah * bl + (double)al * bh;
}

/* Logits z [K] of the gating network at x; f (3 + 6L floats) and h (H) are
 * scratch. */
static void gate_logits(int K, int L, int H, const float *w, const float x[3], float *f, float *h,
                        double *z)
{
    const int P = 3 + 6 * L;
    double g[3 + 6 * 32];
    const double xd[3] = { x[0], x[1], x[2] };
    oracle_posenc(L, xd, g);
    for (int c = 0; c < P; ++c)
        f[c] = (float)g[c];
    const float *W1 = w, *b1 = W1 + (size_t)H * P, *W2 = b1 + H, *b2 = W2 + (size_t)K * H;
    for (int j = 0; j < H; ++j) {
        double acc = b1[j];
        for (int c = 0; c < P; ++c)
            acc += gate_mul(W1[(size_t)j * P + c], f[c]);
        const float v = (float)acc;
        h[j] = v > 0.0f ? v : 0.0f;
    }
    for (int k = 0; k < K; ++k) {
        double acc = b2[k];
        for (int j = 0; j < H; ++j)
            acc += gate_mul(W2[(size_t)k * H + j], h[j]);
        z[k] = acc;
    }
}

/* The gated head (first largest logit) and, in *gap, the difference between
 * the two largest logits (infinite for one head): how near the decision is
 * to a tie. */
static int gate_argmax(int K, const double *z, double *gap)
{
    int best = 0;
    for (int k = 1; k < K; ++k)
        if (z[k] > z[best])
            best = k;
    if (gap) {
        double second = -INFINITY;
        for (int k = 0; k < K; ++k)
            if (k != best && z[k] > second)
                second = z[k];
        *gap = K > 1 ? z[best] - second : INFINITY;
    }
    return best;
}

/* Logits [M][K] of the gating network at the points x [M][3]; -1 for bad
 * sizes. */
int oracle_gate_logits(int K, int L, int H, const float *w, long long M, const float *x,
                       double *z)
{
    if (K < 1 || L < 0 || L > 32 || H < 1 || M < 0)
        return -1;
    float *f = malloc(sizeof(float) * (size_t)(3 + 6 * L));
    float *h = malloc(sizeof(float) * (size_t)H);
    if (!f || !h) {
        free(f);
        free(h);
        return -3;
    }
    for (long long m = 0; m < M; ++m)
        gate_logits(K, L, H, w, x + 3 * m, f, h, z + (size_t)m * K);
    free(f);
    free(h);
    return 0;
}

/* x = o + t d per sample (float32, one fma per component) for depths t [M]
 * of the rays o, d [M][3]. */
void oracle_sample_points(long long M, const float *o, const float *d, const float *t, float *x)
{
    for (long long m = 0; m < M; ++m)
        sample_point(o + 3 * m, d + 3 * m, t[m], x + 3 * m);
}

/* ----------------------------------------------------------- rendering --- */

typedef struct {
    int K;
    const float *sites;
    const oracle_arch *arch;
    const float *weights; /* K x weights_count, head-major */
    float near_t, far_t;
    int n_coarse, n_fine;
    uint64_t seed;
    int perturb;
    double *contrib; /* soft mode, optional: per-ray head contributions [R][K] (Eq. 6) */
    const unsigned char *empty; /* optional [K]: nonzero = 0-capacity head (no density) */
    /* optional per-head architectures (heads of different capacities): */
    const oracle_arch *archs;   /* [K], or NULL: every head is *arch */
    const long long *woff;      /* [K] offset of head k's weights */
    size_t mix_scratch;         /* doubles of scratch one head evaluation uses */
    int mix_pos, mix_dir;       /* largest encoding lengths over the heads */
    /* optional gating network (MODE_GATED): packed weights, L and H */
    const float *gate_w;
    int gate_L, gate_H;
} render_args;

/* Head k at x (view direction dh): its density and colour, or zero for a
 * 0-capacity head (the empty-space head of Sec. 5).  gx, gd: the encodings
 * of x and dh for the shared architecture; with per-head architectures each
 * head encodes with its own frequencies. */
static void eval_head(const render_args *A, int k, const double xd[3], const double dh[3],
                      const double *gx, const double *gd, double *sigma, double rgb[3],
                      double *scratch)
{
    if (A->empty && A->empty[k]) {
        *sigma = 0.0;
        rgb[0] = rgb[1] = rgb[2] = 0.0;
        return;
    }
    if (A->archs) {
        const oracle_arch *a = &A->archs[k];
        double *gxk = scratch + A->mix_scratch, *gdk = gxk + A->mix_pos;
        oracle_posenc(a->pos_freqs, xd, gxk);
        oracle_posenc(a->dir_freqs, dh, gdk);
        oracle_head_eval(a, A->weights + A->woff[k], gxk, gdk, sigma, rgb, scratch);
        return;
    }
    oracle_head_eval(A->arch, A->weights + (size_t)k * oracle_weights_count(A->arch), gx, gd,
                     sigma, rgb, scratch);
}

enum { MODE_DERF = 0, MODE_PLAIN = 1, MODE_SOFT = 2, MODE_DIRECT = 3, MODE_BACK = 4, MODE_GATED = 5 };

/* Evaluate the field at every sample of one ray: cell, sigma, rgb. */
static void eval_samples(const render_args *A, int mode, double beta, const float o[3],
                         const float d[3], const double dh[3], const double *gd, int n,
                         const float *t, int *cell, double *sigma, double *rgb, double *gx,
                         double *scratch, double *soft_w)
{
    const oracle_arch *a = A->arch;
    for (int i = 0; i < n; ++i) {
        float x[3];
        sample_point(o, d, t[i], x);
        double xd[3] = { x[0], x[1], x[2] };
        oracle_posenc(a->pos_freqs, xd, gx);
        if (mode == MODE_PLAIN) {
            cell[i] = 0;
            eval_head(A, 0, xd, dh, gx, gd, &sigma[i], &rgb[3 * i], scratch);
        } else if (mode == MODE_SOFT) {
            /* Eq. 4-5 with the soft Voronoi weights of Eq. 8 */
            double dist_min = INFINITY;
            for (int k = 0; k < A->K; ++k) {
                double ex = xd[0] - A->sites[3 * k], ey = xd[1] - A->sites[3 * k + 1],
                       ez = xd[2] - A->sites[3 * k + 2];
                double dk = sqrt(ex * ex + ey * ey + ez * ez);
                if (dk < dist_min)
                    dist_min = dk;
            }
            double z = 0.0, s = 0.0, c[3] = {0.0, 0.0, 0.0};
            for (int k = 0; k < A->K; ++k) {
                double ex = xd[0] - A->sites[3 * k], ey = xd[1] - A->sites[3 * k + 1],
                       ez = xd[2] - A->sites[3 * k + 2];
                double dk = sqrt(ex * ex + ey * ey + ez * ez);
                double wk = exp(-beta * (dk - dist_min));
                z += wk;
                if (wk == 0.0)
                    continue;
                double sk, ck[3];
                eval_head(A, k, xd, dh, gx, gd, &sk, ck, scratch);
                s += wk * sk;
                c[0] += wk * ck[0];
                c[1] += wk * ck[1];
                c[2] += wk * ck[2];
            }
            sigma[i] = s / z;
            rgb[3 * i + 0] = c[0] / z;
            rgb[3 * i + 1] = c[1] / z;
            rgb[3 * i + 2] = c[2] / z;
            cell[i] = 0;
            if (soft_w) {
                /* the normalised weights of Eq. 8 at this sample */
                for (int k = 0; k < A->K; ++k) {
                    double ex = xd[0] - A->sites[3 * k], ey = xd[1] - A->sites[3 * k + 1],
                           ez = xd[2] - A->sites[3 * k + 2];
                    soft_w[(size_t)i * A->K + k] =
                        exp(-beta * (sqrt(ex * ex + ey * ey + ez * ez) - dist_min)) / z;
                }
            }
        } else if (mode == MODE_GATED) {
            float f[3 + 6 * 32], h[256];
            double z[256];
            gate_logits(A->K, A->gate_L, A->gate_H, A->gate_w, x, f, h, z);
            cell[i] = gate_argmax(A->K, z, NULL);
            eval_head(A, cell[i], xd, dh, gx, gd, &sigma[i], &rgb[3 * i], scratch);
        } else {
            cell[i] = oracle_nearest_site(A->K, A->sites, x);
            eval_head(A, cell[i], xd, dh, gx, gd, &sigma[i], &rgb[3 * i], scratch);
        }
    }
}

static void finish(int mode, int n, const int *cell, const float *t, const double *sigma,
                   const double *rgb, const double *delta, double *o_rgb, double *o_depth,
                   double *o_opac, double *w_out)
{
    if (mode == MODE_DERF || mode == MODE_GATED)
        composite_segments(n, cell, t, sigma, rgb, delta, o_rgb, o_depth, o_opac, w_out);
    else if (mode == MODE_BACK)
        composite_back_to_front(n, t, sigma, rgb, delta, o_rgb, o_depth, o_opac);
    else
        composite_direct(n, t, sigma, rgb, delta, o_rgb, o_depth, o_opac, w_out);
}

/* Render rays [0, R).  Outputs are double; the optional per-sample arrays
 * (any may be NULL) hold the final sample list of every ray (N = n_coarse +
 * n_fine entries): depth t, owning cell, sigma, rgb (3 per sample) and the
 * distance of the sample to its cell boundary.  ray_ids (optional) gives the
 * global ray index of each row, used as the RNG counter. */
static int render_impl(const render_args *A, int mode, double beta, long long R,
                       const float *rays_o, const float *rays_d, const long long *ray_ids,
                       double *out_rgb, double *out_depth, double *out_opacity, float *dbg_t,
                       int *dbg_cell, double *dbg_sigma, double *dbg_rgb, double *dbg_margin,
                       int nthreads)
{
    const oracle_arch *a = A->arch;
    int nc = A->n_coarse, nf = A->n_fine, N = nc + nf;
    if (nc < 1 || nf < 0 || (nf > 0 && nc < 2) || R < 0)
        return -1;
    int P = 3 + 6 * a->pos_freqs, Dd = 3 + 6 * a->dir_freqs;
    size_t scratch_len = 4 * (size_t)(P + a->width + Dd + a->rgb_hidden + 8);
    if (A->archs) {
        /* per-head encodings go after the head evaluation's own scratch */
        P = A->mix_pos;
        Dd = A->mix_dir;
        scratch_len = A->mix_scratch + (size_t)P + (size_t)Dd;
    }
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int failed = 0;
#pragma omp parallel
    {
        float *tc = malloc(sizeof(float) * (size_t)N);
        float *tf = malloc(sizeof(float) * (size_t)N);
        float *tm = malloc(sizeof(float) * (size_t)N);
        int *cell = malloc(sizeof(int) * (size_t)N);
        double *sigma = malloc(sizeof(double) * (size_t)N);
        double *rgb = malloc(sizeof(double) * 3 * (size_t)N);
        double *delta = malloc(sizeof(double) * (size_t)N);
        double *w = malloc(sizeof(double) * (size_t)N);
        double *cdf = malloc(sizeof(double) * (size_t)(N + 1));
        double *gx = malloc(sizeof(double) * (size_t)P);
        double *gd = malloc(sizeof(double) * (size_t)Dd);
        double *scratch = malloc(sizeof(double) * scratch_len);
        const int want_w = mode == MODE_SOFT && A->contrib;
        double *soft_w = want_w ? malloc(sizeof(double) * (size_t)N * A->K) : NULL;
        if (!tc || !tf || !tm || !cell || !sigma || !rgb || !delta || !w || !cdf || !gx || !gd ||
            !scratch || (want_w && !soft_w)) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (long long r = 0; r < R; ++r) {
                const float *o = rays_o + 3 * r, *d = rays_d + 3 * r;
                uint64_t rid = ray_ids ? (uint64_t)ray_ids[r] : (uint64_t)r;
                /* encoded unit view direction, Sec. 3.1: c depends on d */
                double dn = sqrt((double)d[0] * d[0] + (double)d[1] * d[1] + (double)d[2] * d[2]);
                double dh[3] = { d[0] / dn, d[1] / dn, d[2] / dn };
                oracle_posenc(a->dir_freqs, dh, gd);

                oracle_sample_depths(A->seed, rid, A->near_t, A->far_t, nc, A->perturb, tc);
                const float *tt = tc;
                int n = nc;
                eval_samples(A, mode, beta, o, d, dh, gd, nc, tc, cell, sigma, rgb, gx, scratch, soft_w);
                intervals(tc, nc, A->near_t, A->far_t, delta);
                double c3[3], dep, op;
                finish(mode, nc, cell, tc, sigma, rgb, delta, c3, &dep, &op, w);
                if (soft_w) {
                    /* Eq. 6 with the quadrature of the render: head k's share of
                     * each sample's rendering weight T_i alpha_i */
                    for (int k = 0; k < A->K; ++k) {
                        double acc = 0.0;
                        for (int i = 0; i < nc; ++i)
                            acc += w[i] * soft_w[(size_t)i * A->K + k];
                        A->contrib[(size_t)r * A->K + k] = acc;
                    }
                }
                if (nf > 0) {
                    if (mode != MODE_DERF)
                        composite_segments(nc, cell, tc, sigma, rgb, delta, c3, &dep, &op, w);
                    fine_depths(A->seed, rid, A->perturb, nc, nf, tc, A->near_t, A->far_t, w, cdf,
                                tf);
                    merge_sorted(tc, nc, tf, nf, tm);
                    tt = tm;
                    n = N;
                    eval_samples(A, mode, beta, o, d, dh, gd, N, tm, cell, sigma, rgb, gx, scratch, NULL);
                    intervals(tm, N, A->near_t, A->far_t, delta);
                    finish(mode, N, cell, tm, sigma, rgb, delta, c3, &dep, &op, NULL);
                }
                out_rgb[3 * r + 0] = c3[0];
                out_rgb[3 * r + 1] = c3[1];
                out_rgb[3 * r + 2] = c3[2];
                out_depth[r] = dep;
                out_opacity[r] = op;
                for (int i = 0; i < n; ++i) {
                    size_t s = (size_t)r * N + i;
                    if (dbg_t)
                        dbg_t[s] = tt[i];
                    if (dbg_cell)
                        dbg_cell[s] = cell[i];
                    if (dbg_sigma)
                        dbg_sigma[s] = sigma[i];
                    if (dbg_rgb) {
                        dbg_rgb[3 * s + 0] = rgb[3 * i + 0];
                        dbg_rgb[3 * s + 1] = rgb[3 * i + 1];
                        dbg_rgb[3 * s + 2] = rgb[3 * i + 2];
                    }
                    if (dbg_margin) {
                        float x[3];
                        sample_point(o, d, tt[i], x);
                        if (mode == MODE_GATED) {
                            /* the gap between the two largest logits */
                            float f[3 + 6 * 32], h[256];
                            double z[256];
                            gate_logits(A->K, A->gate_L, A->gate_H, A->gate_w, x, f, h, z);
                            (void)gate_argmax(A->K, z, &dbg_margin[s]);
                        } else {
                            dbg_margin[s] = (mode == MODE_PLAIN || mode == MODE_SOFT || A->K == 1)
                                                ? INFINITY
                                                : oracle_bisector_margin(A->K, A->sites, x,
                                                                         cell[i]);
                        }
                    }
                }
            }
        }
        free(tc); free(tf); free(tm); free(cell); free(sigma); free(rgb); free(delta);
        free(w); free(cdf); free(gx); free(gd); free(scratch); free(soft_w);
    }
    return failed ? -3 : 0;
}

#define ORACLE_RENDER_ARGS                                                                    \
    int K, const float *sites, const oracle_arch *arch, const float *weights, long long R,     \
        const float *rays_o, const float *rays_d, const long long *ray_ids, float near_t,      \
        float far_t, int n_coarse, int n_fine, uint64_t seed, int perturb, double *out_rgb,    \
        double *out_depth, double *out_opacity, float *dbg_t, int *dbg_cell, double *dbg_sigma, \
        double *dbg_rgb, double *dbg_margin, int nthreads

#define ORACLE_FILL_ARGS                                                                       \
    render_args A = { K, sites, arch, weights, near_t, far_t, n_coarse, n_fine, seed, perturb, \
                      NULL, NULL, NULL, NULL, 0, 0, 0 };

/* DeRF render: nearest-site heads, per-segment integration, Painter's merge. */
int oracle_render(ORACLE_RENDER_ARGS)
{
    ORACLE_FILL_ARGS
    return render_impl(&A, MODE_DERF, 0.0, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* Same heads, direct front-to-back compositing over all samples (no segments). */
int oracle_render_direct(ORACLE_RENDER_ARGS)
{
    ORACLE_FILL_ARGS
    return render_impl(&A, MODE_DIRECT, 0.0, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* Same heads, back-to-front compositing (Painter's order as the paper states it). */
int oracle_render_back_to_front(ORACLE_RENDER_ARGS)
{
    ORACLE_FILL_ARGS
    return render_impl(&A, MODE_BACK, 0.0, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* Plain NeRF: head 0 everywhere, direct compositing, no decomposition. */
int oracle_render_plain(ORACLE_RENDER_ARGS)
{
    ORACLE_FILL_ARGS
    return render_impl(&A, MODE_PLAIN, 0.0, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* Soft Voronoi at temperature beta: every head evaluated, blended by Eq. 8. */
int oracle_render_soft(ORACLE_RENDER_ARGS, double beta)
{
    ORACLE_FILL_ARGS
    return render_impl(&A, MODE_SOFT, beta, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* Any render mode (0 derf, 1 plain, 2 soft at beta, 3 direct, 4
 * back-to-front) with optional 0-capacity heads (empty, [K], nonzero = the
 * head has no density anywhere) and, in soft mode without fine samples,
 * optional per-ray head contributions [R][K]. */
int oracle_render_ex(ORACLE_RENDER_ARGS, int mode, double beta, const unsigned char *empty,
                     double *contrib)
{
    ORACLE_FILL_ARGS
    if (mode < MODE_DERF || mode > MODE_BACK || (contrib && (mode != MODE_SOFT || n_fine != 0)))
        return -1;
    A.contrib = contrib;
    A.empty = empty;
    return render_impl(&A, mode, beta, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* As oracle_render_ex with one architecture per head: arch points to K
 * architectures and weights holds the heads' packed weights one after
 * another (head k's oracle_weights_count(&arch[k]) floats).  Heads of
 * different capacities in one model (Sec. 5). */
int oracle_render_mixed(ORACLE_RENDER_ARGS, int mode, double beta, const unsigned char *empty,
                        double *contrib)
{
    ORACLE_FILL_ARGS
    if (K < 1 || mode < MODE_DERF || mode > MODE_BACK ||
        (contrib && (mode != MODE_SOFT || n_fine != 0)))
        return -1;
    long long *woff = malloc(sizeof(long long) * (size_t)K);
    if (!woff)
        return -3;
    long long off = 0;
    size_t need = 0;
    int mp = 0, md = 0;
    for (int k = 0; k < K; ++k) {
        const oracle_arch *a = &arch[k];
        woff[k] = off;
        off += oracle_weights_count(a);
        const size_t sl = 4 * (size_t)(pos_dim(a) + a->width + dir_dim(a) + a->rgb_hidden + 8);
        need = sl > need ? sl : need;
        mp = pos_dim(a) > mp ? pos_dim(a) : mp;
        md = dir_dim(a) > md ? dir_dim(a) : md;
    }
    A.contrib = contrib;
    A.empty = empty;
    A.archs = arch;
    A.woff = woff;
    A.mix_scratch = need;
    A.mix_pos = mp;
    A.mix_dir = md;
    const int rc = render_impl(&A, mode, beta, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                               out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin,
                               nthreads);
    free(woff);
    return rc;
}

/* Soft Voronoi render (as oracle_render_soft, single pass) that also returns
 * each ray's head contributions W(r) [R][K] of Sec. 3.2 Eq. 6: the integral
 * of T sigma w_k along the ray, with the render's quadrature, so that
 * sum_k W_k(r) equals the ray's opacity. */
int oracle_render_soft_contrib(ORACLE_RENDER_ARGS, double beta, double *contrib)
{
    ORACLE_FILL_ARGS
    if (n_fine != 0 || !contrib)
        return -1;
    A.contrib = contrib;
    return render_impl(&A, MODE_SOFT, beta, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* DeRF render with the gated assignment (Sec. 4, decompositions with MLPs):
 * each sample's head is the gating network's first largest logit instead of
 * the nearest site.  A gated cell need not be convex, so a ray may enter it
 * more than once; its runs are integrated and merged front to back like
 * segments, which is exact for any partition ("over" is associative).
 * dbg_margin (optional) receives the gap between each sample's two largest
 * logits instead of a bisector distance.  Single pass (n_fine = 0), one
 * architecture; at most 256 heads, 256 hidden units and 32 frequencies. */
int oracle_render_gated(ORACLE_RENDER_ARGS, int gate_L, int gate_H, const float *gate_w)
{
    ORACLE_FILL_ARGS
    if (n_fine != 0 || !gate_w || K < 1 || K > 256 || gate_L < 0 || gate_L > 32 || gate_H < 1 ||
        gate_H > 256)
        return -1;
    A.gate_w = gate_w;
    A.gate_L = gate_L;
    A.gate_H = gate_H;
    return render_impl(&A, MODE_GATED, 0.0, R, rays_o, rays_d, ray_ids, out_rgb, out_depth,
                       out_opacity, dbg_t, dbg_cell, dbg_sigma, dbg_rgb, dbg_margin, nthreads);
}

/* ------------------------------------------- Painter's-order culling ---
 * The Painter's order of Sec. 3.3 visits the segments of a ray front to
 * back, so the transmittance in front of a segment is known before its head
 * has to run.  With piece > 0 each segment is cut, from its first sample, into
 * pieces of at most `piece` samples (piece = 0: whole segments).  Level l of a
 * ray holds its piece of ordinal l along the ray (the last level also every
 * later piece).  Before level l > 0 a ray
 * whose transmittance T is below eps stops: its remaining segments are not
 * evaluated.  The result is the Painter's merge of the evaluated segments
 * (a prefix of the ray).  Its colour and opacity differ from the full
 * render's by at most the T at the stop (< eps: colours lie in [0, 1]) and
 * its depth by at most T * far.  With levels = 1 or eps = 0 nothing is
 * skipped and the result is the full render's, operation for operation.
 * Single pass (n_fine = 0), one architecture for every head; empty
 * (optional [K]) marks 0-capacity heads.  evaluated (optional [R]):
 * samples whose head ran, per ray. */
int oracle_render_culled(ORACLE_RENDER_ARGS, double eps, int levels, int piece,
                         const unsigned char *empty, int *evaluated)
{
    ORACLE_FILL_ARGS
    A.empty = empty;
    (void)dbg_t; (void)dbg_cell; (void)dbg_sigma; (void)dbg_rgb; (void)dbg_margin;
    const int n = n_coarse;
    if (n < 1 || n_fine != 0 || levels < 1 || piece < 0 || !(eps >= 0.0) || R < 0)
        return -1;
    const int P = 3 + 6 * arch->pos_freqs, Dd = 3 + 6 * arch->dir_freqs;
    const size_t scratch_len = 4 * (size_t)(P + arch->width + Dd + arch->rgb_hidden + 8);
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int failed = 0;
#pragma omp parallel
    {
        float *t = malloc(sizeof(float) * (size_t)n);
        int *cell = malloc(sizeof(int) * (size_t)n);
        double *sigma = malloc(sizeof(double) * (size_t)n);
        double *rgb = malloc(sizeof(double) * 3 * (size_t)n);
        double *delta = malloc(sizeof(double) * (size_t)n);
        double *gx = malloc(sizeof(double) * (size_t)P);
        double *gd = malloc(sizeof(double) * (size_t)Dd);
        double *scratch = malloc(sizeof(double) * scratch_len);
        if (!t || !cell || !sigma || !rgb || !delta || !gx || !gd || !scratch) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (long long r = 0; r < R; ++r) {
                const float *o = rays_o + 3 * r, *d = rays_d + 3 * r;
                const uint64_t rid = ray_ids ? (uint64_t)ray_ids[r] : (uint64_t)r;
                double dn = sqrt((double)d[0] * d[0] + (double)d[1] * d[1] + (double)d[2] * d[2]);
                double dh[3] = { d[0] / dn, d[1] / dn, d[2] / dn };
                oracle_posenc(arch->dir_freqs, dh, gd);
                oracle_sample_depths(seed, rid, near_t, far_t, n, perturb, t);
                intervals(t, n, near_t, far_t, delta);
                for (int i = 0; i < n; ++i) {
                    float x[3];
                    sample_point(o, d, t[i], x);
                    cell[i] = oracle_nearest_site(K, sites, x);
                }
                double c3[3] = {0.0, 0.0, 0.0}, dep = 0.0, op = 0.0;
                int end = 0;
                for (int level = 0; end < n; ++level) {
                    /* transmittance in front of this level */
                    if (level > 0 && 1.0 - op < eps)
                        break;
                    /* this level's samples: one piece, or all that remain */
                    int stop = end;
                    do {
                        const int first = stop, c = cell[stop];
                        while (stop < n && cell[stop] == c && (piece == 0 || stop - first < piece))
                            ++stop;
                    } while (level == levels - 1 && stop < n);
                    for (int i = end; i < stop; ++i) {
                        float x[3];
                        sample_point(o, d, t[i], x);
                        double xd[3] = { x[0], x[1], x[2] };
                        oracle_posenc(arch->pos_freqs, xd, gx);
                        eval_head(&A, cell[i], xd, dh, gx, gd, &sigma[i], &rgb[3 * i], scratch);
                    }
                    end = stop;
                    /* Painter's merge of the evaluated prefix */
                    composite_segments(end, cell, t, sigma, rgb, delta, c3, &dep, &op, NULL);
                }
                out_rgb[3 * r + 0] = c3[0];
                out_rgb[3 * r + 1] = c3[1];
                out_rgb[3 * r + 2] = c3[2];
                out_depth[r] = dep;
                out_opacity[r] = op;
                if (evaluated)
                    evaluated[r] = end;
            }
        }
        free(t); free(cell); free(sigma); free(rgb); free(delta); free(gx); free(gd);
        free(scratch);
    }
    return failed ? -3 : 0;
}

/* Sample depths and owning cells of every sample of rays [0, R) (no network):
 * the full-frame check of the assignment.  Ray r uses RNG ray index
 * ray_offset + r.  margin (optional) receives each sample's distance to its
 * cell boundary. */
int oracle_sample_assign(int K, const float *sites, long long R, const float *rays_o,
                         const float *rays_d, uint64_t ray_offset, float near_t, float far_t, int n,
                         uint64_t seed, int perturb, float *t_out, int *cell_out,
                         double *margin_out, int nthreads)
{
    if (n < 1 || R < 0 || K < 1)
        return -1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel for schedule(static)
    for (long long r = 0; r < R; ++r) {
        float *t = t_out + (size_t)r * n;
        oracle_sample_depths(seed, ray_offset + (uint64_t)r, near_t, far_t, n, perturb, t);
        for (int i = 0; i < n; ++i) {
            float x[3];
            sample_point(rays_o + 3 * r, rays_d + 3 * r, t[i], x);
            int c = oracle_nearest_site(K, sites, x);
            cell_out[(size_t)r * n + i] = c;
            if (margin_out)
                margin_out[(size_t)r * n + i] =
                    K > 1 ? oracle_bisector_margin(K, sites, x, c) : INFINITY;
        }
    }
    return 0;
}

/* DeRF render of rays [0, R) at given sample depths t [R][n] (sorted per
 * ray, inside [near, far]): each sample's nearest-site head (Sec. 3.2-3.3),
 * midpoint quadrature on [near, far] and the per-segment integration with
 * the Painter's merge (Sec. 3.3) -- the steps that follow sampling, applied
 * to depths that come from elsewhere (e.g. the fine depths of hierarchical
 * sampling).  Per-sample outputs are optional (NULL). */
int oracle_render_depths(int K, const float *sites, const oracle_arch *arch, const float *weights,
                         long long R, const float *rays_o, const float *rays_d, float near_t,
                         float far_t, int n, const float *t, double *out_rgb, double *out_depth,
                         double *out_opacity, int *dbg_cell, double *dbg_sigma, double *dbg_rgb,
                         int nthreads)
{
    if (n < 1 || R < 0 || K < 1)
        return -1;
    render_args A = { K, sites, arch, weights, near_t, far_t, n, 0, 0, 0 };
    int P = 3 + 6 * arch->pos_freqs, Dd = 3 + 6 * arch->dir_freqs;
    size_t scratch_len = 4 * (size_t)(P + arch->width + Dd + arch->rgb_hidden + 8);
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
    int failed = 0;
#pragma omp parallel
    {
        int *cell = malloc(sizeof(int) * (size_t)n);
        double *sigma = malloc(sizeof(double) * (size_t)n);
        double *rgb = malloc(sizeof(double) * 3 * (size_t)n);
        double *delta = malloc(sizeof(double) * (size_t)n);
        double *gx = malloc(sizeof(double) * (size_t)P);
        double *gd = malloc(sizeof(double) * (size_t)Dd);
        double *scratch = malloc(sizeof(double) * scratch_len);
        if (!cell || !sigma || !rgb || !delta || !gx || !gd || !scratch) {
#pragma omp atomic write
            failed = 1;
        } else {
#pragma omp for schedule(dynamic, 16)
            for (long long r = 0; r < R; ++r) {
                const float *o = rays_o + 3 * r, *d = rays_d + 3 * r;
                const float *tr = t + (size_t)r * n;
                double dn = sqrt((double)d[0] * d[0] + (double)d[1] * d[1] + (double)d[2] * d[2]);
                double dh[3] = { d[0] / dn, d[1] / dn, d[2] / dn };
                oracle_posenc(arch->dir_freqs, dh, gd);
                eval_samples(&A, MODE_DERF, 0.0, o, d, dh, gd, n, tr, cell, sigma, rgb, gx, scratch, NULL);
                intervals(tr, n, near_t, far_t, delta);
                composite_segments(n, cell, tr, sigma, rgb, delta, out_rgb + 3 * r, out_depth + r,
                                   out_opacity + r, NULL);
                for (int i = 0; i < n; ++i) {
                    size_t s = (size_t)r * n + i;
                    if (dbg_cell)
                        dbg_cell[s] = cell[i];
                    if (dbg_sigma)
                        dbg_sigma[s] = sigma[i];
                    if (dbg_rgb) {
                        dbg_rgb[3 * s + 0] = rgb[3 * i + 0];
                        dbg_rgb[3 * s + 1] = rgb[3 * i + 1];
                        dbg_rgb[3 * s + 2] = rgb[3 * i + 2];
                    }
                }
            }
        }
        free(cell); free(sigma); free(rgb); free(delta); free(gx); free(gd); free(scratch);
    }
    return failed ? -3 : 0;
}

/* Owning cells of given sample depths t [R][n] (Sec. 3.3 nearest site, at
 * x = o + t d in float32 with one fma per component): the check of the
 * assignment of samples whose depths come from elsewhere, such as the
 * inverse-CDF draws of hierarchical sampling.  margin as above. */
int oracle_assign_depths(int K, const float *sites, long long R, const float *rays_o,
                         const float *rays_d, int n, const float *t, int *cell_out,
                         double *margin_out, int nthreads)
{
    if (n < 1 || R < 0 || K < 1)
        return -1;
#ifdef _OPENMP
    if (nthreads > 0)
        omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
#pragma omp parallel for schedule(static)
    for (long long r = 0; r < R; ++r) {
        for (int i = 0; i < n; ++i) {
            float x[3];
            sample_point(rays_o + 3 * r, rays_d + 3 * r, t[(size_t)r * n + i], x);
            int c = oracle_nearest_site(K, sites, x);
            cell_out[(size_t)r * n + i] = c;
            if (margin_out)
                margin_out[(size_t)r * n + i] =
                    K > 1 ? oracle_bisector_margin(K, sites, x, c) : INFINITY;
        }
    }
    return 0;
}

/* Composite given per-sample fields (pins of the quadrature and of the
 * Painter's merge on hand-made inputs).  mode: 0 segments, 3 direct, 4 back. */
void oracle_composite(int mode, int n, const int *cell, const float *t, const double *sigma,
                      const double *rgb, float near_t, float far_t, double out_rgb[3],
                      double *out_depth, double *out_opacity, double *w_out)
{
    double *delta = malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    intervals(t, n, near_t, far_t, delta);
    if (mode == MODE_DERF)
        composite_segments(n, cell, t, sigma, rgb, delta, out_rgb, out_depth, out_opacity, w_out);
    else if (mode == MODE_BACK)
        composite_back_to_front(n, t, sigma, rgb, delta, out_rgb, out_depth, out_opacity);
    else
        composite_direct(n, t, sigma, rgb, delta, out_rgb, out_depth, out_opacity, NULL);
    free(delta);
}

/* Inverse-CDF fine depths of one ray from given coarse weights (pins). */
void oracle_fine_depths(uint64_t seed, uint64_t ray, int perturb, int nc, int nf, const float *tc,
                        float near_t, float far_t, const double *w, float *tf)
{
    double *cdf = malloc(sizeof(double) * (size_t)(nc + 1));
    fine_depths(seed, ray, perturb, nc, nf, tc, near_t, far_t, w, cdf, tf);
    free(cdf);
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
