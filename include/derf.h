/*
 * derf.h -- C ABI of the MI355X (gfx950) DeRF renderer.
 *
 * DeRF ("Decomposed Radiance Fields", Rebain et al.) splits a NeRF radiance
 * field into the cells of a Voronoi diagram and gives every cell its own
 * small network head (Sec. 3.2, Eq. 4-5).  At inference the decomposition is
 * a hard partition -- each point is owned by its nearest site, the limit of
 * the soft Voronoi weights of Eq. 8 -- so every ray sample is evaluated by
 * exactly one head.  A ray crosses each convex cell in one contiguous
 * segment; each segment is volume-integrated on its own (Eq. 1-2) and the
 * segments are composited front to back in the order the Painter's argument
 * of Sec. 3.3 fixes.
 *
 * Calls:
 *   derf_create   upload sites and per-head weights            (Sec. 3.2-3.3)
 *   derf_create_mixed  the same with one architecture per head  (Sec. 5)
 *   derf_render   render rays: sample, encode, assign, bucket,
 *                 per-head MLP, segment integration, merge      (Sec. 3.1, 3.3)
 *   derf_render_debug  the same, also returning per-sample data
 *   derf_set_empty_heads  mark heads 0-capacity (empty space)     (Sec. 5)
 *   derf_render_soft   the soft decomposition: every head on every sample,
 *                 blended by the soft Voronoi weights, and each ray's
 *                 per-head contributions                    (Sec. 3.2 Eq. 4-6, Eq. 8)
 *   derf_render_culled  derf_render in Painter's order with transmittance
 *                 culling: a ray's later segments are not evaluated once
 *                 it is nearly opaque                       (Sec. 3.3)
 *   derf_set_gate / derf_render_gated  the MLP-gating decomposition:
 *                 a small network picks each sample's head      (Sec. 4)
 *   derf_weights_count  size of one head's packed weights: NeRF's
 *                 network, scaled per head                       (Sec. 4)
 *   derf_set_encoding  gamma(x) fused into the MLP or stored by its
 *                 own pass (the ablation of the fusion)          (Sec. 4)
 *   derf_render_noalloc  derf_render for callers that cannot allocate
 *
 * All functions return a derf_status (0 on success, negative on error),
 * never abort and never print.  derf_last_error() returns a thread-local
 * text describing the last failure of the calling thread.
 */
#ifndef DERF_H
#define DERF_H

#ifdef __cplusplus
extern "C" {
#endif

typedef struct derf_handle derf_handle;

typedef enum {
    DERF_OK = 0,
    DERF_ERR_INVALID_ARG = -1, /* a null pointer, an out-of-range size or value     */
    DERF_ERR_UNSUPPORTED = -2, /* a head architecture with no compiled kernel      */
    DERF_ERR_OOM = -3,         /* device or host allocation failed                  */
    DERF_ERR_HIP = -4          /* a HIP runtime call or kernel launch failed        */
} derf_status;

typedef enum {
    DERF_PREC_FP32 = 0, /* fp32 operands, fp32 MFMA accumulate                      */
    DERF_PREC_BF16 = 1  /* bf16 operands (round to nearest even), fp32 accumulate   */
} derf_precision;

/* Architecture shared by every head (the paper's heads are homogeneous; the
 * head network keeps NeRF's layout, Sec. 4.1).
 *   pos_freqs  L of the positional encoding gamma(x): 3 + 6L inputs
 *   dir_freqs  L of the direction encoding gamma(d / |d|): 3 + 6L inputs
 *   depth      number of hidden ReLU layers
 *   width      units per hidden layer
 *   skip_layer 0-based hidden layer whose input is [gamma(x); h], -1 = none
 *   rgb_hidden width of the ReLU hidden layer of the colour branch on
 *              [h; gamma(d)]; 0 = the colour logits read [h; gamma(d)] directly
 * The compiled kernels cover (pos, dir, depth, width, skip, rgb_hidden) =
 * (6,4,4,64,-1,0), (10,4,8,256,5,128), (10,4,8,128,5,64), (10,4,6,64,-1,32);
 * any other architecture is DERF_ERR_UNSUPPORTED. */
typedef struct {
    int pos_freqs;
    int dir_freqs;
    int depth;
    int width;
    int skip_layer;
    int rgb_hidden;
} derf_head_arch;

/* Sampling of each ray on [near, far] (Sec. 3.1 Eq. 1 bounds).
 *   n_coarse  stratified samples per ray (>= 1, n_coarse + n_fine <= 1024)
 *   n_fine    0: one pass over the n_coarse samples.  > 0 (needs n_coarse
 *             >= 2): hierarchical sampling as in NeRF, which the paper keeps
 *             for its heads (Sec. 4): the coarse pass's quadrature weights
 *             w_i = T_i alpha_i plus 1e-5 define a piecewise-constant
 *             density on the coarse midpoint intervals; n_fine draws
 *             u_j = (j + xi_j) / n_fine (xi_j: stream 1 of the generator
 *             below) go through its inverse CDF (computed in float64); the
 *             coarse and fine depths are merged in order (coarse first on
 *             equal depths), the fine samples are assigned and evaluated,
 *             the coarse heads' outputs are reused, and the result is the
 *             composite of all n_coarse + n_fine samples.
 *   seed      key of the Philox4x32-10 generator of the stratum jitter
 *   perturb   1: t_i = near + (i + xi) (far - near) / n with xi from Philox;
 *             0: xi = 1/2 (stratum midpoints)
 *   ray_offset  frame index of the first ray of the call: the jitter of sample
 *             i of ray r is word i % 4 of Philox4x32-10 at counter
 *             (i / 4, low and high words of ray_offset + r, 0), key = the
 *             seed's low and high words, mapped as (word >> 8) * 2^-24; so a
 *             frame split over several calls renders exactly as one call */
typedef struct {
    int n_coarse;
    int n_fine;
    unsigned long long seed;
    int perturb;
    unsigned long long ray_offset;
} derf_sampling;

/* Number of floats of one head's packed weights for this architecture (a
 * NeRF network of Sec. 4: ReLU layers over gamma(x) with an optional skip
 * input, density from the last hidden layer, colour from it and gamma(d)),
 * or -1 for invalid values.  Per head, in this order: for each hidden layer l,
 * W_l [width][in_l] row-major (out x in) then b_l [width], with in_0 =
 * 3 + 6 pos_freqs and in_skip = (3 + 6 pos_freqs) + width (input order
 * [gamma(x); h]); then w_sigma [width], b_sigma [1]; then, if rgb_hidden > 0,
 * W_v [rgb_hidden][width + 3 + 6 dir_freqs], b_v [rgb_hidden], W_c
 * [3][rgb_hidden], b_c [3], else W_c [3][width + 3 + 6 dir_freqs], b_c [3]
 * (input order [h; gamma(d)]).  Density is ReLU(w_sigma . h + b_sigma),
 * colour is sigmoid of the logits. */
long long derf_weights_count(const derf_head_arch *arch);

/* Create a renderer on the current HIP device.
 *   out        receives the handle (set to NULL on failure)
 *   num_sites  K, number of Voronoi sites = number of heads, 1 <= K <= 256
 *   sites_xyz  host float [K][3]: the sites phi (Sec. 3.3)
 *   arch       head architecture (see above)
 *   weights    host float [K][derf_weights_count(arch)]: head k's packed
 *              weights at weights + k * derf_weights_count(arch)
 *   precision  a derf_precision
 * The host arrays are copied (converted and re-laid-out for the kernels) and
 * may be freed on return.  The call synchronises the device. */
int derf_create(derf_handle **out, int num_sites, const float *sites_xyz,
                const derf_head_arch *arch, const float *weights, int precision);

/* As derf_create, with heads of different capacities (the heterogeneous
 * heads of Sec. 5, limitations and future work):
 *   archs    host [K]: head k's architecture; each must be one derf_create
 *            accepts, and at most 4 distinct ones per renderer
 *   weights  host float: head k's derf_weights_count(&archs[k]) packed
 *            weights, heads one after another in index order
 * A render runs one grouped-MLP launch per distinct architecture, over its
 * heads.  DERF_ERR_UNSUPPORTED for an architecture without a kernel or more
 * than 4 distinct ones; other errors as derf_create. */
int derf_create_mixed(derf_handle **out, int num_sites, const float *sites_xyz,
                      const derf_head_arch *archs, const float *weights, int precision);

/* Render num_rays rays.  All array arguments are device pointers:
 *   rays_o, rays_d   float [R][3] origins and directions (directions need
 *                    not be unit length: samples are o + t d, the colour
 *                    head sees gamma(d / |d|))
 *   out_rgb          float [R][3] composited colour (black background)
 *   out_depth        float [R] expected depth sum_i w_i t_i
 *   out_opacity      float [R] 1 - transmittance after the last sample
 * near_t < far_t; samp as above; hip_stream is a hipStream_t (NULL: the
 * default stream).  The work is enqueued on hip_stream and the call returns
 * without waiting for it; the inputs must stay valid and the outputs
 * untouched until it completes.  Kernel faults surface at the caller's next
 * synchronisation.  num_rays == 0 is a no-op.  num_rays < 2^30 and
 * R * (n_coarse + n_fine) < 2^32; larger frames are rendered in several calls.  Calls on one handle
 * must not run concurrently (they share the handle's workspace, which grows
 * as needed and is reused). */
int derf_render(derf_handle *h, const float *rays_o, const float *rays_d, long long num_rays,
                float near_t, float far_t, const derf_sampling *samp, float *out_rgb,
                float *out_depth, float *out_opacity, void *hip_stream);

/* derf_render for callers that cannot allocate device memory: code under HIP
 * graph capture, serving loops and harnesses that forbid hipMalloc.  The
 * render's scratch memory (sample depths, cells, head outputs, buckets,
 * counts, walk tables) is a fixed device array of
 * DERF_NOALLOC_SCRATCH_BYTES inside the library, one per device, held from
 * the first derf_create on that device until the process ends; the call
 * itself allocates nothing.  Arguments, results and ownership as
 * derf_render (the results are identical).  A frame whose scratch would
 * exceed the array -- about 25 bytes per sample plus 64-600 bytes per ray,
 * e.g. ~12,000 rays of 192 samples -- returns DERF_ERR_INVALID_ARG before any
 * work is enqueued: render it in parts (samp->ray_offset keeps the jitter of
 * a split frame).  Every handle on one device shares that device's array and
 * each call leaves its contents behind, so calls that overlap in time on one
 * device race: enqueue them on one stream, or wait between them.  Stats
 * (derf_get_stats) read the last call's head counts from the array, so they
 * are only valid until the next call on the device. */
#define DERF_NOALLOC_SCRATCH_BYTES (64u << 20)
int derf_render_noalloc(derf_handle *h, const float *rays_o, const float *rays_d,
                        long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                        float *out_rgb, float *out_depth, float *out_opacity, void *hip_stream);

/* Optional per-sample outputs of derf_render_debug: device pointers, any may
 * be NULL.  They are the quantities the integration of Sec. 3.1 (Eq. 1-2)
 * consumes: each sample's depth, its owning site under the nearest-site
 * partition (Sec. 3.3) and that head's density and colour.  N = n_coarse + n_fine samples per ray, in depth order (with
 * hierarchical sampling: the merged coarse and fine samples); sample i of
 * ray r is at index r * N + i. */
typedef struct {
    int *cell;    /* [R][N] owning site of each sample                       */
    float *t;     /* [R][N] sample depth                                     */
    float *sigma; /* [R][N] density from the owning head                     */
    float *rgb;   /* [R][N][3] colour from the owning head                   */
} derf_debug_out;

int derf_render_debug(derf_handle *h, const float *rays_o, const float *rays_d,
                      long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                      float *out_rgb, float *out_depth, float *out_opacity,
                      const derf_debug_out *dbg, void *hip_stream);

/* Mark heads as 0-capacity: a head with flags[k] != 0 represents empty space
 * (the heterogeneous-capacity remark of Sec. 5, limitations and future work): its
 * density and colour are zero everywhere, so it is never evaluated.  The
 * partition is unchanged -- its samples still belong to it -- and every
 * render (single pass, hierarchical, soft) treats it as transparent; its
 * packed weights are ignored.  flags is a host int [K] (copied; NULL clears
 * every mark).  Takes effect for renders enqueued after the call; marks
 * persist until the next call.  Returns DERF_ERR_INVALID_ARG for a NULL
 * handle. */
int derf_set_empty_heads(derf_handle *h, const int *flags);

/* Render with the soft decomposition at temperature beta (Sec. 3.2 Eq. 4-5
 * with the weights of Sec. 3.3 Eq. 8): every head evaluates every sample,
 *   w_k(x) = exp(-beta |x - phi_k|) / sum_j exp(-beta |x - phi_j|),
 *   sigma(x) = sum_k w_k(x) sigma_k(x),  c(x, d) = sum_k w_k(x) c_k(x, d),
 * and the samples are composited front to back (Eq. 1-2, midpoint
 * intervals).  This is the forward pass the decomposition is trained with; it
 * costs K head evaluations per sample.  As beta grows it approaches
 * derf_render.
 *   beta         finite, >= 0 (0: all heads weighted equally)
 *   out_contrib  NULL, or device float [R][K]: the contributions of Sec. 3.2
 *                Eq. 6, W_k(r) = sum_i T_i alpha_i w_k(x_i) with the render's
 *                quadrature, so that sum_k W_k(r) = out_opacity[r]
 * Other arguments as derf_render; samp->n_fine must be 0 (DERF_ERR_UNSUPPORTED
 * otherwise) and R * n_coarse * K must stay below 2^32.  The workspace holds
 * every head's outputs for every sample (16 K bytes per sample).  Stage times
 * go to DERF_STAGE_SAMPLE (sampling), DERF_STAGE_MLP (all heads) and
 * DERF_STAGE_COMPOSITE (blend and composite). */
int derf_render_soft(derf_handle *h, const float *rays_o, const float *rays_d, long long num_rays,
                     float near_t, float far_t, const derf_sampling *samp, float beta,
                     float *out_rgb, float *out_depth, float *out_opacity, float *out_contrib,
                     void *hip_stream);

/* derf_render with the Painter's order put to work (Sec. 3.3: a ray meets its
 * cells in order of distance from its origin, and composites its segments
 * front to back): the ray's pieces are evaluated level by level, level l of a
 * ray being its piece of ordinal l along the ray (level levels - 1: every
 * later piece), and a ray whose transmittance in front of level l > 0 is
 * below eps skips that level and every later one -- its heads do not run
 * there.  A piece is a segment or, with piece > 0, a part of at most piece
 * samples of one, cut from the segment's first sample (the merge of a
 * segment's pieces front to back is the segment's own, since "over" is
 * associative; cutting only adds places where a ray can stop, which matters
 * when a ray crosses few cells).  The result is the Painter's merge of the evaluated segments: colour
 * and opacity within eps of derf_render's (colours lie in [0, 1]), depth
 * within eps * far.  With levels = 1, eps = 0, or a single head in whole
 * segments (every ray is one segment) nothing can be skipped: the call runs
 * derf_render's single pass, and the outputs equal derf_render's bitwise.
 *   eps            finite, >= 0: the transmittance below which a ray stops
 *   levels         1 .. 32: levels (one bucketing, MLP and integration pass
 *                  each)
 *   piece          >= 0: the most samples of one piece; 0: whole segments
 *   out_evaluated  NULL, or device unsigned [R]: samples whose head ran, per
 *                  ray
 * Other arguments and limits as derf_render; samp->n_fine must be 0
 * (DERF_ERR_UNSUPPORTED otherwise).  Stage times: DERF_STAGE_SAMPLE
 * (sampling, assignment and level bounds) and DERF_STAGE_MLP (the whole
 * level loop); head_samples sums every level's evaluations. */
int derf_render_culled(derf_handle *h, const float *rays_o, const float *rays_d,
                       long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                       float eps, int levels, int piece, float *out_rgb, float *out_depth,
                       float *out_opacity, unsigned *out_evaluated, void *hip_stream);

/* The MLP-gating decomposition (Sec. 4, decompositions with MLPs): instead of
 * the nearest site, a small network with a softmax output assigns each
 * sample to a head, the one of largest weight.  The softmax is monotone, so
 * that is the argmax of the logits (ties to the lowest index):
 *   h = ReLU(W1 gamma_L(x) + b1),  logits = W2 h + b2  (K logits)
 * gamma_L is the positional encoding of the heads (p, then sin and cos of
 * pi 2^l p for l < L), evaluated in fp32.  The products run on bf16 matrix
 * cores with each fp32 operand a split into a_hi = bf16(a) and
 * a_lo = bf16(a - a_hi), each product taken as a_hi b_hi + a_hi b_lo +
 * a_lo b_hi and summed in fp32; the hidden units are fp32.  The argmax is
 * decided in that precision.  Gated cells need not be convex, so a ray may
 * enter one cell several times; its runs are merged front to back, which is
 * exact for any partition.
 * derf_set_gate takes the host weights, fp32, packed W1 [H][3 + 6L], b1 [H],
 * W2 [K][H], b2 [K] (derf_gate_weights_count floats), splits them as above
 * into the kernel's layout on the device (12 KB for L = 10, H = 32, K = 16;
 * at most 81 KB); the caller may free them on return.  pos_freqs 6 or 10 and hidden 16, 32 or 64
 * have kernels (DERF_ERR_UNSUPPORTED otherwise); hidden = 0 removes the gate.
 * Non-finite weights: DERF_ERR_INVALID_ARG.  Waits for the handle's last
 * stream before replacing a gate. */
int derf_set_gate(derf_handle *h, int pos_freqs, int hidden, const float *weights);
/* floats of a gating network for K heads; -1 for invalid values */
long long derf_gate_weights_count(int num_sites, int pos_freqs, int hidden);
/* derf_render with the gated assignment: the stratified depths (the same
 * draws as derf_render's) and the gate in one kernel, then per-head buckets,
 * the grouped MLP and front-to-back integration of the runs; no
 * nearest-site search.  Arguments,
 * limits and ownership as derf_render (single pass: samp->n_fine must be 0,
 * DERF_ERR_UNSUPPORTED otherwise); DERF_ERR_INVALID_ARG without a gate.
 *   out_cell   NULL, or device int32 [R][N]: each sample's gated head
 * Stage times: DERF_STAGE_SAMPLE (sampling and the gate) and
 * DERF_STAGE_MLP (bucketing, heads and integration); head_samples counts
 * each head's gated samples. */
int derf_render_gated(derf_handle *h, const float *rays_o, const float *rays_d,
                      long long num_rays, float near_t, float far_t, const derf_sampling *samp,
                      float *out_rgb, float *out_depth, float *out_opacity, int *out_cell,
                      void *hip_stream);

/* Where gamma(x), the positional encoding of each sample (Sec. 4, the
 * encoding the heads take as input), is formed.
 *   DERF_ENCODING_FUSED   (default) inside the grouped MLP, per tile, from
 *                         the sample's depth and ray: no table in HBM.
 *   DERF_ENCODING_STORED  a separate pass after the assignment writes every
 *                         sample's gamma(x) to a table in the workspace
 *                         (128 B per sample in bf16 at L = 10, 256 B in
 *                         fp32) and the MLP reads it back.  The outputs are
 *                         the fused form's bit for bit; the form exists to
 *                         measure what the fusion saves.
 * STORED needs head architectures without a skip layer, all with the same
 * pos_freqs (DERF_ERR_UNSUPPORTED otherwise, the setting unchanged); while
 * it is set, derf_render, derf_render_debug and derf_render_noalloc use it
 * (both passes of hierarchical sampling; the table counts towards the
 * no-allocation render's limit) and derf_render_soft, derf_render_culled
 * and derf_render_gated return DERF_ERR_UNSUPPORTED.  Other modes:
 * DERF_ERR_INVALID_ARG.  Applies to renders issued after the call. */
enum { DERF_ENCODING_FUSED = 0, DERF_ENCODING_STORED = 1 };
int derf_set_encoding(derf_handle *h, int mode);

/* Per-stage GPU time, recorded with HIP events on the render's stream when
 * timing is on (derf_set_timing); accumulated over renders since the last
 * derf_reset_stats.  With hierarchical sampling a stage's time is the sum of
 * its coarse and fine passes; stage_launches counts the renders that ran the
 * stage.  head_samples counts head evaluations of both passes.
 * walk_rays and walk_fallback_rays describe the last render's assignment
 * (Sec. 3.3: a ray crosses each convex cell in one segment): from 17 heads
 * every ray is first walked through its cells; a ray that crosses more than
 * 32 cells, or has a segment with more than 11 near-tied candidate sites, is
 * assigned by the search over all sites instead (same cells, more work).
 * walk_rays is 0 when the render searched all sites for every sample. */
enum {
    DERF_STAGE_SAMPLE = 0,         /* sample + encode + assign (given depths: assign);
                                      the stored gamma(x) pass                        */
    DERF_STAGE_BUCKET_SCAN = 1,    /* per-head counts -> offsets                     */
    DERF_STAGE_BUCKET_SCATTER = 2, /* sample ids into per-head buckets               */
    DERF_STAGE_MLP = 3,            /* grouped per-head MLP                           */
    DERF_STAGE_COMPOSITE = 4,      /* segment integration + Painter's merge          */
    DERF_STAGE_FINE = 5            /* coarse weights -> inverse-CDF fine depths      */
};
#define DERF_NUM_STAGES 6
typedef struct {
    long long renders;                  /* renders since reset              */
    long long samples;                  /* samples since reset              */
    double stage_ms[DERF_NUM_STAGES];   /* summed event time per stage      */
    long long stage_launches[DERF_NUM_STAGES];
    long long head_samples[256];        /* samples per head of the last render */
    long long walk_rays;                /* rays of the last render walked through their cells */
    long long walk_fallback_rays;       /* of those, rays searched over all sites */
} derf_stats;

int derf_set_timing(derf_handle *h, int on);
/* Waits for the last render's stream, then fills *out. */
int derf_get_stats(derf_handle *h, derf_stats *out);
int derf_reset_stats(derf_handle *h);

/* Waits for the handle's last stream, then frees everything.  NULL is a no-op. */
void derf_destroy(derf_handle *h);

const char *derf_status_string(int status);
const char *derf_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DERF_H */
