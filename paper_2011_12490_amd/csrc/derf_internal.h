// Internal interfaces between the host API (derf_api.cpp) and the HIP kernel
// sources.  Nothing here is part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace derf {

// Samples covered by one bucketing block: the counting pass and the scatter
// pass must agree on this partition of the sample range.
constexpr int kBucketBlock = 4096;
// Padded length of the per-ray direction feature vector gamma(d / |d|).
constexpr int kDirPad = 32;
constexpr int kMaxSites = 256;
// Tile counters of the MLP's work queues (one per XCD), for each of at most
// kMaxHeadGroups MLP launches of a render (one per head architecture).
constexpr int kMlpQueues = 8;
constexpr int kMaxHeadGroups = 4;

// Heads marked 0-capacity (empty space: no density anywhere), one bit each.
struct HeadMask {
    unsigned w[kMaxSites / 32];
    __host__ __device__ bool test(int k) const { return (w[k >> 5] >> (k & 31)) & 1u; }
};

// Per-ray cell walk (see ray_walk_kernel): at most kMaxSeg segments per ray,
// each with at most kMaxCand candidate sites.
constexpr int kMaxSeg = 32;
constexpr int kMaxCand = 11;
struct alignas(16) SegRec {
    float t_end;          // the segment covers depths up to t_end
    unsigned char ncand;  // candidate sites, ascending
    unsigned char cand[kMaxCand];
};
// Heads from which the assignment uses the walk instead of all sites (below,
// the search over all sites costs less than the walk and its table lookups).
constexpr int kWalkSites = 17;
struct WalkTable {
    const SegRec *seg;           // [R][kMaxSeg]
    const unsigned char *nseg;   // [R]; 0: the ray takes the search over all sites
};

struct RenderGeometry {
    const float *rays_o;
    const float *rays_d;
    unsigned num_rays;
    unsigned n;          // samples per ray
    unsigned num_samples;
    double inv_n;        // 1.0 / n, for the sample -> (ray, index) split
    float near_t, far_t, step;
    uint64_t seed;
    uint64_t ray_offset;
    int perturb;
};

// ---- MLP gating (kernels_gate.hip) ---------------------------------------
// Gating networks with a compiled kernel: gamma_L(x) with L = 6 or 10 as
// input, one ReLU layer of 16, 32 or 64 units, K logits.
bool gate_shape_supported(int pos_freqs, int hidden);
// Bytes of a gate's weights and biases laid out for the kernel, and the
// layout itself from the packed fp32 order of derf.h (host side).
size_t gate_packed_bytes(int pos_freqs, int hidden, int num_sites);
void gate_pack(int pos_freqs, int hidden, int num_sites, const float *w, unsigned char *out);
// t[s] = the stratified depth of sample s (as the single pass draws it), and
// cell[s] = argmax of the gating logits there; also to out_cell (int32 [S])
// when not null.  packed: gate_pack's layout on the device; cus: compute
// units (the kernel's workgroups are persistent).
hipError_t launch_gate(const RenderGeometry &g, const unsigned char *packed, int pos_freqs,
                       int hidden, int num_sites, float *t, uint8_t *cell, int *out_cell, int cus,
                       hipStream_t s);

// ---- sampling, assignment and bucketing (kernels_sample.hip) -------------
// p[0 .. count) = v (a kernel: no memset node in a captured stream)
hipError_t launch_fill_u32(unsigned *p, unsigned count, unsigned v, hipStream_t s);
hipError_t launch_ray_encode(const RenderGeometry &g, void *dirbuf, bool bf16, hipStream_t s);
// Walk every ray of g through the cells on [near, far] (one lane per ray).
hipError_t launch_ray_walk(const RenderGeometry &g, const float4 *sites, int num_sites,
                           SegRec *seg, unsigned char *nseg, hipStream_t s);
// walk: the table of launch_ray_walk for the same rays, or {nullptr, nullptr}
hipError_t launch_sample_assign(const RenderGeometry &g, const float4 *sites, int num_sites,
                                const WalkTable &walk, float *t, uint8_t *cell,
                                unsigned *counts, unsigned num_blocks, hipStream_t s);
// same, for given depths t (read only): no sampling
hipError_t launch_assign_given(const RenderGeometry &g, const float4 *sites, int num_sites,
                               const WalkTable &walk, const float *t,
                               uint8_t *cell, unsigned *counts, unsigned num_blocks,
                               hipStream_t s);
// also clears the kMlpQueues tile counters of the MLP launch that follows
hipError_t launch_bucket_scan(unsigned *counts, unsigned num_blocks, int num_sites,
                              unsigned *totals, unsigned *mlp_queue, hipStream_t s);
// Samples of 0-capacity heads also get sr = 0 here (the MLP skips those heads).
hipError_t launch_bucket_scatter(const uint8_t *cell, const unsigned *counts,
                                 const unsigned *totals, unsigned num_samples,
                                 unsigned num_blocks, int num_sites,
                                 const HeadMask &empty, unsigned *bucket, float4 *sr,
                                 hipStream_t s);
// Soft decomposition: bucket[i] = i (i < S), totals[k] = S, queue cleared.
hipError_t launch_soft_setup(unsigned S, int num_sites, unsigned *bucket, unsigned *totals,
                             unsigned *queue, hipStream_t s);
// Blend every head's outputs sr[k * S + i] by the soft Voronoi weights and
// composite; contrib (nullable) receives the per-ray head contributions.
hipError_t launch_soft_composite(const RenderGeometry &g, const float4 *sites, int num_sites,
                                 const HeadMask &empty, float beta, const float *t,
                                 const float4 *sr, float *rgb, float *depth, float *opacity,
                                 float *contrib, hipStream_t s);
hipError_t launch_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                            const float4 *sr, float *rgb, float *depth, float *opacity,
                            hipStream_t s);
hipError_t launch_debug_expand(unsigned num_samples, const float *t, const uint8_t *cell,
                               const float4 *sr, int *dcell, float *dt, float *dsigma,
                               float *drgb, hipStream_t s);

// ---- hierarchical sampling (kernels_fine.hip) -----------------------------
// g describes the coarse pass (n = n_coarse).  tf [R][n_fine] receives the
// sorted inverse-CDF depths drawn from the coarse outputs src.
hipError_t launch_fine_sample(const RenderGeometry &g, const float *tc, const float4 *src,
                              unsigned n_fine, float *tf, hipStream_t s);
// Composite of the depth-ordered merge of the coarse (tc, cc, sc) and fine
// (tf, cf, sf) samples; the optional debug arrays receive the merged fields.
hipError_t launch_merge_composite(const RenderGeometry &g, const float *tc, const uint8_t *cc,
                                  const float4 *sc, unsigned n_fine, const float *tf,
                                  const uint8_t *cf, const float4 *sf, float *rgb, float *depth,
                                  float *opacity, int *dcell, float *dt, float *dsigma,
                                  float *drgb, hipStream_t s);

// ---- grouped per-head MLP (mlp_kernel.h, mlp_*.hip) ----------------------
struct HeadArch {
    int pos_freqs, dir_freqs, depth, width, skip_layer, rgb_hidden;
};

struct MlpVariant {
    // bytes of one head's fragment stream and of its resident block
    size_t stream_bytes;
    size_t block_bytes;
    int tile;            // samples per tile
    // Lay out one head's fp32 weights (packed order of derf.h) for the kernel.
    void (*pack)(const float *w, unsigned char *stream, float *block);
    // queue: kMlpQueues tile counters, zero at launch.  soft: every head
    // takes every sample (bucket = 0 .. S-1, totals[k] = S) and writes its
    // outputs to sr[k * S + sample]; otherwise sr[sample].  offsets: null
    // (head k's entries follow head k - 1's), or where each head's totals[k]
    // entries start in bucket (not soft).  gxtab: null, or for the
    // stored-encoding form (which needs it, and takes no soft launch) the
    // table its encode wrote for the same samples.
    hipError_t (*launch)(const unsigned *bucket, const unsigned *totals, const unsigned *offsets,
                         int num_sites,
                         const RenderGeometry &g, const float *t, const void *dirbuf,
                         const void *gxtab, const unsigned char *streams, const float *blocks,
                         float4 *sr, unsigned *queue, int grid, bool soft, const HeadMask &empty,
                         hipStream_t s);
    // The stored-encoding form of this architecture (same packed weights;
    // gamma(x) read from a table instead of encoded per tile), or null.
    const MlpVariant *stored;
    // stored-encoding form only: table bytes per sample, the number of
    // position frequencies, and the kernel that fills the table from the
    // depths t of g's samples (one row per sample)
    size_t gx_bytes;
    int pos_freqs;
    hipError_t (*encode)(const RenderGeometry &g, const float *t, void *gxtab, int cus,
                         hipStream_t s);
};

// Returns nullptr when no kernel is compiled for this architecture/precision.
const MlpVariant *find_mlp_variant(const HeadArch &a, bool bf16);
// the variants of each supported head architecture (one translation unit each;
// nullptr where a precision is not built)
const MlpVariant *mlp_variant_4x64(bool bf16);
const MlpVariant *mlp_variant_6x64(bool bf16);
const MlpVariant *mlp_variant_8x128(bool bf16);
const MlpVariant *mlp_variant_8x256(bool bf16);

}  // namespace derf
