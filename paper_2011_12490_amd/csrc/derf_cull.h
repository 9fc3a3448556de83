// Painter's-order culling (Sec. 3.3): the level loop of derf_render_culled.
#pragma once

// The kernels are in kernels_sample.hip.

#include "derf_internal.h"

namespace derf {

// Level l of a ray is its piece of ordinal l along the ray (the last level:
// every later piece); a piece is a segment, or with piece > 0 a part of at
// most piece samples of one, cut from the segment's start.  lb [R][levels + 1]: the first sample of each level
// (lb[r][levels] = n).  lvl [S]: each sample's level; the level composite that
// closes a ray (its transmittance below eps) marks the ray's later samples
// dead.  trans [R]: the transmittance in front of the level, written by each
// level's composite.  A ray takes part in level l > 0 only while trans >= eps.
struct CullLevel {
    const unsigned *lb;
    uint8_t *lvl;
    float *trans;
    unsigned *evaluated;  // [R] samples evaluated per ray, or null
    unsigned levels;      // 1 .. kMaxLevels
    unsigned level;
    float eps;
};
constexpr int kMaxLevels = 32;
hipError_t launch_level_bounds(const uint8_t *cell, unsigned n, unsigned num_rays,
                               unsigned levels, unsigned piece, unsigned *lb, uint8_t *lvl,
                               hipStream_t s);
// per-block head counts of the samples live at the level (the layout of the
// assignment's counts)
hipError_t launch_level_count(const RenderGeometry &g, const uint8_t *cell, int num_sites,
                              const CullLevel &lv, unsigned *counts,
                              unsigned num_blocks, hipStream_t s);
// One-pass bucketing of every level at once (levels K <= 256 keys): order
// [S] receives the sample ids sorted by (level, head),
// stably; totals [levels K] the samples per key and offsets [levels K] where
// each key's stretch starts; live [levels][K] the level-0 counts (zeros
// after).  Samples of 0-capacity heads get zero density and colour in sr.
// counts: [levels K][num_blocks] scratch.  Clears the MLP's tile counters.
hipError_t launch_level_head_order(const RenderGeometry &g, unsigned levels, int heads,
                                   const uint8_t *lvl, const uint8_t *cell,
                                   const HeadMask &empty, unsigned *counts, unsigned num_blocks,
                                   unsigned *totals, unsigned *order, unsigned *offsets,
                                   unsigned *live, float4 *sr, unsigned *mlp_queue, hipStream_t s);
// Level l >= 1 after the one-pass bucketing: copies the level's entries whose
// ray is still open from order to the same stretches of bucket, each head's
// packed at the front of its stretch, and counts them in live [K] (zero on
// entry).  num_blocks blocks of 4096 entries must cover the level.  Clears
// the MLP's tile counters.
hipError_t launch_level_compact(const RenderGeometry &g, unsigned level, unsigned levels,
                                int heads, const unsigned *order,
                                const unsigned *offsets, const unsigned *totals,
                                const uint8_t *lvl, const uint8_t *cell, unsigned num_blocks,
                                unsigned *live, unsigned *bucket, unsigned *mlp_queue,
                                hipStream_t s);
// A level below the last, bucketed ray by ray (each open ray's samples at
// such a level are one run of one cell, touching at most two blocks): the
// runs are counted into counts [K][num_blocks] (the per-sample counts'
// layout), scanned by bucket_scan into per-block prefixes and totals [K],
// and written to bucket at head_off [K] (K words of scratch: the exclusive
// scan of the totals) plus a position reserved from the prefix of their
// block (runs of one block in no fixed order).  sr gets zeros for
// 0-capacity heads.  Clears the MLP's tile counters.
hipError_t launch_level_ray_bucket(const RenderGeometry &g, const uint8_t *cell, int num_sites,
                                   const HeadMask &empty, const CullLevel &lv, unsigned *counts,
                                   unsigned num_blocks, unsigned *totals, unsigned *head_off,
                                   unsigned *bucket, float4 *sr, unsigned *mlp_queue,
                                   hipStream_t s);
// bucket_scatter over the samples live at the level
hipError_t launch_level_scatter(const RenderGeometry &g, const uint8_t *cell,
                                const unsigned *counts, const unsigned *totals,
                                unsigned num_blocks, int num_sites,
                                const HeadMask &empty, const CullLevel &lv, unsigned *bucket,
                                float4 *sr, hipStream_t s);
// integrates each open ray's samples of the level behind its state in
// rgb / depth / trans (level 0: from the empty state) and sets opacity.
// max_len: a bound on every ray's sample count at this level (the piece
// length), or 0 for none; levels of at most 32 samples take 8 lanes per ray,
// the others 16.
hipError_t launch_level_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                                  const float4 *sr, const CullLevel &lv, unsigned max_len,
                                  float *rgb, float *depth, float *opacity, hipStream_t s);

}  // namespace derf
