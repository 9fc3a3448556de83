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
                              int site_bits, const CullLevel &lv, unsigned *counts,
                              unsigned num_blocks, hipStream_t s);
// bucket_scatter over the samples live at the level
hipError_t launch_level_scatter(const RenderGeometry &g, const uint8_t *cell,
                                const unsigned *counts, const unsigned *totals,
                                unsigned num_blocks, int num_sites, int site_bits,
                                const HeadMask &empty, const CullLevel &lv, unsigned *bucket,
                                float4 *sr, hipStream_t s);
// integrates each open ray's samples of the level behind its state in
// rgb / depth / trans (level 0: from the empty state) and sets opacity.
// max_len: a bound on every ray's sample count at this level (the piece
// length), or 0 for none; short levels take a few lanes per ray.
hipError_t launch_level_composite(const RenderGeometry &g, const float *t, const uint8_t *cell,
                                  const float4 *sr, const CullLevel &lv, unsigned max_len,
                                  float *rgb, float *depth, float *opacity, hipStream_t s);

}  // namespace derf
