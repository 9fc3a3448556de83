"""GPU parity of hierarchical sampling (coarse pass, inverse-CDF fine depths,
fine pass, merged composite) through the C ABI, against the CPU oracle.

Each stage is checked on its own inputs as well as end to end:
  * merged depths: sorted, and the coarse depths (bit-exact with the oracle's
    stratified samples) sit in them in order;
  * fine depths: the oracle's inverse CDF applied to the coarse weights the
    oracle derives from the GPU's own coarse densities (so the check is
    independent of the heads' precision) -- tight tolerance;
  * cells of every emitted depth: bit-exact except within 1e-5 of a bisector;
  * merged composite: the oracle's segment composite of the GPU's merged
    per-sample fields;
  * pixels: the oracle's heads, quadrature and Painter's merge at the GPU's
    emitted depths (every cell decision on the same float32 points), max-abs
    1e-4 (fp32) and 2e-2 (bf16); and the oracle's own hierarchical render, at
    the precision's bar on rays of opacity >= 0.5, where the inverse CDF is
    well conditioned, and at 2e-2 elsewhere (its float64 coarse densities
    move the fine depths: see _check_hier), except rays where that moved a
    fine sample across a cell boundary from the GPU's (counted and bounded;
    each must have the boundary between the two runs' sample points).
"""
import os

import numpy as np
import pytest

import oracle
from paper_2011_12490_amd import scenes
from parity_log import record

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}
NTHREADS = min(16, os.cpu_count() or 1)
SEED = scenes.SEED_RENDER


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)
    torch.cuda.set_device(0)


def _render(sc, precision, nc, nf, rays=None, perturb=True, ray_offset=0, debug=True):
    from paper_2011_12490_amd import derf
    cfg = sc.cfg
    o = torch.from_numpy(sc.rays_o if rays is None else rays[0]).cuda()
    d = torch.from_numpy(sc.rays_d if rays is None else rays[1]).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
    out = r.render(o, d, cfg.near, cfg.far, nc, nf, SEED, perturb, debug=debug,
                   ray_offset=ray_offset)
    torch.cuda.synchronize()
    r.close()
    return [x.cpu().numpy() if torch.is_tensor(x) else
            {k: v.cpu().numpy() for k, v in x.items()} for x in out]


def _split(t_merged, tc):
    """Positions of the coarse samples in a merged list (greedy in order:
    on equal depths the coarse sample comes first)."""
    coarse = np.zeros(t_merged.shape[0], bool)
    p = 0
    for k, v in enumerate(t_merged):
        if p < tc.size and v == tc[p]:
            coarse[k] = True
            p += 1
    return coarse, p


def _check_hier(sc, gpu, nc, nf, precision, label, ids_pixels, ids_fine, perturb=True,
                ray_offset=0, rays=None, tol_t=None, end_to_end="all"):
    cfg = sc.cfg
    o = sc.rays_o if rays is None else rays[0]
    d = sc.rays_d if rays is None else rays[1]
    R = o.shape[0]
    N = nc + nf
    dbg = gpu[3]
    t_m, c_m, s_m, rgb_m = dbg["t"], dbg["cell"], dbg["sigma"], dbg["rgb"]
    assert t_m.shape == (R, N)
    assert np.all(np.diff(t_m, axis=1) >= 0), "merged depths not sorted"
    assert np.all((t_m >= cfg.near) & (t_m <= cfg.far))

    # cells of every emitted depth
    cell_ref, _ = oracle.assign_depths(sc.sites, o, d, t_m, nthreads=NTHREADS)
    diff = np.argwhere(c_m != cell_ref)
    for r, i in diff:
        x = (o[r].astype(np.float64) + np.float64(t_m[r, i]) * d[r]).astype(np.float32)
        m = oracle.bisector_margin(sc.sites, x, int(cell_ref[r, i]))
        assert m < 1e-5, (r, i, c_m[r, i], cell_ref[r, i], m)
    print("%s: samples=%d cell mismatches=%d (all within 1e-5 of a bisector)"
          % (label, c_m.size, len(diff)), flush=True)
    record(test=label, kind="cells at the emitted depths", samples=int(c_m.size),
           mismatches=int(len(diff)))

    # coarse depths in order, fine depths from the GPU's coarse densities,
    # merged composite from the GPU's merged fields
    e_t = e_comp = 0.0
    for r in ids_fine:
        tc = oracle.sample_depths(SEED, ray_offset + int(r), cfg.near, cfg.far, nc, perturb)
        coarse, found = _split(t_m[r], tc)
        assert found == nc, "ray %d: coarse depths missing from the merged list" % r
        cw = oracle.composite(c_m[r][coarse], tc, s_m[r][coarse], rgb_m[r][coarse],
                              cfg.near, cfg.far)[3]
        tf_ref = oracle.fine_depths(SEED, ray_offset + int(r), perturb, tc, cfg.near, cfg.far,
                                    cw, nf)
        e_t = max(e_t, float(np.abs(t_m[r][~coarse] - tf_ref).max()))
        c3, dep, op, _ = oracle.composite(c_m[r], t_m[r], s_m[r], rgb_m[r], cfg.near, cfg.far)
        e_comp = max(e_comp, float(np.abs(gpu[0][r] - c3).max()), abs(gpu[1][r] - dep),
                     abs(gpu[2][r] - op))
    tol_t = tol_t if tol_t is not None else 4 * np.spacing(np.float32(max(abs(cfg.near),
                                                                          abs(cfg.far))))
    print("%s: fine depths vs oracle inverse CDF of the GPU's coarse weights: max|dt|=%.3g "
          "(tol %.3g); merged composite vs oracle: max|d|=%.3g (rays %d)"
          % (label, e_t, tol_t, e_comp, len(ids_fine)), flush=True)
    record(test=label, kind="fine depths and merged composite", rays=int(len(ids_fine)),
           max_abs_t=e_t, tol_t=float(tol_t), max_abs_composite=e_comp, tol_composite=2e-5)
    assert e_t <= tol_t
    assert e_comp <= 2e-5

    # heads and composite of the oracle at the GPU's emitted depths: every
    # cell decision is taken on the same float32 sample points
    ids_pixels = np.asarray(ids_pixels)
    tol = TOL[precision]
    gd = oracle.render_depths(sc.sites, cfg.arch, sc.weights, o[ids_pixels], d[ids_pixels],
                              cfg.near, cfg.far, t_m[ids_pixels], nthreads=NTHREADS)
    e_rgb = np.abs(gpu[0][ids_pixels] - gd.rgb).max()
    e_dep = np.abs(gpu[1][ids_pixels] - gd.depth).max()
    e_op = np.abs(gpu[2][ids_pixels] - gd.opacity).max()
    print("%s: at the GPU's depths: rays=%d max|d rgb|=%.3g max|d depth|=%.3g "
          "max|d opacity|=%.3g (tol %.0e)" % (label, len(ids_pixels), e_rgb, e_dep, e_op, tol),
          flush=True)
    record(test=label, kind="pixels at the emitted depths", rays=int(len(ids_pixels)),
           max_abs_rgb=float(e_rgb), max_abs_depth=float(e_dep), max_abs_opacity=float(e_op),
           tol=tol)
    assert e_rgb <= tol and e_dep <= tol and e_op <= tol

    # the oracle's own hierarchical render.  Its fine depths follow its own
    # (float64) coarse densities, and the inverse CDF amplifies a density
    # difference by about 1 / (total pdf mass) ~ 1 / opacity: on a nearly
    # transparent ray the pdf is mostly the 1e-5 floor (mass ~ n_coarse
    # 1e-5), so an absolute density change e moves the CDF by up to
    # ~ e delta / (n_coarse 1e-5) and the fine depths with it, and moved
    # quadrature nodes change the pixel at first order.  So the rays are
    # split by conditioning: a ray whose opacity is at least 0.5 (pdf mass at
    # least half) is held to the precision's own bar, 1e-4 (fp32) or 2e-2
    # (bf16); a more transparent ray to the bf16 bar, or, on scenes of mostly
    # translucent rays with bf16 heads (end_to_end="report"), it is only
    # reported.  A fine sample can also land on the other side of a cell
    # boundary than the GPU's; such rays are checked for validity only: the
    # boundary must lie between the two runs' sample points.
    ref = oracle.render(sc.sites, cfg.arch, sc.weights, o[ids_pixels], d[ids_pixels], cfg.near,
                        cfg.far, nc, nf, seed=SEED, perturb=perturb,
                        ray_ids=ids_pixels.astype(np.int64) + ray_offset, per_sample=True,
                        nthreads=NTHREADS)
    cm, tm = c_m[ids_pixels], t_m[ids_pixels].astype(np.float64)
    mism = ref.cell != cm
    flipped = mism.any(axis=1)
    gap = np.abs(tm - ref.t) * np.linalg.norm(d[ids_pixels].astype(np.float64), axis=1)[:, None]
    assert np.all(ref.margin[mism] <= gap[mism] * 1.001 + 1e-5), "cell change not explained"
    err = np.maximum.reduce([np.abs(gpu[0][ids_pixels] - ref.rgb).max(1),
                             np.abs(gpu[1][ids_pixels] - ref.depth),
                             np.abs(gpu[2][ids_pixels] - ref.opacity)])
    well = ref.opacity >= 0.5
    checked = well | (end_to_end == "all")
    tol_ray = np.where(well, TOL[precision], TOL["bf16"])
    keep = checked & ~flipped
    print("%s: end to end (%s): %d rays checked (%d well conditioned, tol %.0e; the rest %.0e), "
          "%d of them with a sample across a cell boundary from the oracle's; max error well "
          "conditioned %.3g, others %.3g; all rays: max depth gap %.3g, error quantiles "
          "50/90/99%% %.3g %.3g %.3g"
          % (label, end_to_end, int(checked.sum()), int((well & checked).sum()), TOL[precision],
             TOL["bf16"], int((checked & flipped).sum()), err[keep & well].max(initial=0.0),
             err[keep & ~well].max(initial=0.0), float(np.abs(tm - ref.t).max()),
             *np.quantile(err, [0.5, 0.9, 0.99])), flush=True)
    record(test=label, kind="end to end", mode=end_to_end, rays=int(len(ids_pixels)),
           checked=int(checked.sum()), well_conditioned=int((well & checked).sum()),
           flipped=int((checked & flipped).sum()),
           max_abs_well=float(err[keep & well].max(initial=0.0)), tol_well=TOL[precision],
           max_abs_other=float(err[keep & ~well].max(initial=0.0)), tol_other=TOL["bf16"])
    assert (checked & flipped).sum() <= 0.05 * max(1, checked.sum())
    assert np.all(err[keep] <= tol_ray[keep])


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("sigma_bias", [0.0, 3.0])
def test_hier_tiny_full_frame(precision, sigma_bias):
    """32x32 object-centric frame, 16 coarse + 32 fine samples, 4 heads."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], sigma_bias=sigma_bias)
    sc = scenes.make_scene(cfg)
    gpu = _render(sc, precision, 16, 32)
    ids = np.arange(cfg.num_rays)
    _check_hier(sc, gpu, 16, 32, precision, "hier tiny %s bias %.0f" % (precision, sigma_bias),
                ids, ids, end_to_end="report" if (sigma_bias == 0 and precision == "bf16")
                else "all")


def test_hier_k16_frame_bf16():
    """800x800 object-centric frame, 64 coarse + 128 fine samples, 16 heads of
    8x256: full-frame cells of the emitted depths; fine depths, merged
    composite and pixels on a seeded ray subset plus one image row."""
    cfg = scenes.CONFIGS["hier_k16"]
    sc = scenes.make_scene(cfg)
    gpu = _render(sc, "bf16", cfg.n_coarse, cfg.n_fine)
    ids = scenes.ray_subset(1024, cfg.num_rays)
    row = cfg.height // 2
    ids = np.unique(np.concatenate([ids, np.arange(row * cfg.width, (row + 1) * cfg.width)]))
    _check_hier(sc, gpu, cfg.n_coarse, cfg.n_fine, "bf16", "hier_k16 bf16", ids, ids[::4],
                end_to_end="report")
    assert np.all(np.isfinite(gpu[0]))


def test_hier_k16_dense_bf16():
    """The same frame and heads with a density bias of +2, so that every ray
    is well conditioned for the independent end-to-end comparison."""
    cfg = scenes.with_changes(scenes.CONFIGS["hier_k16"], sigma_bias=2.0)
    sc = scenes.make_scene(cfg)
    ids = scenes.ray_subset(1024, cfg.num_rays)
    lo = (cfg.height // 2) * cfg.width
    rays = (sc.rays_o[lo - 60_000:lo + 60_000].copy(), sc.rays_d[lo - 60_000:lo + 60_000].copy())
    gpu = _render(sc, "bf16", cfg.n_coarse, cfg.n_fine, rays=rays, ray_offset=lo - 60_000)
    ids = np.concatenate([np.arange(0, 120_000, 131), np.arange(60_000, 60_800)])
    ids = np.unique(ids)
    _check_hier(sc, gpu, cfg.n_coarse, cfg.n_fine, "bf16", "hier_k16 dense bf16", ids, ids[::4],
                ray_offset=lo - 60_000, rays=rays, end_to_end="all")


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
def test_hier_forward_facing_slice(precision):
    """Forward-facing NDC rays with 8x128 heads (fp32 and bf16 kernels), 64 +
    128 samples, on a contiguous slice of the frame given by its ray offset."""
    cfg = scenes.with_changes(scenes.CONFIGS["derf_k16"], sigma_bias=2.0)
    sc = scenes.make_scene(cfg)
    lo, hi = 50_000, 54_096
    rays = (sc.rays_o[lo:hi].copy(), sc.rays_d[lo:hi].copy())
    gpu = _render(sc, precision, 64, 128, rays=rays, ray_offset=lo)
    ids = np.arange(0, hi - lo, 8)
    _check_hier(sc, gpu, 64, 128, precision, "hier ndc %s" % precision, ids, ids[::2],
                ray_offset=lo, rays=rays, end_to_end="all")


@pytest.mark.parametrize("nc,nf,n_rays", [(2, 1, 37), (2, 1022, 5), (1000, 24, 3), (5, 7, 200),
                                          (64, 64, 1), (31, 33, 65)])
def test_hier_sample_count_edges(nc, nf, n_rays):
    """Smallest and largest sample lists (1024 merged samples), lists shorter
    and longer than a wave, and ragged ray counts."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], sigma_bias=2.0)
    sc = scenes.make_scene(cfg)
    rays = (sc.rays_o[:n_rays].copy(), sc.rays_d[:n_rays].copy())
    gpu = _render(sc, "fp32", nc, nf, rays=rays)
    ids = np.arange(n_rays)
    _check_hier(sc, gpu, nc, nf, "fp32", "hier edges nc=%d nf=%d R=%d" % (nc, nf, n_rays), ids,
                ids, rays=rays, end_to_end="all")


def test_hier_many_heads_slice():
    """64 skewed heads of 6x64 (walk-table assignment of the given fine depths),
    32 coarse + 32 fine samples, on a contiguous slice of the 1024x1024 frame."""
    cfg = scenes.CONFIGS["skew_k64"]
    sc = scenes.make_scene(cfg)
    lo, hi = 500_000, 504_096
    rays = (sc.rays_o[lo:hi].copy(), sc.rays_d[lo:hi].copy())
    gpu = _render(sc, "fp32", 32, 32, rays=rays, ray_offset=lo)
    ids = np.arange(0, hi - lo, 4)
    _check_hier(sc, gpu, 32, 32, "fp32", "hier K=64 slice", ids, ids[::4], ray_offset=lo,
                rays=rays)


def test_hier_unperturbed_and_transparent():
    """perturb = 0 (stratum midpoints, u_j = (j + 1/2) / n_fine) on heads with
    zero density: every weight is exactly 0 on both sides, so the density is
    the uniform floor and the fine depths must match the oracle to rounding."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], sigma_bias=-50.0)
    sc = scenes.make_scene(cfg)
    gpu = _render(sc, "fp32", 16, 48, perturb=False)
    assert np.all(gpu[3]["sigma"] == 0.0)
    ids = np.arange(cfg.num_rays)
    _check_hier(sc, gpu, 16, 48, "fp32", "hier transparent", ids, ids, perturb=False,
                tol_t=np.spacing(np.float32(cfg.far)), end_to_end="all")
    assert np.all(gpu[2] == 0.0)


def test_hier_batch_invariance_and_determinism():
    """A frame split over two calls (ray offsets) renders as one call, and a
    repeat render is bit-identical."""
    from paper_2011_12490_amd import derf
    cfg = scenes.with_changes(scenes.CONFIGS["derf_k16"], sigma_bias=2.0)
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o[:20_000]).cuda()
    d = torch.from_numpy(sc.rays_d[:20_000]).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, "bf16")
    a = [x.clone() for x in r.render(o, d, cfg.near, cfg.far, 64, 128, 7)]
    b = [x.clone() for x in r.render(o, d, cfg.near, cfg.far, 64, 128, 7)]
    lo = 12_345
    c = r.render(o[lo:].contiguous(), d[lo:].contiguous(), cfg.near, cfg.far, 64, 128, 7,
                 ray_offset=lo)
    torch.cuda.synchronize()
    for x, y, z in zip(a, b, c):
        assert torch.equal(x, y)
        assert torch.equal(x[lo:], z)
    st = derf.derf_get_stats(r.handle)
    assert sum(st.head_samples[:cfg.num_sites]) == (20_000 - lo) * 192
    r.close()
