"""GPU parity of the MLP-gating decomposition (derf_set_gate /
derf_render_gated, Sec. 4 decompositions with MLPs) against the CPU
oracle's gated render, through the C ABI.

Both sides take the argmax in fp32, but their encodings of x may differ in
the last bit, so samples whose two largest oracle logits are within 1e-4 are
excluded from the bit-exact cell comparison and counted, as samples near a
bisector are for the nearest site.  Pixels of rays with no excluded sample
match within max-abs 1e-4 (fp32) / 2e-2 (bf16).
"""
import numpy as np
import pytest

import oracle
from paper_2011_12490_amd import scenes
from parity_log import record
from test_oracle_gate import random_gate, voronoi_gate

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}
GAP = 1e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)
    torch.cuda.set_device(0)


def _derf():
    from paper_2011_12490_amd import derf
    return derf


def _run(sc, precision, L, H, gw, ids, label, empty=None):
    """empty: optional [K] flags of 0-capacity heads on the GPU; the oracle
    then renders those heads with zero weights (the same render, bitwise, in
    the oracle's own pins)."""
    derf = _derf()
    cfg = sc.cfg
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
    weights = sc.weights
    if empty is not None:
        r.set_empty_heads(list(empty))
        weights = np.array(sc.weights, np.float32).reshape(cfg.num_sites, -1)
        weights[np.asarray(empty, bool)] = 0.0
    r.set_gate(L, H, gw)
    rgb, depth, opac, cell = r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse,
                                            seed=scenes.SEED_RENDER, cells=True)
    torch.cuda.synchronize()
    r.close()
    rgb, depth, opac, cell = [x.cpu().numpy() for x in (rgb, depth, opac, cell)]
    ref = oracle.render_gated(cfg.arch, weights, cfg.num_sites, L, H, gw, sc.rays_o[ids],
                              sc.rays_d[ids], cfg.near, cfg.far, cfg.n_coarse,
                              seed=scenes.SEED_RENDER, ray_ids=ids)
    ok = ref.gap >= GAP
    assert np.array_equal(cell[ids][ok], ref.cell[ok])
    clean = ok.all(axis=1)
    err = max(np.abs(rgb[ids] - ref.rgb)[clean].max(), np.abs(depth[ids] - ref.depth)[clean].max(),
              np.abs(opac[ids] - ref.opacity)[clean].max())
    runs = np.mean([1 + np.count_nonzero(np.diff(c)) for c in ref.cell])
    print("%s: rays=%d near-tie samples=%d clean rays=%d runs/ray=%.2f max|d|=%.3g (tol %.0e)"
          % (label, len(ids), int((~ok).sum()), int(clean.sum()), runs, err, TOL[precision]),
          flush=True)
    record(test=label, kind="gated cells and pixels", rays=int(len(ids)),
           near_tie_samples=int((~ok).sum()), clean_rays=int(clean.sum()),
           runs_per_ray=float(runs), max_abs=float(err), tol=TOL[precision])
    assert clean.mean() > 0.9
    assert err <= TOL[precision]
    assert np.all((cell >= 0) & (cell < cfg.num_sites))
    return cell


@pytest.mark.parametrize("H,scale", [(16, 3.0), (32, 8.0), (64, 3.0)])
def test_gated_tiny_fp32(H, scale):
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=8, sigma_bias=1.0)
    sc = scenes.make_scene(cfg)
    gw = random_gate(8, 6, H, 100 + H, scale=scale)
    _run(sc, "fp32", 6, H, gw, np.arange(0, cfg.num_rays, 4), "gated tiny K=8 H=%d" % H)


def test_voronoi_gate_matches_the_nearest_site_render_fp32():
    """A gate computing 2 phi_k . x - |phi_k|^2 gives the Voronoi cells."""
    derf = _derf()
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=6, sigma_bias=1.0)
    sc = scenes.make_scene(cfg)
    gw = voronoi_gate(sc.sites, 6, 16)
    cell = _run(sc, "fp32", 6, 16, gw, np.arange(0, cfg.num_rays, 8), "voronoi gate K=6")
    t, vcell, margin = oracle.sample_assign(sc.sites, sc.rays_o, sc.rays_d, cfg.near, cfg.far,
                                            cfg.n_coarse, scenes.SEED_RENDER, margin=True)
    ok = margin >= 1e-5
    assert (cell[ok] == vcell[ok]).mean() > 0.999


def test_gated_ragged_and_many_heads_fp32():
    """K = 40 (the per-ray walk assigns first, then the gate overwrites),
    67 samples per ray and a ragged ray count."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=40, sigma_bias=1.0, n_coarse=67)
    sc = scenes.make_scene(cfg)
    keep = 1000
    sc.rays_o, sc.rays_d = sc.rays_o[:keep].copy(), sc.rays_d[:keep].copy()
    gw = random_gate(40, 6, 32, 77, scale=6.0)
    _run(sc, "fp32", 6, 32, gw, np.arange(0, keep, 9), "gated K=40 n=67 R=1000")


def test_gated_256_heads_and_empty_heads_fp32():
    """K = 256 (cells use all 8 bits), a quarter of the heads 0-capacity."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=256, sigma_bias=1.0)
    sc = scenes.make_scene(cfg)
    empty = np.zeros(256, int)
    empty[::4] = 1
    gw = random_gate(256, 6, 16, 31, scale=6.0)
    cell = _run(sc, "fp32", 6, 16, gw, np.arange(0, cfg.num_rays, 8), "gated K=256, empty heads",
                empty=empty)
    assert len(np.unique(cell)) > 128


@pytest.mark.parametrize("n", [1, 2, 12])
def test_gated_sample_counts_fp32(n):
    """1 and 2 samples per ray (each lane draws its own jitter), and 12 (four
    samples share a Philox block, drawn once per four lanes), on 31 x 33
    rays, so that with 12 samples the last 256-sample stretch of the gate is
    partial."""
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=8, sigma_bias=1.0, n_coarse=n,
                              width=31, height=33)
    sc = scenes.make_scene(cfg)
    gw = random_gate(8, 6, 32, 41, scale=6.0)
    _run(sc, "fp32", 6, 32, gw, np.arange(0, cfg.num_rays, 4), "gated n=%d" % n)


def test_gated_headline_frame_bf16():
    """The 504x378 frame with 16 heads of 8x128 (bf16) and a gate on
    gamma_10(x) with 32 hidden units: a ray subset against the oracle."""
    cfg = scenes.CONFIGS["derf_k16"]
    sc = scenes.make_scene(cfg)
    gw = random_gate(16, 10, 32, 5, scale=4.0)
    _run(sc, "bf16", 10, 32, gw, scenes.ray_subset(96, cfg.num_rays), "gated derf_k16 bf16")


def test_gated_errors_and_gate_removal():
    derf = _derf()
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=4)
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, "fp32")
    with pytest.raises(derf.DerfError) as e:
        r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse)
    assert e.value.status == derf.DERF_ERR_INVALID_ARG
    gw = random_gate(4, 6, 16, 3)
    for L, H in ((6, 24), (4, 16)):
        with pytest.raises(derf.DerfError) as e:
            r.set_gate(L, H, np.zeros(oracle.gate_weights_count(4, L, H), np.float32))
        assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    bad = gw.copy()
    bad[5] = np.nan
    with pytest.raises(derf.DerfError) as e:
        r.set_gate(6, 16, bad)
    assert e.value.status == derf.DERF_ERR_INVALID_ARG
    r.set_gate(6, 16, gw)
    out = [torch.empty((o.shape[0], 3), device="cuda"), torch.empty(o.shape[0], device="cuda"),
           torch.empty(o.shape[0], device="cuda")]
    with pytest.raises(derf.DerfError) as e:
        derf.derf_render_gated(r.handle, o, d, cfg.near, cfg.far,
                               derf.derf_sampling(16, 16, 1, 1, 0), *out)
    assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    a = r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse, seed=1)
    b = r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse, seed=1)
    empty = r.render_gated(o[:0], d[:0], cfg.near, cfg.far, cfg.n_coarse, seed=1)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x, y)
    assert empty[0].shape == (0, 3)
    r.set_gate(6, 0, None)
    with pytest.raises(derf.DerfError):
        r.render_gated(o, d, cfg.near, cfg.far, cfg.n_coarse)
    torch.cuda.synchronize()
    r.close()
