"""The stored positional encoding (derf_set_encoding): a separate pass writes
every sample's gamma(x) (Sec. 4, the heads' input encoding) to a table and the
grouped MLP reads it back instead of encoding in its tile prologue.

Bars: the stored form's outputs equal the fused form's bit for bit (same
entries, same rounding, same matrix-core order), per sample and per pixel, on
both passes of hierarchical sampling too; and on a ray subset against the
oracle within the fused path's tolerances.  Handles it cannot serve refuse it.
"""
import os

import numpy as np
import pytest

import oracle
from paper_2011_12490_amd import scenes

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}
NTHREADS = min(16, os.cpu_count() or 1)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)
    torch.cuda.set_device(0)


def _derf():
    from paper_2011_12490_amd import derf
    return derf


def _cpu(out):
    return [x.cpu().numpy() if torch.is_tensor(x) else {k: v.cpu().numpy() for k, v in x.items()}
            for x in out]


def _both(r, o, d, cfg, n, nf, debug=True):
    """(fused, stored) outputs of one handle on the same rays."""
    r.set_encoding(False)
    fused = _cpu(r.render(o, d, cfg.near, cfg.far, n, nf, scenes.SEED_RENDER, debug=debug))
    r.set_encoding(True)
    stored = _cpu(r.render(o, d, cfg.near, cfg.far, n, nf, scenes.SEED_RENDER, debug=debug))
    torch.cuda.synchronize()
    return fused, stored


def _assert_bitwise(fused, stored, label):
    for name, a, b in zip(("rgb", "depth", "opacity"), fused[:3], stored[:3]):
        assert np.array_equal(a, b), "%s: %s differs (max %.3g)" % (label, name,
                                                                     np.abs(a - b).max())
    if len(fused) > 3:
        for k in fused[3]:
            assert np.array_equal(fused[3][k], stored[3][k]), "%s: per-sample %s" % (label, k)
    print("%s: stored == fused bitwise (%d rays)" % (label, fused[0].shape[0]), flush=True)


# A frame of the skewed workload's kind (object-centric rays, heads of 6x64
# with a 10-frequency encoding and no skip layer), cut to 37 x 29 rays and 45
# samples: 1073 rays, 48285 samples, a ragged last tile in every head.
def _skew_small():
    return scenes.with_changes(scenes.CONFIGS["skew_k64"], width=37, height=29, n_coarse=45,
                               num_sites=12)


@pytest.mark.parametrize("precision", ["fp32", "bf16"])
@pytest.mark.parametrize("which", ["tiny", "skew_small"])
def test_stored_encoding_equals_fused(which, precision):
    derf = _derf()
    cfg = scenes.CONFIGS["tiny"] if which == "tiny" else _skew_small()
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, precision)
    fused, stored = _both(r, o, d, cfg, cfg.n_coarse, 0)
    r.close()
    _assert_bitwise(fused, stored, "%s %s" % (which, precision))
    ids = scenes.ray_subset(96, cfg.num_rays)
    ref = oracle.render(sc.sites, cfg.arch, sc.weights, sc.rays_o[ids], sc.rays_d[ids], cfg.near,
                        cfg.far, cfg.n_coarse, 0, seed=scenes.SEED_RENDER, ray_ids=ids,
                        nthreads=NTHREADS)
    err = max(np.abs(stored[0][ids] - ref.rgb).max(), np.abs(stored[1][ids] - ref.depth).max(),
              np.abs(stored[2][ids] - ref.opacity).max())
    print("%s %s stored vs oracle: max abs %.3g (tol %.0e)" % (which, precision, err,
                                                                TOL[precision]))
    assert err <= TOL[precision]


def test_stored_encoding_hierarchical_and_empty():
    """Both passes of hierarchical sampling read the table (coarse and fine
    samples written in turn), on a frame of 1000 rays; an empty render is a
    no-op; switching back gives the fused form again."""
    derf = _derf()
    cfg = scenes.with_changes(_skew_small(), width=40, height=25, n_coarse=24, n_fine=40)
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, "bf16")
    fused, stored = _both(r, o, d, cfg, 24, 40)
    _assert_bitwise(fused, stored, "skew_small 24+40 bf16")
    r.set_encoding(True)
    z = torch.empty((0, 3), dtype=torch.float32, device="cuda")
    out = r.render(z, z, cfg.near, cfg.far, 24, 0, scenes.SEED_RENDER)
    assert out[0].shape == (0, 3)
    r.set_encoding(False)
    again = _cpu(r.render(o, d, cfg.near, cfg.far, 24, 40, scenes.SEED_RENDER, debug=True))
    r.close()
    _assert_bitwise(fused, again, "skew_small fused again")


def test_stored_encoding_refused_where_it_has_no_form():
    """Heads with a skip layer, and mixed heads whose encodings differ, have no
    stored form: the setting fails and stays fused.  With it set, the soft,
    culled and gated renders refuse to run."""
    derf = _derf()
    cfg = scenes.CONFIGS["tiny"]
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    w128 = scenes.make_weights(scenes.ARCH_128, cfg.num_sites, seed=11)
    r = derf.Renderer(sc.sites, scenes.ARCH_128, w128, "bf16")
    with pytest.raises(derf.DerfError) as e:
        r.set_encoding(True)
    assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    r.render(o, d, cfg.near, cfg.far, 16, 0, scenes.SEED_RENDER)  # still fused
    r.close()

    archs = [(scenes.ARCH_TINY, scenes.ARCH_SMALL)[k % 2] for k in range(cfg.num_sites)]
    ws = [scenes.make_weights(a, 1, seed=600 + k)[0] for k, a in enumerate(archs)]
    r = derf.Renderer(sc.sites, archs, ws, "fp32")
    with pytest.raises(derf.DerfError) as e:
        r.set_encoding(True)
    assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    r.close()

    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, "fp32")
    with pytest.raises(derf.DerfError) as e:
        derf.derf_set_encoding(r.handle, 7)
    assert e.value.status == derf.DERF_ERR_INVALID_ARG
    r.set_encoding(True)
    calls = (lambda: r.render_soft(o, d, cfg.near, cfg.far, 16, 3.0, scenes.SEED_RENDER),
             lambda: r.render_culled(o, d, cfg.near, cfg.far, 16, 1e-3, 4, scenes.SEED_RENDER))
    for call in calls:
        with pytest.raises(derf.DerfError) as e:
            call()
        assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    gate = np.zeros(derf.lib().derf_gate_weights_count(cfg.num_sites, 6, 16), np.float32)
    r.set_gate(6, 16, gate)
    with pytest.raises(derf.DerfError) as e:
        r.render_gated(o, d, cfg.near, cfg.far, 16, scenes.SEED_RENDER)
    assert e.value.status == derf.DERF_ERR_UNSUPPORTED
    torch.cuda.synchronize()
    r.close()


def test_stored_encoding_in_the_no_allocation_render():
    """The table lives in the no-allocation render's fixed scratch array too:
    a small frame renders there bit for bit as with the fused form, and a
    frame whose table no longer fits is refused where the fused form's
    workspace still fits."""
    derf = _derf()
    cfg = scenes.with_changes(_skew_small(), width=32, height=32, n_coarse=32)
    sc = scenes.make_scene(cfg)
    o = torch.from_numpy(sc.rays_o).cuda()
    d = torch.from_numpy(sc.rays_d).cuda()
    R = o.shape[0]
    r = derf.Renderer(sc.sites, cfg.arch, sc.weights, "bf16")
    samp = derf.derf_sampling(cfg.n_coarse, 0, scenes.SEED_RENDER, 1, 0)

    def outs(n):
        return (torch.empty((n, 3), device="cuda"), torch.empty((n,), device="cuda"),
                torch.empty((n,), device="cuda"))

    fused, stored = outs(R), outs(R)
    r.set_encoding(False)
    derf.derf_render_noalloc(r.handle, o, d, cfg.near, cfg.far, samp, *fused)
    r.set_encoding(True)
    derf.derf_render_noalloc(r.handle, o, d, cfg.near, cfg.far, samp, *stored)
    torch.cuda.synchronize()
    for a, b in zip(fused, stored):
        assert torch.equal(a, b)
    # 49,152 rays x 32 samples: the fused form's 30 B or so per sample fit
    # the 64 MiB array, with the table's 128 B more they do not
    big_o = o.repeat(48, 1)
    big_d = d.repeat(48, 1)
    big = outs(big_o.shape[0])
    big_samp = derf.derf_sampling(32, 0, scenes.SEED_RENDER, 1, 0)
    with pytest.raises(derf.DerfError) as e:
        derf.derf_render_noalloc(r.handle, big_o, big_d, cfg.near, cfg.far, big_samp, *big)
    assert e.value.status == derf.DERF_ERR_INVALID_ARG
    r.set_encoding(False)
    derf.derf_render_noalloc(r.handle, big_o, big_d, cfg.near, cfg.far, big_samp, *big)
    torch.cuda.synchronize()
    r.close()
