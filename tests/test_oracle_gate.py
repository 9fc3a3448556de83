"""Pins of the oracle's MLP-gating decomposition (Sec. 4, decompositions with
MLPs) against what the mathematics fixes:

* a gating network built to compute 2 phi_k . x - |phi_k|^2 (hidden units
  ReLU(+x) and ReLU(-x)) picks the nearest site, so its cells equal the
  brute-force Voronoi assignment away from ties and bisectors, and its render
  equals the Voronoi render;
* with one head, or with logits that never depend on x, every sample has
  one head and the render is that of a single-head model;
* a gated cell need not be convex: its render still equals direct
  front-to-back compositing of all samples (over is associative).
"""
import numpy as np
import pytest

import oracle
from paper_2011_12490_amd import scenes


@pytest.fixture(scope="module", autouse=True)
def _oracle():
    oracle.build(force=False)


def _tiny(K=4, rays=48):
    cfg = scenes.with_changes(scenes.CONFIGS["tiny"], num_sites=K, sigma_bias=1.0)
    sc = scenes.make_scene(cfg)
    ids = np.arange(0, cfg.num_rays, cfg.num_rays // rays)[:rays]
    return sc, ids


def voronoi_gate(sites, L, hidden):
    """Gate weights whose logits are 2 phi_k . x - |phi_k|^2."""
    K = sites.shape[0]
    P = 3 + 6 * L
    W1 = np.zeros((hidden, P), np.float32)
    for c in range(3):
        W1[c, c] = 1.0
        W1[3 + c, c] = -1.0
    b1 = np.zeros(hidden, np.float32)
    W2 = np.zeros((K, hidden), np.float32)
    W2[:, 0:3] = 2.0 * sites
    W2[:, 3:6] = -2.0 * sites
    b2 = -(sites.astype(np.float64) ** 2).sum(1).astype(np.float32)
    return np.concatenate([W1.ravel(), b1, W2.ravel(), b2])


def random_gate(K, L, hidden, seed, scale=3.0):
    rng = np.random.default_rng(seed)
    n = oracle.gate_weights_count(K, L, hidden)
    return (rng.uniform(-1, 1, n) * scale / np.sqrt(3 + 6 * L)).astype(np.float32)


def test_gate_weights_count_and_unpack_order():
    K, L, H = 5, 6, 16
    assert oracle.gate_weights_count(K, L, H) == H * 39 + H + K * H + K
    # b2 alone decides when W2 = 0: the packing puts b2 last
    w = np.zeros(oracle.gate_weights_count(K, L, H), np.float32)
    w[-K:] = [0.0, 1.0, 3.0, 2.0, 3.0]
    cells, gap = oracle.gate_assign(K, L, H, w, np.zeros((4, 3), np.float32))
    assert np.all(cells == 2) and np.all(gap == 0.0)  # tie between 2 and 4: lowest index
    with pytest.raises(ValueError):
        oracle.gate_assign(K, L, H, w[:-1], np.zeros((1, 3), np.float32))


def test_gate_logits_match_a_float64_matrix_chain():
    """The logits in the kernel's arithmetic (each float32 operand split into
    two bf16 values, each product a b taken as a_hi b_hi + a_hi b_lo + a_lo
    b_hi) equal a float64 matrix chain on the same float32 encoding within
    that arithmetic's bound: a dropped term and the rounding of the two low
    parts, at most 3.01 * 2^-18 |a b| per product, summed over each dot
    product, the hidden layer's error (and its float32 rounding) carried
    through W2.  The ReLU acts on the hidden units."""
    K, L, H = 7, 6, 32
    w = random_gate(K, L, H, 11, scale=4.0)
    P = 3 + 6 * L
    W1 = w[:H * P].reshape(H, P).astype(np.float64)
    b1 = w[H * P:H * P + H].astype(np.float64)
    W2 = w[H * P + H:H * P + H + K * H].reshape(K, H).astype(np.float64)
    b2 = w[H * P + H + K * H:].astype(np.float64)
    x = np.random.default_rng(3).uniform(-1.2, 1.2, (500, 3)).astype(np.float32)
    z = oracle.gate_logits(K, L, H, w, x)
    g = np.stack([oracle.posenc(L, xi.astype(np.float64)) for xi in x]).astype(np.float32)
    g = g.astype(np.float64)
    pre = g @ W1.T + b1
    h = np.maximum(pre, 0.0)
    ref = h @ W2.T + b2
    rel = 3.01 * 2.0 ** -18
    # hidden-unit error bound, carried through W2, plus the logits' own terms
    eh = rel * (np.abs(g) @ np.abs(W1).T) + 2.0 ** -24 * np.abs(pre)
    bound = rel * ((h + eh) @ np.abs(W2).T) + eh @ np.abs(W2).T
    assert np.all(np.abs(z - ref) <= 1.01 * bound + 1e-12)
    assert np.abs(z - ref).max() > 1e-7         # the split arithmetic, not a float64 copy
    # a missing ReLU, a dropped hidden or output bias, or a swapped encoding
    # block (sin and cos of one level) leaves the bound by far
    assert np.abs(pre @ W2.T + b2 - z).max() > 1e-3
    assert np.abs(np.maximum(g @ W1.T, 0.0) @ W2.T + b2 - z).max() > 1e-3
    assert np.abs(h @ W2.T - z).max() > 1e-3
    gs = g.copy()
    gs[:, 3:6], gs[:, 6:9] = g[:, 6:9], g[:, 3:6]
    assert np.abs(np.maximum(gs @ W1.T + b1, 0.0) @ W2.T + b2 - z).max() > 1e-3


def test_voronoi_gate_picks_the_nearest_site():
    sc, ids = _tiny(K=6)
    cfg = sc.cfg
    L, H = 6, 16
    w = voronoi_gate(sc.sites, L, H)
    t, cell, margin = oracle.sample_assign(sc.sites, sc.rays_o[ids], sc.rays_d[ids], cfg.near,
                                           cfg.far, cfg.n_coarse, scenes.SEED_RENDER, margin=True)
    x = oracle.sample_points(sc.rays_o[ids], sc.rays_d[ids], t)
    gcell, gap = oracle.gate_assign(cfg.num_sites, L, H, w, x.reshape(-1, 3))
    ok = (margin.ravel() >= 1e-5) & (gap >= 1e-4)
    assert ok.mean() > 0.99
    assert np.array_equal(gcell[ok], cell.ravel()[ok])
    # a sign slip in the -x units moves many samples
    w_bad = w.copy()
    P = 3 + 6 * L
    w_bad[(3 * P):(3 * P) + P] *= -1.0
    bad, _ = oracle.gate_assign(cfg.num_sites, L, H, w_bad, x.reshape(-1, 3))
    assert (bad[ok] != cell.ravel()[ok]).mean() > 0.05


def test_voronoi_gate_render_is_the_voronoi_render():
    sc, ids = _tiny(K=5, rays=24)
    cfg = sc.cfg
    L, H = 6, 16
    w = voronoi_gate(sc.sites, L, H)
    g = oracle.render_gated(cfg.arch, sc.weights, cfg.num_sites, L, H, w, sc.rays_o[ids],
                            sc.rays_d[ids], cfg.near, cfg.far, cfg.n_coarse,
                            seed=scenes.SEED_RENDER, ray_ids=ids)
    v = oracle.render(sc.sites, cfg.arch, sc.weights, sc.rays_o[ids], sc.rays_d[ids], cfg.near,
                      cfg.far, cfg.n_coarse, seed=scenes.SEED_RENDER, ray_ids=ids,
                      per_sample=True)
    same = np.all(g.cell == v.cell, axis=1)
    assert same.mean() > 0.9
    assert np.array_equal(g.t, v.t)
    assert np.abs(g.rgb[same] - v.rgb[same]).max() < 1e-6
    assert np.abs(g.depth[same] - v.depth[same]).max() < 1e-6
    assert np.abs(g.opacity[same] - v.opacity[same]).max() < 1e-6


def test_one_head_or_constant_logits_is_a_single_head_render():
    sc1, ids = _tiny(K=1, rays=16)
    cfg = sc1.cfg
    L, H = 6, 16
    w = random_gate(1, L, H, 7)
    g = oracle.render_gated(cfg.arch, sc1.weights, 1, L, H, w, sc1.rays_o[ids], sc1.rays_d[ids],
                            cfg.near, cfg.far, cfg.n_coarse, seed=scenes.SEED_RENDER,
                            ray_ids=ids)
    p = oracle.render(sc1.sites, cfg.arch, sc1.weights, sc1.rays_o[ids], sc1.rays_d[ids],
                      cfg.near, cfg.far, cfg.n_coarse, seed=scenes.SEED_RENDER, ray_ids=ids,
                      mode="plain")
    assert np.all(g.cell == 0)
    assert np.abs(g.rgb - p.rgb).max() < 1e-6 and np.abs(g.opacity - p.opacity).max() < 1e-6
    # K = 4 with W2 = 0 and b2 largest for head 3: every sample is head 3's,
    # which renders like a one-head model with head 3's weights
    sc4, _ = _tiny(K=4, rays=16)
    w4 = random_gate(4, L, H, 8)
    w4[-4 - 4 * H:-4] = 0.0
    w4[-4:] = [0.0, 0.5, -1.0, 2.0]
    g4 = oracle.render_gated(cfg.arch, sc4.weights, 4, L, H, w4, sc4.rays_o[ids],
                             sc4.rays_d[ids], cfg.near, cfg.far, cfg.n_coarse,
                             seed=scenes.SEED_RENDER, ray_ids=ids)
    w3 = np.ascontiguousarray(sc4.weights, np.float32).reshape(4, -1)[3]
    p3 = oracle.render(sc1.sites, cfg.arch, w3, sc4.rays_o[ids], sc4.rays_d[ids], cfg.near,
                       cfg.far, cfg.n_coarse, seed=scenes.SEED_RENDER, ray_ids=ids, mode="plain")
    assert np.all(g4.cell == 3)
    assert np.abs(g4.rgb - p3.rgb).max() < 1e-6 and np.abs(g4.depth - p3.depth).max() < 1e-6


def test_nonconvex_gated_cells_composite_like_direct():
    sc, ids = _tiny(K=4, rays=12)
    cfg = sc.cfg
    L, H = 6, 32
    w = random_gate(4, L, H, 9, scale=8.0)
    g = oracle.render_gated(cfg.arch, sc.weights, 4, L, H, w, sc.rays_o[ids], sc.rays_d[ids],
                            cfg.near, cfg.far, cfg.n_coarse, seed=scenes.SEED_RENDER,
                            ray_ids=ids)
    # the gate re-enters cells: more runs than distinct cells on some ray
    runs = [(1 + np.count_nonzero(np.diff(c))) for c in g.cell]
    distinct = [len(set(c.tolist())) for c in g.cell]
    assert any(r > d for r, d in zip(runs, distinct))
    wk = np.ascontiguousarray(sc.weights, np.float32).reshape(4, -1)
    for r in range(len(ids)):
        x = oracle.sample_points(sc.rays_o[ids[r]], sc.rays_d[ids[r]], g.t[r])
        dv = sc.rays_d[ids[r]].astype(np.float64)
        gd = oracle.posenc(cfg.arch.dir_freqs, dv / np.sqrt(dv @ dv))
        sig = np.zeros(cfg.n_coarse)
        col = np.zeros((cfg.n_coarse, 3))
        for i in range(cfg.n_coarse):
            sig[i], col[i] = oracle.head_eval(cfg.arch, wk[g.cell[r, i]],
                                              oracle.posenc(cfg.arch.pos_freqs, x[i]), gd)
        rgb, dep, op, _ = oracle.composite(g.cell[r], g.t[r], sig, col, cfg.near, cfg.far,
                                           mode="direct")
        assert np.abs(rgb - g.rgb[r]).max() < 1e-9 and abs(op - g.opacity[r]) < 1e-9
        assert abs(dep - g.depth[r]) < 1e-9
