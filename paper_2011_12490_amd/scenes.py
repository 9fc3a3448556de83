"""Seeded synthetic scenes for the DeRF renderer.

This module produces inputs only: Voronoi sites, per-head MLP weights in the
packed per-head layout of ``include/derf.h``, and camera rays.  It holds none
of the renderer's arithmetic (no sampling, no nearest-site assignment of ray
samples, no network evaluation, no compositing), so both the CPU oracle and
the GPU library can be fed from it.

Stand-ins for the paper's data (DeRF, Rebain et al., Sec. 4.1 uses the
"Real Forward-Facing" scenes; its Table 1 / Table 2 time "fern" and "room"):
the datasets and trained weights are not available, so every scene here is
synthetic and seeded:

* sites: uniform in the cube, a Gaussian-mixture + k-means placement (a
  trained decomposition concentrates sites where the content is), or a skewed
  ball + cube mix; all sites lie in [-1, 1]^3 as Sec. 3.4 ("parameter
  magnitude scaling") prescribes;
* weights: Glorot-uniform, biases zero (density bias configurable);
* rays: a pinhole camera, either forward-facing with the NDC ray mapping of
  NeRF (near plane 1, so depths run over [0, 1]) or object-centric on a sphere
  of radius 4 looking at the origin.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence

import numpy as np

#: Master seed; every sub-seed is derived from it by a fixed offset.
S0 = 2011_12490
SEED_SITES = S0 + 1
SEED_WEIGHTS = S0 + 2
SEED_CAMERA = S0 + 3
SEED_GMM = S0 + 4
SEED_KMEANS = S0 + 5
SEED_RENDER = S0 + 6


@dataclasses.dataclass(frozen=True)
class HeadArch:
    """Architecture shared by every head (the paper uses homogeneous heads).

    ``pos_freqs``/``dir_freqs`` are the positional-encoding frequency counts
    L of gamma(x) and gamma(d); the encodings have 3 + 6L entries.
    ``skip_layer`` is the 0-based hidden layer whose input is
    [gamma(x); h] (-1: none).  ``rgb_hidden`` is the width of the hidden
    layer of the colour branch (0: colour is read directly from [h; gamma(d)]).
    """

    pos_freqs: int
    dir_freqs: int
    depth: int
    width: int
    skip_layer: int
    rgb_hidden: int

    @property
    def pos_dim(self) -> int:
        return 3 + 6 * self.pos_freqs

    @property
    def dir_dim(self) -> int:
        return 3 + 6 * self.dir_freqs

    def layer_shapes(self):
        """(out, in) of every matrix in packing order, with a tag."""
        shapes = []
        for l in range(self.depth):
            if l == 0:
                fan_in = self.pos_dim
            elif l == self.skip_layer:
                fan_in = self.pos_dim + self.width
            else:
                fan_in = self.width
            shapes.append(("hidden%d" % l, self.width, fan_in))
        shapes.append(("sigma", 1, self.width))
        if self.rgb_hidden > 0:
            shapes.append(("rgb_hidden", self.rgb_hidden, self.width + self.dir_dim))
            shapes.append(("rgb_out", 3, self.rgb_hidden))
        else:
            shapes.append(("rgb_out", 3, self.width + self.dir_dim))
        return shapes

    def weights_count(self) -> int:
        """Floats per head: every matrix (out x in, row-major) followed by its bias."""
        return sum(o * i + o for _, o, i in self.layer_shapes())

    def macs_per_sample(self) -> int:
        """Multiply-accumulates of one head evaluation (no padding)."""
        return sum(o * i for _, o, i in self.layer_shapes())

    def as_tuple(self):
        return (self.pos_freqs, self.dir_freqs, self.depth, self.width,
                self.skip_layer, self.rgb_hidden)


@dataclasses.dataclass(frozen=True)
class SceneConfig:
    name: str
    width: int                # image width in pixels
    height: int               # image height in pixels
    camera: str               # "forward" (NDC) or "object"
    fov_x_deg: float
    near: float
    far: float
    n_coarse: int
    n_fine: int
    num_sites: int
    sites: str                # "uniform", "gmm_kmeans", "ball_mix", "origin"
    arch: HeadArch
    precision: str            # "fp32" or "bf16"
    sigma_bias: float = 0.0   # density output bias of every head

    @property
    def num_rays(self) -> int:
        return self.width * self.height

    @property
    def samples_per_ray(self) -> int:
        return self.n_coarse + self.n_fine


ARCH_TINY = HeadArch(pos_freqs=6, dir_freqs=4, depth=4, width=64, skip_layer=-1, rgb_hidden=0)
ARCH_NERF = HeadArch(pos_freqs=10, dir_freqs=4, depth=8, width=256, skip_layer=5, rgb_hidden=128)
ARCH_128 = HeadArch(pos_freqs=10, dir_freqs=4, depth=8, width=128, skip_layer=5, rgb_hidden=64)
ARCH_SMALL = HeadArch(pos_freqs=10, dir_freqs=4, depth=6, width=64, skip_layer=-1, rgb_hidden=32)

CONFIGS = {
    # 32x32 tiny scene, 4 uniform sites, fp32.
    "tiny": SceneConfig("tiny", 32, 32, "object", 40.0, 2.0, 6.0, 32, 0, 4,
                        "uniform", ARCH_TINY, "fp32"),
    # NeRF-equivalent single head on the forward-facing 504x378 frame.
    "nerf_k1": SceneConfig("nerf_k1", 504, 378, "forward", 60.0, 0.0, 1.0, 192, 0, 1,
                           "origin", ARCH_NERF, "bf16"),
    # 16 heads of 8x128 on the same frame: the headline workload.
    "derf_k16": SceneConfig("derf_k16", 504, 378, "forward", 60.0, 0.0, 1.0, 192, 0, 16,
                            "gmm_kmeans", ARCH_128, "bf16"),
    # 800x800 object-centric, 64 coarse + 128 fine, 16 heads of 8x256.
    "hier_k16": SceneConfig("hier_k16", 800, 800, "object", 40.0, 2.0, 6.0, 64, 128, 16,
                            "gmm_kmeans", ARCH_NERF, "bf16"),
    # The headline frame with the grid decomposition: 64 heads of 8x128 whose
    # cells are a fixed 4x4x4 lattice over [-1, 1]^3 (DeRF-Grid).
    "grid_k64": SceneConfig("grid_k64", 504, 378, "forward", 60.0, 0.0, 1.0, 192, 0, 64,
                            "grid", ARCH_128, "bf16"),
    # The headline frame with a density bias of +16: every ray turns opaque
    # part-way (a stand-in for the opaque surfaces of captured scenes), the
    # workload of Painter's-order culling.
    "dense_k16": SceneConfig("dense_k16", 504, 378, "forward", 60.0, 0.0, 1.0, 192, 0, 16,
                             "gmm_kmeans", ARCH_128, "bf16", sigma_bias=16.0),
    # 1024x1024, 256 samples, 64 skewed heads of 6x64, density bias +2.
    "skew_k64": SceneConfig("skew_k64", 1024, 1024, "object", 40.0, 2.0, 6.0, 256, 0, 64,
                            "ball_mix", ARCH_SMALL, "bf16", sigma_bias=2.0),
}


def with_changes(cfg: SceneConfig, **kw) -> SceneConfig:
    return dataclasses.replace(cfg, **kw)


# ---------------------------------------------------------------- sites ----

def _gmm_points(n_points: int, rng: np.random.Generator) -> np.ndarray:
    comps = 8
    means = rng.uniform(-0.6, 0.6, size=(comps, 3))
    stds = rng.uniform(0.08, 0.25, size=comps)
    which = rng.integers(0, comps, size=n_points)
    pts = means[which] + rng.standard_normal((n_points, 3)) * stds[which, None]
    return pts


def _kmeans(points: np.ndarray, k: int, iters: int, rng: np.random.Generator) -> np.ndarray:
    """Lloyd's algorithm in float64; an empty cluster keeps its centre."""
    init = rng.permutation(points.shape[0])[:k]
    centres = points[init].copy()
    for _ in range(iters):
        # squared distances point x centre, chunked to bound memory
        labels = np.empty(points.shape[0], dtype=np.int64)
        for s in range(0, points.shape[0], 16384):
            p = points[s:s + 16384]
            d2 = ((p[:, None, :] - centres[None, :, :]) ** 2).sum(-1)
            labels[s:s + 16384] = np.argmin(d2, axis=1)
        for j in range(k):
            m = labels == j
            if m.any():
                centres[j] = points[m].mean(0)
    return np.clip(centres, -1.0, 1.0)


def make_sites(kind: str, k: int, seed: int = SEED_SITES) -> np.ndarray:
    """Voronoi sites as float32 [k, 3], all inside [-1, 1]^3."""
    if kind == "origin":
        return np.zeros((k, 3), np.float32) if k == 1 else make_sites("uniform", k, seed)
    if kind == "uniform":
        rng = np.random.Generator(np.random.PCG64(seed))
        return rng.uniform(-1.0, 1.0, size=(k, 3)).astype(np.float32)
    if kind == "gmm_kmeans":
        pts = _gmm_points(100_000, np.random.Generator(np.random.PCG64(SEED_GMM)))
        c = _kmeans(pts, k, 10, np.random.Generator(np.random.PCG64(SEED_KMEANS)))
        return c.astype(np.float32)
    if kind == "ball_mix":
        rng = np.random.Generator(np.random.PCG64(seed))
        n_ball = int(round(0.8 * k))
        # uniform in a ball of radius 0.3: direction x radius^(1/3)
        v = rng.standard_normal((n_ball, 3))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        r = 0.3 * rng.uniform(0.0, 1.0, size=(n_ball, 1)) ** (1.0 / 3.0)
        ball = v * r
        cube = rng.uniform(-1.0, 1.0, size=(k - n_ball, 3))
        return np.concatenate([ball, cube]).astype(np.float32)
    if kind == "grid":
        # a regular lattice of n^3 cell centres: the grid decomposition is the
        # Voronoi diagram of these sites
        n = round(k ** (1.0 / 3.0))
        if n ** 3 != k:
            raise ValueError("grid needs a cube number of sites")
        c = (np.arange(n) + 0.5) / n * 2.0 - 1.0
        g = np.stack(np.meshgrid(c, c, c, indexing="ij"), -1).reshape(-1, 3)
        return g.astype(np.float32)
    raise ValueError("unknown site placement %r" % kind)


# -------------------------------------------------------------- weights ----

def make_weights(arch: HeadArch, k: int, seed: int = SEED_WEIGHTS,
                 sigma_bias: float = 0.0) -> np.ndarray:
    """Glorot-uniform weights of k heads as float32 [k, weights_count].

    Per head, in order: every hidden layer's W [out][in] then b [out]; the
    density row w_sigma [W] then b_sigma; the colour branch (hidden W_v, b_v
    then W_c, b_c, or W_c, b_c alone).  Concatenated inputs are ordered
    [gamma(x); h] for the skip layer and [h; gamma(d)] for the colour branch.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    out = np.zeros((k, arch.weights_count()), np.float32)
    for h in range(k):
        pos = 0
        for tag, o, i in arch.layer_shapes():
            lim = math.sqrt(6.0 / (i + o))
            out[h, pos:pos + o * i] = rng.uniform(-lim, lim, size=o * i)
            pos += o * i
            if tag == "sigma":
                out[h, pos] = sigma_bias
            pos += o
        assert pos == arch.weights_count()
    return out


def weight_views(arch: HeadArch, flat: np.ndarray):
    """Split one head's packed float vector into named (W, b) pairs."""
    views = {}
    pos = 0
    for tag, o, i in arch.layer_shapes():
        W = flat[pos:pos + o * i].reshape(o, i)
        pos += o * i
        b = flat[pos:pos + o]
        pos += o
        views[tag] = (W, b)
    return views


# ----------------------------------------------------------------- rays ----

def _pixel_dirs(width: int, height: int, fov_x_deg: float):
    focal = 0.5 * width / math.tan(0.5 * math.radians(fov_x_deg))
    i, j = np.meshgrid(np.arange(width, dtype=np.float64) + 0.5,
                       np.arange(height, dtype=np.float64) + 0.5, indexing="xy")
    # camera looks down -z, y up (OpenGL convention)
    dirs = np.stack([(i - 0.5 * width) / focal, -(j - 0.5 * height) / focal,
                     -np.ones_like(i)], -1).reshape(-1, 3)
    return dirs, focal


def _rot_x(a):
    c, s = math.cos(a), math.sin(a)
    return np.array([[1, 0, 0], [0, c, -s], [0, s, c]], np.float64)


def _rot_y(a):
    c, s = math.cos(a), math.sin(a)
    return np.array([[c, 0, s], [0, 1, 0], [-s, 0, c]], np.float64)


def ndc_rays(o: np.ndarray, d: np.ndarray, width: int, height: int, focal: float,
             near_plane: float = 1.0):
    """NeRF's normalised-device-coordinate ray mapping for forward-facing
    captures (NeRF, Mildenhall et al., appendix): rays are moved to the near
    plane and mapped so that depth t' in [0, 1] spans near plane .. infinity."""
    t = -(near_plane + o[:, 2]) / d[:, 2]
    o = o + t[:, None] * d
    ox, oy, oz = o[:, 0], o[:, 1], o[:, 2]
    dx, dy, dz = d[:, 0], d[:, 1], d[:, 2]
    fx = -focal / (0.5 * width)
    fy = -focal / (0.5 * height)
    o_n = np.stack([fx * ox / oz, fy * oy / oz, 1.0 + 2.0 * near_plane / oz], -1)
    d_n = np.stack([fx * (dx / dz - ox / oz), fy * (dy / dz - oy / oz),
                    -2.0 * near_plane / oz], -1)
    return o_n, d_n


def make_rays(cfg: SceneConfig, seed: int = SEED_CAMERA):
    """Ray origins and directions, float32 [R, 3] each."""
    rng = np.random.Generator(np.random.PCG64(seed))
    dirs_cam, focal = _pixel_dirs(cfg.width, cfg.height, cfg.fov_x_deg)
    if cfg.camera == "forward":
        yaw = math.radians(rng.uniform(-5.0, 5.0))
        pitch = math.radians(rng.uniform(-5.0, 5.0))
        R = _rot_y(yaw) @ _rot_x(pitch)
        centre = rng.uniform(-0.05, 0.05, size=3)
        d = dirs_cam @ R.T
        d /= np.linalg.norm(d, axis=1, keepdims=True)
        o = np.broadcast_to(centre, d.shape).copy()
        o, d = ndc_rays(o, d, cfg.width, cfg.height, focal)
    elif cfg.camera == "object":
        az = rng.uniform(0.0, 2.0 * math.pi)
        el = math.radians(rng.uniform(15.0, 45.0))
        pos = 4.0 * np.array([math.cos(el) * math.cos(az), math.cos(el) * math.sin(az),
                              math.sin(el)])
        fwd = -pos / np.linalg.norm(pos)
        right = np.cross(fwd, np.array([0.0, 0.0, 1.0]))
        right /= np.linalg.norm(right)
        up = np.cross(right, fwd)
        d = (dirs_cam[:, 0:1] * right[None] + dirs_cam[:, 1:2] * up[None]
             - dirs_cam[:, 2:3] * fwd[None])
        d /= np.linalg.norm(d, axis=1, keepdims=True)
        o = np.broadcast_to(pos, d.shape).copy()
    else:
        raise ValueError(cfg.camera)
    return np.ascontiguousarray(o, np.float32), np.ascontiguousarray(d, np.float32)


@dataclasses.dataclass
class Scene:
    cfg: SceneConfig
    sites: np.ndarray      # float32 [K, 3]
    weights: np.ndarray    # float32 [K, weights_count]
    rays_o: np.ndarray     # float32 [R, 3]
    rays_d: np.ndarray     # float32 [R, 3]

    @property
    def arch(self) -> HeadArch:
        return self.cfg.arch


def make_scene(cfg: SceneConfig, rays: bool = True) -> Scene:
    sites = make_sites(cfg.sites, cfg.num_sites)
    w = make_weights(cfg.arch, cfg.num_sites, sigma_bias=cfg.sigma_bias)
    if rays:
        o, d = make_rays(cfg)
    else:
        o = d = np.zeros((0, 3), np.float32)
    return Scene(cfg, sites, w, o, d)


def ray_subset(n: int, total: int, seed: int = S0 + 7) -> np.ndarray:
    """A seeded, sorted subset of ray indices (for oracle-sized checks)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return np.sort(rng.choice(total, size=min(n, total), replace=False))
