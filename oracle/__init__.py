"""CPU oracle of the DeRF renderer -- test infrastructure only.

Loads ``liboracle.so`` (plain C, built from ``derf_oracle.c`` by ``build()``)
through ctypes.  Only the tests, the smoke check and the benchmark's CPU
baseline use this package; the GPU library never imports or links it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "derf_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP over rays, no fp contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wno-unused-function",
               _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Arch(ctypes.Structure):
    _fields_ = [("pos_freqs", ctypes.c_int), ("dir_freqs", ctypes.c_int),
                ("depth", ctypes.c_int), ("width", ctypes.c_int),
                ("skip_layer", ctypes.c_int), ("rgb_hidden", ctypes.c_int)]


_P = ctypes.c_void_p


def _lib_handle():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        render_sig = [ctypes.c_int, _P, ctypes.POINTER(_Arch), _P, ctypes.c_longlong, _P, _P, _P,
                      ctypes.c_float, ctypes.c_float, ctypes.c_int, ctypes.c_int,
                      ctypes.c_uint64, ctypes.c_int, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_int]
        for name in ("oracle_render", "oracle_render_direct", "oracle_render_back_to_front",
                     "oracle_render_plain"):
            f = getattr(lib, name)
            f.argtypes = render_sig
            f.restype = ctypes.c_int
        lib.oracle_render_soft.argtypes = render_sig + [ctypes.c_double]
        lib.oracle_render_soft.restype = ctypes.c_int
        lib.oracle_render_soft_contrib.argtypes = render_sig + [ctypes.c_double, ctypes.c_void_p]
        lib.oracle_render_soft_contrib.restype = ctypes.c_int
        lib.oracle_render_ex.argtypes = render_sig + [ctypes.c_int, ctypes.c_double,
                                                      ctypes.c_void_p, ctypes.c_void_p]
        lib.oracle_render_ex.restype = ctypes.c_int
        lib.oracle_render_mixed.argtypes = lib.oracle_render_ex.argtypes
        lib.oracle_render_mixed.restype = ctypes.c_int
        lib.oracle_render_culled.argtypes = render_sig + [ctypes.c_double, ctypes.c_int,
                                                          ctypes.c_int, ctypes.c_void_p,
                                                          ctypes.c_void_p]
        lib.oracle_render_culled.restype = ctypes.c_int
        lib.oracle_philox4x32_10.argtypes = [_P, _P, _P]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_jitter.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32,
                                      ctypes.c_uint32]
        lib.oracle_jitter.restype = ctypes.c_float
        lib.oracle_sample_depths.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_float,
                                             ctypes.c_float, ctypes.c_int, ctypes.c_int, _P]
        lib.oracle_sample_depths.restype = None
        lib.oracle_nearest_site.argtypes = [ctypes.c_int, _P, _P]
        lib.oracle_nearest_site.restype = ctypes.c_int
        lib.oracle_bisector_margin.argtypes = [ctypes.c_int, _P, _P, ctypes.c_int]
        lib.oracle_bisector_margin.restype = ctypes.c_double
        lib.oracle_posenc.argtypes = [ctypes.c_int, _P, _P]
        lib.oracle_posenc.restype = None
        lib.oracle_weights_count.argtypes = [ctypes.POINTER(_Arch)]
        lib.oracle_weights_count.restype = ctypes.c_longlong
        lib.oracle_head_eval.argtypes = [ctypes.POINTER(_Arch), _P, _P, _P, _P, _P, _P]
        lib.oracle_head_eval.restype = None
        lib.oracle_composite.argtypes = [ctypes.c_int, ctypes.c_int, _P, _P, _P, _P,
                                         ctypes.c_float, ctypes.c_float, _P, _P, _P, _P]
        lib.oracle_composite.restype = None
        lib.oracle_fine_depths.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int,
                                           ctypes.c_int, ctypes.c_int, _P, ctypes.c_float,
                                           ctypes.c_float, _P, _P]
        lib.oracle_fine_depths.restype = None
        lib.oracle_sample_assign.argtypes = [ctypes.c_int, _P, ctypes.c_longlong, _P, _P,
                                             ctypes.c_uint64, ctypes.c_float, ctypes.c_float,
                                             ctypes.c_int, ctypes.c_uint64, ctypes.c_int, _P, _P,
                                             _P, ctypes.c_int]
        lib.oracle_sample_assign.restype = ctypes.c_int
        lib.oracle_assign_depths.argtypes = [ctypes.c_int, _P, ctypes.c_longlong, _P, _P,
                                             ctypes.c_int, _P, _P, _P, ctypes.c_int]
        lib.oracle_assign_depths.restype = ctypes.c_int
        lib.oracle_render_depths.argtypes = [ctypes.c_int, _P, ctypes.POINTER(_Arch), _P,
                                             ctypes.c_longlong, _P, _P, ctypes.c_float,
                                             ctypes.c_float, ctypes.c_int, _P, _P, _P, _P, _P, _P,
                                             _P, ctypes.c_int]
        lib.oracle_render_depths.restype = ctypes.c_int
        lib.oracle_render_gated.argtypes = render_sig + [ctypes.c_int, ctypes.c_int, _P]
        lib.oracle_render_gated.restype = ctypes.c_int
        lib.oracle_gate_weights_count.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        lib.oracle_gate_weights_count.restype = ctypes.c_longlong
        lib.oracle_gate_logits.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, _P,
                                           ctypes.c_longlong, _P, _P]
        lib.oracle_gate_logits.restype = ctypes.c_int
        lib.oracle_sample_points.argtypes = [ctypes.c_longlong, _P, _P, _P, _P]
        lib.oracle_sample_points.restype = None
        lib.oracle_max_threads.argtypes = []
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _arch(arch) -> _Arch:
    t = arch.as_tuple() if hasattr(arch, "as_tuple") else tuple(arch)
    return _Arch(*t)


def max_threads() -> int:
    return _lib_handle().oracle_max_threads()


def philox4x32_10(counter, key) -> np.ndarray:
    c = np.ascontiguousarray(counter, np.uint32)
    k = np.ascontiguousarray(key, np.uint32)
    out = np.zeros(4, np.uint32)
    _lib_handle().oracle_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def jitter(seed: int, ray: int, i: int, stream: int) -> float:
    return _lib_handle().oracle_jitter(seed, ray, i, stream)


def sample_depths(seed: int, ray: int, near: float, far: float, n: int, perturb: bool = True):
    t = np.zeros(n, np.float32)
    _lib_handle().oracle_sample_depths(seed, ray, near, far, n, int(perturb), _ptr(t))
    return t


def nearest_site(sites: np.ndarray, x) -> int:
    s = np.ascontiguousarray(sites, np.float32)
    xx = np.ascontiguousarray(x, np.float32)
    return _lib_handle().oracle_nearest_site(s.shape[0], _ptr(s), _ptr(xx))


def bisector_margin(sites: np.ndarray, x, a: int) -> float:
    s = np.ascontiguousarray(sites, np.float32)
    xx = np.ascontiguousarray(x, np.float32)
    return _lib_handle().oracle_bisector_margin(s.shape[0], _ptr(s), _ptr(xx), a)


def posenc(L: int, p) -> np.ndarray:
    pp = np.ascontiguousarray(p, np.float64)
    out = np.zeros(3 + 6 * L, np.float64)
    _lib_handle().oracle_posenc(L, _ptr(pp), _ptr(out))
    return out


def weights_count(arch) -> int:
    a = _arch(arch)
    return _lib_handle().oracle_weights_count(ctypes.byref(a))


def head_eval(arch, weights: np.ndarray, gx: np.ndarray, gd: np.ndarray):
    """(sigma, rgb[3]) of one head at encoded inputs gx, gd (float64)."""
    a = _arch(arch)
    w = np.ascontiguousarray(weights, np.float32)
    gx = np.ascontiguousarray(gx, np.float64)
    gd = np.ascontiguousarray(gd, np.float64)
    sigma = np.zeros(1, np.float64)
    rgb = np.zeros(3, np.float64)
    scratch = np.zeros(4 * (gx.size + a.width + gd.size + a.rgb_hidden + 8), np.float64)
    _lib_handle().oracle_head_eval(ctypes.byref(a), _ptr(w), _ptr(gx), _ptr(gd), _ptr(sigma),
                                   _ptr(rgb), _ptr(scratch))
    return float(sigma[0]), rgb


_MODES = {"segments": 0, "direct": 3, "back": 4}


def composite(cell, t, sigma, rgb, near: float, far: float, mode: str = "segments"):
    """Composite given per-sample fields of one ray -> (rgb[3], depth, opacity, weights)."""
    n = len(t)
    cell = np.ascontiguousarray(cell, np.int32)
    t = np.ascontiguousarray(t, np.float32)
    sigma = np.ascontiguousarray(sigma, np.float64)
    rgb = np.ascontiguousarray(rgb, np.float64).reshape(n, 3)
    out = np.zeros(3, np.float64)
    dep = np.zeros(1, np.float64)
    op = np.zeros(1, np.float64)
    w = np.zeros(max(n, 1), np.float64)
    _lib_handle().oracle_composite(_MODES[mode], n, _ptr(cell), _ptr(t), _ptr(sigma), _ptr(rgb),
                                   near, far, _ptr(out), _ptr(dep), _ptr(op), _ptr(w))
    return out, float(dep[0]), float(op[0]), w[:n]


def fine_depths(seed: int, ray: int, perturb: bool, tc: np.ndarray, near: float, far: float,
                w: np.ndarray, n_fine: int) -> np.ndarray:
    tc = np.ascontiguousarray(tc, np.float32)
    w = np.ascontiguousarray(w, np.float64)
    tf = np.zeros(n_fine, np.float32)
    _lib_handle().oracle_fine_depths(seed, ray, int(perturb), tc.size, n_fine, _ptr(tc), near,
                                     far, _ptr(w), _ptr(tf))
    return tf


def sample_assign(sites, rays_o, rays_d, near: float, far: float, n: int, seed: int,
                  perturb: bool = True, ray_offset: int = 0, margin: bool = False,
                  nthreads: int = 0):
    """Sample depths t [R, n] (float32), owning cells [R, n] and optionally each
    sample's distance to its cell boundary, for every sample of the rays."""
    sites = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    R = o.shape[0]
    t = np.zeros((R, n), np.float32)
    cell = np.zeros((R, n), np.int32)
    m = np.zeros((R, n), np.float64) if margin else None
    rc = _lib_handle().oracle_sample_assign(sites.shape[0], _ptr(sites), R, _ptr(o), _ptr(d),
                                            ray_offset, near, far, n, seed, int(perturb), _ptr(t),
                                            _ptr(cell), _ptr(m), nthreads)
    if rc != 0:
        raise RuntimeError("oracle sample_assign failed (%d)" % rc)
    return t, cell, m


def assign_depths(sites, rays_o, rays_d, t, margin: bool = False, nthreads: int = 0):
    """Owning cells [R, n] of the given sample depths t [R, n] (and optionally
    each sample's distance to its cell boundary)."""
    sites = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    t = np.ascontiguousarray(t, np.float32)
    R, n = t.shape
    if o.shape[0] != R or d.shape[0] != R:
        raise ValueError("rays and depths disagree on the ray count")
    cell = np.zeros((R, n), np.int32)
    m = np.zeros((R, n), np.float64) if margin else None
    rc = _lib_handle().oracle_assign_depths(sites.shape[0], _ptr(sites), R, _ptr(o), _ptr(d), n,
                                            _ptr(t), _ptr(cell), _ptr(m), nthreads)
    if rc != 0:
        raise RuntimeError("oracle assign_depths failed (%d)" % rc)
    return cell, m


def render_depths(sites, arch, weights, rays_o, rays_d, near: float, far: float, t,
                  per_sample: bool = False, nthreads: int = 0):
    """DeRF render at given sorted sample depths t [R, n]: heads of the owning
    cells, quadrature, segments and Painter's merge (no sampling)."""
    sites = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    weights = np.ascontiguousarray(weights, np.float32)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    t = np.ascontiguousarray(t, np.float32)
    R, n = t.shape
    if o.shape[0] != R or d.shape[0] != R:
        raise ValueError("rays and depths disagree on the ray count")
    rgb = np.zeros((R, 3), np.float64)
    dep = np.zeros(R, np.float64)
    op = np.zeros(R, np.float64)
    cell = np.zeros((R, n), np.int32) if per_sample else None
    sig = np.zeros((R, n), np.float64) if per_sample else None
    srgb = np.zeros((R, n, 3), np.float64) if per_sample else None
    a = _arch(arch)
    rc = _lib_handle().oracle_render_depths(sites.shape[0], _ptr(sites), ctypes.byref(a),
                                            _ptr(weights), R, _ptr(o), _ptr(d), near, far, n,
                                            _ptr(t), _ptr(rgb), _ptr(dep), _ptr(op), _ptr(cell),
                                            _ptr(sig), _ptr(srgb), nthreads)
    if rc != 0:
        raise RuntimeError("oracle render_depths failed (%d)" % rc)
    return RenderResult(rgb, dep, op, t, cell, sig, srgb)


class RenderResult:
    """Outputs of an oracle render (double) plus optional per-sample arrays."""

    def __init__(self, rgb, depth, opacity, t=None, cell=None, sigma=None, srgb=None,
                 margin=None, contrib=None):
        self.rgb, self.depth, self.opacity = rgb, depth, opacity
        self.t, self.cell, self.sigma, self.srgb, self.margin = t, cell, sigma, srgb, margin
        self.contrib = contrib


def render(sites, arch, weights, rays_o, rays_d, near: float, far: float, n_coarse: int,
           n_fine: int = 0, seed: int = 0, perturb: bool = True, ray_ids=None,
           per_sample: bool = False, mode: str = "derf", beta: float = 0.0,
           nthreads: int = 0, contrib: bool = False, empty=None) -> RenderResult:
    """Render rays on the CPU.  mode: derf | direct | back | plain | soft.
    contrib (soft mode, single pass): also return the per-ray head
    contributions W(r) [R, K] of Sec. 3.2 Eq. 6.  empty: optional [K] flags of
    0-capacity heads (no density anywhere).  arch may be a list of K
    architectures (heads of different capacities); weights is then the heads'
    packed weights concatenated in head order."""
    lib = _lib_handle()
    sites = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    mixed = isinstance(arch, (list, tuple)) and not isinstance(arch[0], int)
    if mixed:
        if len(arch) != sites.shape[0]:
            raise ValueError("need one architecture per head")
        weights = np.ascontiguousarray(np.concatenate([np.ravel(w) for w in weights])
                                       if isinstance(weights, (list, tuple)) else weights,
                                       np.float32)
        if weights.size != sum(weights_count(a) for a in arch):
            raise ValueError("weights do not match the architectures")
    else:
        weights = np.ascontiguousarray(weights, np.float32)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    R = o.shape[0]
    N = n_coarse + n_fine
    ids = None if ray_ids is None else np.ascontiguousarray(ray_ids, np.int64)
    rgb = np.zeros((R, 3), np.float64)
    dep = np.zeros(R, np.float64)
    op = np.zeros(R, np.float64)
    if per_sample:
        t = np.zeros((R, N), np.float32)
        cell = np.zeros((R, N), np.int32)
        sig = np.zeros((R, N), np.float64)
        srgb = np.zeros((R, N, 3), np.float64)
        margin = np.zeros((R, N), np.float64)
    else:
        t = cell = sig = srgb = margin = None
    a = (_Arch * len(arch))(*[_arch(x) for x in arch]) if mixed else _arch(arch)
    a_ref = ctypes.cast(a, ctypes.POINTER(_Arch)) if mixed else ctypes.byref(a)
    args = [sites.shape[0], _ptr(sites), a_ref, _ptr(weights), R, _ptr(o), _ptr(d),
            _ptr(ids), near, far, n_coarse, n_fine, seed, int(perturb), _ptr(rgb), _ptr(dep),
            _ptr(op), _ptr(t), _ptr(cell), _ptr(sig), _ptr(srgb), _ptr(margin), nthreads]
    fn = {"derf": lib.oracle_render, "direct": lib.oracle_render_direct,
          "back": lib.oracle_render_back_to_front, "plain": lib.oracle_render_plain}
    W = None
    if contrib:
        if mode != "soft" or n_fine != 0:
            raise ValueError("contributions come from the single-pass soft render")
        W = np.zeros((R, sites.shape[0]), np.float64)
    if empty is not None or mixed:
        e = None
        if empty is not None:
            e = np.ascontiguousarray(np.asarray(empty) != 0, np.uint8)
            if e.shape != (sites.shape[0],):
                raise ValueError("empty needs one flag per head")
        code = {"derf": 0, "plain": 1, "soft": 2, "direct": 3, "back": 4}[mode]
        fn_ex = lib.oracle_render_mixed if mixed else lib.oracle_render_ex
        rc = fn_ex(*args, code, beta, _ptr(e), _ptr(W))
    elif contrib:
        rc = lib.oracle_render_soft_contrib(*args, beta, _ptr(W))
    elif mode == "soft":
        rc = lib.oracle_render_soft(*args, beta)
    else:
        rc = fn[mode](*args)
    if rc != 0:
        raise RuntimeError("oracle render failed (%d)" % rc)
    return RenderResult(rgb, dep, op, t, cell, sig, srgb, margin, W)


def render_culled(sites, arch, weights, rays_o, rays_d, near: float, far: float,
                  n_coarse: int, eps: float, levels: int, seed: int = 0, perturb: bool = True,
                  ray_ids=None, empty=None, nthreads: int = 0, piece: int = 0) -> RenderResult:
    """Single-pass DeRF render with Painter's-order culling (Sec. 3.3): level l
    of a ray is its l-th piece (a segment, or with piece > 0 a part of at most
    `piece` samples of one, cut from the segment's start; the last level takes
    every later piece), and a ray stops before level l > 0 once its
    transmittance is below eps.  The result's ``evaluated`` holds the samples
    whose head ran, per ray."""
    sites = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    weights = np.ascontiguousarray(weights, np.float32)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    R = o.shape[0]
    ids = None if ray_ids is None else np.ascontiguousarray(ray_ids, np.int64)
    e = None
    if empty is not None:
        e = np.ascontiguousarray(np.asarray(empty) != 0, np.uint8)
        if e.shape != (sites.shape[0],):
            raise ValueError("empty needs one flag per head")
    rgb = np.zeros((R, 3), np.float64)
    dep = np.zeros(R, np.float64)
    op = np.zeros(R, np.float64)
    ev = np.zeros(R, np.int32)
    a = _arch(arch)
    rc = _lib_handle().oracle_render_culled(
        sites.shape[0], _ptr(sites), ctypes.byref(a), _ptr(weights), R, _ptr(o), _ptr(d),
        _ptr(ids), near, far, n_coarse, 0, seed, int(perturb), _ptr(rgb), _ptr(dep), _ptr(op),
        None, None, None, None, None, nthreads, float(eps), int(levels), int(piece), _ptr(e),
        _ptr(ev))
    if rc != 0:
        raise RuntimeError("oracle culled render failed (%d)" % rc)
    res = RenderResult(rgb, dep, op)
    res.evaluated = ev
    return res


# ---------------------------------------------------------------- MLP gating
# The decomposition network of Sec. 4 ("Decompositions with MLPs"), computed
# by the C oracle (oracle_gate_logits, oracle_render_gated): an MLP with a
# softmax output gives each point its head weights; at inference a sample
# belongs to the head of largest weight, which (the softmax being monotone)
# is the first largest logit.  The reading of its shape: one ReLU hidden
# layer of H units on the heads' positional encoding gamma_L(x),
#   h = max(0, W1 gamma_L(x) + b1),  logits = W2 h + b2,
# weights (fp32) packed W1 [H][3 + 6L], b1 [H], W2 [K][H], b2 [K].  The
# decision is taken in the precision of the GPU kernel, which runs both
# products on bf16 matrix cores with each fp32 operand split into two bf16
# values: a b = a_hi b_hi + a_hi b_lo + a_lo b_hi (about 16 significant bits
# per operand; see derf_oracle.c).

def gate_weights_count(num_sites: int, L: int, hidden: int) -> int:
    return _lib_handle().oracle_gate_weights_count(num_sites, L, hidden)


def _gate_weights(num_sites: int, L: int, hidden: int, w) -> np.ndarray:
    w = np.ascontiguousarray(w, np.float32).ravel()
    if w.size != gate_weights_count(num_sites, L, hidden):
        raise ValueError("gating weights: expected %d floats, got %d"
                         % (gate_weights_count(num_sites, L, hidden), w.size))
    return w


def sample_points(rays_o, rays_d, t) -> np.ndarray:
    """x = o + t d in float32 with one fused multiply-add per component, for
    depths t [..., n] of rays o, d [..., 3] (the sample points whose cells the
    path decides); returns [..., n, 3]."""
    t = np.ascontiguousarray(t, np.float32)
    o = np.broadcast_to(np.asarray(rays_o, np.float32)[..., None, :], t.shape + (3,))
    d = np.broadcast_to(np.asarray(rays_d, np.float32)[..., None, :], t.shape + (3,))
    o = np.ascontiguousarray(o)
    d = np.ascontiguousarray(d)
    x = np.zeros(t.shape + (3,), np.float32)
    _lib_handle().oracle_sample_points(t.size, _ptr(o), _ptr(d), _ptr(t), _ptr(x))
    return x


def gate_logits(num_sites: int, L: int, hidden: int, w, x) -> np.ndarray:
    """Logits [M, K] (float64) of the gating network at points x [M, 3]."""
    w = _gate_weights(num_sites, L, hidden, w)
    x = np.ascontiguousarray(x, np.float32).reshape(-1, 3)
    z = np.zeros((x.shape[0], num_sites), np.float64)
    rc = _lib_handle().oracle_gate_logits(num_sites, L, hidden, _ptr(w), x.shape[0], _ptr(x),
                                          _ptr(z))
    if rc != 0:
        raise RuntimeError("oracle gate_logits failed (%d)" % rc)
    return z


def gate_assign(num_sites: int, L: int, hidden: int, w, x):
    """(cells [M], gap [M]): each point's gated head (first largest logit)
    and the difference of its two largest logits (inf for one head), which
    says how close the decision is to a tie."""
    z = gate_logits(num_sites, L, hidden, w, x)
    cells = np.argmax(z, axis=1).astype(np.int32)
    if num_sites == 1:
        return cells, np.full(len(cells), np.inf)
    top2 = np.sort(z, axis=1)[:, -2:]
    return cells, top2[:, 1] - top2[:, 0]


def render_gated(arch, weights, num_sites: int, gate_L: int, gate_hidden: int, gate_w, rays_o,
                 rays_d, near: float, far: float, n: int, seed: int = 0, perturb: bool = True,
                 ray_ids=None, nthreads: int = 0) -> RenderResult:
    """Single-pass render with the gated assignment: stratified depths,
    x = o + t d, each sample's gated head, that head's network, quadrature,
    and the front-to-back merge of the ray's runs of one head (a gated cell
    may be entered more than once).  The result also holds t, cell and gap
    [R, n] (gap: the difference of each sample's two largest logits)."""
    sites = np.zeros((num_sites, 3), np.float32)  # not used by the gated assignment
    w = _gate_weights(num_sites, gate_L, gate_hidden, gate_w)
    weights = np.ascontiguousarray(weights, np.float32)
    o = np.ascontiguousarray(rays_o, np.float32).reshape(-1, 3)
    d = np.ascontiguousarray(rays_d, np.float32).reshape(-1, 3)
    R = o.shape[0]
    ids = None if ray_ids is None else np.ascontiguousarray(ray_ids, np.int64)
    rgb = np.zeros((R, 3), np.float64)
    dep = np.zeros(R, np.float64)
    op = np.zeros(R, np.float64)
    T = np.zeros((R, n), np.float32)
    C = np.zeros((R, n), np.int32)
    G = np.zeros((R, n), np.float64)
    a = _arch(arch)
    rc = _lib_handle().oracle_render_gated(
        num_sites, _ptr(sites), ctypes.byref(a), _ptr(weights), R, _ptr(o), _ptr(d), _ptr(ids),
        near, far, n, 0, seed, int(perturb), _ptr(rgb), _ptr(dep), _ptr(op), _ptr(T), _ptr(C),
        None, None, _ptr(G), nthreads, gate_L, gate_hidden, _ptr(w))
    if rc != 0:
        raise RuntimeError("oracle gated render failed (%d)" % rc)
    res = RenderResult(rgb, dep, op)
    res.t, res.cell, res.gap = T, C, G
    return res
