"""ctypes binding of libderf.so (include/derf.h).

Argument marshalling only: every step of a render runs in the HIP library.
torch supplies device memory and streams; it is imported before the library
is loaded so that both share one HIP runtime.  If libderf.so has not been
built this module raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime the library binds to)

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libderf.so")

DERF_OK = 0
DERF_ERR_INVALID_ARG = -1
DERF_ERR_UNSUPPORTED = -2
DERF_ERR_OOM = -3
DERF_ERR_HIP = -4
DERF_PREC_FP32 = 0
DERF_PREC_BF16 = 1
DERF_NUM_STAGES = 6
DERF_NOALLOC_SCRATCH_BYTES = 64 << 20
STAGE_NAMES = ("sample_assign", "bucket_scan", "bucket_scatter", "mlp", "composite", "fine_sample")


class derf_head_arch(ctypes.Structure):
    _fields_ = [("pos_freqs", ctypes.c_int), ("dir_freqs", ctypes.c_int),
                ("depth", ctypes.c_int), ("width", ctypes.c_int),
                ("skip_layer", ctypes.c_int), ("rgb_hidden", ctypes.c_int)]


class derf_sampling(ctypes.Structure):
    _fields_ = [("n_coarse", ctypes.c_int), ("n_fine", ctypes.c_int),
                ("seed", ctypes.c_ulonglong), ("perturb", ctypes.c_int),
                ("ray_offset", ctypes.c_ulonglong)]


class derf_debug_out(ctypes.Structure):
    _fields_ = [("cell", ctypes.c_void_p), ("t", ctypes.c_void_p),
                ("sigma", ctypes.c_void_p), ("rgb", ctypes.c_void_p)]


class derf_stats(ctypes.Structure):
    _fields_ = [("renders", ctypes.c_longlong), ("samples", ctypes.c_longlong),
                ("stage_ms", ctypes.c_double * DERF_NUM_STAGES),
                ("stage_launches", ctypes.c_longlong * DERF_NUM_STAGES),
                ("head_samples", ctypes.c_longlong * 256),
                ("walk_rays", ctypes.c_longlong), ("walk_fallback_rays", ctypes.c_longlong)]


EXPORTS = ("derf_weights_count", "derf_create", "derf_create_mixed", "derf_render",
           "derf_render_debug", "derf_render_noalloc",
           "derf_render_soft", "derf_render_culled", "derf_set_empty_heads", "derf_set_gate",
           "derf_gate_weights_count", "derf_render_gated", "derf_set_encoding", "derf_set_timing",
           "derf_get_stats",
           "derf_reset_stats", "derf_destroy",
           "derf_status_string", "derf_last_error")

_lib: Optional[ctypes.CDLL] = None


class DerfError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d): %s" % (what, lib().derf_status_string(status).decode(),
                                                    status, lib().derf_last_error().decode()))


def lib() -> ctypes.CDLL:
    """Load libderf.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libderf.so is not built (%s); build it with "
                               "python paper_2011_12490_amd/build.py" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.derf_weights_count.argtypes = [ctypes.POINTER(derf_head_arch)]
        L.derf_weights_count.restype = ctypes.c_longlong
        L.derf_create.argtypes = [ctypes.POINTER(P), ctypes.c_int, P,
                                  ctypes.POINTER(derf_head_arch), P, ctypes.c_int]
        L.derf_create.restype = ctypes.c_int
        L.derf_create_mixed.argtypes = L.derf_create.argtypes
        L.derf_create_mixed.restype = ctypes.c_int
        render_args = [P, P, P, ctypes.c_longlong, ctypes.c_float, ctypes.c_float,
                       ctypes.POINTER(derf_sampling), P, P, P]
        L.derf_render.argtypes = render_args + [P]
        L.derf_render.restype = ctypes.c_int
        L.derf_render_debug.argtypes = render_args + [ctypes.POINTER(derf_debug_out), P]
        L.derf_render_debug.restype = ctypes.c_int
        L.derf_render_noalloc.argtypes = render_args + [P]
        L.derf_render_noalloc.restype = ctypes.c_int
        L.derf_render_soft.argtypes = [P, P, P, ctypes.c_longlong, ctypes.c_float, ctypes.c_float,
                                       ctypes.POINTER(derf_sampling), ctypes.c_float, P, P, P, P, P]
        L.derf_render_soft.restype = ctypes.c_int
        L.derf_render_culled.argtypes = [P, P, P, ctypes.c_longlong, ctypes.c_float,
                                         ctypes.c_float, ctypes.POINTER(derf_sampling),
                                         ctypes.c_float, ctypes.c_int, ctypes.c_int, P, P, P,
                                         P, P]
        L.derf_render_culled.restype = ctypes.c_int
        L.derf_set_empty_heads.argtypes = [P, P]
        L.derf_set_empty_heads.restype = ctypes.c_int
        L.derf_set_gate.argtypes = [P, ctypes.c_int, ctypes.c_int, P]
        L.derf_set_gate.restype = ctypes.c_int
        L.derf_gate_weights_count.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.derf_gate_weights_count.restype = ctypes.c_longlong
        L.derf_render_gated.argtypes = [P, P, P, ctypes.c_longlong, ctypes.c_float,
                                        ctypes.c_float, ctypes.POINTER(derf_sampling), P, P, P, P,
                                        P]
        L.derf_render_gated.restype = ctypes.c_int
        L.derf_set_encoding.argtypes = [P, ctypes.c_int]
        L.derf_set_encoding.restype = ctypes.c_int
        L.derf_set_timing.argtypes = [P, ctypes.c_int]
        L.derf_set_timing.restype = ctypes.c_int
        L.derf_get_stats.argtypes = [P, ctypes.POINTER(derf_stats)]
        L.derf_get_stats.restype = ctypes.c_int
        L.derf_reset_stats.argtypes = [P]
        L.derf_reset_stats.restype = ctypes.c_int
        L.derf_destroy.argtypes = [P]
        L.derf_destroy.restype = None
        L.derf_status_string.argtypes = [ctypes.c_int]
        L.derf_status_string.restype = ctypes.c_char_p
        L.derf_last_error.argtypes = []
        L.derf_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int, what: str):
    if status != DERF_OK:
        raise DerfError(status, what)


def _arch(arch) -> derf_head_arch:
    t = arch.as_tuple() if hasattr(arch, "as_tuple") else tuple(arch)
    return derf_head_arch(*t)


def _dptr(x: Optional[torch.Tensor]):
    return None if x is None else ctypes.c_void_p(x.data_ptr())


def check_rays(rays_o: torch.Tensor, rays_d: torch.Tensor) -> int:
    """Ray count of a pair of device ray arrays, after checking that both are
    contiguous float32 [R, 3] tensors on one GPU (ValueError otherwise: the
    library reads 3 R floats from each)."""
    for name, x in (("rays_o", rays_o), ("rays_d", rays_d)):
        if not isinstance(x, torch.Tensor):
            raise ValueError("%s must be a torch tensor" % name)
        if not x.is_cuda or x.dtype != torch.float32 or not x.is_contiguous():
            raise ValueError("%s must be a contiguous float32 GPU tensor" % name)
        if x.dim() != 2 or x.shape[1] != 3:
            raise ValueError("%s must have shape [R, 3], got %s" % (name, tuple(x.shape)))
    if rays_o.shape != rays_d.shape or rays_o.device != rays_d.device:
        raise ValueError("rays_o and rays_d differ in shape or device")
    return rays_o.shape[0]


def check_out(x: Optional[torch.Tensor], name: str, numel: int, dtype, device,
              optional: bool = False):
    """Check an output tensor before its pointer goes to the library, which
    writes `numel` elements of `dtype` to it: a contiguous GPU tensor on the
    rays' device with at least that many elements (ValueError otherwise, so
    that a wrong buffer fails before any GPU work)."""
    if x is None:
        if optional:
            return
        raise ValueError("%s is required" % name)
    if not isinstance(x, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if x.device != device:
        raise ValueError("%s must live on %s (the rays' device)" % (name, device))
    if x.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, x.dtype))
    if not x.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if x.numel() < numel:
        raise ValueError("%s holds %d elements, the render writes %d" % (name, x.numel(), numel))


def _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity) -> int:
    R = check_rays(rays_o, rays_d)
    dev = rays_o.device
    check_out(out_rgb, "out_rgb", 3 * R, torch.float32, dev)
    check_out(out_depth, "out_depth", R, torch.float32, dev)
    check_out(out_opacity, "out_opacity", R, torch.float32, dev)
    return R


# ---- thin wrappers with the C names -------------------------------------------

def derf_weights_count(arch) -> int:
    a = _arch(arch)
    return lib().derf_weights_count(ctypes.byref(a))


def _is_arch_list(arch) -> bool:
    return isinstance(arch, (list, tuple)) and len(arch) > 0 and not isinstance(arch[0], int)


def derf_create(sites, arch, weights, precision: int) -> ctypes.c_void_p:
    """sites: host float32 [K, 3]; weights: host float32 [K, derf_weights_count].
    With arch a list of K architectures (heads of different capacities),
    weights is a list of K per-head arrays or their concatenation."""
    import numpy as np
    s = np.ascontiguousarray(sites, np.float32).reshape(-1, 3)
    h = ctypes.c_void_p()
    if _is_arch_list(arch):
        if isinstance(weights, (list, tuple)):
            weights = np.concatenate([np.ravel(np.asarray(x, np.float32)) for x in weights])
        w = np.ascontiguousarray(weights, np.float32)
        if len(arch) != s.shape[0]:
            raise ValueError("need one architecture per site")
        if any(derf_weights_count(a) < 0 for a in arch):
            raise ValueError("invalid head architecture")
        if w.size != sum(derf_weights_count(a) for a in arch):
            raise ValueError("weights do not match the per-head architectures")
        arr = (derf_head_arch * len(arch))(*[_arch(a) for a in arch])
        _check(lib().derf_create_mixed(ctypes.byref(h), s.shape[0],
                                       s.ctypes.data_as(ctypes.c_void_p),
                                       ctypes.cast(arr, ctypes.POINTER(derf_head_arch)),
                                       w.ctypes.data_as(ctypes.c_void_p), precision),
               "derf_create_mixed")
        return h
    w = np.ascontiguousarray(weights, np.float32)
    a = _arch(arch)
    per_head = derf_weights_count(arch)
    if per_head < 0:
        raise ValueError("invalid head architecture %s" % (tuple(arch.as_tuple() if hasattr(
            arch, "as_tuple") else arch),))
    if w.size != s.shape[0] * per_head:
        raise ValueError("weights hold %d floats; %d heads of this architecture need %d"
                         % (w.size, s.shape[0], s.shape[0] * per_head))
    _check(lib().derf_create(ctypes.byref(h), s.shape[0], s.ctypes.data_as(ctypes.c_void_p),
                             ctypes.byref(a), w.ctypes.data_as(ctypes.c_void_p), precision),
           "derf_create")
    return h


def derf_render(h, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                samp: derf_sampling, out_rgb: torch.Tensor, out_depth: torch.Tensor,
                out_opacity: torch.Tensor, stream=None, debug: Optional[derf_debug_out] = None):
    """Enqueue a render on `stream` (default: torch's current stream)."""
    R = _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity)
    if stream is None:
        stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    args = [h, _dptr(rays_o), _dptr(rays_d), R, near, far, ctypes.byref(samp), _dptr(out_rgb),
            _dptr(out_depth), _dptr(out_opacity)]
    if debug is None:
        _check(lib().derf_render(*args, sp), "derf_render")
    else:
        _check(lib().derf_render_debug(*args, ctypes.byref(debug), sp), "derf_render_debug")


def derf_render_noalloc(h, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                        samp: derf_sampling, out_rgb: torch.Tensor, out_depth: torch.Tensor,
                        out_opacity: torch.Tensor, stream=None):
    """Enqueue a render that allocates nothing (the library's fixed per-device
    scratch array; frames beyond it raise DERF_ERR_INVALID_ARG) on `stream`
    (default: torch's current stream)."""
    _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity)
    if stream is None:
        stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    _check(lib().derf_render_noalloc(h, _dptr(rays_o), _dptr(rays_d), rays_o.shape[0], near, far,
                                     ctypes.byref(samp), _dptr(out_rgb), _dptr(out_depth),
                                     _dptr(out_opacity), sp),
           "derf_render_noalloc")


def derf_render_soft(h, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                     samp: derf_sampling, beta: float, out_rgb: torch.Tensor,
                     out_depth: torch.Tensor, out_opacity: torch.Tensor,
                     out_contrib: Optional[torch.Tensor] = None, stream=None):
    """Enqueue a soft-decomposition render on `stream` (default: torch's current
    stream).  out_contrib: float32 [R, K] or None."""
    R = _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity)
    if out_contrib is not None:
        if out_contrib.dim() != 2:
            raise ValueError("out_contrib must have shape [R, K]")
        check_out(out_contrib, "out_contrib", R * out_contrib.shape[1], torch.float32,
                  rays_o.device)
        if R and out_contrib.shape[0] < R:
            raise ValueError("out_contrib needs a row per ray")
    if stream is None:
        stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    _check(lib().derf_render_soft(h, _dptr(rays_o), _dptr(rays_d), rays_o.shape[0], near, far,
                                  ctypes.byref(samp), beta, _dptr(out_rgb), _dptr(out_depth),
                                  _dptr(out_opacity),
                                  None if out_contrib is None else _dptr(out_contrib), sp),
           "derf_render_soft")


def derf_render_culled(h, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                       samp: derf_sampling, eps: float, levels: int, out_rgb: torch.Tensor,
                       out_depth: torch.Tensor, out_opacity: torch.Tensor,
                       out_evaluated: Optional[torch.Tensor] = None, stream=None,
                       piece: int = 0):
    """Enqueue a Painter's-order render with transmittance culling on `stream`
    (default: torch's current stream).  out_evaluated: int32 [R] or None;
    piece: the most samples of one piece (0: whole segments)."""
    R = _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity)
    check_out(out_evaluated, "out_evaluated", R, torch.int32, rays_o.device, optional=True)
    if stream is None:
        stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    _check(lib().derf_render_culled(h, _dptr(rays_o), _dptr(rays_d), rays_o.shape[0], near, far,
                                    ctypes.byref(samp), eps, levels, piece, _dptr(out_rgb),
                                    _dptr(out_depth), _dptr(out_opacity),
                                    None if out_evaluated is None else _dptr(out_evaluated), sp),
           "derf_render_culled")


def derf_set_empty_heads(h, flags):
    """Mark 0-capacity heads (flags: K truthy values, or None to clear)."""
    if flags is None:
        _check(lib().derf_set_empty_heads(h, None), "derf_set_empty_heads")
        return
    arr = (ctypes.c_int * len(flags))(*[1 if f else 0 for f in flags])
    _check(lib().derf_set_empty_heads(h, ctypes.cast(arr, ctypes.c_void_p)), "derf_set_empty_heads")


def derf_set_gate(h, pos_freqs: int, hidden: int, weights, num_sites: int):
    """Set the MLP-gating network of a renderer of num_sites heads (host
    float32 weights, W1 [H][3 + 6L], b1, W2 [K][H], b2), or remove it with
    hidden = 0."""
    if hidden == 0:
        _check(lib().derf_set_gate(h, pos_freqs, 0, None), "derf_set_gate")
        return
    w = np.ascontiguousarray(weights, np.float32)
    count = lib().derf_gate_weights_count(num_sites, pos_freqs, hidden)
    if count < 0:
        raise ValueError("invalid gate shape (K=%d, L=%d, H=%d)" % (num_sites, pos_freqs, hidden))
    if w.size != count:
        raise ValueError("gating weights hold %d floats, the network needs %d" % (w.size, count))
    _check(lib().derf_set_gate(h, pos_freqs, hidden, w.ctypes.data_as(ctypes.c_void_p)),
           "derf_set_gate")


def derf_render_gated(h, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                      samp: derf_sampling, out_rgb: torch.Tensor, out_depth: torch.Tensor,
                      out_opacity: torch.Tensor, out_cell: Optional[torch.Tensor] = None,
                      stream=None):
    """Enqueue a render with the gated assignment on `stream` (default:
    torch's current stream).  out_cell: int32 [R, N] or None."""
    R = _check_outputs(rays_o, rays_d, out_rgb, out_depth, out_opacity)
    check_out(out_cell, "out_cell", R * (samp.n_coarse + max(0, samp.n_fine)), torch.int32,
              rays_o.device, optional=True)
    if stream is None:
        stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    _check(lib().derf_render_gated(h, _dptr(rays_o), _dptr(rays_d), rays_o.shape[0], near, far,
                                   ctypes.byref(samp), _dptr(out_rgb), _dptr(out_depth),
                                   _dptr(out_opacity),
                                   None if out_cell is None else _dptr(out_cell), sp),
           "derf_render_gated")


DERF_ENCODING_FUSED = 0
DERF_ENCODING_STORED = 1


def derf_set_encoding(h, mode: int):
    _check(lib().derf_set_encoding(h, int(mode)), "derf_set_encoding")


def derf_set_timing(h, on: bool):
    _check(lib().derf_set_timing(h, int(on)), "derf_set_timing")


def derf_get_stats(h) -> derf_stats:
    st = derf_stats()
    _check(lib().derf_get_stats(h, ctypes.byref(st)), "derf_get_stats")
    return st


def derf_reset_stats(h):
    _check(lib().derf_reset_stats(h), "derf_reset_stats")


def derf_destroy(h):
    lib().derf_destroy(h)


# ---- convenience ----------------------------------------------------------------

class Renderer:
    """A renderer handle bound to the current device."""

    def __init__(self, sites, arch, weights, precision: str = "bf16"):
        self.arch = arch
        self.precision = precision
        self.num_sites = len(sites)
        prec = DERF_PREC_BF16 if precision == "bf16" else DERF_PREC_FP32
        self.handle = derf_create(sites, arch, weights, prec)

    def close(self):
        if self.handle is not None and self.handle.value:
            derf_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def render(self, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
               n_coarse: int, n_fine: int = 0, seed: int = 0, perturb: bool = True,
               out=None, debug: bool = False, stream=None, ray_offset: int = 0):
        """Render device rays; returns (rgb [R,3], depth [R], opacity [R]) and, with
        debug=True, a dict of per-sample cell/t/sigma/rgb."""
        R = check_rays(rays_o, rays_d)
        dev = rays_o.device
        if out is None:
            rgb = torch.empty((R, 3), dtype=torch.float32, device=dev)
            depth = torch.empty((R,), dtype=torch.float32, device=dev)
            opac = torch.empty((R,), dtype=torch.float32, device=dev)
        else:
            rgb, depth, opac = out
        samp = derf_sampling(n_coarse, n_fine, seed, int(perturb), ray_offset)
        dbg = None
        extra = None
        if debug:
            N = n_coarse + n_fine
            extra = {"cell": torch.empty((R, N), dtype=torch.int32, device=dev),
                     "t": torch.empty((R, N), dtype=torch.float32, device=dev),
                     "sigma": torch.empty((R, N), dtype=torch.float32, device=dev),
                     "rgb": torch.empty((R, N, 3), dtype=torch.float32, device=dev)}
            dbg = derf_debug_out(_dptr(extra["cell"]), _dptr(extra["t"]),
                                 _dptr(extra["sigma"]), _dptr(extra["rgb"]))
        derf_render(self.handle, rays_o, rays_d, near, far, samp, rgb, depth, opac, stream, dbg)
        if debug:
            return rgb, depth, opac, extra
        return rgb, depth, opac

    def set_gate(self, pos_freqs: int, hidden: int, weights):
        """Assign samples with an MLP-gating network instead of the nearest
        site in render_gated (hidden = 0 removes it)."""
        derf_set_gate(self.handle, pos_freqs, hidden, weights, self.num_sites)

    def render_gated(self, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                     n: int, seed: int = 0, perturb: bool = True, stream=None,
                     ray_offset: int = 0, cells: bool = False):
        """Single-pass render with the gated assignment; returns (rgb, depth,
        opacity) and, with cells, each sample's head [R, n]."""
        R = check_rays(rays_o, rays_d)
        dev = rays_o.device
        rgb = torch.empty((R, 3), dtype=torch.float32, device=dev)
        depth = torch.empty((R,), dtype=torch.float32, device=dev)
        opac = torch.empty((R,), dtype=torch.float32, device=dev)
        cell = torch.empty((R, n), dtype=torch.int32, device=dev) if cells else None
        samp = derf_sampling(n, 0, seed, int(perturb), ray_offset)
        derf_render_gated(self.handle, rays_o, rays_d, near, far, samp, rgb, depth, opac, cell,
                          stream)
        return (rgb, depth, opac, cell) if cells else (rgb, depth, opac)

    def set_encoding(self, stored: bool):
        """gamma(x) encoded inside the MLP (False, the default) or written to a
        table by its own pass and read back (True; heads without a skip layer)."""
        derf_set_encoding(self.handle, DERF_ENCODING_STORED if stored else DERF_ENCODING_FUSED)

    def set_empty_heads(self, flags):
        """Mark 0-capacity heads (K flags; None clears)."""
        if flags is not None and len(flags) != self.num_sites:
            raise ValueError("need one flag per head")
        derf_set_empty_heads(self.handle, flags)

    def render_soft(self, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                    n: int, beta: float, seed: int = 0, perturb: bool = True,
                    contrib: bool = False, stream=None, ray_offset: int = 0):
        """Soft-decomposition render at temperature beta; returns (rgb, depth,
        opacity) and, with contrib=True, the per-ray head contributions [R, K]."""
        R = check_rays(rays_o, rays_d)
        dev = rays_o.device
        rgb = torch.empty((R, 3), dtype=torch.float32, device=dev)
        depth = torch.empty((R,), dtype=torch.float32, device=dev)
        opac = torch.empty((R,), dtype=torch.float32, device=dev)
        W = torch.empty((R, self.num_sites), dtype=torch.float32, device=dev) if contrib else None
        samp = derf_sampling(n, 0, seed, int(perturb), ray_offset)
        derf_render_soft(self.handle, rays_o, rays_d, near, far, samp, beta, rgb, depth, opac, W,
                         stream)
        if contrib:
            return rgb, depth, opac, W
        return rgb, depth, opac

    def render_culled(self, rays_o: torch.Tensor, rays_d: torch.Tensor, near: float, far: float,
                      n: int, eps: float, levels: int, seed: int = 0, perturb: bool = True,
                      stream=None, ray_offset: int = 0, piece: int = 0):
        """Single-pass render in Painter's order with transmittance culling;
        returns (rgb, depth, opacity, evaluated samples per ray).  piece > 0
        cuts segments into pieces of at most that many samples."""
        R = check_rays(rays_o, rays_d)
        dev = rays_o.device
        rgb = torch.empty((R, 3), dtype=torch.float32, device=dev)
        depth = torch.empty((R,), dtype=torch.float32, device=dev)
        opac = torch.empty((R,), dtype=torch.float32, device=dev)
        ev = torch.empty((R,), dtype=torch.int32, device=dev)
        samp = derf_sampling(n, 0, seed, int(perturb), ray_offset)
        derf_render_culled(self.handle, rays_o, rays_d, near, far, samp, eps, levels, rgb, depth,
                           opac, ev, stream, piece)
        return rgb, depth, opac, ev
