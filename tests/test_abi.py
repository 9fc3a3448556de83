"""The C-ABI library: it loads, exports every declared symbol, and rejects bad
arguments before touching a GPU (no compute calls here)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2011_12490_amd import derf, scenes

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "derf.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(derf_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert set(declared_functions()) == set(derf.EXPORTS)


def test_stage_count_agrees_with_the_binding():
    text = open(os.path.join(ROOT, "include", "derf.h")).read()
    n = int(re.search(r"#define DERF_NUM_STAGES (\d+)", text).group(1))
    assert n == derf.DERF_NUM_STAGES == len(derf.STAGE_NAMES)
    stages = re.findall(r"DERF_STAGE_([A-Z_]+) = (\d+)", text)
    assert sorted(int(v) for _, v in stages) == list(range(n))


def test_struct_layouts_match_the_header(tmp_path):
    """The ctypes mirrors of the header's structs have the C compiler's sizes
    and field offsets (a plain C program built with gcc prints them)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("no gcc")
    structs = {"derf_head_arch": derf.derf_head_arch, "derf_sampling": derf.derf_sampling,
               "derf_debug_out": derf.derf_debug_out, "derf_stats": derf.derf_stats}
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "derf.h"', 'int main(void) {']
    for name, cls in structs.items():
        lines.append('printf("%s %%zu\\n", sizeof(%s));' % (name, name))
        for field, _ in cls._fields_:
            lines.append('printf("%s.%s %%zu\\n", offsetof(%s, %s));'
                         % (name, field, name, field))
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = dict(l.split() for l in subprocess.run([str(exe)], check=True, capture_output=True,
                                                 text=True).stdout.splitlines())
    for name, cls in structs.items():
        assert int(got[name]) == ctypes.sizeof(cls), name
        for field, _ in cls._fields_:
            assert int(got["%s.%s" % (name, field)]) == getattr(cls, field).offset, (name, field)


def test_library_exports_every_declared_symbol():
    L = derf.lib()
    for name in declared_functions():
        assert hasattr(L, name), name


@pytest.mark.parametrize("arch", [scenes.ARCH_TINY, scenes.ARCH_128, scenes.ARCH_SMALL,
                                  scenes.ARCH_NERF, scenes.HeadArch(3, 2, 3, 16, 2, 8)])
def test_weights_count_matches_generator_and_oracle(arch):
    assert derf.derf_weights_count(arch) == arch.weights_count() == oracle.weights_count(arch)


@pytest.mark.parametrize("K,L,H", [(1, 6, 16), (16, 10, 32), (256, 10, 64), (7, 6, 24)])
def test_gate_weights_count_matches_oracle(K, L, H):
    assert derf.lib().derf_gate_weights_count(K, L, H) == oracle.gate_weights_count(K, L, H)


def test_weights_count_rejects_bad_values():
    assert derf.derf_weights_count((10, 4, 0, 128, -1, 0)) == -1
    assert derf.derf_weights_count((10, 4, 8, 128, 8, 0)) == -1     # skip beyond depth
    assert derf.lib().derf_weights_count(None) == -1


def _create(K, arch, prec=1, sites=None, weights=None):
    L = derf.lib()
    h = ctypes.c_void_p(1234)
    a = derf.derf_head_arch(*arch) if arch is not None else None
    s = np.zeros((max(K, 1), 3), np.float32) if sites is None else sites
    w = np.zeros(16, np.float32) if weights is None else weights
    rc = L.derf_create(ctypes.byref(h), K, s.ctypes.data_as(ctypes.c_void_p),
                       ctypes.byref(a) if a is not None else None,
                       w.ctypes.data_as(ctypes.c_void_p), prec)
    return rc, h


def test_create_rejects_bad_arguments_without_a_gpu():
    L = derf.lib()
    assert L.derf_create(None, 1, None, None, None, 0) == derf.DERF_ERR_INVALID_ARG
    rc, h = _create(0, (10, 4, 8, 128, 5, 64))
    assert rc == derf.DERF_ERR_INVALID_ARG and h.value is None
    rc, _ = _create(257, (10, 4, 8, 128, 5, 64), sites=np.zeros((257, 3), np.float32))
    assert rc == derf.DERF_ERR_INVALID_ARG
    rc, _ = _create(4, (10, 4, 8, 128, 5, 64), prec=7)
    assert rc == derf.DERF_ERR_INVALID_ARG
    rc, _ = _create(4, None)
    assert rc == derf.DERF_ERR_INVALID_ARG
    bad = np.zeros((4, 3), np.float32)
    bad[2, 1] = np.nan
    rc, _ = _create(4, (10, 4, 8, 128, 5, 64), sites=bad)
    assert rc == derf.DERF_ERR_INVALID_ARG
    rc, _ = _create(4, (10, 4, 8, 96, 5, 64))
    assert rc == derf.DERF_ERR_UNSUPPORTED
    assert b"no bf16 kernel" in L.derf_last_error()
    rc, _ = _create(4, (10, 4, 8, 256, 5, 128), prec=0)       # no fp32 kernel at width 256
    assert rc == derf.DERF_ERR_UNSUPPORTED


def test_render_rejects_bad_arguments_without_a_gpu():
    L = derf.lib()
    samp = derf.derf_sampling(32, 0, 1, 1, 0)
    assert L.derf_render(None, None, None, 1, 2.0, 6.0, ctypes.byref(samp), None, None, None,
                         None) == derf.DERF_ERR_INVALID_ARG
    for fn in ("derf_set_timing", "derf_reset_stats"):
        args = [None] + ([1] if fn == "derf_set_timing" else [])
        assert getattr(L, fn)(*args) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_get_stats(None, None) == derf.DERF_ERR_INVALID_ARG
    L.derf_destroy(None)


def test_mixed_create_soft_culled_render_and_empty_heads_reject_bad_arguments_without_a_gpu():
    L = derf.lib()
    assert L.derf_create_mixed(None, 1, None, None, None, 1) == derf.DERF_ERR_INVALID_ARG
    archs = [scenes.ARCH_128, scenes.ARCH_SMALL, (10, 4, 8, 96, 5, 64)]
    arr = (derf.derf_head_arch * 3)(*[derf.derf_head_arch(*(a.as_tuple() if hasattr(a, "as_tuple")
                                                             else a)) for a in archs])
    sites = np.zeros((3, 3), np.float32)
    w = np.zeros(sum(max(0, derf.derf_weights_count(a)) for a in archs), np.float32)
    h = ctypes.c_void_p(1234)
    rc = L.derf_create_mixed(ctypes.byref(h), 3, sites.ctypes.data_as(ctypes.c_void_p),
                             ctypes.cast(arr, ctypes.POINTER(derf.derf_head_arch)),
                             w.ctypes.data_as(ctypes.c_void_p), 1)
    assert rc == derf.DERF_ERR_UNSUPPORTED and h.value is None
    assert b"head 2" in L.derf_last_error()
    good = (derf.derf_head_arch * 2)(derf.derf_head_arch(*scenes.ARCH_128.as_tuple()),
                                     derf.derf_head_arch(*scenes.ARCH_SMALL.as_tuple()))
    w2 = np.zeros(derf.derf_weights_count(scenes.ARCH_128) +
                  derf.derf_weights_count(scenes.ARCH_SMALL), np.float32)
    w2[-1] = np.inf
    rc = L.derf_create_mixed(ctypes.byref(h), 2, sites.ctypes.data_as(ctypes.c_void_p),
                             ctypes.cast(good, ctypes.POINTER(derf.derf_head_arch)),
                             w2.ctypes.data_as(ctypes.c_void_p), 1)
    assert rc == derf.DERF_ERR_INVALID_ARG and b"non-finite weight" in L.derf_last_error()
    assert L.derf_set_empty_heads(None, None) == derf.DERF_ERR_INVALID_ARG
    samp = derf.derf_sampling(32, 0, 1, 1, 0)
    assert L.derf_render_soft(None, None, None, 1, 2.0, 6.0, ctypes.byref(samp), 1.0, None, None,
                              None, None, None) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_render_culled(None, None, None, 1, 2.0, 6.0, ctypes.byref(samp), 1e-3, 4, 0,
                                None, None, None, None, None) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_set_gate(None, 6, 16, None) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_set_encoding(None, derf.DERF_ENCODING_STORED) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_render_gated(None, None, None, 1, 2.0, 6.0, ctypes.byref(samp), None, None,
                               None, None, None) == derf.DERF_ERR_INVALID_ARG
    assert L.derf_gate_weights_count(4, 6, 16) == 16 * 39 + 16 + 4 * 16 + 4
    assert L.derf_gate_weights_count(0, 6, 16) == -1


def test_binding_checks_host_weights_before_the_library_reads_them():
    """The library reads K * derf_weights_count floats (one architecture) or the
    per-head sum (mixed) from the host weights, and derf_gate_weights_count
    floats from a gate: the binding refuses arrays of any other length before
    the call, so a short array can never be read past its end."""
    sites = np.zeros((4, 3), np.float32)
    n = derf.derf_weights_count(scenes.ARCH_TINY)
    for size in (4 * n - 1, 4 * n + 1, n):
        with pytest.raises(ValueError, match="weights hold"):
            derf.derf_create(sites, scenes.ARCH_TINY, np.zeros(size, np.float32), 0)
    with pytest.raises(ValueError, match="invalid head architecture"):
        derf.derf_create(sites, (10, 4, 0, 128, -1, 0), np.zeros(16, np.float32), 0)
    with pytest.raises(ValueError, match="one architecture per site"):
        derf.derf_create(sites, [scenes.ARCH_TINY] * 3, [np.zeros(n, np.float32)] * 3, 0)
    count = derf.lib().derf_gate_weights_count(4, 6, 16)
    for size in (count - 1, count + 5):
        with pytest.raises(ValueError, match="gating weights hold"):
            derf.derf_set_gate(None, 6, 16, np.zeros(size, np.float32), 4)


def test_binding_checks_ray_and_output_tensors_before_the_call():
    """Rays must be contiguous float32 GPU tensors of shape [R, 3]; every output
    must be a contiguous tensor of the right dtype on the rays' device with at
    least as many elements as the render writes.  These checks run before any
    pointer reaches the library (here on CPU tensors, so no GPU is touched)."""
    torch = pytest.importorskip("torch")
    o = torch.zeros((5, 3))
    with pytest.raises(ValueError, match="GPU tensor"):
        derf.check_rays(o, o)
    with pytest.raises(ValueError, match="GPU tensor"):
        derf.derf_render(None, o, o, 2.0, 6.0, derf.derf_sampling(8, 0, 1, 1, 0), o, o[:, 0],
                         o[:, 1])
    cpu = torch.device("cpu")
    derf.check_out(torch.zeros(15), "out_rgb", 15, torch.float32, cpu)
    derf.check_out(None, "out_cell", 15, torch.int32, cpu, optional=True)
    with pytest.raises(ValueError, match="is required"):
        derf.check_out(None, "out_rgb", 15, torch.float32, cpu)
    with pytest.raises(ValueError, match="holds 14 elements"):
        derf.check_out(torch.zeros(14), "out_rgb", 15, torch.float32, cpu)
    with pytest.raises(ValueError, match="must be torch.float32"):
        derf.check_out(torch.zeros(15, dtype=torch.float64), "out_rgb", 15, torch.float32, cpu)
    with pytest.raises(ValueError, match="must be torch.int32"):
        derf.check_out(torch.zeros(15), "out_cell", 15, torch.int32, cpu)
    with pytest.raises(ValueError, match="contiguous"):
        derf.check_out(torch.zeros((5, 6))[:, ::2], "out_rgb", 15, torch.float32, cpu)
    with pytest.raises(ValueError, match="rays' device"):
        derf.check_out(torch.zeros(15, device="meta"), "out_rgb", 15, torch.float32, cpu)
    with pytest.raises(ValueError, match="must be a torch tensor"):
        derf.check_out(np.zeros(15, np.float32), "out_rgb", 15, torch.float32, cpu)


def test_status_strings():
    L = derf.lib()
    assert L.derf_status_string(0) == b"ok"
    assert L.derf_status_string(-2) == b"unsupported"
    assert L.derf_status_string(-99) == b"unknown status"
