"""The C ABI driven from C++ (tests/abi_driver.cpp), linked with a test build
of the library's host code that can make any allocation fail:

* on the CPU, with the host code built under AddressSanitizer (leak checks
  on): every argument check, the clean-up of a handle whose device setup
  fails, and a failed handle allocation;
* on the GPU (the driver built by ``__graft_entry__.build()`` into the
  package's ``_build/``, without sanitizer): every allocation of derf_create,
  derf_create_mixed, the render workspace and derf_set_gate made to fail in
  turn -- each returns DERF_ERR_OOM, hands out no handle, leaves an existing
  handle working and releases what it had taken.
"""
import os
import subprocess

import pytest

from paper_2011_12490_amd import build

DRIVER = os.path.join(build.BUILD, "abi_driver")


def _run(exe, env=None):
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, **(env or {})))
    print(r.stdout[-3000:], r.stderr[-3000:], flush=True)
    return r


def test_abi_driver_with_host_asan_on_the_cpu(tmp_path):
    """Host code under AddressSanitizer with leak detection; no GPU is used
    (the CPU suite runs where there is none)."""
    exe = build.build_abi_driver(str(tmp_path / "abi_asan"), asan=True)
    r = _run(exe, {"ASAN_OPTIONS": "detect_leaks=1"})
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi driver: 0 failure(s)" in r.stdout
    assert "ERROR: AddressSanitizer" not in r.stderr
    assert "ERROR: LeakSanitizer" not in r.stderr


@pytest.mark.gpu
def test_allocation_failures_on_the_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(DRIVER), "build the test driver first (__graft_entry__.build())"
    r = _run(DRIVER)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi driver: 0 failure(s)" in r.stdout
    assert "render workspace, gate and stored-encoding failures handled" in r.stdout
