"""Build libderf.so (HIP, gfx950) in-tree.

Each source is compiled to an object in _build/ (in parallel), then linked
into paper_2011_12490_amd/libderf.so.  The library links the HIP runtime by
soname, so inside a process that imported torch it shares torch's runtime.
"""
import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libderf.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# the grouped MLP is instantiated per head architecture, one unit each, so
# that its variants compile in parallel
SOURCES = ["mlp_8x256.hip", "mlp_8x128.hip", "mlp_6x64.hip", "mlp_4x64.hip", "kernels_sample.hip",
           "kernels_fine.hip", "kernels_soft.hip", "kernels_gate.hip", "derf_api.cpp"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "--offload-arch=" + ARCH,
          "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
          # no packed-fp32 VALU ops in device code
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-function"]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"]
    cmd = [HIPCC] + lang + COMMON + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s\n%s" % (" ".join(cmd), r.stdout, r.stderr))
    return obj


# The matrix-core throughput probe (csrc/mfma_probe.hip): a library of its
# own, loaded only by the benchmark's --mfma-ceiling report.
PROBE_LIB = os.path.join(PKG, "libderf_probe.so")


def build(jobs: int = 8) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, SOURCES + ["mfma_probe.hip"]))
    probe_obj = objs.pop()
    tmp = PROBE_LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp, probe_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s\n%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, PROBE_LIB)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s\n%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, LIB)
    return LIB


# Test driver of the C ABI (tests/abi_driver.cpp): the library's host code
# compiled with allocation-failure injection, linked with the kernels built
# above.  With asan, the host code (never the device code) is also built with
# AddressSanitizer, for runs on the CPU.
ASAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]


def build_abi_driver(out: str, asan: bool = False) -> str:
    if not os.path.exists(os.path.join(BUILD, "derf_api.o")):
        build()
    tmpdir = os.path.dirname(os.path.abspath(out))
    os.makedirs(tmpdir, exist_ok=True)
    extra = (ASAN_HOST + ["-g", "-O1"]) if asan else ["-O2"]
    api = out + ".api.o"
    drv = out + ".drv.o"
    steps = [
        [HIPCC, "-x", "hip"] + COMMON + extra + ["-DDERF_FAULT_INJECTION", "-c",
                                                  os.path.join(CSRC, "derf_api.cpp"), "-o", api],
        [HIPCC, "-x", "hip"] + COMMON + extra + ["-c", os.path.join(ROOT, "tests", "abi_driver.cpp"),
                                                  "-o", drv],
        [HIPCC, "--offload-arch=" + ARCH] + (ASAN_HOST if asan else []) +
        ["-o", out, drv, api] + [os.path.join(BUILD, os.path.splitext(x)[0] + ".o")
                                 for x in SOURCES if x != "derf_api.cpp"],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("abi driver build failed: %s\n%s\n%s"
                               % (" ".join(cmd), r.stdout, r.stderr))
    for f in (api, drv):
        os.remove(f)
    return out


if __name__ == "__main__":
    print(build())
    sys.exit(0)
