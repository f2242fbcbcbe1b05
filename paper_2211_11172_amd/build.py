"""Build libharl.so (the HIP kernels and the C ABI) for gfx950 with hipcc, in-tree.

Usage: ``python -m paper_2211_11172_amd.build`` (or ``build()`` from Python).  Objects go to
``paper_2211_11172_amd/_build``; the library to ``paper_2211_11172_amd/libharl.so``, and the
visit-loop microbenchmark (``probe/``) to ``paper_2211_11172_amd/libharl_probe.so``.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OUT_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libharl.so")
ARCH = os.environ.get("HARL_OFFLOAD_ARCH", "gfx950")


def hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libharl)")


# -packed-fp32-ops is disabled: the kernels are written without packed fp32 arithmetic and the
# compiler must not introduce it either.  No fast-math: the traversal relies on NaN compares.
CXXFLAGS = ["-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-pass-failed", "-Wno-unused-function"]


def _compile(src: str) -> str:
    obj = os.path.join(OUT_DIR, os.path.basename(src) + ".o")
    cmd = [hipcc(), *CXXFLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    jobs = min(len(srcs), int(os.environ.get("MAX_JOBS", "8")))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIB)
    # the visit-loop microbenchmark (probe/): a separate library only the benchmark loads
    for src in sorted(glob.glob(os.path.join(PKG, "probe", "*.hip"))):
        out = os.path.join(PKG, "lib" + "harl_probe" + ".so")
        tmp = out + ".tmp%d" % os.getpid()
        r = subprocess.run([hipcc(), *CXXFLAGS, "-shared", src, "-o", tmp], capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, r.stdout, r.stderr))
        os.replace(tmp, out)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
