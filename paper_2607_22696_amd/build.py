"""Builds libdsa3d.so (gfx950 HIP kernels + C-ABI host code) in-tree with hipcc, and the
gather-bandwidth microbenchmark libdsa3d_probe.so that bench.py uses for its ceiling."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdsa3d.so")
PROBE_LIB = os.path.join(PKG, "libdsa3d_probe.so")
PROBE_SOURCES = [os.path.join(CSRC, "gather_probe.hip")]

SOURCES = [os.path.join(CSRC, "dsa3d_forward.hip"), os.path.join(CSRC, "dsa3d_backward.hip"),
           os.path.join(CSRC, "dwconv3d.hip"), os.path.join(CSRC, "dsa3d_api.cpp"),
           os.path.join(CSRC, "dwconv3d_api.cpp"), os.path.join(CSRC, "winattn.hip"),
           os.path.join(CSRC, "winattn_api.cpp")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-munsafe-fp-atomics",
    # no packed-FP32 instructions in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def build(verbose: bool = False) -> str:
    _compile(SOURCES, LIB, verbose)
    _compile(PROBE_SOURCES, PROBE_LIB, verbose)
    return LIB


def _compile(sources, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", INCLUDE, "-I", CSRC, *sources, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    errs = [ln for ln in (res.stderr or "").splitlines()
            if "packed-fp32-ops' is not a recognized feature" not in ln]
    if res.returncode != 0:
        sys.stderr.write("\n".join(errs) + "\n")
        raise RuntimeError(f"hipcc failed ({res.returncode})")
    if verbose and errs:
        sys.stderr.write("\n".join(errs) + "\n")
    os.replace(tmp, lib)


if __name__ == "__main__":
    print(build(verbose=True))
