"""Builds libdsa3d.so (gfx950 HIP kernels + C-ABI host code) in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libdsa3d.so")

SOURCES = [os.path.join(CSRC, "dsa3d_forward.hip"), os.path.join(CSRC, "dsa3d_backward.hip"),
           os.path.join(CSRC, "dsa3d_noalloc.hip"),
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
    # no packed-FP32 instructions in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
]


def build(verbose: bool = False) -> str:
    compile_shared(SOURCES, LIB, verbose)
    return LIB


def compile_shared(sources, lib, verbose=False):
    """hipcc the sources into the shared library `lib` (replaced only when the build
    succeeds)."""
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
