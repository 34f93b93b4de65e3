"""Builds libfkv.so (the C-ABI HIP library) in-tree for gfx950 with hipcc.

Every call recompiles; ``python -m paper_2607_07144_amd.build`` does the same
from the command line.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libfkv.so")

SOURCES = ["fkv_codec.cpp", "cgr_kernels.hip", "rvq_kernels.hip", "archive_kernels.hip", "kmeans_kernels.hip",
           "diag_kernels.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

COMMON = ["-O3", "-fPIC", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", "-fno-slp-vectorize",
          "-I" + INCLUDE, "-I" + CSRC]
# Device code: no packed-fp32 instructions; hipcc's host pass warns that it
# does not know the feature, which is harmless.
DEVICE = ["-x", "hip", "--offload-arch=" + ARCH,
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, obj: str) -> None:
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        cmd = [HIPCC] + DEVICE + COMMON + ["-c", path, "-o", obj]
    else:
        # host-only codec setup: libm sin and cos called as written (no sincos fusion)
        cmd = [HIPCC] + COMMON + ["-fno-builtin", "-c", path, "-o", obj]
    subprocess.check_call(cmd)


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libfkv.so next to this file."""
    bdir = os.path.join(PKG, "_build")
    os.makedirs(bdir, exist_ok=True)
    objs = [os.path.join(bdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        list(ex.map(lambda a: _compile(*a), zip(SOURCES, objs)))
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.check_call([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
