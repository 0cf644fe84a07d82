"""Builds libtbs.so (the gfx950 HIP library behind include/tbs.h) in place.

Usage: python -m paper_2211_00484_amd.csrc.build   (or via __graft_entry__.build())
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libtbs.so")
SOURCES = ["api.cpp", "kernels.hip", "lattice.hip", "hyps.hip", "transducer.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-fp32 VALU forms are kept out of the generated code on purpose.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", HERE]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    srcs = []
    for s in SOURCES:
        p = os.path.join(HERE, s)
        srcs += ["-x", "hip", p] if s.endswith(".cpp") else [p]
    cmd = [HIPCC] + FLAGS + srcs + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building libtbs.so")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
