"""Builds libtbs.so (the gfx950 HIP library behind include/tbs.h) in place.

Each source compiles to its own object (in parallel), then hipcc links the shared
library.  Usage: python -m paper_2211_00484_amd.csrc.build   (or via
__graft_entry__.build())
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libtbs.so")
SOURCES = ["api.cpp", "kernels.hip", "lattice.hip", "hyps.hip", "transducer.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-fp32 VALU forms are kept out of the generated code on purpose.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include"), "-I", HERE]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed building libtbs.so: " + " ".join(cmd[-3:]))


def build(verbose: bool = False) -> str:
    with tempfile.TemporaryDirectory(prefix="tbs_build_") as tmpdir:
        jobs = []
        for s in SOURCES:
            src = os.path.join(HERE, s)
            obj = os.path.join(tmpdir, s + ".o")
            lang = ["-x", "hip"] if s.endswith(".cpp") else []
            jobs.append(([HIPCC] + FLAGS + ["-c"] + lang + [src, "-o", obj], obj))
        with ThreadPoolExecutor(max_workers=len(jobs)) as ex:
            for f in [ex.submit(_run, cmd, verbose) for cmd, _ in jobs]:
                f.result()
        tmp = LIB + ".tmp"
        _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + [o for _, o in jobs] +
             ["-o", tmp], verbose)
        os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
