"""Build libA2T.so in-tree with hipcc for gfx950.

Usage: ``python paper_2609_31224_amd/build.py`` (run it as a script: importing
the package itself loads the library).  The library lands next to this file;
a build always recompiles.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libA2T.so")
SOURCES = ["kernels.hip", "a2t.cpp", "distill.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # packed fp32 instructions are disabled for every HIP code object
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    p = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (p.stderr or "").splitlines() if noise not in l)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


def build(verbose: bool = False) -> str:
    """Compile every source and link libA2T.so; returns its path."""
    tmpdir = tempfile.mkdtemp(prefix="a2t_build_")
    try:
        objs = []
        for src in SOURCES:
            obj = os.path.join(tmpdir, src + ".o")
            _run([HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj], verbose)
            objs.append(obj)
        tmp_lib = os.path.join(tmpdir, "libA2T.so")
        _run([HIPCC, *FLAGS, "-shared", *objs, "-o", tmp_lib], verbose)
        shutil.move(tmp_lib, LIB + ".tmp")
        os.replace(LIB + ".tmp", LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
