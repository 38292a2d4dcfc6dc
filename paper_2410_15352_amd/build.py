"""Build the HIP library ``libcompact.so`` in-tree for gfx950.

    python -m paper_2410_15352_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
LIB = os.path.join(PKG_DIR, "libcompact.so")
INCLUDE = os.path.join(ROOT, "include")

# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU ops.
# -ffp-contract=off: every fp32 expression rounds once per operation, so the
#   projection stream and the update epilogue are reproducible bit for bit.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]

# Translation units and their extra flags.  The persistent GEMM's K steps are
# written in issue order, so its unit is compiled with the machine scheduler off.
UNITS = [
    ("compact_api.hip", []),
    ("kernels_w4.hip", ["-mllvm", "-enable-misched=false", "-mllvm", "-enable-post-misched=false"]),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the CompAct HIP library cannot be built")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + res.stdout + res.stderr)


def build_library(verbose: bool = False) -> str:
    """Compile the units in csrc/ (and the headers they include) to libcompact.so."""
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="compact_build_") as objdir:
        objs = []
        for name, extra in UNITS:
            obj = os.path.join(objdir, name.replace(".hip", ".o"))
            _run([hipcc(), *FLAGS, *extra, "-I", INCLUDE, "-c", os.path.join(CSRC, name), "-o", obj], verbose)
            objs.append(obj)
        _run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build_library(verbose="-v" in sys.argv))
