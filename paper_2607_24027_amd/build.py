"""Build libsolattn.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2607_24027_amd.build   (or call build()).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libsolattn.so")
SOURCES = ["sol_attn_kernels.hip", "sol_attn_baselines.hip", "sol_attn_noalloc.hip", "sol_attn_api.cpp"]
ARCH = os.environ.get("SOL_ATTN_ARCH", "gfx950")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    objs = []
    common = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
              "-I", os.path.join(ROOT, "include"),
              # packed-f32 VALU forms are kept out of the generated code
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    build_dir = os.path.join(HERE, "_build")
    os.makedirs(build_dir, exist_ok=True)
    for src in SOURCES:
        obj = os.path.join(build_dir, src + ".o")
        # Kernels never see NaN by contract (NaN inputs are invalid); this lets max() skip
        # NaN canonicalisation of MFMA results.  Infinities keep their IEEE meaning.
        extra = ["-fno-honor-nans"] if src.endswith(".hip") else []
        cmd = [hipcc(), "-x", "hip", *common, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
        _run(cmd, verbose)
        objs.append(obj)
    tmp = LIB + ".tmp"
    _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    # An unresolved kernel handle (e.g. a kernel the host pass dropped) only shows up at
    # load time: load the fresh library once so such a build fails here.
    import ctypes
    ctypes.CDLL(tmp)
    os.replace(tmp, LIB)
    return LIB


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)


if __name__ == "__main__":
    print(build(verbose=True))
