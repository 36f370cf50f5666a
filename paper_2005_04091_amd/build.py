"""Build libspconv.so (HIP for gfx950) in-tree with hipcc.

``python -m paper_2005_04091_amd.build`` compiles the kernels and the C-ABI in
``csrc/`` into ``paper_2005_04091_amd/libspconv.so``.
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
INCLUDE = ROOT / "include"
LIB_PATH = PKG / "libspconv.so"
SOURCES = [CSRC / "spconv.hip", CSRC / "dense.hip", CSRC / "pack.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-FP32 VALU instructions are disabled for all device code: hipcc would
# otherwise form v_pk_fma_f32 / v_pk_add_f32 / v_pk_mul_f32 from scalar float code.
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(verbose: bool = False) -> Path:
    tmp = LIB_PATH.with_name(LIB_PATH.name + f".tmp{os.getpid()}")
    cmd = [HIPCC, "-O3", "-std=c++17", "-fPIC", "-shared", *DEVICE_FLAGS, "-I", str(INCLUDE),
           *map(str, SOURCES), "-o", str(tmp)]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the device-only feature name; that warning is harmless.
    noise = "'-packed-fp32-ops' is not a recognized feature for this target (ignoring feature)"
    err = "\n".join(l for l in res.stderr.splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{err}")
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
