"""Compile the HIP library ``libssm_adjoint.so`` for gfx950 with hipcc.

Usage: ``python -m paper_2501_00692_amd.build`` (or ``build()`` from Python).
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
SRC = [CSRC / "scan.hip", CSRC / "scan_grad_f32_full.hip", CSRC / "scan_grad_f32_trunc.hip",
       CSRC / "scan_grad_bf16_full.hip", CSRC / "scan_grad_bf16_trunc.hip", CSRC / "gemm.hip", CSRC / "pairs.hip", CSRC / "stack.hip",
       CSRC / "noalloc.hip", CSRC / "layer.hip", CSRC / "da_debug.hip", CSRC / "unstructured.hip", CSRC / "head.hip", CSRC / "abi.cpp", CSRC / "timing.cpp"]
OBJ = PKG / "_build"
LIB = PKG / "libssm_adjoint.so"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", str(ROOT / "include"),
    "-I", str(PKG / "csrc"),
]


def _compile(src: Path, verbose: bool) -> Path:
    obj = OBJ / (src.name + ".o")
    cmd = [HIPCC, *FLAGS, "-c", "-o", str(obj), str(src)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return obj


def build(verbose: bool = False, jobs: int | None = None) -> Path:
    """Compile every source (in parallel) and link the shared library."""
    from concurrent.futures import ThreadPoolExecutor

    OBJ.mkdir(exist_ok=True)
    jobs = jobs or min(len(SRC), os.cpu_count() or 1)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SRC))
    tmp = LIB.with_suffix(".so.tmp")
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", str(tmp), *map(str, objs)]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    print(LIB, file=sys.stderr)
