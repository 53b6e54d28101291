"""Shared helpers of the GPU parity tests (inputs from the seeded generator, the
oracle on the host, and the per-tensor relative-L2 metric)."""
from __future__ import annotations

import sys

import numpy as np
import torch

# Tolerances (rel-L2 per output tensor): fp32 inputs, and bf16 inputs with fp32
# accumulation.
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().double().numpy()


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    if den == 0.0:
        return float(num)
    return float(num / den)


def check(name: str, got, ref, tol: float, report: dict | None = None):
    e = rel_l2(got, ref)
    if report is not None:
        report[name] = e
    assert np.all(np.isfinite(np.asarray(got, dtype=np.float64))), f"{name}: non-finite values"
    assert e <= tol, f"{name}: rel-L2 {e:.3e} > {tol:.1e}"
    return e
