"""Plain fp64 CPU oracle for the per-layer adjoint gradient of a selective
diagonal SSM layer (adjoint sharding, arXiv 2501.00692).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``.  It never imports the HIP package
and the HIP package never imports it.

What each function follows (sections, propositions and equations of the paper):

* :func:`forward` -- Sec. 3.1, the five SSM steps, sequential in t.
* :func:`bptt` -- the exact gradient of ``L = sum dy * out`` by backpropagation
  through time (the nested expansion in Sec. 3.3, evaluated from the outer
  step inwards; Prop. 1's recurrence for the state cotangent).
* :func:`adjoint_sum` -- Prop. 2 taken literally, and with ``tbar`` the
  truncated estimator of Eq. "capped" taken literally: for every loss term t
  the adjoint states ``lambda^{t,i} = C^t A^t ... A^{i+1}`` for i = t, t-1, ...
  down to the window edge, each vjp accumulated.  O(T * Tbar) per channel.
* :func:`trunc_tail` -- the same truncated estimator rewritten with the tail
  identity ``sum_{t=i}^{i+Tbar-1} g_t lambda^{t,i} = mu_i - P(i,i+Tbar) mu_{i+Tbar}``
  where ``mu_i = sum_{t>=i} g_t lambda^{t,i}`` obeys ``mu_i = g_i C_i + a_{i+1} mu_{i+1}``
  and ``P(i,j) = prod_{k=i+1}^{j} a_k``.  O(T) per channel; pinned against
  :func:`adjoint_sum` by the tests.
* :func:`layer_grad` -- the chain rule through the input projections (the
  A, B, C networks as single-layer maps, Sec. 4.5) and the SiLU gate, with
  numpy fp64 matmuls as the library primitive.
* :func:`proj_dw`, :func:`proj_dx` -- ``dW = X^T dZ`` and ``dX = dZ W^T`` on
  sampled entries, from bf16 operands upcast exactly.
* :func:`vjp_count_full`, :func:`vjp_count_truncated` -- the number of
  (t, i) VJP pairs of Sec. 4.3, written as plain sums.

Readings of the paper used here (where it is silent or garbled):

* window edges: for t > Tbar the truncated sum keeps i in [t+1-Tbar, t]
  (exactly Tbar terms); for t <= Tbar it keeps i in [1, t]; Tbar >= T is the
  full gradient;
* the vjp_C term is never truncated;
* the truncated VJPs use the true full-history states h;
* dx is the B-path cotangent summed over the state (the paper differentiates
  only the parameters);
* dh0 exists for the full gradient only;
* the discretisation is a = exp(-Delta e^{A_log}) and h = a h + B x, with no
  Delta factor on B; two variants are selectable: ``a_scalar`` (the "scalar
  SSM" row of Table 1: one decay per channel, ``A_log`` of shape [D]) and
  ``b_delta`` (the input term scaled by the step size, ``h = a h + Delta B x``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_HERE = Path(__file__).resolve().parent
_SRC = _HERE / "oracle.c"
_LIB = _HERE / "liboracle.so"
_lib = None


def build(force: bool = False) -> Path:
    """Compile ``liboracle.so`` with gcc (OpenMP).  Rebuilds when stale."""
    if force or not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
        tmp = _LIB.with_suffix(".so.tmp")
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
               "-o", str(tmp), str(_SRC), "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(str(_LIB))
        i64, dp, ip = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int
        lib.oracle_forward.argtypes = [i64, i64, i64, i64, dp, dp, ip, dp, dp, dp, dp, dp, dp, dp, ip]
        grad_args = [dp, dp, ip, dp, dp, dp, dp, dp, dp, dp, dp, dp, dp, dp, dp, dp, dp, ip]
        lib.oracle_bptt.argtypes = [i64, i64, i64, i64] + grad_args
        lib.oracle_adjoint_sum.argtypes = [i64, i64, i64, i64, i64] + grad_args
        lib.oracle_trunc_tail.argtypes = [i64, i64, i64, i64, i64] + grad_args
        lib.oracle_proj_dw.argtypes = [i64, i64, i64, dp, i64, dp, i64, i64, dp, dp, dp, ip]
        lib.oracle_proj_dx.argtypes = [i64, i64, i64, dp, i64, dp, i64, i64, dp, dp, ip]
        lib.oracle_max_threads.argtypes = []
        for f in ("oracle_forward", "oracle_bptt", "oracle_adjoint_sum", "oracle_trunc_tail",
                  "oracle_proj_dw", "oracle_proj_dx", "oracle_max_threads"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def max_threads() -> int:
    return _load().oracle_max_threads()


def _f64(a):
    if a is None:
        return None
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


# variant bits of the C oracle's `flags` argument
_SOFTPLUS, _A_SCALAR, _B_DELTA = 1, 2, 4


def _flags(delta_softplus, a_scalar, b_delta):
    return (_SOFTPLUS if delta_softplus else 0) | (_A_SCALAR if a_scalar else 0) | (_B_DELTA if b_delta else 0)


def forward(x, delta, A_log, B, C, h0=None, z=None, delta_softplus=False, nthreads=0, a_scalar=False,
            b_delta=False):
    """Sec. 3.1 forward.  Returns ``(out, h_last)``; ``out = y`` or ``y*silu(z)``."""
    x, delta, A_log, B, C, h0, z = map(_f64, (x, delta, A_log, B, C, h0, z))
    nb, T, D = x.shape
    N = B.shape[-1]
    assert A_log.shape == ((D,) if a_scalar else (D, N))
    out = np.empty((nb, T, D))
    h_last = np.empty((nb, D, N))
    rc = _load().oracle_forward(nb, T, D, N, _ptr(x), _ptr(delta), _flags(delta_softplus, a_scalar, b_delta), _ptr(A_log),
                                _ptr(B), _ptr(C), _ptr(h0), _ptr(z), _ptr(out), _ptr(h_last), nthreads)
    if rc:
        raise ValueError(f"oracle_forward failed ({rc})")
    return out, h_last


def _grad(fn, with_tbar, tbar, x, delta, A_log, B, C, dy, h0, z, delta_softplus, want_dh0, nthreads,
          a_scalar=False, b_delta=False, want_da=False):
    x, delta, A_log, B, C, h0, z, dy = map(_f64, (x, delta, A_log, B, C, h0, z, dy))
    nb, T, D = x.shape
    N = B.shape[-1]
    assert A_log.shape == ((D,) if a_scalar else (D, N))
    out = {
        "dx": np.empty((nb, T, D)), "ddelta": np.empty((nb, T, D)), "dA_log": np.empty(A_log.shape),
        "dB": np.empty((nb, T, N)), "dC": np.empty((nb, T, N)),
    }
    out["dz"] = np.empty((nb, T, D)) if z is not None else None
    out["dh0"] = np.empty((nb, D, N)) if want_dh0 else None
    out["da"] = np.empty((nb, T, D, N)) if want_da else None
    head = (nb, T, D, N, int(tbar)) if with_tbar else (nb, T, D, N)
    rc = fn(*head, _ptr(x), _ptr(delta), _flags(delta_softplus, a_scalar, b_delta), _ptr(A_log), _ptr(B),
            _ptr(C), _ptr(h0),
            _ptr(z), _ptr(dy), _ptr(out["dx"]), _ptr(out["ddelta"]), _ptr(out["dA_log"]), _ptr(out["dB"]),
            _ptr(out["dC"]), _ptr(out["dz"]), _ptr(out["dh0"]), _ptr(out["da"]), nthreads)
    if rc:
        raise ValueError(f"oracle gradient failed ({rc})")
    return out


def bptt(x, delta, A_log, B, C, dy, h0=None, z=None, delta_softplus=False, want_dh0=True, nthreads=0,
         a_scalar=False, b_delta=False, want_da=False):
    """Exact full gradient by backpropagation through time (dict of arrays).
    ``want_da`` adds ``da`` [b, T, D, N], the cotangent of the decay a_t itself."""
    return _grad(_load().oracle_bptt, False, 0, x, delta, A_log, B, C, dy, h0, z, delta_softplus,
                 want_dh0, nthreads, a_scalar, b_delta, want_da)


def adjoint_sum(x, delta, A_log, B, C, dy, tbar=0, h0=None, z=None, delta_softplus=False,
                want_dh0=None, nthreads=0, a_scalar=False, b_delta=False, want_da=False):
    """Prop. 2 (``tbar<=0`` or ``tbar>=T``) / Eq. "capped" double sum, literally."""
    T = np.shape(x)[1]
    full = tbar <= 0 or tbar >= T
    if want_dh0 is None:
        want_dh0 = full
    return _grad(_load().oracle_adjoint_sum, True, tbar, x, delta, A_log, B, C, dy, h0, z,
                 delta_softplus, want_dh0, nthreads, a_scalar, b_delta, want_da)


def trunc_tail(x, delta, A_log, B, C, dy, tbar=0, h0=None, z=None, delta_softplus=False,
               want_dh0=None, nthreads=0, a_scalar=False, b_delta=False, want_da=False):
    """Truncated estimator via the tail identity (O(T) per channel)."""
    T = np.shape(x)[1]
    full = tbar <= 0 or tbar >= T
    if want_dh0 is None:
        want_dh0 = full
    return _grad(_load().oracle_trunc_tail, True, tbar, x, delta, A_log, B, C, dy, h0, z,
                 delta_softplus, want_dh0, nthreads, a_scalar, b_delta, want_da)


def silu(z):
    return z / (1.0 + np.exp(-z))


def layer_forward(u, W_in, W_x, A_log, N, h0=None):
    """Layer forward with projections: ``[x | z] = u W_in``, ``[Delta_pre | B | C] = x W_x``,
    ``Delta = softplus(Delta_pre)``, ``out = y * silu(z)``.  fp64 throughout."""
    u, W_in, W_x = _f64(u), _f64(W_in), _f64(W_x)
    D = W_x.shape[0]
    xz = u @ W_in
    x, z = xz[..., :D], xz[..., D:]
    pj = x @ W_x
    dpre, B, C = pj[..., :D], pj[..., D:D + N], pj[..., D + N:]
    out, h_last = forward(x, dpre, A_log, B, C, h0=h0, z=z, delta_softplus=True)
    return out, dict(x=x, z=z, dpre=dpre, B=B, C=C, h_last=h_last)


def layer_grad(u, x, z, dpre, B, C, W_x, A_log, dy, W_in=None, tbar=0, scan=None, a_scalar=False,
               b_delta=False):
    """Gradient of ``L = sum dy * out`` for the layer with input projections.

    ``scan`` selects the scan gradient: ``bptt`` (default, full), ``trunc_tail`` or
    ``adjoint_sum`` (truncated with ``tbar``).  Chain rule (matmul = library primitive):
    ``dZx = [dDelta_pre | dB | dC]``, ``dW_x = x^T dZx``, ``dx_total = dx_scan + dZx W_x^T``,
    ``dW_in = u^T [dx_total | dz]``, ``du = [dx_total | dz] W_in^T``.
    """
    u, x, z, dpre, B, C, W_x, dy = map(_f64, (u, x, z, dpre, B, C, W_x, dy))
    v = dict(a_scalar=a_scalar, b_delta=b_delta)
    if scan is None:
        g = bptt(x, dpre, A_log, B, C, dy, z=z, delta_softplus=True, want_dh0=False, **v)
    else:
        g = scan(x, dpre, A_log, B, C, dy, tbar=tbar, z=z, delta_softplus=True, want_dh0=False, **v)
    nb, T, D = x.shape
    M = nb * T
    dZx = np.concatenate([g["ddelta"], g["dB"], g["dC"]], axis=-1).reshape(M, -1)
    xf = x.reshape(M, D)
    dW_x = xf.T @ dZx
    dx_total = g["dx"].reshape(M, D) + dZx @ W_x.T
    dxz = np.concatenate([dx_total, g["dz"].reshape(M, D)], axis=-1)
    dW_in = u.reshape(M, -1).T @ dxz
    res = dict(g)
    res.update(dZx=dZx, dW_x=dW_x, dx_total=dx_total, dxz=dxz, dW_in=dW_in)
    if W_in is not None:
        res["du"] = dxz @ _f64(W_in).T
    return res


def proj_dw(X, dZ, kk, jj, nthreads=0):
    """``dW[k, j] = sum_m X[m, k] dZ[m, j]`` for the sampled (k, j) pairs.

    ``X`` and ``dZ`` are 2-D uint16 arrays holding bf16 bit patterns."""
    X = np.ascontiguousarray(X, dtype=np.uint16)
    dZ = np.ascontiguousarray(dZ, dtype=np.uint16)
    kk = np.ascontiguousarray(kk, dtype=np.int64)
    jj = np.ascontiguousarray(jj, dtype=np.int64)
    M, K = X.shape
    Nout = dZ.shape[1]
    out = np.empty(len(kk))
    rc = _load().oracle_proj_dw(M, K, Nout, _ptr(X), K, _ptr(dZ), Nout, len(kk), _ptr(kk), _ptr(jj),
                                _ptr(out), nthreads)
    if rc:
        raise ValueError("oracle_proj_dw failed")
    return out


def proj_dx(dZ, W, rows, nthreads=0):
    """``dX[m, :] = dZ[m, :] W^T`` for the sampled rows; ``W`` is [K, Nout] (bf16 bits)."""
    dZ = np.ascontiguousarray(dZ, dtype=np.uint16)
    W = np.ascontiguousarray(W, dtype=np.uint16)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    M, Nout = dZ.shape
    K = W.shape[0]
    out = np.empty((len(rows), K))
    rc = _load().oracle_proj_dx(M, K, Nout, _ptr(dZ), Nout, _ptr(W), Nout, len(rows), _ptr(rows),
                                _ptr(out), nthreads)
    if rc:
        raise ValueError("oracle_proj_dx failed")
    return out


def vjp_count_full(T: int) -> int:
    """Number of (t, i) pairs of the A/B vjps in the full sum of Prop. 2, summed over t."""
    return sum(t for t in range(1, T + 1))


def vjp_count_truncated(T: int, tbar: int) -> int:
    """Number of (t, i) pairs kept by Eq. "capped": min(t, Tbar) per t."""
    return sum(min(t, tbar) for t in range(1, T + 1))
