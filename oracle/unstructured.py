"""Oracle for the unstructured SSM of Table 1 (test infrastructure only).

Plain numpy fp64 with a Python loop over time.  Only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline may import it; it
shares nothing with the HIP library.

The layer is the general SSM of Sec. 3.1 with an N-dimensional state shared by
the P channels and input-dependent matrices (the outputs of the A, B, C
networks at each step, taken here as given):

    h_t = A_t h_{t-1} + B_t x_t,   y_t = C_t h_t,
    A_t in R^{N x N},  B_t in R^{N x P},  C_t in R^{P x N},  x_t, y_t in R^P,

with h_{-1} = h0 (zero unless given) and the loss L = sum_{b,t} <dy_t, y_t>.
Gradients are taken with respect to the per-step matrices and inputs:
dA [b,T,N,N], dB [b,T,N,P], dC [b,T,P,N], dx [b,T,P] and dh0 [b,N] (the
chain through the networks' parameters is a product with the networks'
inputs, as for the diagonal layer's projections).

* :func:`un_forward`   -- the recurrence, step by step.
* :func:`un_bptt`      -- backpropagation through time: the state cotangent
  mu_t = C_t^T dy_t + A_{t+1}^T mu_{t+1} (Prop. 1's recurrence), then
  dA_t = mu_t h_{t-1}^T, dB_t = mu_t x_t^T, dx_t = B_t^T mu_t, dC_t = dy_t h_t^T.
* :func:`un_adjoint_sum` -- Prop. 2 and Eq. "capped" literally: for each loss
  term t the adjoint state lambda^{t,i} = (C_t A_t ... A_{i+1})^T dy_t for
  i = t, t-1, ... down to the window edge (i >= t - Tbar + 1 when truncated),
  with the A-, B- and x-path vjps of step i accumulated; the C term is never
  truncated.
"""
from __future__ import annotations

import numpy as np


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def un_forward(A, B, C, x, h0=None):
    """Returns (y [b,T,P], h_last [b,N], hs [b,T+1,N]) with hs[:, 0] = h0."""
    A, B, C, x, h0 = map(_f64, (A, B, C, x, h0))
    nb, T, N, P = B.shape
    hs = np.zeros((nb, T + 1, N))
    if h0 is not None:
        hs[:, 0] = h0
    y = np.zeros((nb, T, P))
    for t in range(T):
        for b in range(nb):
            hs[b, t + 1] = A[b, t] @ hs[b, t] + B[b, t] @ x[b, t]
            y[b, t] = C[b, t] @ hs[b, t + 1]
    return y, hs[:, T].copy(), hs


def un_bptt(A, B, C, x, dy, h0=None, want_dh0=True):
    """Exact gradient of L = sum <dy, y> by backpropagation through time."""
    A, B, C, x, dy = map(_f64, (A, B, C, x, dy))
    nb, T, N, P = B.shape
    _, _, hs = un_forward(A, B, C, x, h0)
    out = dict(dA=np.zeros_like(A), dB=np.zeros_like(B), dC=np.zeros_like(C), dx=np.zeros_like(x),
               dh0=np.zeros((nb, N)) if want_dh0 else None)
    for b in range(nb):
        lam = np.zeros(N)  # A_{t+1}^T mu_{t+1}
        for t in range(T - 1, -1, -1):
            mu = C[b, t].T @ dy[b, t] + lam
            out["dA"][b, t] = np.outer(mu, hs[b, t])
            out["dB"][b, t] = np.outer(mu, x[b, t])
            out["dx"][b, t] = B[b, t].T @ mu
            out["dC"][b, t] = np.outer(dy[b, t], hs[b, t + 1])
            lam = A[b, t].T @ mu
        if want_dh0:
            out["dh0"][b] = lam
    return out


def un_adjoint_sum(A, B, C, x, dy, tbar=0, h0=None, want_dh0=None):
    """Prop. 2 (tbar <= 0 or tbar >= T) and Eq. "capped" (truncated), taken
    literally as a double sum over (loss term t, step i)."""
    A, B, C, x, dy = map(_f64, (A, B, C, x, dy))
    nb, T, N, P = B.shape
    full = tbar <= 0 or tbar >= T
    if want_dh0 is None:
        want_dh0 = full
    if want_dh0 and not full:
        raise ValueError("dh0 is defined for the full gradient only")
    _, _, hs = un_forward(A, B, C, x, h0)
    out = dict(dA=np.zeros_like(A), dB=np.zeros_like(B), dC=np.zeros_like(C), dx=np.zeros_like(x),
               dh0=np.zeros((nb, N)) if want_dh0 else None)
    for b in range(nb):
        for t in range(T):
            out["dC"][b, t] = np.outer(dy[b, t], hs[b, t + 1])  # vjp_C, all t
            lam = C[b, t].T @ dy[b, t]                          # lambda^{t,t}
            i_lo = 0 if full else max(0, t - tbar + 1)
            for i in range(t, i_lo - 1, -1):
                out["dA"][b, i] += np.outer(lam, hs[b, i])      # h_{i-1} is hs[i]
                out["dB"][b, i] += np.outer(lam, x[b, i])
                out["dx"][b, i] += B[b, i].T @ lam
                lam = A[b, i].T @ lam                           # lambda^{t,i-1}
            if want_dh0:
                out["dh0"][b] += lam
    return out


def un_trunc_at(A, B, C, x, dy, tbar, steps, h0=None):
    """Eq. "capped" at the given steps i only (sequence b, step i pairs): the
    windowed adjoint mubar_i = sum_{t=i}^{i+tbar-1} lambda^{t,i}, each lambda^{t,i}
    built from C_t^T dy_t by the transposed decays A_t^T ... A_{i+1}^T, and the
    vjps dA_i = mubar_i h_{i-1}^T, dB_i = mubar_i x_i^T, dx_i = B_i^T mubar_i.
    Returns dict of arrays indexed like ``steps``."""
    A, B, C, x, dy = map(_f64, (A, B, C, x, dy))
    nb, T, N, P = B.shape
    _, _, hs = un_forward(A, B, C, x, h0)
    out = dict(dA=[], dB=[], dx=[])
    for b, i in steps:
        mub = np.zeros(N)
        for t in range(i, min(T, i + tbar)):
            lam = C[b, t].T @ dy[b, t]
            for j in range(t, i, -1):  # A_t^T ... A_{i+1}^T, innermost first
                lam = A[b, j].T @ lam
            mub += lam
        out["dA"].append(np.outer(mub, hs[b, i]))
        out["dB"].append(np.outer(mub, x[b, i]))
        out["dx"].append(B[b, i].T @ mub)
    return {k: np.array(v) for k, v in out.items()}


__all__ = ["un_forward", "un_bptt", "un_adjoint_sum", "un_trunc_at"]
