"""Oracle for the language head and its loss (test infrastructure only).

Plain numpy fp64.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s CPU baseline may import it; it shares nothing with the HIP
library.

Sec. 3.2 puts a head Omega (vocabulary V x width P) on the last residual
output: the prediction for token t is o^t = Omega Norm(y_K^t) (Alg. 1 writes
it without the normalisation; ``norm=False`` gives that form).  Alg. 1 then
evaluates the per-token losses l(o^t) and their gradients dl/dy_K^t once, and
hands the latter to every layer.  The paper leaves l open; here it is the
cross-entropy of the softmax of o^t against a target token,

    l^t = log sum_v exp(o^t_v) - o^t_{target_t},

with dl/do^t = softmax(o^t) - onehot(target_t).  A negative target marks a
token without a loss (l = 0, no gradient); a target >= V gives l = NaN and no
gradient.  Norm is the stack's root-mean-square normalisation (no learned
scale).  Gradients: dy [M][P] = Norm'(y)^T (G Omega) and dOmega [V][P] = G^T u
with G [M][V] the logit gradients and u = Norm(y).

``round_bf16`` rounds u and G to bf16 (round to nearest even) where the GPU
path stores them as the operands of its bf16 matrix products; the normalisation
backward still uses the unrounded u = y r, as the GPU path recomputes it in
fp32 from y.
"""
from __future__ import annotations

import numpy as np

from .stack import bf16, rms_norm, rms_norm_vjp


def head_forward(y, omega, norm=True, round_bf16=False):
    """Returns (logits [M][V], u [M][P], r [M][1] or None): u is the input of
    the head (Norm(y), rounded to bf16 when asked)."""
    y = np.asarray(y, dtype=np.float64)
    om = np.asarray(omega, dtype=np.float64)
    if norm:
        u, r = rms_norm(y)
    else:
        u, r = y, None
    if round_bf16:
        u = bf16(u)
    return u @ om.T, u, r


def head_loss_grad(y, omega, targets, norm=True, round_bf16=False, want_domega=True):
    """Per-token losses [M], dy [M][P] and dOmega [V][P] (None unless asked)."""
    y = np.asarray(y, dtype=np.float64)
    om = np.asarray(omega, dtype=np.float64)
    t = np.asarray(targets, dtype=np.int64)
    M, V = y.shape[0], om.shape[0]
    o, u, r = head_forward(y, om, norm=norm, round_bf16=round_bf16)
    m = o.max(axis=1, keepdims=True)
    e = np.exp(o - m)
    s = e.sum(axis=1, keepdims=True)
    lse = (m + np.log(s))[:, 0]
    valid = (t >= 0) & (t < V)
    loss = np.zeros(M)
    rows = np.nonzero(valid)[0]
    loss[rows] = lse[rows] - o[rows, t[rows]]
    loss[t >= V] = np.nan
    G = e / s
    G[rows, t[rows]] -= 1.0
    G[~valid] = 0.0
    if round_bf16:
        G = bf16(G)
    dU = G @ om
    dy = rms_norm_vjp(y, r, dU) if norm else dU
    domega = G.T @ u if want_domega else None
    return dict(loss=loss, dy=dy, domega=domega)


__all__ = ["head_forward", "head_loss_grad"]
