"""Oracle for a stack of K residual SSM layers (test infrastructure only).

Plain numpy fp64, built on the single-layer oracle (``layer_forward``,
``layer_grad``).  Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
CPU baseline may import it.

The model follows the residual network of Sec. 3.2 with the SSM layers of
Sec. 3.1, as the forward of Alg. 1 computes it:

    y_0 given;  for k = 1..K:  u_k = Norm(y_{k-1}),  y_k = y_{k-1} + SSM_k(u_k)

with Norm the root-mean-square normalisation over the channels (no learned
scale; the paper gives none) and SSM_k the selective layer with input
projections ([x | z] = u W_in, [Delta_pre | B | C] = x W_x, out = y * silu(z)).
The residual width equals the SSM's channel count D (the paper's SSM maps P to
P).  The upstream gradient g_K = dL/dy_K is an input (Alg. 1 computes it once
from the language head and hands it to every device).

Two gradients of L = sum g_K * y_K with respect to every layer's parameters:
  * ``adjoint``: Prop. 3 -- every layer's vjps are taken with the upstream
    g_K and the layer's own stored input u_k, independently of the other
    layers (the sum over k of Prop. 2 applied to y_K = y_0 + sum_k SSM_k(u_k)
    with each u_k held fixed);
  * ``exact``: backpropagation through the whole stack, where layer k's
    upstream is g_k = dL/dy_k = g_{k+1} + Norm'(y_k)^T du_{k+1}.
The two agree for the last layer and for K = 1; elsewhere their difference is
the contribution of the paths through later layers, which Prop. 3 omits.

``round_bf16`` rounds the activations that the GPU path stores in bf16 (the
normalised input u, the projections x, z, Delta_pre, B, C, the layer output and
the upstream passed to each layer) to bf16, round to nearest even; with it off
the functions compute the exact fp64 model.
"""
from __future__ import annotations

import numpy as np

from . import forward, layer_grad, trunc_tail

EPS = 1e-6


def bf16(a):
    """Round to the nearest bf16 value (ties to even), returned as fp64."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).astype(np.float64)
    nan = np.isnan(f)
    out[nan] = np.nan
    return out


def rms_norm(y):
    """u = y / sqrt(mean over channels of y^2 + eps) and the factor 1/rms."""
    y = np.asarray(y, dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + EPS)
    return y * r, r


def rms_norm_vjp(y, r, du):
    """Cotangent of y for u = y r(y): (du - u mean(du u)) r, with u = y r."""
    u = y * r
    return (du - u * np.mean(du * u, axis=-1, keepdims=True)) * r


def stack_forward(y0, W_in, W_x, A_log, N, round_bf16=True):
    """Forward of Alg. 1 over the K layers.  Returns y_K and, per layer, the
    stored activations (u, x, z, dpre, B, C) and the layer input y_{k-1}."""
    rd = bf16 if round_bf16 else (lambda a: np.asarray(a, dtype=np.float64))
    y = np.asarray(y0, dtype=np.float64)
    acts = []
    for k in range(len(W_in)):
        u = rd(rms_norm(y)[0])
        D = W_x[k].shape[0]
        xz = u @ np.asarray(W_in[k], dtype=np.float64)
        x, z = rd(xz[..., :D]), rd(xz[..., D:])
        pj = x @ np.asarray(W_x[k], dtype=np.float64)
        dpre, B, C = rd(pj[..., :D]), rd(pj[..., D:D + N]), rd(pj[..., D + N:])
        out, _ = forward(x, dpre, A_log[k], B, C, z=z, delta_softplus=True)
        acts.append(dict(y_in=y, u=u, x=x, z=z, dpre=dpre, B=B, C=C))
        y = y + rd(out)
    return y, acts


def stack_grad(acts, W_in, W_x, A_log, gK, mode="adjoint", tbar=0, round_bf16=True):
    """Parameter gradients dW_in, dW_x, dA_log of every layer (lists, layer 1
    first) for ``mode`` "adjoint" (Prop. 3) or "exact" (backpropagation)."""
    rd = bf16 if round_bf16 else (lambda a: np.asarray(a, dtype=np.float64))
    K = len(W_in)
    scan = trunc_tail if tbar > 0 else None
    out = [None] * K
    g = np.asarray(gK, dtype=np.float64)
    for k in reversed(range(K)):
        a = acts[k]
        up = gK if mode == "adjoint" else g
        r = layer_grad(a["u"], a["x"], a["z"], a["dpre"], a["B"], a["C"], W_x[k], A_log[k], rd(up),
                       W_in=W_in[k], tbar=tbar, scan=scan)
        out[k] = dict(dW_in=r["dW_in"], dW_x=r["dW_x"], dA_log=r["dA_log"])
        if mode == "exact" and k > 0:
            _, rr = rms_norm(a["y_in"])
            du = r["du"].reshape(a["y_in"].shape)
            g = g + rms_norm_vjp(a["y_in"], rr, du)
    return out


__all__ = ["bf16", "rms_norm", "rms_norm_vjp", "stack_forward", "stack_grad"]
