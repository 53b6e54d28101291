"""Pins of the unstructured-SSM oracle (Table 1's N x N row) against facts fixed
by mathematics: central differences, torch autograd of an independently written
loop, Prop. 2 against backpropagation, the truncated estimator against per-loss
truncated backpropagation, closed forms, and the diagonal special case against
the diagonal layer's own (separately pinned) oracle.  CPU only."""
import numpy as np
import pytest
import torch

import oracle
from oracle.unstructured import un_adjoint_sum, un_bptt, un_forward, un_trunc_at


def _inputs(rng, nb=2, T=6, N=3, P=2, h0=True, scale=0.6):
    A = rng.standard_normal((nb, T, N, N)) * scale / np.sqrt(N)
    B = rng.standard_normal((nb, T, N, P))
    C = rng.standard_normal((nb, T, P, N))
    x = rng.standard_normal((nb, T, P))
    dy = rng.standard_normal((nb, T, P))
    hz = rng.standard_normal((nb, N)) if h0 else None
    return dict(A=A, B=B, C=C, x=x, dy=dy, h0=hz)


def _loss(inp):
    y, _, _ = un_forward(inp["A"], inp["B"], inp["C"], inp["x"], inp["h0"])
    return float(np.sum(inp["dy"] * y))


def _relerr(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def test_forward_identity_transition_is_cumsum(rng):
    """A_t = I makes h_t = h0 + cumsum_t(B_t x_t)."""
    inp = _inputs(rng, T=9)
    nb, T, N, _ = inp["B"].shape
    A = np.broadcast_to(np.eye(N), (nb, T, N, N)).copy()
    _, _, hs = un_forward(A, inp["B"], inp["C"], inp["x"], inp["h0"])
    bx = np.einsum("btnp,btp->btn", inp["B"], inp["x"])
    assert _relerr(hs[:, 1:], inp["h0"][:, None] + np.cumsum(bx, axis=1)) < 1e-13


def test_bptt_matches_central_differences(rng):
    inp = _inputs(rng)
    g = un_bptt(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], inp["h0"])
    eps = 1e-6
    for key, gkey in (("A", "dA"), ("B", "dB"), ("C", "dC"), ("x", "dx"), ("h0", "dh0")):
        fd = np.zeros_like(inp[key])
        for idx in np.ndindex(*inp[key].shape):
            p, m = dict(inp), dict(inp)
            p[key] = inp[key].copy()
            m[key] = inp[key].copy()
            p[key][idx] += eps
            m[key][idx] -= eps
            fd[idx] = (_loss(p) - _loss(m)) / (2 * eps)
        assert _relerr(g[gkey], fd) < 1e-7, key


def test_bptt_matches_torch_autograd(rng):
    inp = _inputs(rng, nb=2, T=11, N=4, P=3)
    ts = {k: torch.tensor(inp[k], dtype=torch.float64, requires_grad=True) for k in ("A", "B", "C", "x", "h0")}
    h = ts["h0"]
    L = 0.0
    for t in range(inp["x"].shape[1]):
        h = torch.einsum("bij,bj->bi", ts["A"][:, t], h) + torch.einsum("bip,bp->bi", ts["B"][:, t], ts["x"][:, t])
        y = torch.einsum("bpi,bi->bp", ts["C"][:, t], h)
        L = L + (torch.tensor(inp["dy"][:, t]) * y).sum()
    L.backward()
    g = un_bptt(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], inp["h0"])
    for key, gkey in (("A", "dA"), ("B", "dB"), ("C", "dC"), ("x", "dx"), ("h0", "dh0")):
        assert _relerr(g[gkey], ts[key].grad.numpy()) < 1e-12, key


def test_double_sum_full_equals_bptt(rng):
    """Prop. 2: the sum of the per-pair vjps over all (t, i) is the gradient."""
    inp = _inputs(rng, T=12, N=4, P=3)
    a = un_adjoint_sum(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], h0=inp["h0"])
    b = un_bptt(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], inp["h0"])
    for k in ("dA", "dB", "dC", "dx", "dh0"):
        assert _relerr(a[k], b[k]) < 1e-12, k


def test_dot_product_identity(rng):
    """L = sum_i <mu_i, B_i x_i> + <A_0^T mu_0, h0>: the loss is linear in (B, h0)
    jointly, so L = <dB, B> + <dh0, h0>."""
    inp = _inputs(rng, T=15, N=5, P=3)
    g = un_bptt(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], inp["h0"])
    lhs = _loss(inp)
    rhs = float(np.sum(g["dB"] * inp["B"]) + np.sum(g["dh0"] * inp["h0"]))
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # and linear in C alone: L = <dC, C>
    assert abs(lhs - float(np.sum(g["dC"] * inp["C"]))) <= 1e-12 * max(1.0, abs(lhs))


def test_truncated_limits(rng):
    """tbar >= T is the full gradient; tbar = 1 keeps only lambda^{t,t} = C_t^T dy_t."""
    inp = _inputs(rng, T=8, N=3, P=2, h0=False)
    args = (inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"])
    full = un_bptt(*args, want_dh0=False)
    for tb in (8, 20):
        tr = un_adjoint_sum(*args, tbar=tb)
        for k in ("dA", "dB", "dC", "dx"):
            assert _relerr(tr[k], full[k]) < 1e-12, (tb, k)
    one = un_adjoint_sum(*args, tbar=1)
    _, _, hs = un_forward(*args[:4])
    mu = np.einsum("btpn,btp->btn", inp["C"], inp["dy"])
    assert _relerr(one["dA"], np.einsum("bti,btj->btij", mu, hs[:, :-1])) < 1e-13
    assert _relerr(one["dx"], np.einsum("btnp,btn->btp", inp["B"], mu)) < 1e-13
    assert _relerr(one["dC"], full["dC"]) < 1e-13  # the C term is never truncated


def test_truncated_equals_sum_of_per_loss_truncated_backprop(rng):
    """Eq. "capped": for each loss term, backpropagate through its last Tbar
    transitions only (the state entering that window detached), summed over t."""
    nb, T, N, P, tbar = 1, 10, 3, 2, 3
    inp = _inputs(rng, nb=nb, T=T, N=N, P=P)
    ts = {k: torch.tensor(inp[k], dtype=torch.float64, requires_grad=True) for k in ("A", "B", "C", "x")}
    dy = torch.tensor(inp["dy"])
    for t in range(T):
        h = torch.tensor(inp["h0"])
        for i in range(t + 1):
            if i == t - tbar + 1:
                h = h.detach()
            h = torch.einsum("bij,bj->bi", ts["A"][:, i], h) + torch.einsum("bip,bp->bi", ts["B"][:, i],
                                                                            ts["x"][:, i])
        y = torch.einsum("bpi,bi->bp", ts["C"][:, t], h)
        (dy[:, t] * y).sum().backward()
    g = un_adjoint_sum(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], tbar=tbar, h0=inp["h0"])
    for key, gkey in (("A", "dA"), ("B", "dB"), ("C", "dC"), ("x", "dx")):
        assert _relerr(g[gkey], ts[key].grad.numpy()) < 1e-12, key


@pytest.mark.parametrize("tbar", [0, 4])
def test_diagonal_special_case_equals_diagonal_layer(rng, tbar):
    """With one channel (P = 1) and diagonal A_t = diag(a_t), the unstructured
    SSM is the diagonal layer with D = 1: dx, dB, dC and the diagonal of dA
    equal the diagonal layer's dx, dB, dC and decay cotangent da."""
    nb, T, N = 2, 9, 4
    x = rng.standard_normal((nb, T, 1))
    dl = np.log1p(np.exp(rng.standard_normal((nb, T, 1))))  # Delta > 0
    A_log = rng.uniform(0.0, np.log(16.0), (1, N))
    Bd = rng.standard_normal((nb, T, N)) * 0.5
    Cd = rng.standard_normal((nb, T, N)) * 0.5
    dy = rng.standard_normal((nb, T, 1))
    a = np.exp(-dl[..., 0, None] * np.exp(A_log[0])[None, None])  # [b,T,N]
    A = np.zeros((nb, T, N, N))
    idx = np.arange(N)
    A[:, :, idx, idx] = a
    B = Bd[..., None]       # [b,T,N,1]
    C = Cd[:, :, None, :]   # [b,T,1,N]
    un = un_adjoint_sum(A, B, C, x, dy, tbar=tbar, want_dh0=False)
    kw = dict(want_da=True, want_dh0=False)
    dg = (oracle.bptt(x, dl, A_log, Bd, Cd, dy, **kw) if tbar == 0
          else oracle.adjoint_sum(x, dl, A_log, Bd, Cd, dy, tbar=tbar, **kw))
    assert _relerr(un["dx"], dg["dx"]) < 1e-12
    assert _relerr(un["dB"][..., 0], dg["dB"]) < 1e-12
    assert _relerr(un["dC"][:, :, 0, :], dg["dC"]) < 1e-12
    assert _relerr(un["dA"][:, :, idx, idx], dg["da"][:, :, 0, :]) < 1e-12


def test_sampled_truncated_steps_equal_double_sum(rng):
    """un_trunc_at (the window sum at chosen steps, for the long workloads) equals
    the full double sum at those steps."""
    inp = _inputs(rng, nb=2, T=20, N=4, P=3)
    args = (inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"])
    for tbar in (1, 5, 30):
        full = un_adjoint_sum(*args, tbar=tbar, h0=inp["h0"], want_dh0=False)
        steps = [(0, 0), (1, 7), (0, 19), (1, 15)]
        got = un_trunc_at(*args, tbar=tbar, steps=steps, h0=inp["h0"])
        for k in ("dA", "dB", "dx"):
            ref = np.array([full[k][b, i] for b, i in steps])
            assert _relerr(got[k], ref) < 1e-12, (tbar, k)
