"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Each test checks the oracle against something other than itself: finite
differences, a library autograd, closed forms that reduce to numpy's cumsum /
convolve, exact algebraic identities, brute-force counts and the numbers the
paper prints.  They run on the CPU only.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny(rng, nb=2, T=10, D=3, N=4, gate=True, softplus=True, h0=True, slow=False, a_scalar=False,
         b_delta=False):
    x = rng.standard_normal((nb, T, D))
    dpre = rng.standard_normal((nb, T, D)) - (3.0 if slow else 0.0)
    if not softplus:
        dpre = np.log1p(np.exp(dpre))
    A_log = rng.uniform(0.0, math.log(16.0), (D,) if a_scalar else (D, N))
    B = rng.standard_normal((nb, T, N)) * 0.5
    C = rng.standard_normal((nb, T, N)) * 0.5
    z = rng.standard_normal((nb, T, D)) if gate else None
    hz = rng.standard_normal((nb, D, N)) if h0 else None
    dy = rng.standard_normal((nb, T, D))
    return dict(x=x, delta=dpre, A_log=A_log, B=B, C=C, z=z, h0=hz, dy=dy, delta_softplus=softplus,
                a_scalar=a_scalar, b_delta=b_delta)


def variant(inp):
    return dict(a_scalar=inp.get("a_scalar", False), b_delta=inp.get("b_delta", False))


def loss(inp):
    out, _ = oracle.forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], h0=inp["h0"],
                            z=inp["z"], delta_softplus=inp["delta_softplus"], **variant(inp))
    return float(np.sum(inp["dy"] * out))


def relerr(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def bptt_of(inp, **kw):
    return oracle.bptt(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], h0=inp["h0"],
                       z=inp["z"], delta_softplus=inp["delta_softplus"], **variant(inp), **kw)


# --------------------------------------------------------------------------
# Forward: closed forms (Sec. 3.1)
# --------------------------------------------------------------------------
def test_forward_unit_decay_is_cumsum(rng):
    """Delta = 0 makes every a_t = 1, so h_t = h_0 + cumsum(B x)."""
    nb, T, D, N = 2, 17, 3, 5
    x = rng.standard_normal((nb, T, D))
    B = rng.standard_normal((nb, T, N))
    C = rng.standard_normal((nb, T, N))
    h0 = rng.standard_normal((nb, D, N))
    A_log = rng.uniform(0, 2.7, (D, N))
    out, h_last = oracle.forward(x, np.zeros((nb, T, D)), A_log, B, C, h0=h0)
    bx = x[:, :, :, None] * B[:, :, None, :]               # [b,T,D,N]
    h = h0[:, None] + np.cumsum(bx, axis=1)
    np.testing.assert_allclose(out, np.einsum("btdn,btn->btd", h, C), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(h_last, h[:, -1], rtol=1e-12, atol=1e-12)


def test_forward_constant_decay_is_convolution(rng):
    """Constant Delta and A_log = 0 give a = alpha, so h is the causal
    convolution of B x with alpha^k plus alpha^{t+1} h_0."""
    nb, T, D, N = 1, 23, 2, 3
    delta = 0.3
    alpha = math.exp(-delta)
    x = rng.standard_normal((nb, T, D))
    B = rng.standard_normal((nb, T, N))
    C = rng.standard_normal((nb, T, N))
    h0 = rng.standard_normal((nb, D, N))
    out, _ = oracle.forward(x, np.full((nb, T, D), delta), np.zeros((D, N)), B, C, h0=h0)
    kern = alpha ** np.arange(T)
    ref = np.zeros((nb, T, D))
    for d in range(D):
        for n in range(N):
            bx = x[0, :, d] * B[0, :, n]
            h = np.convolve(bx, kern)[:T] + alpha ** np.arange(1, T + 1) * h0[0, d, n]
            ref[0, :, d] += C[0, :, n] * h
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# Full gradient: finite differences and a library autograd
# --------------------------------------------------------------------------
@pytest.mark.parametrize("gate,softplus", [(True, True), (False, False)])
def test_bptt_matches_central_differences(rng, gate, softplus):
    inp = tiny(rng, nb=2, T=9, D=3, N=4, gate=gate, softplus=softplus, h0=True)
    g = bptt_of(inp)
    names = [("x", "dx"), ("delta", "ddelta"), ("A_log", "dA_log"), ("B", "dB"), ("C", "dC"), ("h0", "dh0")]
    if gate:
        names.append(("z", "dz"))
    eps = 1e-6
    for src, dst in names:
        arr = inp[src]
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps
            lp = loss(inp)
            arr[idx] = keep - eps
            lm = loss(inp)
            arr[idx] = keep
            fd[idx] = (lp - lm) / (2 * eps)
        assert relerr(g[dst], fd) < 1e-6, (src, relerr(g[dst], fd))


def _torch_naive_loss(x, dl, A_log, B, C, z, h0, dy, softplus):
    """The five steps of Sec. 3.1 as a plain torch loop; autograd differentiates it."""
    nb, T, D = x.shape
    delta = torch.nn.functional.softplus(dl) if softplus else dl
    h = h0.clone()
    L = 0.0
    for t in range(T):
        a = torch.exp(-delta[:, t, :, None] * torch.exp(A_log)[None])
        h = a * h + B[:, t, None, :] * x[:, t, :, None]
        y = (C[:, t, None, :] * h).sum(-1)
        out = y * torch.nn.functional.silu(z[:, t]) if z is not None else y
        L = L + (dy[:, t] * out).sum()
    return L


def test_bptt_matches_torch_autograd(rng):
    inp = tiny(rng, nb=2, T=13, D=4, N=3, gate=True, softplus=True, h0=True)
    ts = {k: torch.tensor(inp[k], dtype=torch.float64, requires_grad=True)
          for k in ("x", "delta", "A_log", "B", "C", "z", "h0")}
    L = _torch_naive_loss(ts["x"], ts["delta"], ts["A_log"], ts["B"], ts["C"], ts["z"], ts["h0"],
                          torch.tensor(inp["dy"]), True)
    L.backward()
    g = bptt_of(inp)
    for src, dst in [("x", "dx"), ("delta", "ddelta"), ("A_log", "dA_log"), ("B", "dB"), ("C", "dC"),
                     ("z", "dz"), ("h0", "dh0")]:
        assert relerr(g[dst], ts[src].grad.numpy()) < 1e-12, src


def test_homogeneity_identities(rng):
    """L = sum_t g_t . y_t is linear in C, and jointly linear in (x, h0) and in
    (B, h0); Euler's identity for each gives an exact check of dC, dx, dB, dh0
    (and of the adjoint dot-product identity sum<g,y> = sum<mu, Bx> + <a_1 mu_1, h0>)."""
    inp = tiny(rng, nb=2, T=31, D=5, N=4, gate=False, softplus=True, h0=True)
    g = bptt_of(inp)
    L = loss(inp)
    assert abs(np.sum(g["dC"] * inp["C"]) - L) < 1e-12 * max(1.0, abs(L)) * 100
    assert abs(np.sum(g["dx"] * inp["x"]) + np.sum(g["dh0"] * inp["h0"]) - L) < 1e-10
    assert abs(np.sum(g["dB"] * inp["B"]) + np.sum(g["dh0"] * inp["h0"]) - L) < 1e-10


# --------------------------------------------------------------------------
# Prop. 2: the literal double sum equals backpropagation
# --------------------------------------------------------------------------
@pytest.mark.parametrize("gate", [True, False])
def test_doublesum_full_equals_bptt(rng, gate):
    inp = tiny(rng, nb=2, T=20, D=3, N=4, gate=gate, softplus=True, h0=True)
    ref = bptt_of(inp)
    ds = oracle.adjoint_sum(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"],
                            tbar=0, h0=inp["h0"], z=inp["z"], delta_softplus=True)
    for k in ("dx", "ddelta", "dA_log", "dB", "dC", "dh0") + (("dz",) if gate else ()):
        assert relerr(ds[k], ref[k]) < 1e-12, k


# --------------------------------------------------------------------------
# Eq. "capped": truncated estimator
# --------------------------------------------------------------------------
def _trunc_both(inp, tbar):
    args = (inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"])
    kw = dict(tbar=tbar, h0=inp["h0"], z=inp["z"], delta_softplus=inp["delta_softplus"])
    return oracle.adjoint_sum(*args, **kw), oracle.trunc_tail(*args, **kw)


def test_truncated_window_at_least_T_is_full(rng):
    inp = tiny(rng, nb=1, T=12, D=2, N=3, gate=True, slow=True)
    full = bptt_of(inp, want_dh0=False)
    for tbar in (12, 13, 1000):
        ds, tl = _trunc_both(inp, tbar)
        for k in ("dx", "ddelta", "dA_log", "dB", "dC", "dz"):
            assert relerr(ds[k], full[k]) < 1e-12 and relerr(tl[k], full[k]) < 1e-12, (tbar, k)


def _gC(inp):
    return inp["dy"][..., :, None] * inp["C"][:, :, None, :]      # [b,T,D,N], no gate


@pytest.mark.parametrize("tbar", [1, 2, 5, 11])
def test_truncated_unit_decay_is_box_filter(rng, tbar):
    """a = 1 (Delta = 0): the kept cotangent at step i is the sum of g_t C_t over
    the window t in [i, i+Tbar-1], a box filter (numpy.convolve)."""
    nb, T, D, N = 1, 19, 3, 2
    inp = tiny(rng, nb=nb, T=T, D=D, N=N, gate=False, softplus=False, h0=True)
    inp["delta"] = np.zeros((nb, T, D))
    s = _gC(inp)
    mubar = np.zeros_like(s)
    for d in range(D):
        for n in range(N):
            mubar[0, :, d, n] = np.convolve(s[0, :, d, n], np.ones(tbar))[tbar - 1:tbar - 1 + T]
    h = inp["h0"][:, None] + np.cumsum(inp["x"][..., None] * inp["B"][:, :, None, :], axis=1)
    hprev = np.concatenate([inp["h0"][:, None], h[:, :-1]], axis=1)
    ds, tl = _trunc_both(inp, tbar)
    ref_dx = np.einsum("btdn,btn->btd", mubar, inp["B"])
    ref_dB = np.einsum("btdn,btd->btn", mubar, inp["x"])
    ref_dd = -np.einsum("btdn,dn->btd", mubar * hprev, np.exp(inp["A_log"]))
    for got in (ds, tl):
        assert relerr(got["dx"], ref_dx) < 1e-12
        assert relerr(got["dB"], ref_dB) < 1e-12
        assert relerr(got["ddelta"], ref_dd) < 1e-12
        assert np.max(np.abs(got["dA_log"])) == 0.0     # Delta = 0 kills the A_log path


@pytest.mark.parametrize("tbar", [1, 3, 8])
def test_truncated_constant_decay_is_truncated_geometric_kernel(rng, tbar):
    """a = alpha: the kept cotangent is sum_{k<Tbar} alpha^k g_{i+k} C_{i+k}."""
    nb, T, D, N = 1, 21, 2, 3
    dconst = 0.2
    alpha = math.exp(-dconst)
    inp = tiny(rng, nb=nb, T=T, D=D, N=N, gate=False, softplus=False, h0=False)
    inp["delta"] = np.full((nb, T, D), dconst)
    inp["A_log"] = np.zeros((D, N))
    s = _gC(inp)
    kern = alpha ** (tbar - 1 - np.arange(tbar))
    mubar = np.zeros_like(s)
    for d in range(D):
        for n in range(N):
            mubar[0, :, d, n] = np.convolve(s[0, :, d, n], kern)[tbar - 1:tbar - 1 + T]
    ds, tl = _trunc_both(inp, tbar)
    for got in (ds, tl):
        assert relerr(got["dx"], np.einsum("btdn,btn->btd", mubar, inp["B"])) < 1e-12
        assert relerr(got["dB"], np.einsum("btdn,btd->btn", mubar, inp["x"])) < 1e-12


def test_truncated_equals_sum_of_per_loss_truncated_backprop(rng):
    """Truncated adjoint sharding generalises T-BPTT (Sec. 2 and Sec. 4.3): for
    each loss term l^t, backpropagate through the last Tbar transitions only
    (the state entering that window is detached) and sum over t; torch autograd."""
    nb, T, D, N, tbar = 1, 14, 2, 3, 4
    inp = tiny(rng, nb=nb, T=T, D=D, N=N, gate=True, softplus=True, h0=True)
    ts = {k: torch.tensor(inp[k], dtype=torch.float64, requires_grad=True)
          for k in ("x", "delta", "A_log", "B", "C", "z")}
    h0 = torch.tensor(inp["h0"])
    dy = torch.tensor(inp["dy"])
    for t in range(T):
        delta = torch.nn.functional.softplus(ts["delta"])
        h = h0
        for i in range(t + 1):
            if i == t - tbar + 1:
                h = h.detach()
            a = torch.exp(-delta[:, i, :, None] * torch.exp(ts["A_log"])[None])
            h = a * h + ts["B"][:, i, None, :] * ts["x"][:, i, :, None]
        y = (ts["C"][:, t, None, :] * h).sum(-1)
        lt = (dy[:, t] * y * torch.nn.functional.silu(ts["z"][:, t])).sum()
        lt.backward()
    ds, tl = _trunc_both(inp, tbar)
    for src, dst in [("x", "dx"), ("delta", "ddelta"), ("A_log", "dA_log"), ("B", "dB"), ("C", "dC"),
                     ("z", "dz")]:
        ref = ts[src].grad.numpy()
        assert relerr(ds[dst], ref) < 1e-12, ("doublesum", src)
        assert relerr(tl[dst], ref) < 1e-12, ("tail", src)


@pytest.mark.parametrize("tbar", [1, 2, 31, 32, 33, 63, 64, 100])
def test_tail_form_equals_literal_double_sum(rng, tbar):
    inp = tiny(rng, nb=2, T=64, D=3, N=4, gate=True, softplus=True, h0=False, slow=True)
    ds, tl = _trunc_both(inp, tbar)
    for k in ("dx", "ddelta", "dA_log", "dB", "dC", "dz"):
        assert relerr(tl[k], ds[k]) < 1e-11, k


def test_truncation_leaves_C_path_and_gate_untouched(rng):
    """The vjp_C term of Eq. "capped" runs over every t, so dC (and dz) do not
    depend on the window."""
    inp = tiny(rng, nb=1, T=30, D=3, N=4, gate=True, slow=True)
    full = bptt_of(inp, want_dh0=False)
    ds, tl = _trunc_both(inp, 5)
    for got in (ds, tl):
        assert relerr(got["dC"], full["dC"]) < 1e-13
        assert relerr(got["dz"], full["dz"]) < 1e-13
        assert relerr(got["dx"], full["dx"]) > 1e-3      # the window is visible


def test_truncated_rejects_dh0(rng):
    inp = tiny(rng, nb=1, T=8, D=2, N=2, gate=False, h0=True)
    with pytest.raises(ValueError):
        oracle.adjoint_sum(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], tbar=3,
                           h0=inp["h0"], delta_softplus=True, want_dh0=True)


# --------------------------------------------------------------------------
# VJP counts (Sec. 4.3) against the printed numbers
# --------------------------------------------------------------------------
def _golden(name):
    vals = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                k, v = line.split()
                vals[k] = int(v)
    return vals


def test_vjp_counts_reproduce_printed_reduction():
    g = _golden("vjp_counts.txt")
    T, tbar = g["T"], g["tbar"]
    full = oracle.vjp_count_full(T)
    trunc = oracle.vjp_count_truncated(T, tbar)
    assert full == (1 + T) * T // 2                                   # Sec. 4.3 full count
    assert trunc == tbar * T - tbar * (tbar - 1) // 2                 # the closed form with '-'
    assert round(100 * (1 - trunc / full)) == g["removed_percent"]    # 64 %
    plus = tbar * T + tbar * (tbar - 1) // 2                          # the printed sign
    assert round(100 * (1 - plus / full)) != g["removed_percent"]


@pytest.mark.parametrize("T,tbar", [(1, 1), (5, 1), (5, 5), (7, 3), (40, 13)])
def test_vjp_count_closed_form_small(T, tbar):
    brute = sum(1 for t in range(1, T + 1) for i in range(1, t + 1) if i >= t + 1 - tbar)
    assert oracle.vjp_count_truncated(T, tbar) == brute
    assert oracle.vjp_count_full(T) == sum(1 for t in range(1, T + 1) for i in range(1, t + 1))


# --------------------------------------------------------------------------
# Projections and the whole layer
# --------------------------------------------------------------------------
def _bf16_bits(a):
    t = torch.tensor(a, dtype=torch.float32).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16), t.to(torch.float64).numpy()


def test_proj_sampled_entries_match_numpy_matmul(rng):
    M, K, Nout = 37, 11, 13
    Xb, X = _bf16_bits(rng.standard_normal((M, K)))
    Zb, Z = _bf16_bits(rng.standard_normal((M, Nout)))
    Wb, W = _bf16_bits(rng.standard_normal((K, Nout)))
    kk = rng.integers(0, K, 50)
    jj = rng.integers(0, Nout, 50)
    np.testing.assert_allclose(oracle.proj_dw(Xb, Zb, kk, jj), (X.T @ Z)[kk, jj], rtol=1e-13, atol=1e-12)
    rows = np.array([0, 5, 36])
    np.testing.assert_allclose(oracle.proj_dx(Zb, Wb, rows), (Z @ W.T)[rows], rtol=1e-13, atol=1e-12)


def test_layer_gradient_matches_central_differences(rng):
    nb, T, dm, D, N = 1, 6, 3, 4, 2
    u = rng.standard_normal((nb, T, dm))
    W_in = rng.standard_normal((dm, 2 * D)) / math.sqrt(dm)
    W_x = rng.standard_normal((D, D + 2 * N)) / math.sqrt(D)
    A_log = rng.uniform(0, 1.5, (D, N))
    dy = rng.standard_normal((nb, T, D))

    def L():
        out, _ = oracle.layer_forward(u, W_in, W_x, A_log, N)
        return float(np.sum(dy * out))

    _, act = oracle.layer_forward(u, W_in, W_x, A_log, N)
    g = oracle.layer_grad(u, act["x"], act["z"], act["dpre"], act["B"], act["C"], W_x, A_log, dy, W_in=W_in)
    eps = 1e-6
    for arr, key in [(u, "du"), (W_in, "dW_in"), (W_x, "dW_x"), (A_log, "dA_log")]:
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps
            lp = L()
            arr[idx] = keep - eps
            lm = L()
            arr[idx] = keep
            fd[idx] = (lp - lm) / (2 * eps)
        got = g[key].reshape(fd.shape)
        assert relerr(got, fd) < 1e-6, key


# --------------------------------------------------------------------------
# Variants: the scalar-decay SSM of Table 1 and the step-size-scaled input
# --------------------------------------------------------------------------
VARIANTS = [(True, False), (False, True), (True, True)]


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
def test_variant_bptt_matches_central_differences(rng, a_scalar, b_delta):
    inp = tiny(rng, nb=2, T=8, D=3, N=4, gate=True, softplus=True, h0=True, a_scalar=a_scalar, b_delta=b_delta)
    g = bptt_of(inp)
    eps = 1e-6
    for src, dst in [("x", "dx"), ("delta", "ddelta"), ("A_log", "dA_log"), ("B", "dB"), ("C", "dC"),
                     ("h0", "dh0"), ("z", "dz")]:
        arr = inp[src]
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps
            lp = loss(inp)
            arr[idx] = keep - eps
            lm = loss(inp)
            arr[idx] = keep
            fd[idx] = (lp - lm) / (2 * eps)
        assert relerr(g[dst], fd) < 1e-6, (src, relerr(g[dst], fd))


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
def test_variant_bptt_matches_torch_autograd(rng, a_scalar, b_delta):
    inp = tiny(rng, nb=2, T=11, D=3, N=4, gate=True, softplus=True, h0=True, a_scalar=a_scalar, b_delta=b_delta)
    ts = {k: torch.tensor(inp[k], dtype=torch.float64, requires_grad=True)
          for k in ("x", "delta", "A_log", "B", "C", "z", "h0")}
    delta = torch.nn.functional.softplus(ts["delta"])
    rate = torch.exp(ts["A_log"])
    rate = rate[:, None].expand(-1, 4) if a_scalar else rate
    h = ts["h0"].clone()
    L = 0.0
    for t in range(ts["x"].shape[1]):
        a = torch.exp(-delta[:, t, :, None] * rate[None])
        u = ts["x"][:, t] * (delta[:, t] if b_delta else 1.0)
        h = a * h + ts["B"][:, t, None, :] * u[:, :, None]
        y = (ts["C"][:, t, None, :] * h).sum(-1)
        L = L + (torch.tensor(inp["dy"][:, t]) * y * torch.nn.functional.silu(ts["z"][:, t])).sum()
    L.backward()
    g = bptt_of(inp)
    for src, dst in [("x", "dx"), ("delta", "ddelta"), ("A_log", "dA_log"), ("B", "dB"), ("C", "dC"),
                     ("z", "dz"), ("h0", "dh0")]:
        assert relerr(g[dst], ts[src].grad.numpy()) < 1e-12, src


def test_scalar_decay_equals_diagonal_with_shared_rates(rng):
    """A scalar decay per channel is the diagonal decay with A_log[d, n] = A_log[d]
    for every n: same outputs and gradients, and dA_log is the row sum."""
    inp = tiny(rng, nb=2, T=15, D=3, N=5, gate=True, softplus=True, h0=True, a_scalar=True)
    g = bptt_of(inp)
    diag = dict(inp, A_log=np.repeat(inp["A_log"][:, None], 5, axis=1), a_scalar=False)
    gd = bptt_of(diag)
    assert abs(loss(inp) - loss(diag)) < 1e-12 * max(1.0, abs(loss(diag)))
    for k in ("dx", "ddelta", "dB", "dC", "dz", "dh0"):
        assert relerr(g[k], gd[k]) < 1e-13, k
    assert relerr(g["dA_log"], gd["dA_log"].sum(axis=1)) < 1e-13


def test_step_scaled_input_equals_rescaled_x(rng):
    """h = a h + Delta B x is the plain layer run on x' = Delta x: same outputs,
    dx = Delta dx', and the input path adds dx' x to dDelta."""
    inp = tiny(rng, nb=2, T=14, D=3, N=4, gate=True, softplus=False, h0=True, b_delta=True)
    g = bptt_of(inp)
    plain = dict(inp, x=inp["x"] * inp["delta"], b_delta=False)
    gp = bptt_of(plain)
    assert abs(loss(inp) - loss(plain)) < 1e-12 * max(1.0, abs(loss(plain)))
    assert relerr(g["dx"], gp["dx"] * inp["delta"]) < 1e-13
    assert relerr(g["ddelta"], gp["ddelta"] + gp["dx"] * inp["x"]) < 1e-13
    for k in ("dA_log", "dB", "dC", "dz", "dh0"):
        assert relerr(g[k], gp[k]) < 1e-13, k


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
def test_variant_doublesum_and_tail_agree(rng, a_scalar, b_delta):
    """Prop. 2 and the tail identity hold for the variants too."""
    inp = tiny(rng, nb=2, T=24, D=3, N=4, gate=True, softplus=True, h0=True, slow=True, a_scalar=a_scalar,
               b_delta=b_delta)
    args = (inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"])
    kw = dict(h0=inp["h0"], z=inp["z"], delta_softplus=True, a_scalar=a_scalar, b_delta=b_delta)
    ref = bptt_of(inp)
    full = oracle.adjoint_sum(*args, tbar=0, **kw)
    for k in ("dx", "ddelta", "dA_log", "dB", "dC", "dz", "dh0"):
        assert relerr(full[k], ref[k]) < 1e-12, k
    for tbar in (1, 5, 13):
        ds = oracle.adjoint_sum(*args, tbar=tbar, **kw)
        tl = oracle.trunc_tail(*args, tbar=tbar, **kw)
        for k in ("dx", "ddelta", "dA_log", "dB", "dC", "dz"):
            assert relerr(tl[k], ds[k]) < 1e-11, (tbar, k)


# --------------------------------------------------------------------------
# The decay cotangent da_i = mubar_i h_{i-1} (Prop. 2's vjp_A before the chain
# into Delta and A_log)
# --------------------------------------------------------------------------
def _loss_with_decays(inp, a):
    """L = sum dy * out for the layer with the decays a [b, T, D, N] given
    directly (a plain loop, written here independently of the oracle)."""
    nb, T, D = inp["x"].shape
    N = inp["B"].shape[-1]
    h = np.array(inp["h0"]) if inp["h0"] is not None else np.zeros((nb, D, N))
    L = 0.0
    for t in range(T):
        h = a[:, t] * h + inp["B"][:, t, None, :] * inp["x"][:, t, :, None]
        y = (inp["C"][:, t, None, :] * h).sum(-1)
        if inp["z"] is not None:
            y = y * inp["z"][:, t] / (1.0 + np.exp(-inp["z"][:, t]))
        L += float(np.sum(inp["dy"][:, t] * y))
    return L


def _decays(inp):
    dl = np.log1p(np.exp(inp["delta"])) if inp["delta_softplus"] else inp["delta"]
    return np.exp(-dl[..., None] * np.exp(inp["A_log"])[None, None])


def test_decay_cotangent_matches_central_differences(rng):
    """Full mode: da[b, i, d, n] = dL/da_i[d, n] with every decay an independent
    input; central differences (step 1e-6) on every entry of a small layer."""
    inp = tiny(rng, nb=2, T=7, D=2, N=3, gate=True, softplus=True, h0=True)
    got = bptt_of(inp, want_dh0=False, want_da=True)["da"]
    a = _decays(inp)
    fd = np.zeros_like(a)
    eps = 1e-6
    for idx in np.ndindex(*a.shape):
        ap, am = a.copy(), a.copy()
        ap[idx] += eps
        am[idx] -= eps
        fd[idx] = (_loss_with_decays(inp, ap) - _loss_with_decays(inp, am)) / (2 * eps)
    assert relerr(got, fd) < 1e-7
    ds = oracle.adjoint_sum(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], h0=inp["h0"],
                            z=inp["z"], delta_softplus=True, want_da=True)["da"]
    assert relerr(ds, got) < 1e-12  # Prop. 2's double sum, literally


def test_truncated_decay_cotangent_is_sum_of_per_loss_truncated_backprop(rng):
    """Truncated mode: da is the sum over loss terms l^t of the gradient of l^t
    with respect to the decays of its last Tbar steps only (the state entering
    that window detached): torch autograd with the decays as leaves."""
    nb, T, D, N, tbar = 1, 13, 2, 3, 4
    inp = tiny(rng, nb=nb, T=T, D=D, N=N, gate=True, softplus=True, h0=True)
    a = torch.tensor(_decays(inp), dtype=torch.float64, requires_grad=True)
    Bt, Ct, xt = (torch.tensor(inp[k]) for k in ("B", "C", "x"))
    zt, dyt = torch.tensor(inp["z"]), torch.tensor(inp["dy"])
    for t in range(T):
        h = torch.tensor(inp["h0"])
        for i in range(t + 1):
            if i == t - tbar + 1:
                h = h.detach()
            h = a[:, i] * h + Bt[:, i, None, :] * xt[:, i, :, None]
        y = (Ct[:, t, None, :] * h).sum(-1)
        (dyt[:, t] * y * torch.nn.functional.silu(zt[:, t])).sum().backward()
    ref = a.grad.numpy()
    kw = dict(tbar=tbar, h0=inp["h0"], z=inp["z"], delta_softplus=True, want_da=True)
    args = (inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"])
    assert relerr(oracle.adjoint_sum(*args, **kw)["da"], ref) < 1e-12
    assert relerr(oracle.trunc_tail(*args, **kw)["da"], ref) < 1e-11
