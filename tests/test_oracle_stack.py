"""Pins of the K-layer stack oracle (oracle/stack.py) against torch float64
autograd of an independently written naive model, and against the relations
between Prop. 3's gradient and backpropagation."""
import numpy as np
import pytest
import torch

from oracle import stack as ostack

K, B_, T, D, N = 3, 2, 10, 8, 4


@pytest.fixture(scope="module")
def model():
    r = np.random.default_rng(692300)
    y0 = r.standard_normal((B_, T, D))
    W_in = [r.standard_normal((D, 2 * D)) / np.sqrt(D) for _ in range(K)]
    W_x = [r.standard_normal((D, D + 2 * N)) / np.sqrt(D) for _ in range(K)]
    A_log = [r.uniform(0.0, np.log(16.0), (D, N)) for _ in range(K)]
    gK = r.standard_normal((B_, T, D))
    return y0, W_in, W_x, A_log, gK


def _torch_stack(y0, W_in, W_x, A_log, detach_inputs):
    """The residual stack of Sec. 3.2 written as plain torch ops with a step
    loop for the recurrence; with ``detach_inputs`` each layer's normalised
    input is computed from a detached y_{k-1} (no gradient flows into earlier
    layers through it)."""
    y = torch.tensor(y0)
    for k in range(K):
        src = y.detach() if detach_inputs else y
        u = src / torch.sqrt((src * src).mean(-1, keepdim=True) + ostack.EPS)
        xz = u @ W_in[k]
        x, z = xz[..., :D], xz[..., D:]
        pj = x @ W_x[k]
        dl = torch.nn.functional.softplus(pj[..., :D])
        Bm, Cm = pj[..., D:D + N], pj[..., D + N:]
        h = torch.zeros(B_, D, N, dtype=torch.float64)
        outs = []
        for t in range(T):
            a = torch.exp(-dl[:, t, :, None] * torch.exp(A_log[k]))
            h = a * h + Bm[:, t, None, :] * x[:, t, :, None]
            outs.append((h * Cm[:, t, None, :]).sum(-1))
        yk = torch.stack(outs, 1)
        y = y + yk * z * torch.sigmoid(z)
    return y


def _autograd(model, detach_inputs):
    y0, W_in, W_x, A_log, gK = model
    Wi = [torch.tensor(w, requires_grad=True) for w in W_in]
    Wx = [torch.tensor(w, requires_grad=True) for w in W_x]
    Al = [torch.tensor(a, requires_grad=True) for a in A_log]
    yK = _torch_stack(y0, Wi, Wx, Al, detach_inputs)
    (yK * torch.tensor(gK)).sum().backward()
    return [dict(dW_in=Wi[k].grad.numpy(), dW_x=Wx[k].grad.numpy(), dA_log=Al[k].grad.numpy()) for k in range(K)]


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def _oracle(model, mode):
    y0, W_in, W_x, A_log, gK = model
    yK, acts = ostack.stack_forward(y0, W_in, W_x, A_log, N, round_bf16=False)
    return yK, ostack.stack_grad(acts, W_in, W_x, A_log, gK, mode=mode, round_bf16=False)


def test_forward_matches_torch(model):
    y0, W_in, W_x, A_log, gK = model
    yK, _ = _oracle(model, "exact")
    ref = _torch_stack(y0, [torch.tensor(w) for w in W_in], [torch.tensor(w) for w in W_x],
                       [torch.tensor(a) for a in A_log], False).numpy()
    assert _rel(yK, ref) < 1e-12


def test_exact_mode_is_backpropagation(model):
    _, got = _oracle(model, "exact")
    ref = _autograd(model, detach_inputs=False)
    for k in range(K):
        for n in ("dW_in", "dW_x", "dA_log"):
            assert _rel(got[k][n], ref[k][n]) < 1e-10, (k, n)


def test_adjoint_mode_is_prop3(model):
    """Prop. 3 takes every layer's vjps with the upstream dL/dy_K and the layer's
    stored input: the gradient of L with each layer input held fixed."""
    _, got = _oracle(model, "adjoint")
    ref = _autograd(model, detach_inputs=True)
    for k in range(K):
        for n in ("dW_in", "dW_x", "dA_log"):
            assert _rel(got[k][n], ref[k][n]) < 1e-10, (k, n)


def test_modes_agree_on_last_layer_and_differ_below(model):
    _, ad = _oracle(model, "adjoint")
    _, ex = _oracle(model, "exact")
    for n in ("dW_in", "dW_x", "dA_log"):
        assert _rel(ad[K - 1][n], ex[K - 1][n]) < 1e-12
        assert _rel(ad[0][n], ex[0][n]) > 1e-3  # the omitted paths are visible


def test_single_layer_modes_agree(model):
    y0, W_in, W_x, A_log, gK = model
    _, acts = ostack.stack_forward(y0, W_in[:1], W_x[:1], A_log[:1], N, round_bf16=False)
    ad = ostack.stack_grad(acts, W_in[:1], W_x[:1], A_log[:1], gK, mode="adjoint", round_bf16=False)
    ex = ostack.stack_grad(acts, W_in[:1], W_x[:1], A_log[:1], gK, mode="exact", round_bf16=False)
    for n in ("dW_in", "dW_x", "dA_log"):
        assert _rel(ad[0][n], ex[0][n]) == 0.0


def test_bf16_rounding_matches_torch():
    r = np.random.default_rng(1)
    v = np.concatenate([r.standard_normal(10000) * 10.0 ** r.integers(-6, 6, 10000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38]])
    ref = torch.tensor(v, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(ostack.bf16(v), ref)
