"""Pins of the language-head oracle (Sec. 3.2's Omega with the cross-entropy
loss) against facts fixed by mathematics: central differences, torch autograd
of an independently written head, closed forms (a zero head, two-token
vocabularies), invariants (softmax rows sum to one; the normalised head is
scale invariant), and the handling of ignored and out-of-range targets.  CPU
only."""
import numpy as np
import pytest
import torch

from oracle.head import head_forward, head_loss_grad
from oracle.stack import EPS


def _inputs(rng, M=5, P=6, V=7, ignore=True):
    y = rng.standard_normal((M, P)) * 1.5
    om = rng.standard_normal((V, P)) / np.sqrt(P)
    t = rng.integers(0, V, M)
    if ignore:
        t[1] = -1
    return y, om, t


def _relerr(a, b):
    a, b = np.asarray(a, float), np.asarray(b, float)
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def _total(y, om, t, norm):
    return float(np.sum(head_loss_grad(y, om, t, norm=norm, want_domega=False)["loss"]))


@pytest.mark.parametrize("norm", [True, False])
def test_head_grad_matches_central_differences(rng, norm):
    y, om, t = _inputs(rng)
    g = head_loss_grad(y, om, t, norm=norm)
    eps = 1e-6
    for name, arr, ref in (("y", y, g["dy"]), ("omega", om, g["domega"])):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(*arr.shape):
            p, m = arr.copy(), arr.copy()
            p[idx] += eps
            m[idx] -= eps
            args_p = (p, om) if name == "y" else (y, p)
            args_m = (m, om) if name == "y" else (y, m)
            fd[idx] = (_total(*args_p, t, norm) - _total(*args_m, t, norm)) / (2 * eps)
        assert _relerr(ref, fd) < 1e-7, name


@pytest.mark.parametrize("norm", [True, False])
def test_head_matches_torch_autograd(rng, norm):
    y, om, t = _inputs(rng, M=9, P=8, V=11)
    ty = torch.tensor(y, requires_grad=True)
    to = torch.tensor(om, requires_grad=True)
    u = ty / torch.sqrt((ty * ty).mean(dim=1, keepdim=True) + EPS) if norm else ty
    logits = u @ to.T
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(t), ignore_index=-1, reduction="none")
    loss.sum().backward()
    g = head_loss_grad(y, om, t, norm=norm)
    assert _relerr(g["loss"], loss.detach().numpy()) < 1e-13
    assert _relerr(g["dy"], ty.grad.numpy()) < 1e-12
    assert _relerr(g["domega"], to.grad.numpy()) < 1e-12


def test_zero_head_closed_form(rng):
    """Omega = 0: every logit is 0, so l = log V, G = 1/V - onehot, dy = 0 and
    dOmega[v] = sum_m (1/V - [t_m = v]) u_m."""
    y, om, t = _inputs(rng, M=6, P=5, V=9, ignore=False)
    om[:] = 0.0
    g = head_loss_grad(y, om, t)
    assert np.allclose(g["loss"], np.log(9.0), rtol=0, atol=1e-14)
    assert np.abs(g["dy"]).max() == 0.0
    u = y / np.sqrt(np.mean(y * y, axis=1, keepdims=True) + EPS)
    ref = np.tile(u.sum(axis=0) / 9.0, (9, 1))
    for m in range(6):
        ref[t[m]] -= u[m]
    assert _relerr(g["domega"], ref) < 1e-14


def test_two_token_vocabulary_is_logistic(rng):
    """V = 2: the cross-entropy is the logistic loss of the margin,
    l = log(1 + exp(o_other - o_target))."""
    y, om, t = _inputs(rng, M=8, P=4, V=2, ignore=False)
    o, _, _ = head_forward(y, om)
    margin = o[np.arange(8), 1 - t] - o[np.arange(8), t]
    g = head_loss_grad(y, om, t)
    assert _relerr(g["loss"], np.logaddexp(0.0, margin)) < 1e-14


def test_softmax_rows_sum_to_one(rng):
    """Each valid row of G sums to 0, so the rows of dOmega sum to the zero
    vector over the vocabulary."""
    y, om, t = _inputs(rng, M=7, P=6, V=13)
    g = head_loss_grad(y, om, t)
    col = g["domega"].sum(axis=0)
    assert np.abs(col).max() < 1e-13 * np.abs(g["domega"]).max() * 13


def test_normalised_head_is_scale_invariant(rng):
    """With Norm, l(c y) = l(y) up to the epsilon of the normalisation, and
    dy is orthogonal to y up to the same epsilon: <dy, y> = r <dU, y> eps/(ms + eps)."""
    y, om, t = _inputs(rng, M=6, P=32, V=10, ignore=False)
    a = head_loss_grad(y, om, t)
    b = head_loss_grad(3.0 * y, om, t)
    assert np.abs(a["loss"] - b["loss"]).max() < 1e-5
    dots = np.abs(np.sum(a["dy"] * y, axis=1))
    norms = np.linalg.norm(a["dy"], axis=1) * np.linalg.norm(y, axis=1)
    assert (dots <= 1e-5 * norms).all()


def test_ignored_and_out_of_range_targets(rng):
    y, om, t = _inputs(rng, M=5, P=6, V=7, ignore=False)
    t[0], t[3] = -1, 7
    g = head_loss_grad(y, om, t)
    assert g["loss"][0] == 0.0 and np.isnan(g["loss"][3])
    assert np.abs(g["dy"][[0, 3]]).max() == 0.0
    keep = [1, 2, 4]
    ref = head_loss_grad(y[keep], om, t[keep])
    assert _relerr(g["domega"], ref["domega"]) < 1e-14
    assert _relerr(g["loss"][keep], ref["loss"]) < 1e-15


def test_rounded_operands_stay_close(rng):
    """round_bf16 changes only the stored operands: the result stays within the
    bf16 budget of the exact one."""
    y, om, t = _inputs(rng, M=64, P=48, V=200)
    a = head_loss_grad(y, om, t)
    b = head_loss_grad(y, om, t, round_bf16=True)
    for k in ("loss", "dy", "domega"):
        assert _relerr(b[k], a[k]) < 2e-2, k
