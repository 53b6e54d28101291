"""GPU parity of the gradient's debug output da [b, T, D, N], the cotangent of
each decay value da_t = mubar_t h_{t-1} (Prop. 2's vjp_A term before it is
chained into Delta and A_log), against the oracle's, which is pinned by
central differences (full) and by per-loss truncated backpropagation
(truncated) in tests/test_oracle_pins.py."""
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import WORKLOADS, Workload, make_inputs

from gpu_helpers import TOL_F32, TOL_SCAN_BF16, check, say, to_np

pytestmark = pytest.mark.gpu

SLOW = WORKLOADS["small_slow"]
RAGGED = Workload("ragged_da", 2, 250, 50, 5, 50, 0, False, False, 692140, delta_scale=0.25)
GATE16 = Workload("gate16_da", 2, 300, 40, 16, 40, 0, True, True, 692141)


def _oracle_da(inp, w, tbar, a_scalar=False, b_delta=False):
    args = [to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C", "dy")]
    kw = dict(h0=to_np(inp["h0"]) if "h0" in inp else None, z=to_np(inp["z"]) if "z" in inp else None,
              delta_softplus=w.proj, want_da=True, a_scalar=a_scalar, b_delta=b_delta)
    if tbar <= 0 or tbar >= w.T:
        return oracle.bptt(*args, want_dh0=False, **kw)["da"]
    return oracle.adjoint_sum(*args, tbar=tbar, **kw)["da"]


def _gpu(fn, inp, w, tbar, b_delta=False):
    g = fn(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], h0=inp.get("h0"), z=inp.get("z"),
           softplus=w.proj, tbar=tbar, want_da=True, b_delta=b_delta)
    torch.cuda.synchronize()
    return g


@pytest.mark.parametrize("tbar", [0, 1, 32, 100])
def test_da_small_slow(tbar):
    w = SLOW
    say(f"[da] {w.name} tbar={tbar}")
    inp = make_inputs(w, device="cuda")
    g = _gpu(ssm.ssm_adjoint_grad, inp, w, tbar)
    check("da", to_np(g["da"]), _oracle_da(inp, w, tbar), TOL_F32)


@pytest.mark.parametrize("tbar", [0, 37])
def test_da_ragged_h0_and_entry_points(tbar):
    """Ragged shape (N = 5, D = 50, b = 2) with h0; the same output through the
    pair formulation and the entry point without a workspace."""
    w = RAGGED
    say(f"[da ragged] tbar={tbar}")
    inp = make_inputs(w, device="cuda", h0=True)
    ref = _oracle_da(inp, w, tbar)
    for name, fn in (("scan", ssm.ssm_adjoint_grad), ("pairs", ssm.ssm_adjoint_grad_pairs),
                     ("noalloc", ssm.ssm_adjoint_grad_noalloc)):
        g = _gpu(fn, inp, w, tbar)
        check(f"da[{name}]", to_np(g["da"]), ref, TOL_F32)


@pytest.mark.parametrize("tbar", [0, 64])
def test_da_bf16_gate_softplus(tbar):
    w = GATE16
    say(f"[da bf16 gate] tbar={tbar}")
    inp = make_inputs(w, device="cuda")
    g = _gpu(ssm.ssm_adjoint_grad, inp, w, tbar)
    check("da", to_np(g["da"]), _oracle_da(inp, w, tbar), TOL_SCAN_BF16)


@pytest.mark.parametrize("a_scalar,b_delta", [(True, False), (False, True)])
def test_da_variants(a_scalar, b_delta):
    w = SLOW.with_(T=200, D=48)
    say(f"[da variants] a_scalar={a_scalar} b_delta={b_delta}")
    inp = make_inputs(w, device="cuda")
    if a_scalar:
        inp["A_log"] = inp["A_log"][:, 0].contiguous()
    for tbar in (0, 30):
        g = _gpu(ssm.ssm_adjoint_grad, inp, w, tbar, b_delta=b_delta)
        check(f"da[tbar={tbar}]", to_np(g["da"]), _oracle_da(inp, w, tbar, a_scalar, b_delta), TOL_F32)
