"""GPU parity of the language head (ssm_lm_head_grad: Sec. 3.2's Omega with the
cross-entropy loss, the products on the bf16 MFMA GEMMs) against the fp64
oracle in oracle/head.py, whose pins are in tests/test_oracle_head.py.

Two references: the oracle with Norm(y) and the logit gradients rounded to bf16
where the GPU stores them (round_bf16=True), where only fp32 against fp64
arithmetic differs, and the exact fp64 model, within the bf16 budget.  Bound of
the first: the logit gradients are computed in fp32 to about 2^-22 relative
before their rounding to bf16, so a fraction of about 2^-22 / 2^-8 = 2^-14 of
them round to the neighbouring bf16 value on one side only, each a change of
2^-8 relative: a rel-L2 of about 2^-7 * 2^-8 = 3e-5 in dy and dOmega; 2e-4 leaves
a factor of 6 above it."""
import numpy as np
import pytest
import torch

import paper_2501_00692_amd as ssm
from oracle.head import head_loss_grad
from paper_2501_00692_amd.synth import HEAD_WORKLOADS, make_head_inputs

from gpu_helpers import TOL_BF16, check, say, to_np

pytestmark = pytest.mark.gpu

TOL_HEAD_ROUNDED = 2e-4


def _run(inp, norm, block_rows=0):
    o = ssm.ssm_lm_head_grad(inp["y"], inp["omega"], inp["targets"], norm=norm, block_rows=block_rows)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in o.items()}


def _compare(o, y, om, t, norm, valid):
    for rnd, tol in ((True, TOL_HEAD_ROUNDED), (False, TOL_BF16)):
        ref = head_loss_grad(y, om, t, norm=norm, round_bf16=rnd)
        tag = "rounded" if rnd else "exact"
        check(f"loss[{tag}]", o["loss"][valid], ref["loss"][valid], tol)
        check(f"dy[{tag}]", o["dy"], ref["dy"], tol)
        check(f"domega[{tag}]", o["domega"], ref["domega"], tol)


@pytest.mark.parametrize("norm", [True, False])
def test_head_small(norm):
    """Ragged shapes (M = 300, P = 96, V = 1000: partial GEMM tiles in every
    dimension), one ignored and one out-of-range target."""
    M, P, V = HEAD_WORKLOADS["head_small"]
    say(f"[head small] M={M} P={P} V={V} norm={norm}")
    inp = make_head_inputs(M, P, V, 692300, device="cuda")
    inp["targets"][5] = -1
    inp["targets"][17] = V
    o = _run(inp, norm)
    y, om, t = to_np(inp["y"]), to_np(inp["omega"]), inp["targets"].cpu().numpy()
    assert o["loss"][5] == 0.0 and np.isnan(o["loss"][17])
    assert np.abs(o["dy"][[5, 17]]).max() == 0.0
    valid = (t >= 0) & (t < V)
    _compare(o, y, om, t, norm, valid)


@pytest.mark.parametrize("extra", [0, 3])
def test_head_row_blocks(extra):
    """Four row blocks of 256, dOmega adding the blocks.  The last block has 232
    rows, or 235, which is not a multiple of 8: its logits then take the dX form
    while the full blocks' take the weight-gradient form from the transposed
    Norm(y), so one call runs both paths."""
    M, P, V = HEAD_WORKLOADS["head_blocks"]
    M += extra
    say(f"[head blocks] M={M} P={P} V={V} block_rows=256")
    inp = make_head_inputs(M, P, V, 692301, device="cuda")
    o = _run(inp, True, block_rows=256)
    y, om, t = to_np(inp["y"]), to_np(inp["omega"]), inp["targets"].cpu().numpy()
    _compare(o, y, om, t, True, np.ones(M, bool))


@pytest.mark.parametrize("block_rows", [0, 1024])
def test_head_medium(block_rows):
    """4,096 tokens, a 32,000-token vocabulary: one block, and four blocks."""
    M, P, V = HEAD_WORKLOADS["head_medium"]
    say(f"[head medium] M={M} P={P} V={V} block_rows={block_rows}")
    inp = make_head_inputs(M, P, V, 692302, device="cuda")
    o = _run(inp, True, block_rows=block_rows)
    y, om, t = to_np(inp["y"]), to_np(inp["omega"]), inp["targets"].cpu().numpy()
    ref = head_loss_grad(y, om, t, norm=True, round_bf16=True)
    check("loss[rounded]", o["loss"], ref["loss"], TOL_HEAD_ROUNDED)
    check("dy[rounded]", o["dy"], ref["dy"], TOL_HEAD_ROUNDED)
    check("domega[rounded]", o["domega"], ref["domega"], TOL_HEAD_ROUNDED)


def test_head_repeat_is_bitwise_identical():
    M, P, V = HEAD_WORKLOADS["head_small"]
    inp = make_head_inputs(M, P, V, 692303, device="cuda")
    a = _run(inp, True)
    b = _run(inp, True)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("V", [6000, 12000, 50304, 80000])
def test_head_row_kernel_paths(V):
    """The loss kernel holds a row in registers for vocabularies up to 65,536
    (2, 4 and 16 float4 pieces per thread here) and reads it twice above that
    (80,000): each against the oracle with the GPU's bf16 rounding."""
    M, P = 48, 64
    say(f"[head row kernel] M={M} P={P} V={V}")
    inp = make_head_inputs(M, P, V, 692304, device="cuda")
    inp["targets"][0] = V - 1
    inp["targets"][1] = 0
    o = _run(inp, True)
    y, om, t = to_np(inp["y"]), to_np(inp["omega"]), inp["targets"].cpu().numpy()
    ref = head_loss_grad(y, om, t, norm=True, round_bf16=True)
    for k in ("loss", "dy", "domega"):
        check(f"{k}[rounded]", o[k], ref[k], TOL_HEAD_ROUNDED)
