"""GPU parity of the one-lane-per-channel chunk-aggregate and forward kernels
against the fp64 oracle.  Those kernels run on grids of at least 2,048 waves at
one lane per channel (64-channel blocks x chunks x batch); smaller grids take the
quad layout, which the other small-size tests cover.  Chunks of 16 steps let
T = 32,768 steps and 64 channels reach that size at a cost the oracle finishes
in seconds.  Cases: fp32 and bf16 inputs; 16 states (wide scalar loads of B and
C) and fewer (per-state scalar loads, odd element offsets in bf16); gate and
softplus; the scalar decay and the step-size-scaled input; ragged last chunks
(11 steps, and 2: shorter than a group of 4) with padding channels; full and
truncated gradients; the forward output."""
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import Workload, make_inputs

from gpu_helpers import TOL_F32, TOL_SCAN_BF16, check, say, to_np

pytestmark = pytest.mark.gpu

CHUNK = 16
# name, b, T, D, N, d_model, tbar, gate+softplus, bf16, seed
F32 = Workload("lanes_f32", 1, 32768, 64, 16, 64, 100, False, False, 692301, delta_scale=0.25)
# ragged: T ends inside a chunk and its last group, 60 channels end inside the block
RAGGED = Workload("lanes_ragged", 1, 32763, 60, 12, 60, 100, False, False, 692302, delta_scale=0.25)
BF16 = Workload("lanes_bf16", 1, 32768, 64, 16, 64, 300, True, True, 692303)
# the last chunk has 2 steps: no whole 4-step group, only the per-step tail
BF16_N7 = Workload("lanes_bf16_n7", 1, 32754, 64, 7, 64, 300, True, True, 692304)


def _waves(w):
    return (w.D + 63) // 64 * -(-w.T // CHUNK) * w.b


def _inputs(w, a_scalar=False):
    assert _waves(w) >= 2048, "the shape must select the one-lane-per-channel kernels"
    inp = make_inputs(w, device="cuda")
    if a_scalar:
        inp["A_log"] = inp["A_log"][:, 0].contiguous()
    torch.cuda.synchronize()
    return inp


def _args(inp):
    return [to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C", "dy")]


def _grad_case(w, tbar, a_scalar, b_delta, tol):
    inp = _inputs(w, a_scalar)
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], z=inp.get("z"),
                             softplus=w.proj, tbar=tbar, chunk=CHUNK, b_delta=b_delta)
    torch.cuda.synchronize()
    kw = dict(z=to_np(inp["z"]) if "z" in inp else None, delta_softplus=w.proj, a_scalar=a_scalar,
              b_delta=b_delta)
    if tbar <= 0:
        ref = oracle.bptt(*_args(inp), want_dh0=False, **kw)
    else:
        ref = oracle.trunc_tail(*_args(inp), tbar=tbar, want_dh0=False, **kw)
    rep = {}
    for k in ("dx", "ddelta", "dA_log", "dB", "dC") + (("dz",) if w.proj else ()):
        check(k, to_np(g[k]), ref[k], tol, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


@pytest.mark.parametrize("tbar", [0, 100])
def test_lanes_f32(tbar):
    say(f"[lanes f32] T={F32.T} D={F32.D} chunk={CHUNK} tbar={tbar}")
    _grad_case(F32, tbar, False, False, TOL_F32)


@pytest.mark.parametrize("a_scalar,b_delta", [(False, False), (True, False), (False, True), (True, True)])
def test_lanes_ragged_variants(a_scalar, b_delta):
    say(f"[lanes ragged] T={RAGGED.T} D={RAGGED.D} N={RAGGED.N} a_scalar={a_scalar} b_delta={b_delta}")
    _grad_case(RAGGED, RAGGED.tbar, a_scalar, b_delta, TOL_F32)


@pytest.mark.parametrize("w", [BF16, BF16_N7], ids=["n16", "n7"])
@pytest.mark.parametrize("tbar", [0, 300])
def test_lanes_bf16_gate(w, tbar):
    # bf16 inputs read as the same bits on both sides: fp32 against fp64 arithmetic
    say(f"[lanes bf16 gate] T={w.T} D={w.D} N={w.N} tbar={tbar}")
    _grad_case(w, tbar, False, False, TOL_SCAN_BF16)


@pytest.mark.parametrize("w", [F32, RAGGED, BF16, BF16_N7], ids=["f32", "ragged", "bf16", "bf16_n7"])
def test_lanes_forward(w):
    say(f"[lanes forward] {w.name} T={w.T} D={w.D} N={w.N}")
    inp = _inputs(w)
    y, hl = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], z=inp.get("z"),
                                    softplus=w.proj, chunk=CHUNK, want_h_last=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")),
                            z=to_np(inp["z"]) if "z" in inp else None, delta_softplus=w.proj)
    # bf16 y carries one rounding (2^-9 relative): held to half of that
    check("y", to_np(y), ry, 2e-3 if w.bf16 else TOL_F32)
    check("h_last", to_np(hl), rh, TOL_SCAN_BF16 if w.bf16 else TOL_F32)
