"""GPU parity of the layer variants against the fp64 oracle: the scalar-decay
SSM of Table 1 (one decay rate per channel, A_log of shape [D]) and the
step-size-scaled input (h = a h + Delta B x), alone and together, in full and
truncated form, with ragged shapes, fp32 and bf16 inputs, and through the whole
layer with projections."""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import WORKLOADS, Workload, make_inputs

from gpu_helpers import TOL_BF16, TOL_F32, TOL_SCAN_BF16, check, say, to_np

pytestmark = pytest.mark.gpu

VARIANTS = [(True, False), (False, True), (True, True)]


def _inputs(w, a_scalar, h0=False):
    inp = make_inputs(w, device="cuda", h0=h0)
    if a_scalar:
        inp["A_log"] = inp["A_log"][:, 0].contiguous()
    torch.cuda.synchronize()
    return inp


def _oracle(inp, w, tbar, a_scalar, b_delta, want_dh0=False):
    args = [to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C", "dy")]
    kw = dict(h0=to_np(inp["h0"]) if "h0" in inp else None, z=to_np(inp["z"]) if "z" in inp else None,
              delta_softplus=w.proj, a_scalar=a_scalar, b_delta=b_delta)
    if tbar <= 0 or tbar >= w.T:
        return oracle.bptt(*args, want_dh0=want_dh0, **kw)
    return oracle.adjoint_sum(*args, tbar=tbar, want_dh0=False, **kw)


def _gpu(inp, w, tbar, chunk, b_delta, want_dh0=False):
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"],
                             h0=inp.get("h0"), z=inp.get("z"), softplus=w.proj, tbar=tbar, chunk=chunk,
                             want_dh0=want_dh0, b_delta=b_delta)
    torch.cuda.synchronize()
    return g


def _compare(g, ref, tol, gate, dh0=False):
    rep = {}
    for k in ("dx", "ddelta", "dA_log", "dB", "dC") + (("dz",) if gate else ()) + (("dh0",) if dh0 else ()):
        check(k, to_np(g[k]), ref[k], tol, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


SMALL = WORKLOADS["small"]
RAGGED = Workload("ragged_v", 2, 250, 50, 5, 50, 0, False, False, 692110, delta_scale=0.25)
GATED32 = Workload("gated32_v", 2, 300, 40, 16, 40, 0, True, False, 692111)
BF16MID = Workload("bf16mid_v", 2, 1000, 256, 16, 128, 0, True, True, 692112)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
@pytest.mark.parametrize("chunk", [16, 128])
def test_variant_forward(a_scalar, b_delta, chunk):
    w = SMALL
    say(f"[variant forward] a_scalar={a_scalar} b_delta={b_delta} chunk={chunk}")
    inp = _inputs(w, a_scalar, h0=True)
    y, hl = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], h0=inp["h0"],
                                    chunk=chunk, want_h_last=True, b_delta=b_delta)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")), h0=to_np(inp["h0"]),
                            a_scalar=a_scalar, b_delta=b_delta)
    check("y", to_np(y), ry, TOL_F32)
    check("h_last", to_np(hl), rh, TOL_F32)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
@pytest.mark.parametrize("chunk,tbar", [(64, 0), (16, 0), (256, 0), (64, 32), (128, 32)])
def test_variant_grad_small(a_scalar, b_delta, chunk, tbar):
    w = SMALL
    say(f"[variant grad] a_scalar={a_scalar} b_delta={b_delta} chunk={chunk} tbar={tbar}")
    inp = _inputs(w, a_scalar, h0=tbar == 0)
    full = tbar == 0
    g = _gpu(inp, w, tbar, chunk, b_delta, want_dh0=full)
    _compare(g, _oracle(inp, w, tbar, a_scalar, b_delta, want_dh0=full), TOL_F32, False, dh0=full)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
@pytest.mark.parametrize("chunk,tbar", [(64, 0), (32, 100), (16, 249)])
def test_variant_grad_ragged(a_scalar, b_delta, chunk, tbar):
    """T not a multiple of the chunk, D not a multiple of 16, N < 16."""
    w = RAGGED
    say(f"[variant ragged] a_scalar={a_scalar} b_delta={b_delta} chunk={chunk} tbar={tbar}")
    inp = _inputs(w, a_scalar, h0=tbar == 0)
    full = tbar == 0
    g = _gpu(inp, w, tbar, chunk, b_delta, want_dh0=full)
    _compare(g, _oracle(inp, w, tbar, a_scalar, b_delta, want_dh0=full), TOL_F32, False, dh0=full)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
@pytest.mark.parametrize("tbar", [0, 20])
def test_variant_grad_gate_softplus_fp32(a_scalar, b_delta, tbar):
    w = GATED32
    say(f"[variant gate fp32] a_scalar={a_scalar} b_delta={b_delta} tbar={tbar}")
    inp = _inputs(w, a_scalar)
    g = _gpu(inp, w, tbar, 64, b_delta)
    _compare(g, _oracle(inp, w, tbar, a_scalar, b_delta), TOL_F32, True)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
def test_variant_grad_bf16(a_scalar, b_delta):
    w = BF16MID
    say(f"[variant bf16] a_scalar={a_scalar} b_delta={b_delta}")
    inp = _inputs(w, a_scalar)
    g = _gpu(inp, w, 64, 0, b_delta)
    _compare(g, _oracle(inp, w, 64, a_scalar, b_delta), TOL_SCAN_BF16, True)


LAYER_V = Workload("layer_v", 2, 192, 96, 16, 64, 0, True, True, 692113)


@pytest.mark.parametrize("a_scalar,b_delta", VARIANTS)
def test_variant_layer(a_scalar, b_delta):
    w = LAYER_V
    say(f"[variant layer] a_scalar={a_scalar} b_delta={b_delta}")
    inp = _inputs(w, a_scalar)
    o = ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"],
                           inp["A_log"], inp["dy"], want_scan=True, b_delta=b_delta)
    torch.cuda.synchronize()
    h = {k: to_np(v) for k, v in inp.items()}
    ref = oracle.layer_grad(h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"],
                            a_scalar=a_scalar, b_delta=b_delta)
    M = w.b * w.T
    rep = {}
    for k in ("dx", "ddelta", "dB", "dC", "dz", "dA_log"):
        check(k, to_np(o[k]), ref[k], TOL_SCAN_BF16, rep)
    check("dx_total", to_np(o["dx_total"]).reshape(M, -1), ref["dx_total"], TOL_BF16, rep)
    check("dW_x", to_np(o["dW_x"]), ref["dW_x"], TOL_BF16, rep)
    check("dW_in", to_np(o["dW_in"]), ref["dW_in"], TOL_BF16, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))
