"""GPU parity against the fp64 oracle at sizes the oracle finishes in seconds:
several chunks and 16-channel tiles, ragged tails, every chunk size, full and
truncated forms, gate and softplus, fp32 and bf16 inputs."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import WORKLOADS, Workload, make_inputs

from gpu_helpers import TOL_BF16, TOL_F32, TOL_SCAN_BF16, check, say, to_np

pytestmark = pytest.mark.gpu


def _inputs(w: Workload, h0=False):
    inp = make_inputs(w, device="cuda", h0=h0)
    torch.cuda.synchronize()
    return inp


def _oracle_grad(inp, w, tbar, literal=False, want_dh0=False):
    args = [to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C", "dy")]
    kw = dict(h0=to_np(inp["h0"]) if "h0" in inp else None,
              z=to_np(inp["z"]) if "z" in inp else None, delta_softplus=w.proj)
    if tbar <= 0 or tbar >= w.T:
        return oracle.bptt(*args, want_dh0=want_dh0, **kw)
    fn = oracle.adjoint_sum if literal else oracle.trunc_tail
    return fn(*args, tbar=tbar, want_dh0=False, **kw)


def _gpu_grad(inp, w, tbar, chunk, want_dh0=False):
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"],
                             h0=inp.get("h0"), z=inp.get("z"), softplus=w.proj, tbar=tbar, chunk=chunk,
                             want_dh0=want_dh0)
    torch.cuda.synchronize()
    return g


def _compare(g, ref, tol, gate, dh0=False):
    rep = {}
    for k in ("dx", "ddelta", "dA_log", "dB", "dC") + (("dz",) if gate else ()) + (("dh0",) if dh0 else ()):
        check(k, to_np(g[k]), ref[k], tol, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


SMALL = WORKLOADS["small"]
SLOW = WORKLOADS["small_slow"]


@pytest.mark.parametrize("chunk", [16, 32, 64, 128, 256])
def test_forward_small(chunk):
    w = SMALL
    say(f"[forward] workload={w.name} chunk={chunk}")
    inp = _inputs(w, h0=True)
    y, hl = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], h0=inp["h0"],
                                    chunk=chunk, want_h_last=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")), h0=to_np(inp["h0"]))
    check("y", to_np(y), ry, TOL_F32)
    check("h_last", to_np(hl), rh, TOL_F32)


# the layer's forward configuration (bf16 inputs, softplus, gate) with ragged
# length and channel count (T = 300 ends inside a chunk, 72 channels end inside a
# 64-channel workgroup); y is bf16, the state fp32
GATE_BF16 = Workload("fwd_gate_bf16", 2, 300, 72, 16, 32, 0, True, True, 692151)


@pytest.mark.parametrize("chunk", [16, 128])
def test_forward_gate_bf16(chunk):
    w = GATE_BF16
    say(f"[forward gate bf16] T={w.T} D={w.D} chunk={chunk}")
    inp = _inputs(w, h0=True)
    y, hl = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], h0=inp["h0"],
                                    z=inp["z"], softplus=True, chunk=chunk, want_h_last=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")), h0=to_np(inp["h0"]),
                            z=to_np(inp["z"]), delta_softplus=True)
    # y is stored in bf16 (one rounding, 2^-9 relative): held to half of that
    check("y", to_np(y), ry, 2e-3)
    check("h_last", to_np(hl), rh, TOL_SCAN_BF16)


@pytest.mark.parametrize("chunk", [16, 64, 128, 256])
def test_grad_small_full(chunk):
    w = SMALL
    say(f"[grad full] workload={w.name} chunk={chunk}")
    inp = _inputs(w, h0=True)
    g = _gpu_grad(inp, w, 0, chunk, want_dh0=True)
    _compare(g, _oracle_grad(inp, w, 0, want_dh0=True), TOL_F32, False, dh0=True)


@pytest.mark.parametrize("chunk", [16, 64, 128, 256])
def test_grad_small_truncated_literal(chunk):
    w = SMALL
    say(f"[grad trunc] workload={w.name} tbar={w.tbar} chunk={chunk}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, w.tbar, chunk)
    _compare(g, _oracle_grad(inp, w, w.tbar, literal=True), TOL_F32, False)


@pytest.mark.parametrize("tbar", [1, 2, 31, 32, 33, 255, 256, 300])
@pytest.mark.parametrize("chunk", [16, 128])
def test_grad_slow_decay_truncated(tbar, chunk):
    w = SLOW
    say(f"[grad trunc slow] workload={w.name} tbar={tbar} chunk={chunk}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, tbar, chunk)
    ref = _oracle_grad(inp, w, tbar, literal=True)
    _compare(g, ref, TOL_F32, False)
    if 1 < tbar <= w.T // 4:
        full = _oracle_grad(inp, w, 0)
        assert np.linalg.norm(ref["dx"] - full["dx"]) > 1e-3 * np.linalg.norm(full["dx"])  # window visible


# Chunks of 256 steps (16-step segments) over several chunks, with windows below,
# at and above one chunk: the shifted C rows of a segment come from the next
# chunks, and windows that are not a multiple of the chunk sweep the adjoint
# carry back from the end of the chunk holding t + tbar.  Slow decay (Delta / 512:
# horizons of up to about 1,300 steps) keeps the window visible at every tbar.
SLOW1K = Workload("slow1k", 1, 1000, 64, 16, 64, 0, False, False, 692120, delta_scale=1.0 / 512)


@pytest.mark.parametrize("tbar", [37, 255, 256, 300, 512, 700])
def test_grad_chunk256_truncated_multichunk(tbar):
    w = SLOW1K
    say(f"[grad trunc chunk 256] T={w.T} D={w.D} tbar={tbar}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, tbar, 256)
    ref = _oracle_grad(inp, w, tbar, literal=True)
    _compare(g, ref, TOL_F32, False)
    full = _oracle_grad(inp, w, 0)
    assert np.linalg.norm(ref["dx"] - full["dx"]) > 1e-3 * np.linalg.norm(full["dx"])  # window visible


# the same over bf16 inputs, without and with the gate and softplus (b = 2,
# ragged last chunk); the oracle reads the same bf16 bits
SLOW_BF16_256 = Workload("slow_bf16_256", 2, 1800, 96, 16, 96, 0, False, True, 692121, delta_scale=1.0 / 512)
GATE_BF16_256 = Workload("gate_bf16_256", 2, 1800, 96, 16, 96, 0, True, True, 692122)


@pytest.mark.parametrize("tbar", [0, 200, 256, 600])
@pytest.mark.parametrize("w", [SLOW_BF16_256, GATE_BF16_256], ids=["slow", "gate"])
def test_grad_bf16_chunk256(w, tbar):
    say(f"[grad bf16 chunk 256] {w.name} T={w.T} D={w.D} tbar={tbar}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, tbar, 256)
    _compare(g, _oracle_grad(inp, w, tbar), TOL_SCAN_BF16, w.proj)


# fp32, long sequence, slow decay (Delta / 2048: horizons of 150 to 2,500 steps)
# and a short window: the full adjoint is several times larger than the windowed
# one, so any formation of the windowed adjoint as a difference of full-horizon
# fp32 sums would lose the tolerance.
SLOW8K = Workload("slow8k", 1, 8192, 64, 16, 64, 32, False, False, 692123, delta_scale=1.0 / 2048)


@pytest.mark.parametrize("chunk", [128, 256])
def test_grad_fp32_long_slow_short_window(chunk):
    w = SLOW8K
    say(f"[grad trunc fp32 long slow] T={w.T} D={w.D} tbar={w.tbar} chunk={chunk}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, w.tbar, chunk)
    ref = _oracle_grad(inp, w, w.tbar, literal=True)
    _compare(g, ref, TOL_F32, False)
    full = _oracle_grad(inp, w, 0)
    ratio = np.linalg.norm(full["dx"]) / np.linalg.norm(ref["dx"])
    say(f"   |full dx| / |truncated dx| = {ratio:.2f}")
    assert ratio > 2.0


RAGGED = Workload("ragged", 2, 250, 50, 5, 50, 0, False, False, 692100, delta_scale=0.25)


@pytest.mark.parametrize("chunk,tbar", [(64, 0), (16, 0), (64, 37), (32, 100), (16, 249), (128, 250)])
def test_grad_ragged_shapes(chunk, tbar):
    """T not a multiple of the chunk, D not a multiple of 16, N < 16, batch 2, h0."""
    w = RAGGED
    say(f"[grad ragged] T={w.T} D={w.D} N={w.N} b={w.b} chunk={chunk} tbar={tbar}")
    inp = _inputs(w, h0=True)
    full = tbar == 0 or tbar >= w.T
    g = _gpu_grad(inp, w, tbar, chunk, want_dh0=full)
    _compare(g, _oracle_grad(inp, w, tbar, literal=True, want_dh0=full), TOL_F32, False, dh0=full)


GATED32 = Workload("gated32", 2, 300, 40, 16, 40, 0, True, False, 692101)


@pytest.mark.parametrize("chunk,tbar", [(64, 0), (128, 20), (256, 0)])
def test_grad_gate_softplus_fp32(chunk, tbar):
    w = GATED32
    say(f"[grad gate fp32] chunk={chunk} tbar={tbar}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, tbar, chunk)
    _compare(g, _oracle_grad(inp, w, tbar, literal=True), TOL_F32, True)
    y = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], z=inp["z"],
                                softplus=True, chunk=chunk)
    torch.cuda.synchronize()
    ry, _ = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")), z=to_np(inp["z"]),
                           delta_softplus=True)
    check("y", to_np(y), ry, TOL_F32)


BF16MID = Workload("bf16mid", 2, 1000, 256, 16, 128, 0, True, True, 692102)


@pytest.mark.parametrize("tbar", [0, 64])
def test_grad_bf16_gate(tbar):
    w = BF16MID
    say(f"[grad bf16 gate] T={w.T} D={w.D} tbar={tbar}")
    inp = _inputs(w)
    g = _gpu_grad(inp, w, tbar, 0)
    _compare(g, _oracle_grad(inp, w, tbar), TOL_SCAN_BF16, True)


def test_grad_deterministic():
    w = BF16MID
    say("[determinism] two identical calls")
    inp = _inputs(w)
    a = _gpu_grad(inp, w, 64, 0)
    b = _gpu_grad(inp, w, 64, 0)
    for k in a:
        assert torch.equal(a[k], b[k]), k


def _bf16(shape, seed, std=1.0):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return (torch.randn(*shape, generator=g, device="cuda") * std).to(torch.bfloat16)


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


# The GEMMs read exactly the bf16 values the oracle reads, so the only difference
# is fp32 accumulation (relative error of order sqrt(reduction) * 2^-24): a dropped
# reduction step or tile shows up far above this bound.
TOL_GEMM = 1e-5


# shapes: ragged rows and columns, reductions that are not a multiple of the
# 32-deep LDS stage (200, 24, 8, 1000, 700, 333), a reduction split over workgroups
# (8192 rows onto a 256 x 256 output; 5000 rows, whose last split is short and
# ends inside a stage; a 16-column dX over a 1536-long reduction, split too), and
# the smallest legal sizes
@pytest.mark.parametrize("M,K,N", [(1000, 136, 200), (100, 64, 24), (4096, 256, 384), (333, 8, 8),
                                   (700, 264, 1568), (8192, 256, 256), (5000, 264, 136), (4096, 16, 1536)])
def test_proj_grad_matches_oracle(M, K, N):
    say(f"[proj] M={M} K={K} N={N}")
    X = _bf16((M, K), 11)
    dZ = _bf16((M, N), 12)
    W = _bf16((K, N), 13, 0.1)
    dW, dX = ssm.ssm_proj_grad(X, dZ, W, want_dW=True, want_dX=True)
    torch.cuda.synchronize()
    kk, jj = np.meshgrid(np.arange(K), np.arange(N), indexing="ij")
    ref_dW = oracle.proj_dw(_bits(X), _bits(dZ), kk.ravel(), jj.ravel()).reshape(K, N)
    ref_dX = oracle.proj_dx(_bits(dZ), _bits(W), np.arange(M))
    say("   rel-L2 dW=%.2e dX=%.2e" % (check("dW", to_np(dW), ref_dW, TOL_GEMM),
                                         check("dX", to_np(dX), ref_dX, TOL_GEMM)))
    # accumulate flags add onto the existing contents
    dW2, dX2 = ssm.ssm_proj_grad(X, dZ, W, want_dW=True, want_dX=True, dW=dW.clone(), dX=dX.clone(),
                                 accum_dW=True, accum_dX=True)
    torch.cuda.synchronize()
    check("dW accum", to_np(dW2), 2 * ref_dW, TOL_GEMM)
    check("dX accum", to_np(dX2), 2 * ref_dX, TOL_GEMM)


LAYER_SMALL = Workload("layer_small", 2, 300, 64, 16, 32, 40, True, True, 692103)


@pytest.mark.parametrize("tbar", [0, 40])
def test_layer_grad_small(tbar):
    w = LAYER_SMALL
    say(f"[layer] b={w.b} T={w.T} D={w.D} d_model={w.d_model} tbar={tbar}")
    inp = _inputs(w)
    o = ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"],
                           inp["A_log"], inp["dy"], tbar=tbar, want_du=True, want_scan=True)
    torch.cuda.synchronize()
    h = {k: to_np(v) for k, v in inp.items()}
    ref = oracle.layer_grad(h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"],
                            W_in=h["W_in"], tbar=tbar, scan=oracle.adjoint_sum if tbar else None)
    M = w.b * w.T
    rep = {}
    for k in ("dx", "ddelta", "dB", "dC", "dz", "dA_log"):
        check(k, to_np(o[k]), ref[k], TOL_SCAN_BF16, rep)
    # downstream of the bf16 rounding of the GEMM operands
    check("dx_total", to_np(o["dx_total"]).reshape(M, -1), ref["dx_total"], TOL_BF16, rep)
    check("dW_x", to_np(o["dW_x"]), ref["dW_x"], TOL_BF16, rep)
    check("dW_in", to_np(o["dW_in"]), ref["dW_in"], TOL_BF16, rep)
    check("du", to_np(o["du"]).reshape(M, -1), ref["du"], TOL_BF16, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


@pytest.mark.parametrize("tbar", [0, 40])
def test_layer_grad_optional_outputs(tbar):
    """Parameter gradients do not depend on which optional outputs are asked for:
    none (only the bf16 copies of dDelta_pre and dz are written, no fp32 dx_total),
    some, or all; bit-identical across the three calls and equal to the oracle."""
    w = LAYER_SMALL
    say(f"[layer optional outputs] b={w.b} T={w.T} D={w.D} tbar={tbar}")
    inp = _inputs(w)
    args = (inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"], inp["A_log"],
            inp["dy"])
    full = ssm.ssm_layer_grad(*args, tbar=tbar, want_du=True, want_scan=True)
    none = ssm.ssm_layer_grad(*args, tbar=tbar)
    f32 = dict(dtype=torch.float32, device="cuda")
    some_out = {"ddelta": torch.empty(w.b, w.T, w.D, **f32), "dx_total": torch.empty(w.b, w.T, w.D, **f32)}
    some = ssm.ssm_layer_grad(*args, tbar=tbar, out=some_out)
    torch.cuda.synchronize()
    for k in ("dW_in", "dW_x", "dA_log"):
        assert torch.equal(full[k], none[k]), k
        assert torch.equal(full[k], some[k]), k
    assert torch.equal(full["ddelta"], some["ddelta"])
    assert torch.equal(full["dx_total"], some["dx_total"])
    h = {k: to_np(v) for k, v in inp.items()}
    ref = oracle.layer_grad(h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"],
                            W_in=h["W_in"], tbar=tbar, scan=oracle.adjoint_sum if tbar else None)
    rep = {}
    for k in ("dW_in", "dW_x", "dA_log"):
        check(k, to_np(none[k]), ref[k], TOL_BF16, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))
