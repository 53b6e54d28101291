"""GPU parity against the fp64 oracle on the degenerate shapes of the scan: one
step, one channel, one state, a sequence shorter than one chunk or one step
past it, a window of one step, batch entries of a few steps.  Every entry point
of the scan (forward, fused gradient, explicit pairs) on each shape; the
smallest projection GEMM (one row)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import Workload, make_inputs

from gpu_helpers import TOL_BF16, TOL_F32, check, say, to_np

pytestmark = pytest.mark.gpu

# (workload, chunk, tbar); tbar 0 is the full gradient (with dL/dh0)
CASES = [
    (Workload("one_step", 1, 1, 1, 1, 1, 0, False, False, 692700), 16, 0),
    (Workload("one_step_n16", 1, 1, 1, 16, 1, 0, False, False, 692701), 256, 0),
    (Workload("two_steps", 1, 2, 1, 1, 1, 0, False, False, 692702), 16, 1),
    (Workload("chunk_plus_one", 1, 17, 3, 1, 3, 0, False, False, 692703), 16, 0),
    (Workload("chunk_plus_one_w", 1, 17, 3, 1, 3, 0, False, False, 692703), 16, 16),
    (Workload("short_batch", 3, 5, 2, 16, 2, 0, False, False, 692704), 256, 2),
    (Workload("state_one", 2, 100, 17, 1, 17, 0, False, False, 692705, delta_scale=0.25), 16, 7),
    (Workload("gate_bf16_one_channel", 1, 3, 1, 2, 1, 0, True, True, 692706), 16, 0),
    (Workload("gate_bf16_short", 2, 9, 8, 3, 8, 0, True, True, 692707), 64, 4),
]
IDS = [f"{w.name}-c{c}-tbar{t}" for w, c, t in CASES]


def _inputs(w, h0):
    inp = make_inputs(w, device="cuda", h0=h0)
    torch.cuda.synchronize()
    return inp


def _oracle(inp, w, tbar, want_dh0, a_scalar=False):
    args = [to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C", "dy")]
    kw = dict(h0=to_np(inp["h0"]) if "h0" in inp else None, z=to_np(inp["z"]) if "z" in inp else None,
              delta_softplus=w.proj, a_scalar=a_scalar)
    if tbar <= 0 or tbar >= w.T:
        return oracle.bptt(*args, want_dh0=want_dh0, **kw)
    return oracle.adjoint_sum(*args, tbar=tbar, want_dh0=False, **kw)


def _compare(g, ref, tol, gate, dh0):
    rep = {}
    for k in ("dx", "ddelta", "dA_log", "dB", "dC") + (("dz",) if gate else ()) + (("dh0",) if dh0 else ()):
        check(k, to_np(g[k]), ref[k], tol, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


@pytest.mark.parametrize("w,chunk,tbar", CASES, ids=IDS)
def test_degenerate_forward(w, chunk, tbar):
    say(f"[degenerate forward] b={w.b} T={w.T} D={w.D} N={w.N} chunk={chunk} gate={w.proj} bf16={w.bf16}")
    inp = _inputs(w, h0=True)
    y, hl = ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], h0=inp["h0"],
                                    z=inp.get("z"), softplus=w.proj, chunk=chunk, want_h_last=True)
    torch.cuda.synchronize()
    ry, rh = oracle.forward(*(to_np(inp[k]) for k in ("x", "delta", "A_log", "B", "C")), h0=to_np(inp["h0"]),
                            z=to_np(inp["z"]) if "z" in inp else None, delta_softplus=w.proj)
    check("y", to_np(y), ry, TOL_BF16 if w.bf16 else TOL_F32)
    check("h_last", to_np(hl), rh, TOL_F32)


@pytest.mark.parametrize("pairs", [False, True], ids=["scan", "pairs"])
@pytest.mark.parametrize("w,chunk,tbar", CASES, ids=IDS)
def test_degenerate_grad(w, chunk, tbar, pairs):
    say(f"[degenerate grad] {'pairs' if pairs else 'scan'} b={w.b} T={w.T} D={w.D} N={w.N} "
        f"chunk={chunk} tbar={tbar} gate={w.proj} bf16={w.bf16}")
    full = tbar == 0
    inp = _inputs(w, h0=full)
    fn = ssm.ssm_adjoint_grad_pairs if pairs else ssm.ssm_adjoint_grad
    g = fn(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], h0=inp.get("h0"), z=inp.get("z"),
           softplus=w.proj, tbar=tbar, chunk=chunk, want_dh0=full)
    torch.cuda.synchronize()
    _compare(g, _oracle(inp, w, tbar, full), TOL_F32, w.proj, full)


@pytest.mark.parametrize("w,chunk,tbar", CASES[:6], ids=IDS[:6])
def test_degenerate_grad_scalar_decay(w, chunk, tbar):
    say(f"[degenerate grad scalar A] b={w.b} T={w.T} D={w.D} N={w.N} chunk={chunk} tbar={tbar}")
    full = tbar == 0
    inp = _inputs(w, h0=full)
    inp["A_log"] = inp["A_log"][:, 0].contiguous()
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], h0=inp.get("h0"),
                             softplus=w.proj, tbar=tbar, chunk=chunk, want_dh0=full)
    torch.cuda.synchronize()
    _compare(g, _oracle(inp, w, tbar, full, a_scalar=True), TOL_F32, False, full)


def test_degenerate_proj_one_row():
    """One row of activations: dW is the outer product x^T dz, dX one row."""
    say("[degenerate proj] M=1 K=8 N=8")
    g = torch.Generator().manual_seed(692708)
    X = torch.randn(1, 8, generator=g).to(torch.bfloat16).cuda()
    dZ = torch.randn(1, 8, generator=g).to(torch.bfloat16).cuda()
    W = (0.1 * torch.randn(8, 8, generator=g)).to(torch.bfloat16).cuda()
    dW, dX = ssm.ssm_proj_grad(X, dZ, W, want_dW=True, want_dX=True)
    torch.cuda.synchronize()
    xb, zb, wb = (t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16) for t in (X, dZ, W))
    kk, jj = np.meshgrid(np.arange(8), np.arange(8), indexing="ij")
    check("dW", to_np(dW), oracle.proj_dw(xb, zb, kk.ravel(), jj.ravel()).reshape(8, 8), 1e-5)
    check("dX", to_np(dX), oracle.proj_dx(zb, wb, np.arange(1)), 1e-5)


# The language head on degenerate shapes: one token, the smallest vocabulary and
# width (8), a ragged 257-row block, every target ignored.
HEAD_CASES = [(1, 8, 8, True), (257, 16, 8, False), (3, 8, 16, True)]


@pytest.mark.parametrize("M,P,V,norm", HEAD_CASES, ids=[f"M{m}-P{p}-V{v}-norm{n}" for m, p, v, n in HEAD_CASES])
def test_degenerate_head(M, P, V, norm):
    from oracle.head import head_loss_grad
    from paper_2501_00692_amd.synth import make_head_inputs
    say(f"[degenerate head] M={M} P={P} V={V} norm={norm}")
    inp = make_head_inputs(M, P, V, 692710, device="cuda")
    inp["targets"][0] = V - 1
    o = ssm.ssm_lm_head_grad(inp["y"], inp["omega"], inp["targets"], norm=norm)
    torch.cuda.synchronize()
    ref = head_loss_grad(to_np(inp["y"]), to_np(inp["omega"]), inp["targets"].cpu().numpy(), norm=norm,
                         round_bf16=True)
    rep = {}
    for k in ("loss", "dy", "domega"):
        check(k, to_np(o[k]), ref[k], 2e-4, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


def test_degenerate_head_all_targets_ignored():
    """No token has a loss: every loss, dy and dOmega is exactly zero."""
    from paper_2501_00692_amd.synth import make_head_inputs
    inp = make_head_inputs(64, 32, 64, 692711, device="cuda")
    inp["targets"].fill_(-1)
    o = ssm.ssm_lm_head_grad(inp["y"], inp["omega"], inp["targets"])
    torch.cuda.synchronize()
    for k in ("loss", "dy", "domega"):
        assert float(o[k].abs().max()) == 0.0, k


# The unstructured SSM on degenerate shapes: (b, T, P, chunk, tbar); tbar 0 is the
# full gradient (with dh0): one step, one step past a chunk, a window of one step,
# a window one step shorter than the sequence, the smallest channel count (16).
UN_CASES = [(1, 1, 16, 16, 0), (2, 17, 16, 16, 0), (2, 17, 16, 16, 16), (1, 33, 16, 16, 1), (3, 5, 32, 16, 4),
            (1, 300, 16, 256, 299)]


@pytest.mark.parametrize("b,T,P,chunk,tbar", UN_CASES, ids=[f"b{b}-T{t}-P{p}-c{c}-tbar{tb}" for b, t, p, c, tb in UN_CASES])
def test_degenerate_unstructured(b, T, P, chunk, tbar):
    from oracle.unstructured import un_adjoint_sum, un_bptt
    from paper_2501_00692_amd.synth import make_unstructured_inputs
    say(f"[degenerate unstructured] b={b} T={T} P={P} chunk={chunk} tbar={tbar}")
    inp = make_unstructured_inputs(b, T, P, 692712, device="cuda", h0=True)
    full = tbar == 0
    o = ssm.ssm_unstructured_grad(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], h0=inp["h0"], tbar=tbar,
                                  chunk=chunk, want_dh0=full)
    torch.cuda.synchronize()
    h = {k: to_np(v) for k, v in inp.items()}
    if full:
        ref = un_bptt(h["A"], h["B"], h["C"], h["x"], h["dy"], h["h0"])
    else:
        ref = un_adjoint_sum(h["A"], h["B"], h["C"], h["x"], h["dy"], tbar=tbar, h0=h["h0"])
    rep = {}
    for k in ("dA", "dB", "dC", "dx") + (("dh0",) if full else ()):
        check(k, to_np(o[k]), ref[k], TOL_F32, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))
