"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times.  Where the fp64 oracle cannot run over the whole problem in
seconds, it checks sampled outputs it can compute exactly:

* per-channel outputs (dx, ddelta, dz, the dA_log row) of sampled channels, with
  the oracle run over the full sequence for those channels only (channels are
  independent except through dB and dC);
* all-channel outputs (dB, dC and every per-channel output) on sampled time
  windows, with the oracle run on a slice that starts PRE steps before the
  window from a zero state and ends POST steps after it.  The states' decay makes
  the slice exact to far below the tolerance: each step multiplies the carried
  state by a <= exp(-Delta) with Delta = softplus(N(0,1)), so PRE = POST = 512
  steps leave a factor of about exp(-400); the truncated adjoint only reaches
  tbar steps ahead, which POST covers;
* projection-gradient columns whose upstream factor is per-channel (dW_x
  columns of dDelta_pre, dW_in columns of dz), and dx_total / du rows on the
  sampled windows.
The whole-layer chain is compared on every entry at the "layer" workload."""
import numpy as np
import pytest
import torch

import oracle
import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import WORKLOADS, make_inputs

from gpu_helpers import TOL_BF16, TOL_SCAN_BF16, check, say, to_np

pytestmark = pytest.mark.gpu

PRE = 512
POST = 512


def _sel_channels(D, k=16, seed=5):
    rng = np.random.default_rng(seed)
    return np.sort(rng.choice(D, size=min(k, D), replace=False))


def _windows(T, tbar, k=2, width=256, seed=7):
    rng = np.random.default_rng(seed)
    starts = [0, T - width]  # the sequence edges
    for _ in range(k):
        starts.append(int(rng.integers(PRE, max(PRE + 1, T - width - POST - tbar))))
    return sorted(set(starts))


def _scan_fn(tbar, T):
    return oracle.bptt if tbar <= 0 or tbar >= T else oracle.trunc_tail


def _oracle_channels(inp, w, tbar, sel):
    """Per-channel oracle outputs for channels `sel` over the full sequence."""
    s = torch.as_tensor(sel, device="cuda")
    host = {k: to_np(inp[k].index_select(-1, s)) for k in ("x", "delta", "dy")}
    if "z" in inp:
        host["z"] = to_np(inp["z"].index_select(-1, s))
    A = to_np(inp["A_log"])[sel]
    B, C = to_np(inp["B"]), to_np(inp["C"])
    fn = _scan_fn(tbar, w.T)
    kw = dict(z=host.get("z"), delta_softplus=w.proj)
    if fn is oracle.bptt:
        return fn(host["x"], host["delta"], A, B, C, host["dy"], want_dh0=False, **kw)
    return fn(host["x"], host["delta"], A, B, C, host["dy"], tbar=tbar, **kw)


def _oracle_window(inp, w, tbar, t0, t1):
    """All-channel oracle on the slice [t0-PRE, t1+POST+tbar) (clipped), zero state
    at its start; returns outputs restricted to [t0, t1)."""
    post = POST + (tbar if 0 < tbar < w.T else 0)
    a, e = max(0, t0 - PRE), min(w.T, t1 + post)
    sl = slice(a, e)
    h = {k: to_np(inp[k][:, sl]) for k in ("x", "delta", "dy", "B", "C")}
    z = to_np(inp["z"][:, sl]) if "z" in inp else None
    A = to_np(inp["A_log"])
    fn = _scan_fn(tbar, w.T)
    kw = dict(z=z, delta_softplus=w.proj)
    if fn is oracle.bptt:
        r = fn(h["x"], h["delta"], A, h["B"], h["C"], h["dy"], want_dh0=False, **kw)
    else:
        r = fn(h["x"], h["delta"], A, h["B"], h["C"], h["dy"], tbar=tbar, **kw)
    cut = slice(t0 - a, t1 - a)
    return {k: (v[:, cut] if v is not None and v.ndim == 3 else v) for k, v in r.items()}


def _check_scan_sampled(g, inp, w, tbar, rep):
    sel = _sel_channels(w.D)
    say(f"   oracle on {len(sel)} sampled channels, full sequence")
    rc = _oracle_channels(inp, w, tbar, sel)
    s = torch.as_tensor(sel, device="cuda")
    for k in ("dx", "ddelta") + (("dz",) if w.proj else ()):
        check(f"{k}[ch]", to_np(g[k].index_select(-1, s)), rc[k], TOL_SCAN_BF16, rep)
    check("dA_log[ch]", to_np(g["dA_log"])[sel], rc["dA_log"], TOL_SCAN_BF16, rep)
    wins = _windows(w.T, tbar if 0 < tbar < w.T else 0)
    for t0 in wins:
        t1 = t0 + 256
        say(f"   oracle on window [{t0}, {t1}) over all channels")
        rw = _oracle_window(inp, w, tbar, t0, t1)
        for k in ("dB", "dC", "dx", "ddelta") + (("dz",) if w.proj else ()):
            check(f"{k}[t{t0}]", to_np(g[k][:, t0:t1]), rw[k], TOL_SCAN_BF16, rep)
    return sel, wins


@pytest.mark.parametrize("tbar", [0])
def test_layer_workload_every_entry(tbar):
    """b=2, T=4096, D=1536, d_model=768, N=16, full gradient with projections."""
    w = WORKLOADS["layer"]
    say(f"[layer full-size] {w}")
    inp = make_inputs(w, device="cuda")
    o = ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"],
                           inp["W_in"], inp["A_log"], inp["dy"], tbar=tbar, want_du=True, want_scan=True)
    torch.cuda.synchronize()
    h = {k: to_np(v) for k, v in inp.items()}
    ref = oracle.layer_grad(h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"],
                            W_in=h["W_in"])
    M = w.M
    rep = {}
    for k in ("dx", "ddelta", "dB", "dC", "dz", "dA_log"):
        check(k, to_np(o[k]), ref[k], TOL_SCAN_BF16, rep)
    # downstream of the bf16 rounding of the GEMM operands
    check("dx_total", to_np(o["dx_total"]).reshape(M, -1), ref["dx_total"], TOL_BF16, rep)
    for k in ("dW_x", "dW_in"):
        check(k, to_np(o[k]), ref[k], TOL_BF16, rep)
    check("du", to_np(o["du"]).reshape(M, -1), ref["du"], TOL_BF16, rep)
    del o
    # the call as the benchmark makes it (no per-token outputs requested)
    bare = ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"],
                              inp["W_in"], inp["A_log"], inp["dy"], tbar=tbar)
    torch.cuda.synchronize()
    check("dA_log(bench call)", to_np(bare["dA_log"]), ref["dA_log"], TOL_SCAN_BF16, rep)
    for k in ("dW_x", "dW_in"):
        check(f"{k}(bench call)", to_np(bare[k]), ref[k], TOL_BF16, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


def test_layer_workload_deterministic():
    """Two calls at the layer workload (channel splits of the scan, a split
    reduction in both dW GEMMs, the multi-slice dA_log sum) give bit-identical
    outputs: every reduction runs in a fixed order."""
    w = WORKLOADS["layer"]
    say(f"[layer determinism] {w}")
    inp = make_inputs(w, device="cuda")
    args = (inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"], inp["A_log"],
            inp["dy"])
    a = ssm.ssm_layer_grad(*args, want_du=True, want_scan=True)
    b = ssm.ssm_layer_grad(*args, want_du=True, want_scan=True)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k


def _layer_sampled(name, tbar, chunk=0):
    w = WORKLOADS[name]
    say(f"[layer sampled] {w} tbar={tbar} chunk={chunk}")
    inp = make_inputs(w, device="cuda")
    args = (inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"], inp["A_log"],
            inp["dy"])
    o = ssm.ssm_layer_grad(*args, tbar=tbar, chunk=chunk, want_du=True, want_scan=True)
    # the call as the benchmark makes it (no per-token outputs: the scan writes only
    # the GEMMs' bf16 operands and its fp32 dx addend) gives the same parameter
    # gradients bit for bit
    bare = ssm.ssm_layer_grad(*args, tbar=tbar, chunk=chunk)
    torch.cuda.synchronize()
    for k in ("dW_in", "dW_x", "dA_log"):
        assert torch.equal(o[k], bare[k]), k
    del bare
    rep = {}
    sel, wins = _check_scan_sampled(o, inp, w, tbar, rep)
    # dW_x columns of dDelta_pre for the sampled channels; dW_in columns of dz
    rc = _oracle_channels(inp, w, tbar, sel)
    M, D, N = w.M, w.D, w.N
    x = to_np(inp["x"]).reshape(M, D)
    u = to_np(inp["u"]).reshape(M, -1)
    check("dW_x[:,ch]", to_np(o["dW_x"])[:, sel], x.T @ rc["ddelta"].reshape(M, -1), TOL_BF16, rep)
    check("dW_in[:,D+ch]", to_np(o["dW_in"])[:, D + sel], u.T @ rc["dz"].reshape(M, -1), TOL_BF16, rep)
    del x, u
    Wx, Win = to_np(inp["W_x"]), to_np(inp["W_in"])
    for t0 in wins:
        t1 = t0 + 256
        rw = _oracle_window(inp, w, tbar, t0, t1)
        dzx = np.concatenate([rw["ddelta"], rw["dB"], rw["dC"]], axis=-1)
        dxt = rw["dx"] + dzx @ Wx.T
        check(f"dx_total[t{t0}]", to_np(o["dx_total"][:, t0:t1]), dxt, TOL_BF16, rep)
        du = np.concatenate([dxt, rw["dz"]], axis=-1) @ Win.T
        check(f"du[t{t0}]", to_np(o["du"][:, t0:t1]), du, TOL_BF16, rep)
    say("   rel-L2 max:", f"{max(rep.values()):.2e}", "over", len(rep), "checks")


@pytest.mark.parametrize("chunk", [0, 256])
def test_long_workload_truncated_sampled(chunk):
    """b=2, T=65536, D=1536, d_model=768, truncated tbar=2048 with projections;
    with the default chunk and with chunks of 256 steps."""
    _layer_sampled("long", WORKLOADS["long"].tbar, chunk)


@pytest.mark.parametrize("tbar", [0, 4096])
def test_slice_workload_sampled(tbar):
    """b=1, T=262144, D=4096, d_model=2048: full and truncated (tbar=4096)."""
    _layer_sampled("slice", tbar)


def test_vlong_workload_truncated_sampled():
    """b=1, T=1,048,576, D=3072, truncated tbar=8192, scan only."""
    w = WORKLOADS["vlong"]
    say(f"[vlong sampled] {w}")
    inp = make_inputs(w, device="cuda")
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], tbar=w.tbar)
    torch.cuda.synchronize()
    rep = {}
    _check_scan_sampled(g, inp, w, w.tbar, rep)
    say("   rel-L2 max:", f"{max(rep.values()):.2e}", "over", len(rep), "checks")


@pytest.mark.parametrize("tbar", [2048, 2000])
def test_long_slow_decay_truncated(tbar):
    """Slow decay (Delta / 2048) so that the window is visible: full shape on
    sampled channels, and every output on a reduced shape.  2000 is not a
    multiple of the 128-step chunk: every tile then also sweeps the adjoint carry
    back from the end of the chunk that holds t + tbar, up to 127 steps, and the
    last chunks' sweeps run past the end of the sequence."""
    w = WORKLOADS["long_slow"].with_(tbar=tbar)
    say(f"[long_slow] {w}")
    inp = make_inputs(w, device="cuda")
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], tbar=w.tbar)
    torch.cuda.synchronize()
    rep = {}
    sel = _sel_channels(w.D)
    rc = _oracle_channels(inp, w, w.tbar, sel)
    s = torch.as_tensor(sel, device="cuda")
    for k in ("dx", "ddelta"):
        check(f"{k}[ch]", to_np(g[k].index_select(-1, s)), rc[k], TOL_SCAN_BF16, rep)
    check("dA_log[ch]", to_np(g["dA_log"])[sel], rc["dA_log"], TOL_SCAN_BF16, rep)
    full = _oracle_channels(inp, w, 0, sel)
    assert np.linalg.norm(rc["dx"] - full["dx"]) > 1e-2 * np.linalg.norm(full["dx"])  # window visible
    del g, inp
    small = w.with_(name="long_slow_small", b=1, T=8192, D=512)
    inp = make_inputs(small, device="cuda")
    g = ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], tbar=w.tbar)
    torch.cuda.synchronize()
    h = {k: to_np(v) for k, v in inp.items()}
    ref = oracle.trunc_tail(h["x"], h["delta"], h["A_log"], h["B"], h["C"], h["dy"], tbar=w.tbar)
    for k in ("dx", "ddelta", "dA_log", "dB", "dC"):
        check(k, to_np(g[k]), ref[k], TOL_SCAN_BF16, rep)
    say("   rel-L2 max:", f"{max(rep.values()):.2e}", "over", len(rep), "checks")


def test_proj_grad_slice_shapes_sampled():
    """The projection GEMMs at the slice workload's shapes (M = 262,144 rows):
    sampled dW entries and dX rows against the oracle's plain loops."""
    M, D, N, dm = 262144, 4096, 16, 2048
    say(f"[proj sampled] M={M} K={D} N={D + 2 * N}")
    g = torch.Generator(device="cuda")
    g.manual_seed(4242)
    X = torch.randn(M, D, generator=g, device="cuda").to(torch.bfloat16)
    dZ = torch.randn(M, D + 2 * N, generator=g, device="cuda").to(torch.bfloat16)
    W = (torch.randn(D, D + 2 * N, generator=g, device="cuda") / 64).to(torch.bfloat16)
    dW, dX = ssm.ssm_proj_grad(X, dZ, W, want_dW=True, want_dX=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    kk = rng.integers(0, D, 4096)
    jj = rng.integers(0, D + 2 * N, 4096)
    rows = np.sort(rng.choice(M, 256, replace=False))
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    Xb, Zb, Wb = bits(X), bits(dZ), bits(W)
    rep = {}
    # exact bf16 inputs on both sides: only fp32 accumulation differs, of relative
    # order 2^-24 sqrt(n) for a reduction of n = 262,144 terms (about 3e-5 at worst)
    tol = 1e-4
    check("dW[sampled]", to_np(dW)[kk, jj], oracle.proj_dw(Xb, Zb, kk, jj), tol, rep)
    check("dX[rows]", to_np(dX[torch.as_tensor(rows, device="cuda")]), oracle.proj_dx(Zb, Wb, rows), tol, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))

def test_proj_grad_wide_dw_tiles_sampled():
    """dW with an output of 2040 x 8184 over a 4096-long reduction: about 256
    output tiles, so the planner takes the 256-column tiles of the dW product; the
    last row block and column block are ragged.  Sampled entries, including the
    output's last row and column, against the oracle's plain loops."""
    M, K, N = 4096, 2040, 8184
    say(f"[proj wide dW] M={M} K={K} N={N}")
    g = torch.Generator(device="cuda")
    g.manual_seed(4243)
    X = torch.randn(M, K, generator=g, device="cuda").to(torch.bfloat16)
    dZ = torch.randn(M, N, generator=g, device="cuda").to(torch.bfloat16)
    dW, _ = ssm.ssm_proj_grad(X, dZ, None, want_dW=True, want_dX=False)
    torch.cuda.synchronize()
    rng = np.random.default_rng(4)
    kk = np.concatenate([rng.integers(0, K, 4096), [K - 1, K - 1, 0]])
    jj = np.concatenate([rng.integers(0, N, 4096), [N - 1, 0, N - 1]])
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    rep = {}
    check("dW[sampled]", to_np(dW)[kk, jj], oracle.proj_dw(bits(X), bits(dZ), kk, jj), 1e-5, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


def test_proj_grad_wide_dx_tiles_sampled():
    """dX = dZ W^T with an output of 4000 x 8184 over a 2040-long reduction (not a
    multiple of the 32-step stage): 512 output tiles of 256 x 256, so the planner
    takes the four-wave kernel for the plain dX epilogue; the last row block and
    column block are ragged.  Sampled rows, the last one included, against the
    oracle's plain loops, written and accumulated."""
    M, K, N = 4000, 8184, 2040
    say(f"[proj wide dX] M={M} K={K} N={N}")
    g = torch.Generator(device="cuda")
    g.manual_seed(4244)
    dZ = torch.randn(M, N, generator=g, device="cuda").to(torch.bfloat16)
    W = (torch.randn(K, N, generator=g, device="cuda") / 32).to(torch.bfloat16)
    _, dX = ssm.ssm_proj_grad(None, dZ, W, want_dW=False, want_dX=True)
    _, dX2 = ssm.ssm_proj_grad(None, dZ, W, want_dW=False, want_dX=True, dX=dX.clone(), accum_dX=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(5)
    rows = np.sort(np.concatenate([rng.choice(M - 1, 128, replace=False), [M - 1]]))
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = oracle.proj_dx(bits(dZ), bits(W), rows)
    idx = torch.as_tensor(rows, device="cuda")
    rep = {}
    check("dX[rows]", to_np(dX[idx]), ref, 1e-5, rep)
    check("dX accum[rows]", to_np(dX2[idx]), 2 * ref, 1e-5, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))


@pytest.mark.parametrize("form", ["dW", "dX"])
def test_proj_grad_every_main_loop_residue(form):
    """The four-wave kernel's main loop runs four passes over its five-stage LDS
    ring per iteration (20 reduction steps of 32), then single passes, then the
    last stages one by one.  Reductions of 32 n + 7 for n = 24..43 put every
    residue of that schedule (and a ragged last stage) into one 256 x 256-tile
    launch: dW of 2048 x 8192 (256 output tiles) and plain dX of 4096 x 4096 (256
    output tiles, so both take 256-column tiles and no split; dX's reduction must
    be a multiple of 8, so there it is 32 n + 8).  Sampled entries,
    each output's corners included, against the oracle's plain loops."""
    g = torch.Generator(device="cuda")
    g.manual_seed(4245 if form == "dW" else 4246)
    rng = np.random.default_rng(6)
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    rep = {}
    for n in range(24, 44):
        red = 32 * n + (7 if form == "dW" else 8)
        if form == "dW":
            K, N = 2048, 8192
            say(f"[proj residue dW] M={red} K={K} N={N}")
            X = torch.randn(red, K, generator=g, device="cuda").to(torch.bfloat16)
            dZ = torch.randn(red, N, generator=g, device="cuda").to(torch.bfloat16)
            dW, _ = ssm.ssm_proj_grad(X, dZ, None, want_dW=True, want_dX=False)
            torch.cuda.synchronize()
            kk = np.concatenate([rng.integers(0, K, 256), [0, 0, K - 1, K - 1]])
            jj = np.concatenate([rng.integers(0, N, 256), [0, N - 1, 0, N - 1]])
            check(f"dW[n={n}]", to_np(dW)[kk, jj], oracle.proj_dw(bits(X), bits(dZ), kk, jj), 1e-5, rep)
        else:
            M, K = 4096, 4096
            say(f"[proj residue dX] M={M} K={K} N={red}")
            dZ = torch.randn(M, red, generator=g, device="cuda").to(torch.bfloat16)
            W = (torch.randn(K, red, generator=g, device="cuda") / 32).to(torch.bfloat16)
            _, dX = ssm.ssm_proj_grad(None, dZ, W, want_dW=False, want_dX=True)
            torch.cuda.synchronize()
            rows = np.sort(np.concatenate([rng.choice(M - 1, 6, replace=False), [0, M - 1]]))
            ref = oracle.proj_dx(bits(dZ), bits(W), rows)
            check(f"dX[n={n}]", to_np(dX[torch.as_tensor(rows, device="cuda")]), ref, 1e-5, rep)
    say("   worst rel-L2: %.2e" % max(rep.values()))


def test_layer_workload_weight_grads_exact_sampled():
    """The layer's weight gradients against the products of the bf16 operands the
    layer hands over, at the layer workload (one launch over the M = 8192 rows).
    With d_model < D the input projection's gradient is reassociated:
    dW_x = x^T dZx, dW_in[:, D:] = u^T dz and dW_in[:, :D] = u^T dx + (u^T dZx)
    W_x^T, with dZx = bf16([dDelta_pre | dB | dC]), dx and dz in bf16 (round to
    nearest even).  The layer's own fp32 outputs, rounded to bf16, rebuild those
    operands exactly, so sampled entries (with every row's and column's last
    one) are checked against the oracle's plain loops: the pure products at the
    GEMM tolerance, the reassociated block (whose d_model x (D+2N) factor enters
    the second product as two bf16 parts, about 2^-17 relative) at 1e-4."""
    w = WORKLOADS["layer"]
    say(f"[layer weight gradients] {w}")
    inp = make_inputs(w, device="cuda")
    o = ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"],
                           inp["W_in"], inp["A_log"], inp["dy"], want_scan=True)
    torch.cuda.synchronize()
    M, D, dm = w.M, w.D, w.d_model
    assert dm < D  # the reassociated form
    bits = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    dzx = bits(torch.cat([o["ddelta"], o["dB"], o["dC"]], dim=-1).reshape(M, -1).to(torch.bfloat16))
    dx16 = bits(o["dx"].reshape(M, D).to(torch.bfloat16))
    dz16 = bits(o["dz"].reshape(M, D).to(torch.bfloat16))
    xb, ub = bits(inp["x"].reshape(M, D)), bits(inp["u"].reshape(M, dm))
    rng = np.random.default_rng(11)
    rep = {}
    nx = dzx.shape[1]
    kk = np.concatenate([rng.integers(0, D, 2048), [D - 1, D - 1, 0]])
    jj = np.concatenate([rng.integers(0, nx, 2048), [nx - 1, 0, nx - 1]])
    check("dW_x[sampled]", to_np(o["dW_x"])[kk, jj], oracle.proj_dw(xb, dzx, kk, jj), 1e-5, rep)
    kk = np.concatenate([rng.integers(0, dm, 2048), [dm - 1, dm - 1, 0]])
    jj = np.concatenate([rng.integers(0, D, 2048), [D - 1, 0, D - 1]])
    check("dW_in[:,D:][sampled]", to_np(o["dW_in"])[kk, D + jj], oracle.proj_dw(ub, dz16, kk, jj), 1e-5, rep)
    # the reassociated block on 24 sampled rows of dW_in (all of each row's
    # u^T dZx, then its product with W_x^T) and 64 sampled columns
    rows = np.concatenate([np.sort(rng.choice(dm, 23, replace=False)), [dm - 1]])
    cols = np.concatenate([np.sort(rng.choice(D, 63, replace=False)), [D - 1]])
    rr, cc = np.meshgrid(rows, np.arange(nx), indexing="ij")
    gz = oracle.proj_dw(ub, dzx, rr.ravel(), cc.ravel()).reshape(len(rows), nx)
    wx = to_np(inp["W_x"])[cols]  # [cols][nx]
    r2, c2 = np.meshgrid(rows, cols, indexing="ij")
    ref = oracle.proj_dw(ub, dx16, r2.ravel(), c2.ravel()).reshape(len(rows), len(cols)) + gz @ wx.T
    check("dW_in[:,:D][sampled]", to_np(o["dW_in"])[np.ix_(rows, cols)], ref, 1e-4, rep)
    say("   rel-L2:", " ".join(f"{k}={v:.2e}" for k, v in rep.items()))
