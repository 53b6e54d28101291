"""Benchmark of the per-layer adjoint gradient on one MI355X.

One step = the layer's two gradients over one batch of the "slice" workload
(a 1.27B-class layer slice: b=1, T=262,144, d_model=2,048, D=4,096, N=16, with
input projections and the SiLU gate; bf16 activations, fp32 accumulation): one
``ssm_layer_grad`` call in full mode (Prop. 2) and one in truncated mode
(Eq. "capped", window 4,096).  Together they run every step of the hot path:
the decay in registers, the chunked forward recomputation with its two-level
carry, the reverse adjoint (full) and the windowed adjoint (truncated) with the
vjp epilogue, the activation vjps into projection space and the projection-
gradient GEMMs.  Inputs are seeded synthetic tensors already resident in HBM.
``value`` is tokens of gradient computed per second, 2 b T per step (the two
modes' rates combined harmonically); each mode's own rate is in ``modes``.
Per-kernel times come from hipEvents recorded around every launch on its
stream during the timed steps.  The other workloads are reported under "extra".

Prints ONE JSON line.  ``--gpus`` above 1 is not supported (one GPU).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 MFMA
# MI355X fp32 vector arithmetic: 256 CUs x 4 SIMDs x 32 lanes per cycle x 2 (FMA)
# x 2.4 GHz = 157.3 TFLOP/s (reported beside the HBM fraction of the scan kernels)
FP32_VECTOR_PEAK_TFS = 157.3
HEADLINE = "slice"


def scan_flops_per_state_step(trunc):
    """fp32 operations per (state, token) of the fused gradient (an FMA counts 2,
    exp counts 1): forward recompute a = exp(Delta c) (2), h = a h + B x (3),
    y += C h (2), dC contribution and channel sum (2); reverse adjoint mu = g C +
    a mu (3), dx += mu B (2), s = mu (a h) (2), ddelta += s w (2), dA += s Delta
    (2), dB contribution and sum (2) -> 22.  The truncated form adds the window
    product P = exp(W c) (2) and the step leaving the window, - P g' C' (3)."""
    return 22 + (5 if trunc else 0)


def scan_bytes_per_token(D, N, s, gate):
    """Compulsory HBM bytes per token of the scan gradient at the C ABI's dtypes:
    every input read once and every output written once (outputs fp32).  With the
    gate: reads x, Delta_pre, dy, z, writes dx, dDelta_pre, dz; without: reads x,
    Delta, dy, writes dx, dDelta; both read B, C and write dB, dC."""
    per_ch = 4 * s + 12 if gate else 3 * s + 8
    return D * per_ch + N * (2 * s + 8)


def layer_scan_bytes_per_token(D, N, s, dm):
    """Compulsory bytes per token of the scan kernel inside the whole-layer call
    (reads x, Delta_pre, dy, z, B, C), which writes the projection GEMMs' bf16
    operands dDelta_pre, dz, dB, dC (plus dB, dC in fp32) and dx: in bf16 when
    d_model < D (the reassociated input-projection gradient reads it as an
    operand), else in fp32 (the addend of dx_total)."""
    return D * (4 * s + (2 if dm < D else 4) + 2 + 2) + N * (2 * s + 8 + 4)


def layer_gemm_flops(M, D, N, dm):
    """Flops per launch of the layer's projection products, by timing name.  With
    d_model < D the input projection's gradient is reassociated: one weight-
    gradient launch computes dW_x = x^T dZx and G = u^T [dx | dz | dZx], and two
    small launches add (u^T dZx) W_x^T (its bf16 hi and lo parts) into dW_in.
    Otherwise: dx_total = dx + dZx W_x^T (the dX launch), then dW_x and dW_in =
    u^T [dx_total | dz] in one launch."""
    nx = D + 2 * N
    if dm < D:
        return {"gemm_dw": 2 * M * D * nx + 2 * M * dm * (3 * D + 2 * N), "gemm_dwin_fix": 2 * dm * nx * D}
    return {"gemm_dw": 2 * M * D * nx + 2 * M * dm * 2 * D, "gemm_dx": 2 * M * nx * D}


def _timed(fn, steps, warmup, torch):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def _timed_kernels(fn, steps, warmup, ssm, torch):
    """Time `steps` calls of `fn` (ms per call) with every library kernel launch
    bracketed by hipEvents on its own stream; returns the per-call time and the
    per-kernel launches and durations of the same calls."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ssm.timing_summary()  # clear
    ssm.timing_enable(True)
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    ssm.timing_enable(False)
    ms = start.elapsed_time(stop) / steps
    kt = {}
    for name, (n, tot) in ssm.timing_summary().items():
        kt[name] = {"launches": n, "total_ms": tot, "avg_ms": tot / n, "launches_per_step": n / steps,
                    "ms_per_step": tot / steps}
    return ms, kt


def _timed_each(fn, reps, warmup, torch, flush=None):
    """Median, p10 and p90 of per-rep times (ms), each rep bracketed by its own
    events; with `flush`, a 512 MB write runs before every rep (outside the
    events) so that the rep starts with cold L2 and MALL caches."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    times = []
    for _ in range(reps):
        if flush is not None:
            flush()
        start = torch.cuda.Event(enable_timing=True)
        stop = torch.cuda.Event(enable_timing=True)
        start.record()
        fn()
        stop.record()
        stop.synchronize()
        times.append(start.elapsed_time(stop))
    times.sort()
    pick = lambda q: times[min(len(times) - 1, int(q * (len(times) - 1) + 0.5))]
    return {"median": pick(0.5), "p10": pick(0.1), "p90": pick(0.9), "reps": reps}


def layer_step(w, inp, ssm, torch, tbar=0, b_delta=False, chunk=0, ws=None):
    """One whole-layer gradient; ``inp["A_log"]`` of shape [D] selects the scalar-decay variant."""
    D, N, dm = w.D, w.N, w.d_model
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dW_in": torch.empty(dm, 2 * D, **f32), "dW_x": torch.empty(D, D + 2 * N, **f32),
           "dA_log": torch.empty(*inp["A_log"].shape, **f32)}
    if ws is None:
        desc = ssm.make_desc(inp["x"], N, True, True, chunk, inp["A_log"].dim() == 1, b_delta)
        ws = torch.empty(ssm.layer_workspace_size(desc, tbar, dm), dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"],
                           inp["W_in"], inp["A_log"], inp["dy"], tbar=tbar, chunk=chunk, out=out, workspace=ws,
                           b_delta=b_delta)
    return step


def vjp_pairs(T, tbar):
    """(t, i) adjoint-state pairs of one sequence: T(T+1)/2 in full mode, else
    tbar T - tbar (tbar - 1) / 2 (the paper's VJP counts, Sec. 4.3)."""
    if tbar <= 0 or tbar >= T:
        return T * (T + 1) // 2
    return tbar * T - tbar * (tbar - 1) // 2


def scan_step(w, inp, ssm, torch, tbar=0, b_delta=False, pairs=False, chunk=0):
    """One scan gradient; ``inp["A_log"]`` of shape [D] selects the scalar-decay variant;
    ``pairs`` evaluates it by the explicit pair formulation instead of the adjoint scan."""
    b, T, D, N = w.b, w.T, w.D, w.N
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dx": torch.empty(b, T, D, **f32), "ddelta": torch.empty(b, T, D, **f32),
           "dA_log": torch.empty(*inp["A_log"].shape, **f32), "dB": torch.empty(b, T, N, **f32),
           "dC": torch.empty(b, T, N, **f32)}
    z = inp.get("z") if w.proj else None
    if z is not None:
        out["dz"] = torch.empty(b, T, D, **f32)
    desc = ssm.make_desc(inp["x"], N, w.proj, z is not None, chunk, inp["A_log"].dim() == 1, b_delta)
    ws = torch.empty(ssm.grad_workspace_size(desc, tbar, pairs), dtype=torch.uint8, device="cuda")
    fn = ssm.ssm_adjoint_grad_pairs if pairs else ssm.ssm_adjoint_grad

    def step():
        fn(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], z=z, softplus=w.proj, tbar=tbar,
           chunk=chunk, out=out, workspace=ws, b_delta=b_delta)
    return step


def un_bytes_per_token(N, P):
    """Compulsory HBM bytes per token (sequence step) of the unstructured SSM's
    gradient call, fp32: reads A_t, B_t, C_t, x_t, dy_t; writes dA_t, dB_t, dC_t, dx_t."""
    return 4 * (2 * N * N + 4 * N * P + 3 * P)


def un_step(b, T, P, tbar, ssm, torch, chunk=0):
    """One gradient call of the unstructured SSM (Table 1, 16 states) on seeded inputs."""
    from paper_2501_00692_amd.synth import make_unstructured_inputs
    inp = make_unstructured_inputs(b, T, P, 692210, device="cuda")
    out = {"dA": torch.empty_like(inp["A"]), "dB": torch.empty_like(inp["B"]), "dC": torch.empty_like(inp["C"]),
           "dx": torch.empty_like(inp["x"])}
    desc = ssm.SsmDesc(b, T, P, 16, chunk, ssm.SSM_F32, 0)
    import ctypes
    n = ctypes.c_size_t()
    mode = ssm.SSM_TRUNCATED if tbar > 0 else ssm.SSM_FULL
    ssm.load_library().ssm_unstructured_grad_workspace_size(ctypes.byref(desc), mode, int(tbar), ctypes.byref(n))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_unstructured_grad(inp["A"], inp["B"], inp["C"], inp["x"], inp["dy"], tbar=tbar, chunk=chunk, out=out,
                                  workspace=ws)
    return step


def forward_bytes_per_token(D, N, s, gate):
    """Compulsory HBM bytes per token of the forward: reads x, Delta (and z), B, C;
    writes y (input dtype)."""
    return D * (3 * s + (s if gate else 0)) + 2 * N * s


def forward_step(w, inp, ssm, torch):
    """One forward (y only) of the scan with the workload's options."""
    z = inp.get("z") if w.proj else None
    desc = ssm.make_desc(inp["x"], w.N, w.proj, z is not None, 0, False, False)
    ws = torch.empty(ssm.forward_workspace_size(desc), dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_adjoint_forward(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], z=z, softplus=w.proj,
                                workspace=ws)
    return step


def stack_step(K, b, T, D, N, ssm, torch, exact):
    """One whole K-layer step: the forward of every layer, then every layer's
    parameter gradient (Prop. 3 or backpropagation)."""
    from paper_2501_00692_amd.synth import make_stack_inputs
    inp = make_stack_inputs(K, b, T, D, N, 692500, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dW_in": [torch.empty(D, 2 * D, **f32) for _ in range(K)],
           "dW_x": [torch.empty(D, D + 2 * N, **f32) for _ in range(K)],
           "dA_log": [torch.empty(D, N, **f32) for _ in range(K)]}
    desc = ssm.SsmDesc(b, T, D, N, 0, ssm.SSM_BF16, 0)
    grad = ssm.SSM_STACK_EXACT if exact else ssm.SSM_STACK_ADJOINT
    ws = torch.empty(ssm.stack_workspace_size(desc, K, grad), dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_stack_grad(inp["y0"], inp["W_in"], inp["W_x"], inp["A_log"], inp["gK"], N, exact=exact, out=out,
                           workspace=ws)
    return step, inp, out


def measured_traffic(kern, workload):
    """HBM-side bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"traffic_{kern}_{workload}.txt")
    if not os.path.exists(path):
        return None
    rec = {}
    for line in open(path):
        if line.strip() and not line.startswith("#"):
            k, v = line.split(None, 1)
            rec[k] = v.strip()
    src = os.path.join(ROOT, "paper_2501_00692_amd", "csrc", rec.get("source", ""))
    if not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec.get("source_sha256"):
        return None
    return int(rec["bytes_per_launch"])


# The gradient modes each workload is defined with: the timed step runs one call
# of each on the same batch.
MODES = {"small": ("full", "truncated"), "layer": ("full",), "long": ("truncated",),
         "slice": ("full", "truncated"), "vlong": ("truncated",)}


def workload_tag(w, chunk=0):
    return f"{w.name}-b{w.b}-T{w.T}-D{w.D}" + (f"-L{chunk}" if chunk else "")


def workload_text(w, modes):
    kind = ("one selective diagonal SSM layer with input projections and SiLU gate" if w.proj
            else "one selective diagonal SSM scan (per-layer gradients only, no projections)")
    dm = f", d_model={w.d_model}" if w.proj else ""
    call = "ssm_layer_grad" if w.proj else "ssm_adjoint_grad"
    what = " and one ".join(f"truncated (tbar={w.tbar})" if m == "truncated" else "full" for m in modes)
    return (f"{w.name}: {kind}, b={w.b}, T={w.T}{dm}, D={w.D}, N={w.N}; each step one {what} {call} call "
            f"on the same batch")


def rooflines(kt, w, layer, tag=None):
    """Roofline entries of the kernels with an algorithmic work figure: the scan
    gradient kernels against HBM (compulsory bytes per launch / average launch
    duration), the projection GEMMs against bf16 MFMA (flops per launch / average
    launch duration).  One launch of each per gradient call."""
    s = 2 if w.bf16 else 4
    out = {}
    for kern in ("grad_fused", "grad_fused_trunc"):
        if kern not in kt:
            continue
        avg = kt[kern]["avg_ms"] * 1e-3
        bpt = scan_bytes_per_token(w.D, w.N, s, w.proj)
        per_launch = bpt * w.M
        gbs = per_launch / avg / 1e9
        flops = scan_flops_per_state_step(kern.endswith("trunc")) * w.M * w.D * w.N
        e = {"kernel": kern, "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": gbs / HBM_PEAK_GBS, "traffic": measured_traffic(kern, tag) if tag else None,
             "avg_ms": kt[kern]["avg_ms"], "bytes_per_token": bpt, "tokens_per_launch": w.M,
             "algorithmic_bytes_per_launch": per_launch,
             "valu_TFLOPs": flops / avg / 1e12, "valu_frac": flops / avg / 1e12 / FP32_VECTOR_PEAK_TFS}
        if layer:
            lb = layer_scan_bytes_per_token(w.D, w.N, s, w.d_model)
            e["layer_path_bytes_per_token"] = lb
            e["layer_path_frac"] = lb * w.M / avg / 1e9 / HBM_PEAK_GBS
        out[kern] = e
    if layer:
        for kern, f in layer_gemm_flops(w.M, w.D, w.N, w.d_model).items():
            if kern not in kt:
                continue
            avg = kt[kern]["avg_ms"] * 1e-3
            ach = f / avg / 1e12
            out[kern] = {"kernel": kern, "bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFS,
                         "unit": "TFLOP/s", "frac": ach / MFMA_BF16_PEAK_TFS,
                         "traffic": measured_traffic(kern, tag) if tag else None, "avg_ms": kt[kern]["avg_ms"],
                         "algorithmic_flops_per_launch": f}
    return out


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, T_all=8192, T_one=1024, ch_one=512):
    """The fp64 oracle as it stands, on the host cores, on bounded samples of the
    headline workload (the first tokens of its sequence, its layer shape):
      * all cores: the layer's full gradient (BPTT scan + projection products)
        and its truncated gradient (tail-form scan, window w.tbar + projections)
        on T_all tokens, all channels; ``value`` combines the two like the GPU's;
      * one core: the full and the truncated scan gradient (no projections) on
        T_all tokens of ch_one channels (channels are independent in the scan;
        the rate is scaled to all channels and labelled so), and the full layer
        gradient on T_one tokens."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    from paper_2501_00692_amd.synth import make_inputs

    ws = w.with_(T=T_all)
    inp = make_inputs(ws, device="cpu")
    h = {k: v.float().double().numpy() for k, v in inp.items()}
    del inp
    nthreads = oracle.max_threads()
    args = (h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"])
    t0 = time.perf_counter()
    oracle.layer_grad(*args)
    t1 = time.perf_counter()
    oracle.layer_grad(*args, tbar=w.tbar, scan=oracle.trunc_tail)
    t2 = time.perf_counter()
    full_all, trunc_all = t1 - t0, t2 - t1
    legs = {"layer_full_all_cores": {"tokens_per_s": T_all / full_all, "s": full_all, "tokens": T_all},
            "layer_trunc_all_cores": {"tokens_per_s": T_all / trunc_all, "s": trunc_all, "tokens": T_all,
                                      "tbar": w.tbar}}
    with threadpool_limits(limits=1):
        sl = {k: np.ascontiguousarray(h[k][..., :ch_one]) for k in ("x", "delta", "dy", "z")}
        A = np.ascontiguousarray(h["A_log"][:ch_one])
        kw = dict(z=sl["z"], delta_softplus=True, nthreads=1)
        t0 = time.perf_counter()
        oracle.bptt(sl["x"], sl["delta"], A, h["B"], h["C"], sl["dy"], want_dh0=False, **kw)
        t1 = time.perf_counter()
        oracle.trunc_tail(sl["x"], sl["delta"], A, h["B"], h["C"], sl["dy"], tbar=w.tbar, **kw)
        t2 = time.perf_counter()
        scale = ch_one / w.D
        legs["scan_full_1core"] = {"tokens_per_s": T_all / (t1 - t0) * scale, "s": t1 - t0,
                                   "sample": f"{T_all} tokens x {ch_one} of {w.D} channels, rate scaled to "
                                             f"all channels (extrapolated)"}
        legs["scan_trunc_1core"] = {"tokens_per_s": T_all / (t2 - t1) * scale, "s": t2 - t1, "tbar": w.tbar,
                                    "sample": f"{T_all} tokens x {ch_one} of {w.D} channels, rate scaled to "
                                              f"all channels (extrapolated)"}
        one = {k: np.ascontiguousarray(v[:, :T_one]) if v.ndim == 3 else v for k, v in h.items()}
        t0 = time.perf_counter()
        oracle.layer_grad(one["u"], one["x"], one["z"], one["delta"], one["B"], one["C"], one["W_x"],
                          one["A_log"], one["dy"])
        t1 = time.perf_counter()
        legs["layer_full_1core"] = {"tokens_per_s": T_one / (t1 - t0), "s": t1 - t0, "tokens": T_one}
    oracle.max_threads()  # (the OpenMP team size is set per call; later calls pass their own)
    value = 2 * T_all / (full_all + trunc_all)
    return {"value": value, "unit": "tokens/s", "cores": nthreads, "kind": "oracle",
            "sample": f"fp64 oracle, layer gradient of the {w.name} workload's shape (D={w.D}, d_model={w.d_model}) "
                      f"on its first {T_all} tokens: one full (BPTT scan + projection products) and one "
                      f"truncated (tail-form scan, tbar={w.tbar}) call, {full_all:.1f} s + {trunc_all:.1f} s on "
                      f"{nthreads} OpenMP threads (numpy BLAS for the projection products); value = 2 x "
                      f"{T_all} tokens / total",
            "cpu_model": _cpu_model(), "nproc": os.cpu_count(), "legs": legs}


def unstructured_measure(ssm, torch, steps, warmup, chunk=0):
    """Full and truncated gradient of the unstructured SSM workload: per-call
    time, tokens/s, per-kernel times and the whole call's HBM fraction by
    compulsory bytes."""
    from paper_2501_00692_amd.synth import UN_WORKLOADS
    b, T, P, tbar = UN_WORKLOADS["unstructured"]
    res = {"config": f"b={b}, T={T}, P={P} channels, N=16 states, fp32, tbar={tbar}"}
    for mode, tb in (("full", 0), ("truncated", tbar)):
        st = un_step(b, T, P, tb, ssm, torch, chunk)
        m, kt = _timed_kernels(st, steps, warmup, ssm, torch)
        bpt = un_bytes_per_token(16, P)
        res[mode] = {"ms": m, "tokens_per_s": b * T / (m * 1e-3), "bytes_per_token": bpt,
                     "hbm_frac_call": bpt * b * T / (m * 1e-3) / (HBM_PEAK_GBS * 1e9),
                     "kernels_ms": {k: v["avg_ms"] for k, v in kt.items()}}
        del st
        torch.cuda.empty_cache()
    return res


def copy_bandwidth(torch, nbytes=1 << 30, reps=10):
    """Achievable HBM bandwidth as context for the HBM fractions: a plain device
    copy of nbytes (read + write counted), timed with events over reps copies."""
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    gbps = 2 * nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbps


def head_measure(ssm, torch, steps, warmup):
    """The language head with its loss at the head workload: per-call time,
    tokens/s, the MFMA fraction of its three products (logits, dU, dOmega:
    3 x 2 M P V flops) and the per-kernel split."""
    import ctypes

    from paper_2501_00692_amd.synth import HEAD_WORKLOADS, make_head_inputs
    M, P, V = HEAD_WORKLOADS["head"]
    inp = make_head_inputs(M, P, V, 692310, device="cuda")
    out = {"loss": torch.empty(M, dtype=torch.float32, device="cuda"),
           "dy": torch.empty(M, P, dtype=torch.float32, device="cuda"),
           "domega": torch.empty(V, P, dtype=torch.float32, device="cuda")}
    n = ctypes.c_size_t()
    ssm.load_library().ssm_lm_head_grad_workspace_size(M, P, V, ssm.SSM_HEAD_NORM, 0, ctypes.byref(n))
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_lm_head_grad(inp["y"], inp["omega"], inp["targets"], out=out, workspace=ws)

    m, kt = _timed_kernels(step, steps, warmup, ssm, torch)
    flops = 3 * 2 * M * P * V
    res = {"config": f"M={M} tokens, P={P}, V={V}, RMS-normalised input, bf16 products, fp32 accumulation",
           "ms": m, "tokens_per_s": M / (m * 1e-3), "tflops": flops / (m * 1e-3) / 1e12,
           "mfma_frac_call": flops / (m * 1e-3) / (MFMA_BF16_PEAK_TFS * 1e12),
           "kernels_ms": {k: v["ms_per_step"] for k, v in kt.items()}}
    del inp, out, ws
    torch.cuda.empty_cache()
    return res


def unstructured_line(args, ssm, torch):
    """The JSON line of ``--workload unstructured`` (for profiling that variant)."""
    r = unstructured_measure(ssm, torch, args.steps, args.warmup, args.chunk)
    ms = r["full"]["ms"] + r["truncated"]["ms"]
    return {"metric": "SSM-layer adjoint-gradient tokens/sec (full & truncated Tbar); % HBM/MFMA peak",
            "value": 2 * 8 * 16384 / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "fp32", "data": "synthetic",
            "config": {"workload": "unstructured SSM of Table 1 (16 states shared by 64 channels, per-step matrices), "
                                   + r["config"] + "; each step one full and one truncated ssm_unstructured_grad call"},
            "extra": r}


def head_line(args, ssm, torch):
    """The JSON line of ``--workload head`` (for profiling the language head)."""
    from paper_2501_00692_amd.synth import HEAD_WORKLOADS
    r = head_measure(ssm, torch, args.steps, args.warmup)
    M = HEAD_WORKLOADS["head"][0]
    return {"metric": "language-head loss and gradient tokens/sec; % MFMA peak",
            "value": M / (r["ms"] * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": r["ms"], "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16-in/fp32-acc", "data": "synthetic",
            "config": {"workload": "language head of Sec. 3.2 with cross-entropy loss, " + r["config"]
                                   + "; each step one ssm_lm_head_grad call"},
            "extra": r}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--workload", default=HEADLINE,
                    help="workload of the timed step (default: slice); the step runs the gradient modes the "
                         "workload is defined with (see MODES)")
    ap.add_argument("--chunk", type=int, default=0, help="carry chunk of the timed step (0: the library default)")
    ap.add_argument("--quick", action="store_true",
                    help="only the warmup and the timed steps (for profiler runs): no per-mode, spread or "
                         "graph timings")
    ap.add_argument("--copy-calib", action="store_true",
                    help="first run a plain 256 MiB device copy (torch copy_) three times, as the known-size "
                         "reference for HBM traffic counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: this library measures one GPU only "
              f"(the multi-GPU sharding is a design, not an implementation)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2501_00692_amd as ssm
    from paper_2501_00692_amd.synth import WORKLOADS, make_inputs

    torch.cuda.set_device(0)
    if args.copy_calib:
        src = torch.ones(64 * 1024 * 1024, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if args.workload == "unstructured":
        print(json.dumps(unstructured_line(args, ssm, torch)), flush=True)
        return
    if args.workload == "head":
        print(json.dumps(head_line(args, ssm, torch)), flush=True)
        return
    w = WORKLOADS[args.workload]
    tbar = w.tbar
    inp = make_inputs(w, device="cuda")
    calls = {}
    for mode in MODES[w.name]:
        tb = tbar if mode == "truncated" else 0
        if w.proj:
            calls[mode] = layer_step(w, inp, ssm, torch, tbar=tb, chunk=args.chunk)
        else:
            calls[mode] = scan_step(w, inp, ssm, torch, tbar=tb, chunk=args.chunk)

    def step():
        for fn in calls.values():
            fn()

    print(f"bench: {w.name} workload ({', '.join(calls)}), warmup", file=sys.stderr, flush=True)
    ms, ktimes = _timed_kernels(step, args.steps, args.warmup, ssm, torch)
    print(f"bench: {w.name} timed {args.steps} steps, {ms:.3f} ms/step", file=sys.stderr, flush=True)
    tag = workload_tag(w, args.chunk)
    roofs = rooflines(ktimes, w, w.proj, tag)
    dom = max(roofs, key=lambda k: ktimes[k]["ms_per_step"])
    value = len(calls) * w.M / (ms * 1e-3)
    extra = {"kernels": ktimes, "roofline_other": {k: v for k, v in roofs.items() if k != dom}}
    modes = {}
    if not args.quick:
        extra["ms_per_step_without_kernel_events"] = _timed(step, args.steps, 1, torch)
        for mode, fn in calls.items():
            m = _timed(fn, args.steps, 1, torch)
            modes[mode] = {"ms": m, "tokens_per_s": w.M / (m * 1e-3)}
            if mode == "truncated":
                modes[mode]["tbar"] = tbar
        scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        extra["ms_per_step_warm"] = _timed_each(step, 10, 1, torch)
        extra["ms_per_step_cold"] = _timed_each(step, 10, 1, torch, flush=lambda: scratch.fill_(1))
        del scratch
        extra["hbm_copy_GBps"] = copy_bandwidth(torch)
    del inp, calls
    torch.cuda.empty_cache()

    if not args.no_extra:
        # (workload, kind, tbar, chunk, variant); variant "scalarA+deltaB" is the scalar-decay
        # SSM of Table 1 with the step-size-scaled input
        runs = [("small", "scan", 0, 0, ""), ("small", "scan", 32, 0, ""), ("layer", "layer", 0, 0, ""),
                ("long", "layer", 2048, 256, ""), ("long", "layer", 2048, 0, ""), ("long", "scan", 2048, 0, ""),
                ("long_slow", "scan", 2048, 0, ""), ("vlong", "scan", 8192, 0, ""),
                ("layer", "layer", 0, 0, "scalarA+deltaB"), ("long", "scan", 2048, 0, "scalarA+deltaB"),
                ("small", "pairs", 0, 0, ""), ("small", "pairs", 32, 0, ""), ("pairs", "pairs", 256, 0, ""),
                ("pairs", "scan", 256, 0, "")]
        res = {}
        for name, kind, tb, chunk, variant in runs:
            wl = WORKLOADS[name]
            print(f"bench: extra {name}/{kind}/tbar={tb}/chunk={chunk} {variant}", file=sys.stderr, flush=True)
            x = make_inputs(wl, device="cuda")
            if variant:
                x["A_log"] = x["A_log"][:, 0].contiguous()
            if kind == "layer":
                st = layer_step(wl, x, ssm, torch, tbar=tb, b_delta=bool(variant), chunk=chunk)
            else:
                st = scan_step(wl, x, ssm, torch, tbar=tb, b_delta=bool(variant), pairs=kind == "pairs",
                               chunk=chunk)
            steps = 5 if wl.M >= 262144 else 10
            m, kt = _timed_kernels(st, steps, 2, ssm, torch)
            entry = {"ms_per_step": m, "tokens_per_s": wl.M / (m * 1e-3), "tbar": tb, "chunk": chunk or "default",
                     "kernels_ms": {k: v["avg_ms"] for k, v in kt.items()}}
            if kind == "pairs":
                # the paper's unit of work: one (t, i) adjoint state over all D x N states
                entry["vjp_pairs_per_s"] = wl.b * vjp_pairs(wl.T, tb) / (m * 1e-3)
            elif not variant:
                for k, r in rooflines(kt, wl, kind == "layer").items():
                    entry[f"{k}_frac"] = r["frac"]
                    entry[f"{k}_{r['unit'].replace('/', 'per')}"] = r["achieved"]
            res[f"{name}/{kind}/tbar={tb}" + (f"/chunk={chunk}" if chunk else "") +
                (f"/{variant}" if variant else "")] = entry
            del x, st
            torch.cuda.empty_cache()
        # the unstructured SSM of Table 1
        print("bench: extra unstructured", file=sys.stderr, flush=True)
        res["unstructured"] = unstructured_measure(ssm, torch, 5, 2)
        # the language head of Sec. 3.2 with the cross-entropy loss
        print("bench: extra head", file=sys.stderr, flush=True)
        res["head"] = head_measure(ssm, torch, 5, 2)
        # the forward alone (y only), reported beside the gradients
        fwd = {}
        for name in ("layer", "long"):
            wl = WORKLOADS[name]
            x = make_inputs(wl, device="cuda")
            st = forward_step(wl, x, ssm, torch)
            m = _timed(st, 10, 2, torch)
            bpt = forward_bytes_per_token(wl.D, wl.N, 2 if wl.bf16 else 4, wl.proj)
            fwd[name] = {"ms": m, "tokens_per_s": wl.M / (m * 1e-3), "bytes_per_token": bpt,
                         "hbm_frac_algorithmic": bpt * wl.M / (m * 1e-3) / (HBM_PEAK_GBS * 1e9)}
            del x, st
            torch.cuda.empty_cache()
        res["forward"] = fwd
        # the K-layer residual stack (forward + gradients of every layer), Prop. 3 and
        # backpropagation, and how far apart their parameter gradients are
        K, b, T, D, N = 4, 2, 4096, 1536, 16
        st_res = {}
        grads = {}
        for exact in (False, True):
            st, sinp, sout = stack_step(K, b, T, D, N, ssm, torch, exact)
            m = _timed(st, 5, 2, torch)
            st_res["exact" if exact else "adjoint"] = {"ms_per_step": m, "tokens_per_s": b * T / (m * 1e-3)}
            grads[exact] = [x.clone() for x in sout["dW_in"]]
            del st, sinp, sout
            torch.cuda.empty_cache()
        st_res["dW_in_rel_diff_per_layer"] = [
            float((grads[False][k] - grads[True][k]).norm() / grads[True][k].norm()) for k in range(K)]
        st_res["config"] = f"K={K} layers, b={b}, T={T}, D={D} (residual width = channels), N={N}, bf16, full"
        res["stack"] = st_res
        extra["workloads"] = res

    line = {
        "metric": "SSM-layer adjoint-gradient tokens/sec (full & truncated Tbar); % HBM/MFMA peak",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16-in/fp32-acc" if w.bf16 else "fp32",
        "data": "synthetic",
        "config": {"workload": workload_text(w, list(MODES[w.name])),
                   "batch": w.b, "seq_len": w.T, "d_model": w.d_model if w.proj else None, "channels": w.D,
                   "dstate": w.N, "tbar": tbar, "inputs": "bf16" if w.bf16 else "fp32", "accumulate": "fp32",
                   "chunk": args.chunk or "default (128)", "tokens_per_step": len(MODES[w.name]) * w.M},
        "modes": modes,
        "roofline": roofs[dom],
    }
    if not args.no_cpu and w.proj:
        print("bench: cpu baseline", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(w)
    line["extra"] = extra
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
