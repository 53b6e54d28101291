"""Benchmark of the per-layer adjoint gradient on one MI355X.

One step = one whole-layer gradient call (``ssm_layer_grad``): the chunked
forward recomputation, the reverse adjoint scan with its vjp epilogue, and the
projection-gradient GEMMs, on the "layer" workload (b=2, T=4096, d_model=768,
D=1536, N=16, full gradient; bf16 activations, fp32 accumulation).  Inputs are
seeded synthetic tensors already resident in HBM.  The other workloads are
reported under "extra".

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
# x 2.4 GHz = 157.3 TFLOP/s.  On gfx950 an ordinary (non-packed) wave64 fp32
# add, mul or FMA issues every 2 cycles per SIMD, so this peak needs no packed
# instructions (which this library's kernels are built without).
FP32_VECTOR_PEAK_TFS = 157.3


def scan_flops_per_state_step(trunc):
    """Algorithmic fp32 operations per (state, token) of the fused gradient (an FMA
    counts 2, exp counts 1): forward recompute a = exp(Delta c) (2), h = a h + B x (3),
    y += C h (2), dC contribution and channel sum (2); reverse mu = g C + a mu (3),
    dx += mu B (2), s = mu (a h) (2), ddelta += s w (2), dA += s Delta (2), dB
    contribution and sum (2) -> 22.  The truncated window adds the window product
    P = exp(W c) (2), the tail nu = P g' C' + a nu (4) and mubar = mu - nu (1)."""
    return 22 + (7 if trunc else 0)


def scan_bytes_per_token(D, N, s, gate, layer=False):
    """Compulsory HBM bytes per token of the scan gradient: every input read once
    and every output written once at the ABI's dtypes (outputs fp32).  Inside the
    whole-layer call with no scan outputs requested (``layer``), the kernel writes
    dx in fp32 (the projection GEMM's addend) and dDelta_pre, dz, dB, dC as the
    bf16 operands of the projection GEMMs, plus fp32 dB, dC."""
    if layer:  # reads x, Delta_pre, dy, z; writes dx (fp32), dDelta_pre, dz (bf16)
        return D * (4 * s + 4 + 2 + 2) + N * (2 * s + 8 + 4)
    if gate:  # reads x, Delta_pre, dy, z; writes dx, dDelta_pre, dz
        per_ch = 4 * s + 12
    else:     # reads x, Delta, dy; writes dx, dDelta
        per_ch = 3 * s + 8
    return D * per_ch + N * (2 * s + 8)  # reads B, C; writes dB, dC


def layer_gemm_flops(M, D, N, dm, with_du=False):
    f = 2 * M * D * (D + 2 * N)        # dW_x = x^T dZx
    f += 2 * M * (D + 2 * N) * D       # dx_total = dx + dZx W_x^T
    f += 2 * M * dm * 2 * D            # dW_in = u^T [dx_total | dz]
    if with_du:
        f += 2 * M * 2 * D * dm
    return f


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


def _timed_graph(fn, steps, warmup, torch):
    """Per-step time of `fn` captured once in a HIP graph and replayed `steps`
    times (launch overheads between the step's kernels removed)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fn()
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        graph.replay()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def _kernel_times(fn, steps, ssm, torch):
    """Per-kernel average launch duration (ms) from hipEvents recorded on the
    launch stream around every kernel of `steps` calls."""
    torch.cuda.synchronize()
    ssm.timing_summary()
    ssm.timing_enable(True)
    for _ in range(steps):
        fn()
    ssm.timing_enable(False)
    torch.cuda.synchronize()
    out = {}
    for name, (n, ms) in ssm.timing_summary().items():
        out[name] = {"launches": n, "total_ms": ms, "avg_ms": ms / n, "launches_per_step": n / steps}
    return out


def layer_step(w, inp, ssm, torch, tbar=0, b_delta=False):
    """One whole-layer gradient; ``inp["A_log"]`` of shape [D] selects the scalar-decay variant."""
    b, T, D, N, dm = w.b, w.T, w.D, w.N, w.d_model
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dW_in": torch.empty(dm, 2 * D, **f32), "dW_x": torch.empty(D, D + 2 * N, **f32),
           "dA_log": torch.empty(*inp["A_log"].shape, **f32)}
    desc = ssm.make_desc(inp["x"], N, True, True, 0, inp["A_log"].dim() == 1, b_delta)
    ws = torch.empty(ssm.layer_workspace_size(desc, tbar, dm), dtype=torch.uint8, device="cuda")

    def step():
        ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"],
                           inp["W_in"], inp["A_log"], inp["dy"], tbar=tbar, out=out, workspace=ws, b_delta=b_delta)
    return step


def vjp_pairs(T, tbar):
    """(t, i) adjoint-state pairs of one sequence: T(T+1)/2 in full mode, else
    tbar T - tbar (tbar - 1) / 2 (the paper's VJP counts, Sec. 4.3)."""
    if tbar <= 0 or tbar >= T:
        return T * (T + 1) // 2
    return tbar * T - tbar * (tbar - 1) // 2


def scan_step(w, inp, ssm, torch, tbar=0, b_delta=False, pairs=False):
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
    desc = ssm.make_desc(inp["x"], N, w.proj, z is not None, 0, inp["A_log"].dim() == 1, b_delta)
    ws = torch.empty(ssm.grad_workspace_size(desc, tbar, pairs), dtype=torch.uint8, device="cuda")
    fn = ssm.ssm_adjoint_grad_pairs if pairs else ssm.ssm_adjoint_grad

    def step():
        fn(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], z=z, softplus=w.proj, tbar=tbar,
           out=out, workspace=ws, b_delta=b_delta)
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


def tbar_of(kind):
    """`kind` is "layer"/"scan" (full) or a (kind, tbar) tuple."""
    return kind[1] if isinstance(kind, tuple) else 0


def roofline_for(kern, ktimes, w, kind):
    """Roofline entry for kernel `kern` (algorithmic work per launch / average
    launch duration)."""
    kt = ktimes[kern]
    s = 2 if w.bf16 else 4
    if kern == "grad_fused":
        layer = (kind[0] if isinstance(kind, tuple) else kind) == "layer"
        per_launch = scan_bytes_per_token(w.D, w.N, s, w.proj, layer) * w.M  # bytes
        gbs = per_launch / (kt["avg_ms"] * 1e-3) / 1e9
        flops = scan_flops_per_state_step(0 < tbar_of(kind) < w.T) * w.M * w.D * w.N
        tfs = flops / (kt["avg_ms"] * 1e-3) / 1e12
        return {"kernel": kern, "bound": "alu", "achieved": tfs, "peak": FP32_VECTOR_PEAK_TFS, "unit": "TFLOP/s",
                "frac": tfs / FP32_VECTOR_PEAK_TFS, "traffic": None, "avg_ms": kt["avg_ms"],
                "algorithmic_flops_per_launch": flops, "algorithmic_bytes_per_launch": per_launch,
                "hbm_GBps_algorithmic": gbs, "hbm_frac_algorithmic": gbs / HBM_PEAK_GBS}
    if kern in ("gemm_dw", "gemm_dx"):
        M, D, N, dm = w.M, w.D, w.N, w.d_model
        if kern == "gemm_dw":
            flops = 2 * M * D * (D + 2 * N) + 2 * M * dm * 2 * D
        else:
            flops = 2 * M * (D + 2 * N) * D
        per_launch = flops / kt["launches_per_step"]
        ach = per_launch / (kt["avg_ms"] * 1e-3) / 1e12
        return {"kernel": kern, "bound": "mfma", "achieved": ach, "peak": MFMA_BF16_PEAK_TFS, "unit": "TFLOP/s",
                "frac": ach / MFMA_BF16_PEAK_TFS, "traffic": None, "avg_ms": kt["avg_ms"],
                "algorithmic_flops_per_launch": per_launch}
    return None


def cpu_baseline(w, T_sample=256):
    """The fp64 oracle (layer gradient incl. projections) on the first T_sample
    tokens of every batch row of the workload, all channels."""
    import numpy as np

    import oracle
    from paper_2501_00692_amd.synth import make_inputs

    ws = w.with_(T=T_sample)
    inp = make_inputs(ws, device="cpu")
    h = {k: v.float().double().numpy() for k, v in inp.items()}
    nthreads = oracle.max_threads()
    t0 = time.perf_counter()
    if w.proj:
        oracle.layer_grad(h["u"], h["x"], h["z"], h["delta"], h["B"], h["C"], h["W_x"], h["A_log"], h["dy"],
                          tbar=w.tbar, scan=oracle.trunc_tail if w.tbar else None)
    else:
        oracle.trunc_tail(h["x"], h["delta"], h["A_log"], h["B"], h["C"], h["dy"], tbar=w.tbar)
    dt = time.perf_counter() - t0
    del np
    return {"value": ws.b * T_sample / dt, "unit": "tokens/s", "cores": nthreads, "kind": "oracle",
            "sample": f"fp64 oracle layer gradient (BPTT scan + projection chain) on b={ws.b} x T={T_sample} "
                      f"tokens of the {w.name} workload, all {w.D} channels; {dt:.2f} s wall on {nthreads} "
                      f"OpenMP threads (numpy BLAS for the projection products)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-extra", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-tokens", type=int, default=4096)
    ap.add_argument("--copy-calib", action="store_true",
                    help="first run a plain 256 MiB device copy (torch copy_) three times, as the known-size "
                         "reference for HBM traffic counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: this build measures one GPU only "
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
    w = WORKLOADS["layer"]
    inp = make_inputs(w, device="cuda")
    step = layer_step(w, inp, ssm, torch, tbar=0)
    ms = _timed(step, args.steps, args.warmup, torch)
    # the same step captured in a HIP graph and replayed, reported beside it (the
    # gaps between dependent kernels are on the GPU side: replay gains nothing)
    ms_graph = _timed_graph(step, args.steps, args.warmup, torch)
    # per-rep spread, warm and with the L2 and MALL flushed before every rep
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    spread_warm = _timed_each(step, 20, 3, torch)
    spread_cold = _timed_each(step, 20, 3, torch, flush=lambda: scratch.fill_(1))
    del scratch
    ktimes = _kernel_times(step, args.steps, ssm, torch)
    dom = max(ktimes, key=lambda k: ktimes[k]["total_ms"])
    roof = roofline_for(dom, ktimes, w, "layer")
    if roof is not None:
        roof["traffic"] = measured_traffic(dom, "layer-b2-T4096-D1536")
    value = w.M / (ms * 1e-3)

    other = {k: roofline_for(k, ktimes, w, "layer") for k in ("grad_fused", "gemm_dw", "gemm_dx")
             if k in ktimes and k != dom}
    for k, r in other.items():
        r["traffic"] = measured_traffic(k, "layer-b2-T4096-D1536")
    extra = {"ms_per_step_graph_replay": ms_graph, "ms_per_step_warm": spread_warm,
             "ms_per_step_cold": spread_cold, "kernels_layer": ktimes,
             "roofline_other": other,
             "gemm_tflops_layer": layer_gemm_flops(w.M, w.D, w.N, w.d_model) / 1e12}
    del inp, step
    torch.cuda.empty_cache()

    if not args.no_extra:
        # (workload, kind, tbar, variant); variant "scalarA+deltaB" is the scalar-decay SSM of
        # Table 1 with the step-size-scaled input
        runs = [("small", "scan", 0, ""), ("small", "scan", 32, ""), ("long", "layer", 2048, ""),
                ("long", "scan", 2048, ""), ("long_slow", "scan", 2048, ""), ("slice", "layer", 0, ""),
                ("slice", "layer", 4096, ""), ("vlong", "scan", 8192, ""),
                ("layer", "layer", 0, "scalarA+deltaB"), ("long", "scan", 2048, "scalarA+deltaB"),
                ("small", "pairs", 0, ""), ("small", "pairs", 32, ""), ("pairs", "pairs", 256, ""),
                ("pairs", "scan", 256, "")]
        res = {}
        for name, kind, tbar, variant in runs:
            wl = WORKLOADS[name]
            x = make_inputs(wl, device="cuda")
            if variant:
                x["A_log"] = x["A_log"][:, 0].contiguous()
            if kind == "layer":
                st = layer_step(wl, x, ssm, torch, tbar=tbar, b_delta=bool(variant))
            else:
                st = scan_step(wl, x, ssm, torch, tbar=tbar, b_delta=bool(variant), pairs=kind == "pairs")
            steps = 5 if wl.M >= 262144 else 10
            m = _timed(st, steps, 2, torch)
            kt = _kernel_times(st, 2, ssm, torch)
            entry = {"ms_per_step": m, "tokens_per_s": wl.M / (m * 1e-3), "tbar": tbar,
                     "grad_fused_avg_ms": kt.get("grad_fused", {}).get("avg_ms")}
            if kind == "pairs":
                # the paper's unit of work: one (t, i) adjoint state over all D x N states
                entry["vjp_pairs_per_s"] = wl.b * vjp_pairs(wl.T, tbar) / (m * 1e-3)
                entry["pairs_kernel_avg_ms"] = kt.get("pairs", {}).get("avg_ms")
            r = None if (variant or kind == "pairs") else roofline_for("grad_fused", kt, wl, (kind, tbar))
            if r:
                entry["grad_fused_TFLOPs"] = r["achieved"]
                entry["grad_fused_alu_frac"] = r["frac"]
                entry["grad_fused_GBps"] = r["hbm_GBps_algorithmic"]
                entry["grad_fused_hbm_frac"] = r["hbm_frac_algorithmic"]
            for g in ("gemm_dw", "gemm_dx"):
                if g in kt:
                    rg = roofline_for(g, kt, wl, kind)
                    entry[f"{g}_TFLOPs"] = rg["achieved"]
            res[f"{name}/{kind}/tbar={tbar}" + (f"/{variant}" if variant else "")] = entry
            del x, st
            torch.cuda.empty_cache()
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
        "dtype": "fp32",
        "data": "synthetic",
        "config": {"workload": "layer: one selective diagonal SSM layer with input projections and SiLU gate, "
                               "b=2, T=4096, d_model=768, D=1536, N=16, full adjoint gradient; each step one "
                               "ssm_layer_grad call",
                   "batch": w.b, "seq_len": w.T, "d_model": w.d_model, "channels": w.D, "dstate": w.N,
                   "inputs": "bf16", "accumulate": "fp32", "chunk": 128},
        "roofline": roof,
    }
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_tokens)
    line["extra"] = extra
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
