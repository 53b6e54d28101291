"""The gradient entry points captured in a HIP graph (through torch's graph
capture on the calling stream): every replay, with unrelated eager work and
synchronisations between replays, must reproduce the eager result bit for bit
(the library is deterministic and its calls enqueue kernels only)."""
import pytest
import torch

import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import WORKLOADS, Workload, make_inputs

from gpu_helpers import say

pytestmark = pytest.mark.gpu

LAYER_SMALL = Workload("layer_graph", 2, 512, 128, 16, 64, 0, True, True, 692600)


def _capture_and_replay(call, outs, nreplay=3):
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in outs.items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call()
    junk = torch.randn(1 << 20, device="cuda")
    for r in range(nreplay):
        for v in outs.values():
            v.fill_(float("nan"))
        junk.mul_(1.0001).add_(0.5)  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in outs:
            assert torch.equal(outs[k], eager[k]), f"replay {r}: {k} differs from the eager result"
        say(f"   replay {r}: identical")


@pytest.mark.parametrize("tbar", [0, 64])
def test_layer_grad_graph_replays(tbar):
    w = LAYER_SMALL
    inp = make_inputs(w, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dW_in": torch.empty(w.d_model, 2 * w.D, **f32), "dW_x": torch.empty(w.D, w.D + 2 * w.N, **f32),
           "dA_log": torch.empty(w.D, w.N, **f32)}
    desc = ssm.make_desc(inp["x"], w.N, True, True, 0, False, False)
    ws = torch.empty(ssm.layer_workspace_size(desc, tbar, w.d_model), dtype=torch.uint8, device="cuda")

    def call():
        ssm.ssm_layer_grad(inp["u"], inp["x"], inp["z"], inp["delta"], inp["B"], inp["C"], inp["W_x"], inp["W_in"],
                           inp["A_log"], inp["dy"], tbar=tbar, out=out, workspace=ws)
    say(f"[graph layer] tbar={tbar}")
    _capture_and_replay(call, out)


def test_adjoint_grad_graph_replays():
    w = WORKLOADS["small_slow"]
    inp = make_inputs(w, device="cuda")
    f32 = dict(dtype=torch.float32, device="cuda")
    out = {"dx": torch.empty(w.b, w.T, w.D, **f32), "ddelta": torch.empty(w.b, w.T, w.D, **f32),
           "dA_log": torch.empty(w.D, w.N, **f32), "dB": torch.empty(w.b, w.T, w.N, **f32),
           "dC": torch.empty(w.b, w.T, w.N, **f32)}
    desc = ssm.make_desc(inp["x"], w.N, False, False, 0, False, False)
    ws = torch.empty(ssm.grad_workspace_size(desc, 32), dtype=torch.uint8, device="cuda")

    def call():
        ssm.ssm_adjoint_grad(inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"], tbar=32, out=out,
                             workspace=ws)
    say("[graph adjoint grad] tbar=32")
    _capture_and_replay(call, out)
