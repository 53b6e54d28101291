"""The gradient entry point that allocates nothing (its scratch is a fixed
device array inside the library) against ssm_adjoint_grad with a caller
workspace: two calls in a row, the second on a smaller problem, each equal to
the workspace entry point's outputs bit for bit (the same kernels on the same
inputs) and so within the oracle tolerance of them."""
import pytest
import torch

import paper_2501_00692_amd as ssm
from paper_2501_00692_amd.synth import Workload, make_inputs

from gpu_helpers import TOL_F32, check, say, to_np

pytestmark = pytest.mark.gpu

# first a larger bf16 call with the gate, softplus and a window, then a smaller
# fp32 call without them (full gradient with h0 and dh0): the second call finds
# the first call's contents in the scratch
FIRST = Workload("noalloc_first", 2, 2000, 256, 16, 256, 64, True, True, 692130)
SECOND = Workload("noalloc_second", 1, 700, 96, 16, 96, 0, False, False, 692131, delta_scale=1.0 / 32)


def _args(inp, w):
    return (inp["x"], inp["delta"], inp["A_log"], inp["B"], inp["C"], inp["dy"])


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_entry(order):
    for w, tbar, h0 in ((FIRST, FIRST.tbar, False), (SECOND, 0, True)):
        say(f"[noalloc] {w.name} b={w.b} T={w.T} D={w.D} tbar={tbar}")
        inp = make_inputs(w, device="cuda", h0=h0)
        kw = dict(h0=inp.get("h0"), z=inp.get("z"), softplus=w.proj, tbar=tbar, want_dh0=h0)
        ref = ssm.ssm_adjoint_grad(*_args(inp, w), **kw)
        got = ssm.ssm_adjoint_grad_noalloc(*_args(inp, w), **kw)
        torch.cuda.synchronize()
        assert set(got) == set(ref)
        rep = {}
        for k in ref:
            if ref[k] is None:
                continue
            check(k, to_np(got[k]), to_np(ref[k]), TOL_F32, rep)
            assert torch.equal(got[k], ref[k]), k
        say("   rel-L2 vs workspace entry:", " ".join(f"{k}={v:.1e}" for k, v in rep.items()))


def test_noalloc_rejects_oversize():
    """A problem whose scratch exceeds the fixed array is refused on the host
    (SSM_ERR_WORKSPACE) before anything is enqueued."""
    b, T, D, N = 1, 1 << 18, 1024, 16
    desc = ssm.SsmDesc(b, T, D, N, 0, ssm.SSM_BF16, 0)
    assert ssm.grad_workspace_size(desc, 0) > (64 << 20)
    big = {k: torch.empty(b, T, D if k in ("x", "delta", "dy") else N, dtype=torch.bfloat16, device="cuda")
           for k in ("x", "delta", "B", "C", "dy")}
    A = torch.zeros(D, N, device="cuda")
    with pytest.raises(ssm.SsmError) as e:
        ssm.ssm_adjoint_grad_noalloc(big["x"], big["delta"], A, big["B"], big["C"], big["dy"])
    assert e.value.status == 5
