"""Seeded synthetic inputs for the selective diagonal SSM layer.

This module only draws random tensors with the shapes and value distributions
of the layer workloads; it holds none of the gradient arithmetic, and both the
HIP path and the oracle read the very tensors it returns (the oracle after an
exact upcast to fp64).

Workloads (b batch, T length, D channels, N state, d_model, window Tbar):

=======  ====  =========  =====  ==  =======  =====  =====  ========
name     b     T          D      N   d_model  Tbar   proj   dtype
=======  ====  =========  =====  ==  =======  =====  =====  ========
small    1     256        64     16  64       32     no     fp32
layer    2     4,096      1536   16  768      --     yes    bf16
long     2     65,536     1536   16  768      2048   yes    bf16
slice    1     262,144    4096   16  2048     4096   yes    bf16
vlong    1     1,048,576  3072   16  --       8192   no     bf16
pairs    2     4,096      1536   16  --       256    no     bf16
=======  ====  =========  =====  ==  =======  =====  =====  ========

Distributions: x ~ N(0,1); Delta = softplus(N(0,1)) (drawn as Delta_pre ~ N(0,1)
when the layer applies the softplus itself); A_log ~ U(log 1, log 16) per (d, n);
upstream gradient ~ N(0,1); B, C ~ N(0, 1/N) without projections and N(0,1) with
them (the marginals of x W_B with W_B ~ N(0, 1/fan_in)).  With projections the
stored activations x, z, Delta_pre, B, C are drawn directly from those marginals
(rather than computed from u and the weights), u ~ N(0,1), and
W ~ N(0, 1/fan_in).  ``delta_scale`` < 1 gives the slow-decay variants in which
the truncation window is visible (Delta / 32 for "small", Delta / 2048 for "long").
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    b: int
    T: int
    D: int
    N: int
    d_model: int
    tbar: int           # 0: full gradient only
    proj: bool          # input projections and SiLU gate
    bf16: bool          # bf16 inputs (else fp32)
    seed: int
    delta_scale: float = 1.0

    @property
    def M(self) -> int:
        return self.b * self.T

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "small": Workload("small", 1, 256, 64, 16, 64, 32, False, False, 692000),
    "layer": Workload("layer", 2, 4096, 1536, 16, 768, 0, True, True, 692001),
    "long": Workload("long", 2, 65536, 1536, 16, 768, 2048, True, True, 692002),
    "slice": Workload("slice", 1, 262144, 4096, 16, 2048, 4096, True, True, 692003),
    "vlong": Workload("vlong", 1, 1048576, 3072, 16, 1536, 8192, False, True, 692004),
}
# the explicit pair formulation's workload: the layer's scan shape with a 256-step window
WORKLOADS["pairs"] = Workload("pairs", 2, 4096, 1536, 16, 768, 256, False, True, 692005)
WORKLOADS["small_slow"] = WORKLOADS["small"].with_(name="small_slow", delta_scale=1.0 / 32)
WORKLOADS["long_slow"] = WORKLOADS["long"].with_(name="long_slow", proj=False, delta_scale=1.0 / 2048)


def make_inputs(w: Workload, device="cpu", seed: int | None = None, h0: bool = False):
    """Draw the inputs of one gradient call.

    Returns a dict of tensors on ``device``: ``x, delta, A_log, B, C, dy`` and, with
    projections, ``z, u, W_x, W_in``; ``h0`` when asked.  ``delta`` holds Delta_pre
    (the layer applies softplus) when ``w.proj`` and Delta itself otherwise.
    Activations are bf16 (round-to-nearest-even from fp32) or fp32; ``A_log`` and
    ``h0`` are fp32.
    """
    g = torch.Generator(device=device)
    g.manual_seed(w.seed if seed is None else seed)
    dt = torch.bfloat16 if w.bf16 else torch.float32
    b, T, D, N = w.b, w.T, w.D, w.N

    def randn(*shape, std=1.0):
        t = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
        return t.mul_(std) if std != 1.0 else t

    out = {}
    out["x"] = randn(b, T, D).to(dt)
    pre = randn(b, T, D)
    if w.proj:
        out["delta"] = pre.to(dt)
    else:
        d = torch.nn.functional.softplus(pre)
        if w.delta_scale != 1.0:
            d.mul_(w.delta_scale)
        out["delta"] = d.to(dt)
    del pre
    out["A_log"] = (torch.rand(D, N, generator=g, device=device, dtype=torch.float32)
                    .mul_(math.log(16.0)))
    bc_std = 1.0 if w.proj else 1.0 / math.sqrt(N)
    out["B"] = randn(b, T, N, std=bc_std).to(dt)
    out["C"] = randn(b, T, N, std=bc_std).to(dt)
    out["dy"] = randn(b, T, D).to(dt)
    if w.proj:
        out["z"] = randn(b, T, D).to(dt)
        out["u"] = randn(b, T, w.d_model).to(dt)
        out["W_x"] = randn(D, D + 2 * N, std=1.0 / math.sqrt(D)).to(dt)
        out["W_in"] = randn(w.d_model, 2 * D, std=1.0 / math.sqrt(w.d_model)).to(dt)
    if h0:
        out["h0"] = randn(b, D, N)
    return out


def make_stack_inputs(K: int, b: int, T: int, D: int, N: int, seed: int, device="cpu"):
    """Inputs of a K-layer residual stack: y0 ~ N(0,1) [b, T, D] (fp32); per layer
    W_in ~ N(0, 1/D) [D, 2D], W_x ~ N(0, 1/D) [D, D+2N] (bf16, round to nearest
    even) and A_log ~ U(log 1, log 16) [D, N] (fp32); the upstream gK ~ N(0,1)."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device)
    y0 = torch.randn(b, T, D, generator=g, **f32)
    W_in = [(torch.randn(D, 2 * D, generator=g, **f32) / math.sqrt(D)).to(torch.bfloat16) for _ in range(K)]
    W_x = [(torch.randn(D, D + 2 * N, generator=g, **f32) / math.sqrt(D)).to(torch.bfloat16) for _ in range(K)]
    A_log = [torch.rand(D, N, generator=g, **f32) * math.log(16.0) for _ in range(K)]
    gK = torch.randn(b, T, D, generator=g, **f32)
    return dict(y0=y0, W_in=W_in, W_x=W_x, A_log=A_log, gK=gK)


# The unstructured SSM of Table 1 (16 states shared by P channels, per-step
# matrices): (b, T, P, tbar).  "unstructured" is the measured workload.
UN_WORKLOADS = {
    "un_small": (2, 300, 32, 64),
    "unstructured": (8, 16384, 64, 256),
}


def make_unstructured_inputs(b: int, T: int, P: int, seed: int, N: int = 16, device="cpu", h0: bool = False):
    """Per-step matrices and inputs of the unstructured SSM, fp32: A_t with
    entries N(0, 0.81/N) (a random transition of spectral radius about 0.9, so
    the state neither grows nor vanishes over long sequences), B_t ~ N(0, 1/P),
    C_t ~ N(0, 1/N), x, dy ~ N(0, 1), and h0 ~ N(0, 1) when asked."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device)
    out = {
        "A": torch.randn(b, T, N, N, generator=g, **f32).mul_(0.9 / math.sqrt(N)),
        "B": torch.randn(b, T, N, P, generator=g, **f32).mul_(1.0 / math.sqrt(P)),
        "C": torch.randn(b, T, P, N, generator=g, **f32).mul_(1.0 / math.sqrt(N)),
        "x": torch.randn(b, T, P, generator=g, **f32),
        "dy": torch.randn(b, T, P, generator=g, **f32),
    }
    if h0:
        out["h0"] = torch.randn(b, N, generator=g, **f32)
    return out


# The language head of Sec. 3.2: (rows M, width P, vocabulary V).  "head" is the
# measured workload (32,768 tokens of a 2,048-wide model, a 32,000-token
# vocabulary); the others are parity cases.
HEAD_WORKLOADS = {
    "head_small": (300, 96, 1000),
    "head_blocks": (1000, 64, 1024),
    "head_medium": (4096, 512, 32000),
    "head": (32768, 2048, 32000),
}


def make_head_inputs(M: int, P: int, V: int, seed: int, device="cpu"):
    """Inputs of the head: y ~ N(0, 1) fp32 [M][P] (the last residual output),
    Omega ~ N(0, 4/P) as bf16 [V][P] (logits of standard deviation about 2 on
    the normalised input), targets uniform over the vocabulary (int32 [M])."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device)
    return {
        "y": torch.randn(M, P, generator=g, **f32),
        "omega": torch.randn(V, P, generator=g, **f32).mul_(2.0 / math.sqrt(P)).to(torch.bfloat16),
        "targets": torch.randint(0, V, (M,), generator=g, device=device, dtype=torch.int32),
    }
