"""MI355X (gfx950) per-layer adjoint gradient of a selective diagonal SSM layer.

Thin ctypes binding over the C ABI in ``include/ssm_adjoint.h`` (library
``libssm_adjoint.so`` in this package directory).  The functions here only
marshal arguments: they check tensors, allocate outputs and workspace with
torch, and call the C entry point of the same name on torch's current stream.
Every step of the computation runs in the library's HIP kernels; there is no
other implementation behind this module, and it raises if the library is not
built.

Entry points (names as in the C ABI): :func:`ssm_adjoint_forward`,
:func:`ssm_adjoint_grad`, :func:`ssm_adjoint_grad_noalloc`, :func:`ssm_adjoint_grad_pairs`,
:func:`ssm_unstructured_grad`, :func:`ssm_proj_grad`,
:func:`ssm_layer_grad`, :func:`ssm_stack_grad`, :func:`ssm_lm_head_grad`.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

_PKG = Path(__file__).resolve().parent
LIB_PATH = _PKG / "libssm_adjoint.so"

SSM_F32, SSM_BF16 = 0, 1
SSM_FULL, SSM_TRUNCATED = 0, 1
SSM_DELTA_SOFTPLUS, SSM_GATE_SILU, SSM_A_SCALAR, SSM_B_DELTA = 1, 2, 4, 8
SSM_ACCUM_DW, SSM_ACCUM_DX = 1, 2
SSM_STACK_ADJOINT, SSM_STACK_EXACT, SSM_STACK_FORWARD = 0, 1, 2
SSM_HEAD_NORM = 1

STATUS = {0: "SSM_OK", 1: "SSM_ERR_NULL", 2: "SSM_ERR_SHAPE", 3: "SSM_ERR_DTYPE",
          4: "SSM_ERR_UNSUPPORTED", 5: "SSM_ERR_WORKSPACE", 6: "SSM_ERR_ALIGN", 7: "SSM_ERR_HIP"}

EXPORTED = (
    "ssm_adjoint_forward_workspace_size", "ssm_adjoint_grad_workspace_size", "ssm_adjoint_forward",
    "ssm_adjoint_grad", "ssm_adjoint_grad_noalloc", "ssm_adjoint_grad_pairs_workspace_size",
    "ssm_adjoint_grad_pairs",
    "ssm_unstructured_grad_workspace_size", "ssm_unstructured_grad",
    "ssm_proj_grad_workspace_size", "ssm_proj_grad",
    "ssm_layer_grad_workspace_size", "ssm_layer_grad", "ssm_stack_grad_workspace_size", "ssm_stack_grad",
    "ssm_lm_head_grad_workspace_size", "ssm_lm_head_grad",
    "ssm_timing_enable", "ssm_timing_summary",
    "ssm_last_error",
)


class SsmError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {msg}")
        self.status = status


class SsmDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int64), ("seqlen", ctypes.c_int64), ("channels", ctypes.c_int64),
                ("dstate", ctypes.c_int64), ("chunk", ctypes.c_int64), ("in_dtype", ctypes.c_int32),
                ("flags", ctypes.c_uint32)]


_lib = None


def load_library():
    """Load ``libssm_adjoint.so``; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not LIB_PATH.exists():
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2501_00692_amd.build` "
                           "(there is no fallback implementation)")
    lib = ctypes.CDLL(str(LIB_PATH))
    vp, i64, i32, u32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
    dp = ctypes.POINTER(SsmDesc)
    szp = ctypes.POINTER(ctypes.c_size_t)
    sig = {
        "ssm_adjoint_forward_workspace_size": [dp, szp],
        "ssm_adjoint_grad_workspace_size": [dp, i32, i64, szp],
        "ssm_adjoint_forward": [dp] + [vp] * 9 + [vp, sz, vp],
        "ssm_adjoint_grad": [dp, i32, i64] + [vp] * 16 + [vp, sz, vp],
        "ssm_adjoint_grad_noalloc": [dp, i32, i64] + [vp] * 16 + [vp],
        "ssm_adjoint_grad_pairs_workspace_size": [dp, i32, i64, szp],
        "ssm_adjoint_grad_pairs": [dp, i32, i64] + [vp] * 16 + [vp, sz, vp],
        "ssm_unstructured_grad_workspace_size": [dp, i32, i64, szp],
        "ssm_unstructured_grad": [dp, i32, i64] + [vp] * 11 + [vp, sz, vp],
        "ssm_proj_grad_workspace_size": [i64, i64, i64, u32, szp],
        "ssm_proj_grad": [i64, i64, i64, vp, i64, vp, i64, vp, i64, vp, vp, u32, vp, sz, vp],
        "ssm_layer_grad_workspace_size": [dp, i32, i64, i64, szp],
        "ssm_layer_grad": [dp, i32, i64, i64] + [vp] * 20 + [vp, sz, vp],
        "ssm_stack_grad_workspace_size": [dp, i64, i32, i32, i64, szp],
        "ssm_stack_grad": [dp, i64, i32, i32, i64] + [vp] * 9 + [vp, sz, vp],
        "ssm_lm_head_grad_workspace_size": [i64, i64, i64, u32, i64, szp],
        "ssm_lm_head_grad": [i64, i64, i64, u32, i64] + [vp] * 6 + [vp, sz, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.ssm_timing_enable.argtypes = [i32]
    lib.ssm_timing_enable.restype = ctypes.c_int
    lib.ssm_timing_summary.argtypes = [ctypes.c_char_p, sz]
    lib.ssm_timing_summary.restype = ctypes.c_int
    lib.ssm_last_error.argtypes = []
    lib.ssm_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().ssm_last_error().decode()


def timing_enable(on: bool = True):
    """Bracket every library kernel launch with hipEvents on its stream (profiling)."""
    load_library().ssm_timing_enable(1 if on else 0)


def timing_summary() -> dict:
    """Per-kernel ``{name: (launches, total_ms)}`` of the launches recorded since the
    last summary (waits for their events)."""
    buf = ctypes.create_string_buffer(1 << 16)
    rc = load_library().ssm_timing_summary(buf, len(buf))
    if rc != 0:
        raise SsmError(rc, "ssm_timing_summary", "event timing failed")
    out = {}
    for line in buf.value.decode().splitlines():
        name, n, ms = line.split()
        out[name] = (int(n), float(ms))
    return out


def _check(rc: int, where: str):
    if rc != 0:
        raise SsmError(rc, where, last_error())


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SSM_F32
    if t.dtype == torch.bfloat16:
        return SSM_BF16
    raise TypeError(f"activations must be float32 or bfloat16, got {t.dtype}")


def _need(t, name, dtype=None, shape=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def make_desc(x: torch.Tensor, N: int, softplus=False, gate=False, chunk=0, a_scalar=False,
              b_delta=False) -> SsmDesc:
    b, T, D = x.shape
    flags = ((SSM_DELTA_SOFTPLUS if softplus else 0) | (SSM_GATE_SILU if gate else 0) |
             (SSM_A_SCALAR if a_scalar else 0) | (SSM_B_DELTA if b_delta else 0))
    return SsmDesc(b, T, D, N, chunk, _dtype_code(x), flags)


def _alog_shape(A_log, D, N):
    """A_log is [D, N], or [D] for one decay rate per channel (the scalar variant)."""
    return (D,) if A_log.dim() == 1 else (D, N)


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns blocks aligned to at least 512 bytes
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def grad_workspace_size(desc: SsmDesc, tbar: int = 0, pairs: bool = False) -> int:
    n = ctypes.c_size_t()
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    name = "ssm_adjoint_grad_pairs_workspace_size" if pairs else "ssm_adjoint_grad_workspace_size"
    _check(getattr(load_library(), name)(ctypes.byref(desc), mode, int(tbar), ctypes.byref(n)), name)
    return n.value


def forward_workspace_size(desc: SsmDesc) -> int:
    n = ctypes.c_size_t()
    _check(load_library().ssm_adjoint_forward_workspace_size(ctypes.byref(desc), ctypes.byref(n)),
           "ssm_adjoint_forward_workspace_size")
    return n.value


def ssm_adjoint_forward(x, delta, A_log, B, C, h0=None, z=None, softplus=False, chunk=0, want_h_last=False,
                        workspace=None, b_delta=False):
    """Forward pass; returns ``y`` (and ``h_last`` if asked).  ``y`` has x's dtype.
    ``A_log`` of shape [D] selects one decay rate per channel; ``b_delta`` the
    input term Delta B x."""
    lib = load_library()
    dt = x.dtype
    b, T, D = x.shape
    N = B.shape[-1]
    _need(x, "x", dt)
    _need(delta, "delta", dt, (b, T, D))
    _need(A_log, "A_log", torch.float32, _alog_shape(A_log, D, N))
    _need(B, "B", dt, (b, T, N))
    _need(C, "C", dt, (b, T, N))
    _need(h0, "h0", torch.float32, (b, D, N))
    _need(z, "z", dt, (b, T, D))
    desc = make_desc(x, N, softplus, z is not None, chunk, A_log.dim() == 1, b_delta)
    n = ctypes.c_size_t()
    _check(lib.ssm_adjoint_forward_workspace_size(ctypes.byref(desc), ctypes.byref(n)),
           "ssm_adjoint_forward_workspace_size")
    ws = workspace if workspace is not None else _workspace(n.value, x.device)
    y = torch.empty_like(x)
    h_last = torch.empty(b, D, N, dtype=torch.float32, device=x.device) if want_h_last else None
    _check(lib.ssm_adjoint_forward(ctypes.byref(desc), _p(x), _p(delta), _p(A_log), _p(B), _p(C), _p(h0), _p(z),
                                   _p(y), _p(h_last), _p(ws), ws.numel(), _stream()), "ssm_adjoint_forward")
    return (y, h_last) if want_h_last else y


def ssm_adjoint_grad(x, delta, A_log, B, C, dy, h0=None, z=None, softplus=False, tbar=0, chunk=0,
                     want_dh0=False, out=None, workspace=None, b_delta=False, want_da=False):
    """Per-layer adjoint gradient.  ``tbar > 0`` selects the truncated form.
    ``A_log`` of shape [D] selects one decay rate per channel (and dA_log is [D]);
    ``b_delta`` the input term Delta B x.

    Returns a dict with fp32 ``dx, ddelta, dA_log, dB, dC`` (+ ``dz`` with a gate,
    ``dh0`` if asked, the debug output ``da`` [b, T, D, N] if ``want_da``).  ``out``
    may hold preallocated outputs under the same keys."""
    return _adjoint_grad(False, x, delta, A_log, B, C, dy, h0, z, softplus, tbar, chunk, want_dh0, out, workspace,
                         b_delta, want_da=want_da)


def ssm_adjoint_grad_noalloc(x, delta, A_log, B, C, dy, h0=None, z=None, softplus=False, tbar=0, chunk=0,
                             want_dh0=False, out=None, b_delta=False, want_da=False):
    """:func:`ssm_adjoint_grad` through the C entry point that takes no workspace
    (its scratch is a fixed device array inside the library); arguments and
    results as there.  Raises :class:`SsmError` with SSM_ERR_WORKSPACE when the
    problem needs more scratch than the library holds."""
    return _adjoint_grad(False, x, delta, A_log, B, C, dy, h0, z, softplus, tbar, chunk, want_dh0, out, None,
                         b_delta, noalloc=True, want_da=want_da)


def ssm_adjoint_grad_pairs(x, delta, A_log, B, C, dy, h0=None, z=None, softplus=False, tbar=0, chunk=0,
                           want_dh0=False, out=None, workspace=None, b_delta=False, want_da=False):
    """The same gradient as :func:`ssm_adjoint_grad`, evaluated by the explicit
    pair formulation (every adjoint state of the window formed and its VJPs
    accumulated); arguments and results as there."""
    return _adjoint_grad(True, x, delta, A_log, B, C, dy, h0, z, softplus, tbar, chunk, want_dh0, out, workspace,
                         b_delta, want_da=want_da)


def _adjoint_grad(pairs, x, delta, A_log, B, C, dy, h0, z, softplus, tbar, chunk, want_dh0, out, workspace,
                  b_delta, noalloc=False, want_da=False):
    lib = load_library()
    dt = x.dtype
    b, T, D = x.shape
    N = B.shape[-1]
    _need(x, "x", dt)
    _need(delta, "delta", dt, (b, T, D))
    _need(A_log, "A_log", torch.float32, _alog_shape(A_log, D, N))
    _need(B, "B", dt, (b, T, N))
    _need(C, "C", dt, (b, T, N))
    _need(dy, "dy", dt, (b, T, D))
    _need(h0, "h0", torch.float32, (b, D, N))
    _need(z, "z", dt, (b, T, D))
    desc = make_desc(x, N, softplus, z is not None, chunk, A_log.dim() == 1, b_delta)
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    dev = x.device
    f32 = dict(dtype=torch.float32, device=dev)
    o = dict(out) if out else {}
    o.setdefault("dx", torch.empty(b, T, D, **f32))
    o.setdefault("ddelta", torch.empty(b, T, D, **f32))
    o.setdefault("dA_log", torch.empty(*A_log.shape, **f32))
    o.setdefault("dB", torch.empty(b, T, N, **f32))
    o.setdefault("dC", torch.empty(b, T, N, **f32))
    if z is not None:
        o.setdefault("dz", torch.empty(b, T, D, **f32))
    if want_dh0:
        o.setdefault("dh0", torch.empty(b, D, N, **f32))
    if want_da:
        o.setdefault("da", torch.empty(b, T, D, N, **f32))
    args = (ctypes.byref(desc), mode, int(tbar), _p(x), _p(delta), _p(A_log), _p(B), _p(C), _p(h0), _p(z), _p(dy),
            _p(o["dx"]), _p(o["ddelta"]), _p(o["dA_log"]), _p(o["dB"]), _p(o["dC"]), _p(o.get("dz")),
            _p(o.get("dh0")), _p(o.get("da")))
    if noalloc:
        _check(lib.ssm_adjoint_grad_noalloc(*args, _stream()), "ssm_adjoint_grad_noalloc")
        return o
    ws = workspace if workspace is not None else _workspace(grad_workspace_size(desc, tbar, pairs), dev)
    name = "ssm_adjoint_grad_pairs" if pairs else "ssm_adjoint_grad"
    _check(getattr(lib, name)(*args, _p(ws), ws.numel(), _stream()), name)
    return o


def ssm_unstructured_grad(A, B, C, x, dy, h0=None, tbar=0, chunk=0, want_dh0=False, out=None, workspace=None):
    """Adjoint gradient of the unstructured SSM (16 states, per-step matrices
    A [b,T,16,16], B [b,T,16,P], C [b,T,P,16]; x, dy [b,T,P]; fp32).  Returns a dict
    with ``dA, dB, dC, dx`` (+ ``dh0`` if asked, full mode)."""
    lib = load_library()
    b, T, N, P = B.shape
    f32 = torch.float32
    _need(A, "A", f32, (b, T, N, N))
    _need(B, "B", f32)
    _need(C, "C", f32, (b, T, P, N))
    _need(x, "x", f32, (b, T, P))
    _need(dy, "dy", f32, (b, T, P))
    _need(h0, "h0", f32, (b, N))
    desc = SsmDesc(b, T, P, N, chunk, SSM_F32, 0)
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    n = ctypes.c_size_t()
    _check(lib.ssm_unstructured_grad_workspace_size(ctypes.byref(desc), mode, int(tbar), ctypes.byref(n)),
           "ssm_unstructured_grad_workspace_size")
    ws = workspace if workspace is not None else _workspace(n.value, A.device)
    o = dict(out) if out else {}
    for k, t in (("dA", A), ("dB", B), ("dC", C), ("dx", x)):
        o.setdefault(k, torch.empty_like(t))
    if want_dh0:
        o.setdefault("dh0", torch.empty(b, N, dtype=f32, device=A.device))
    _check(lib.ssm_unstructured_grad(ctypes.byref(desc), mode, int(tbar), _p(A), _p(B), _p(C), _p(x), _p(h0), _p(dy),
                                     _p(o["dA"]), _p(o["dB"]), _p(o["dC"]), _p(o["dx"]), _p(o.get("dh0")), _p(ws),
                                     ws.numel(), _stream()), "ssm_unstructured_grad")
    return o


def ssm_proj_grad(X, dZ, W=None, want_dW=True, want_dX=False, dW=None, dX=None, accum_dW=False,
                  accum_dX=False):
    """``dW = X^T dZ`` and/or ``dX = dZ W^T`` (bf16 operands, fp32 results)."""
    lib = load_library()
    M, Nout = dZ.shape
    _need(dZ, "dZ", torch.bfloat16)
    K = (X.shape[1] if X is not None else W.shape[0])
    if want_dW:
        _need(X, "X", torch.bfloat16, (M, K))
        dW = dW if dW is not None else torch.empty(K, Nout, dtype=torch.float32, device=dZ.device)
    if want_dX:
        _need(W, "W", torch.bfloat16, (K, Nout))
        dX = dX if dX is not None else torch.empty(M, K, dtype=torch.float32, device=dZ.device)
    flags = (SSM_ACCUM_DW if accum_dW else 0) | (SSM_ACCUM_DX if accum_dX else 0)
    n = ctypes.c_size_t()
    _check(lib.ssm_proj_grad_workspace_size(M, K, Nout, flags, ctypes.byref(n)), "ssm_proj_grad_workspace_size")
    ws = _workspace(n.value, dZ.device)
    _check(lib.ssm_proj_grad(M, K, Nout, _p(X if want_dW else None), K, _p(dZ), Nout, _p(W if want_dX else None),
                             Nout, _p(dW if want_dW else None), _p(dX if want_dX else None), flags, _p(ws),
                             ws.numel(), _stream()), "ssm_proj_grad")
    return (dW if want_dW else None), (dX if want_dX else None)


def layer_workspace_size(desc: SsmDesc, tbar: int, d_model: int) -> int:
    n = ctypes.c_size_t()
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    _check(load_library().ssm_layer_grad_workspace_size(ctypes.byref(desc), mode, int(tbar), int(d_model),
                                                        ctypes.byref(n)), "ssm_layer_grad_workspace_size")
    return n.value


def ssm_layer_grad(u, x, z, delta_pre, B, C, W_x, W_in, A_log, dy, tbar=0, chunk=0, want_du=False,
                   want_scan=False, out=None, workspace=None, b_delta=False):
    """Whole-layer gradient with input projections (bf16 activations).

    Returns a dict with fp32 ``dW_in, dW_x, dA_log`` (+ ``du`` if asked; + the scan
    gradients ``dx, ddelta, dB, dC, dz`` and ``dx_total`` if ``want_scan``)."""
    lib = load_library()
    b, T, D = x.shape
    N = B.shape[-1]
    dm = u.shape[-1]
    bf = torch.bfloat16
    _need(u, "u", bf, (b, T, dm))
    _need(x, "x", bf)
    _need(z, "z", bf, (b, T, D))
    _need(delta_pre, "delta_pre", bf, (b, T, D))
    _need(B, "B", bf, (b, T, N))
    _need(C, "C", bf, (b, T, N))
    _need(W_x, "W_x", bf, (D, D + 2 * N))
    _need(W_in, "W_in", bf, (dm, 2 * D))
    _need(A_log, "A_log", torch.float32, _alog_shape(A_log, D, N))
    _need(dy, "dy", bf, (b, T, D))
    desc = make_desc(x, N, True, True, chunk, A_log.dim() == 1, b_delta)
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    dev = x.device
    f32 = dict(dtype=torch.float32, device=dev)
    o = dict(out) if out else {}
    o.setdefault("dW_in", torch.empty(dm, 2 * D, **f32))
    o.setdefault("dW_x", torch.empty(D, D + 2 * N, **f32))
    o.setdefault("dA_log", torch.empty(*A_log.shape, **f32))
    if want_du:
        o.setdefault("du", torch.empty(b, T, dm, **f32))
    if want_scan:
        for k, shp in (("dx", (b, T, D)), ("ddelta", (b, T, D)), ("dB", (b, T, N)), ("dC", (b, T, N)),
                       ("dz", (b, T, D)), ("dx_total", (b, T, D))):
            o.setdefault(k, torch.empty(*shp, **f32))
    ws = workspace if workspace is not None else _workspace(layer_workspace_size(desc, tbar, dm), dev)
    _check(lib.ssm_layer_grad(ctypes.byref(desc), mode, int(tbar), dm, _p(u), _p(x), _p(z), _p(delta_pre), _p(B),
                              _p(C), _p(W_x), _p(W_in), _p(A_log), _p(dy), _p(o["dW_in"]), _p(o["dW_x"]),
                              _p(o["dA_log"]), _p(o.get("du")), _p(o.get("dx")), _p(o.get("ddelta")), _p(o.get("dB")),
                              _p(o.get("dC")), _p(o.get("dz")), _p(o.get("dx_total")), _p(ws), ws.numel(),
                              _stream()), "ssm_layer_grad")
    return o


def _ptr_array(ts):
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])


def stack_workspace_size(desc: SsmDesc, K: int, grad: int, tbar: int = 0) -> int:
    n = ctypes.c_size_t()
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    _check(load_library().ssm_stack_grad_workspace_size(ctypes.byref(desc), int(K), int(grad), mode, int(tbar),
                                                        ctypes.byref(n)), "ssm_stack_grad_workspace_size")
    return n.value


def ssm_stack_grad(y0, W_in, W_x, A_log, gK, N, exact=False, tbar=0, chunk=0, want_yK=False, out=None,
                   workspace=None, forward_only=False):
    """Parameter gradients of a K-layer residual stack (lists ``W_in``, ``W_x``,
    ``A_log`` of K tensors) for the upstream ``gK = dL/dy_K``: Prop. 3 (each layer
    under gK, ``exact=False``) or backpropagation (``exact=True``).  ``y0`` and
    ``gK`` are fp32 [b, T, D]; the projections bf16.  Returns a dict with lists
    ``dW_in, dW_x, dA_log`` (+ ``yK`` if asked).  ``forward_only`` runs the
    forward alone (SSM_STACK_FORWARD; gK may be None) and returns ``yK`` only."""
    lib = load_library()
    b, T, D = y0.shape
    K = len(W_in)
    assert len(W_x) == K and len(A_log) == K
    _need(y0, "y0", torch.float32)
    if not forward_only:
        _need(gK, "gK", torch.float32, (b, T, D))
    for k in range(K):
        _need(W_in[k], "W_in[k]", torch.bfloat16, (D, 2 * D))
        _need(W_x[k], "W_x[k]", torch.bfloat16, (D, D + 2 * N))
        _need(A_log[k], "A_log[k]", torch.float32, (D, N))
    desc = SsmDesc(b, T, D, N, chunk, SSM_BF16, 0)
    grad = SSM_STACK_FORWARD if forward_only else (SSM_STACK_EXACT if exact else SSM_STACK_ADJOINT)
    mode = SSM_TRUNCATED if tbar > 0 else SSM_FULL
    dev = y0.device
    f32 = dict(dtype=torch.float32, device=dev)
    o = dict(out) if out else {}
    if not forward_only:
        o.setdefault("dW_in", [torch.empty(D, 2 * D, **f32) for _ in range(K)])
        o.setdefault("dW_x", [torch.empty(D, D + 2 * N, **f32) for _ in range(K)])
        o.setdefault("dA_log", [torch.empty(D, N, **f32) for _ in range(K)])
    else:
        o = {k: v for k, v in o.items() if k == "yK"}
    if want_yK or forward_only:
        o.setdefault("yK", torch.empty(b, T, D, **f32))
    ws = workspace if workspace is not None else _workspace(stack_workspace_size(desc, K, grad, tbar), dev)
    keep = [_ptr_array(W_in), _ptr_array(W_x), _ptr_array(A_log)]
    keep += [None] * 3 if forward_only else [_ptr_array(o["dW_in"]), _ptr_array(o["dW_x"]), _ptr_array(o["dA_log"])]
    _check(lib.ssm_stack_grad(ctypes.byref(desc), K, grad, mode, int(tbar), _p(y0), *[ctypes.cast(a, ctypes.c_void_p)
                                                                                    for a in keep[:3]],
                              _p(gK), *[ctypes.cast(a, ctypes.c_void_p) for a in keep[3:]], _p(o.get("yK")), _p(ws),
                              ws.numel(), _stream()), "ssm_stack_grad")
    return o


def ssm_lm_head_grad(y, omega, targets, norm=True, want_domega=True, block_rows=0, out=None, workspace=None):
    """Language head with the cross-entropy loss: y fp32 [M, P], omega bf16
    [V, P], targets int32 [M] (negative: no loss).  Returns a dict with ``loss``
    [M], ``dy`` [M, P] and (if asked) ``domega`` [V, P], all fp32."""
    lib = load_library()
    M, P = y.shape
    V = omega.shape[0]
    _need(y, "y", torch.float32, (M, P))
    _need(omega, "omega", torch.bfloat16, (V, P))
    _need(targets, "targets", torch.int32, (M,))
    flags = SSM_HEAD_NORM if norm else 0
    n = ctypes.c_size_t()
    _check(lib.ssm_lm_head_grad_workspace_size(M, P, V, flags, int(block_rows), ctypes.byref(n)),
           "ssm_lm_head_grad_workspace_size")
    ws = workspace if workspace is not None else _workspace(n.value, y.device)
    o = dict(out) if out else {}
    o.setdefault("loss", torch.empty(M, dtype=torch.float32, device=y.device))
    o.setdefault("dy", torch.empty(M, P, dtype=torch.float32, device=y.device))
    if want_domega:
        o.setdefault("domega", torch.empty(V, P, dtype=torch.float32, device=y.device))
    _check(lib.ssm_lm_head_grad(M, P, V, flags, int(block_rows), _p(y), _p(omega), _p(targets), _p(o["loss"]), _p(o["dy"]),
                                _p(o.get("domega")), _p(ws), ws.numel(), _stream()), "ssm_lm_head_grad")
    return o
