"""C-ABI contract checks that need no GPU: the library loads, exports every
function the header declares, and rejects bad arguments on the host (before
any HIP call) with the documented status codes."""
import ctypes
import os
import re

import pytest

import paper_2501_00692_amd as ssm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssm_adjoint.h")


@pytest.fixture(scope="module")
def lib():
    if not ssm.LIB_PATH.exists():
        pytest.fail("libssm_adjoint.so is not built (run __graft_entry__.build())")
    return ssm.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssm_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert sorted(ssm.EXPORTED) == declared_functions()


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_binding_declares_every_signature(lib):
    # without argtypes ctypes would pass 64-bit sizes as C ints
    for name in ssm.EXPORTED:
        assert getattr(lib, name).argtypes is not None, name


def desc(**kw):
    d = dict(batch=1, seqlen=256, channels=64, dstate=16, chunk=0, in_dtype=ssm.SSM_F32, flags=0)
    d.update(kw)
    return ssm.SsmDesc(**d)


FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: every call below fails validation
MISALIGNED = ctypes.c_void_p(0x100004)


def grad_call(lib, dsc, mode=ssm.SSM_FULL, tbar=0, x=FAKE, dh0=None, z=None, dz=None, ws=FAKE,
              ws_bytes=1 << 40, entry="ssm_adjoint_grad", da=None):
    return getattr(lib, entry)(ctypes.byref(dsc) if dsc is not None else None, mode, tbar, x, FAKE, FAKE, FAKE,
                               FAKE, None, z, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, dz, dh0, da, ws, ws_bytes, None)


GRAD_ENTRIES = ["ssm_adjoint_grad", "ssm_adjoint_grad_pairs"]


@pytest.mark.parametrize("entry", GRAD_ENTRIES)
def test_null_and_shape_errors(lib, entry):
    call = lambda *a, **k: grad_call(*a, entry=entry, **k)
    assert call(lib, None) == 1
    assert "desc" in ssm.last_error()
    assert call(lib, desc(batch=0)) == 2
    assert call(lib, desc(seqlen=0)) == 2
    assert call(lib, desc(dstate=17)) == 4
    assert call(lib, desc(in_dtype=7)) == 3
    assert call(lib, desc(chunk=100)) == 4
    assert call(lib, desc(flags=16)) == 2
    assert call(lib, desc(), x=None) == 1
    assert "x is NULL" in ssm.last_error()
    assert call(lib, desc(), x=MISALIGNED) == 6
    assert call(lib, desc(), da=MISALIGNED) == 6


@pytest.mark.parametrize("entry", GRAD_ENTRIES)
def test_mode_errors(lib, entry):
    call = lambda *a, **k: grad_call(*a, entry=entry, **k)
    assert call(lib, desc(), mode=5) == 2
    assert call(lib, desc(), mode=ssm.SSM_TRUNCATED, tbar=0) == 2
    # dh0 exists for the full gradient only
    assert call(lib, desc(), mode=ssm.SSM_TRUNCATED, tbar=32, dh0=FAKE) == 4
    # gate flag and z must agree
    assert call(lib, desc(flags=ssm.SSM_GATE_SILU)) == 1
    assert call(lib, desc(), z=FAKE, dz=FAKE) == 2


@pytest.mark.parametrize("entry", GRAD_ENTRIES)
def test_workspace_errors(lib, entry):
    d = desc()
    assert grad_call(lib, d, ws=None, entry=entry) == 5
    assert grad_call(lib, d, ws_bytes=16, entry=entry) == 5
    assert grad_call(lib, d, ws=ctypes.c_void_p(0x100010), entry=entry) == 6


def test_workspace_queries(lib):
    n = ctypes.c_size_t()
    d = desc()
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(d), ssm.SSM_FULL, 0, ctypes.byref(n)) == 0
    full = n.value
    assert full > 0
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(d), ssm.SSM_TRUNCATED, 32, ctypes.byref(n)) == 0
    assert n.value >= full
    # tbar >= T is the full gradient
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(d), ssm.SSM_TRUNCATED, 256, ctypes.byref(n)) == 0
    assert n.value == full
    assert lib.ssm_adjoint_forward_workspace_size(ctypes.byref(d), ctypes.byref(n)) == 0
    assert 0 < n.value <= full
    assert lib.ssm_adjoint_grad_pairs_workspace_size(ctypes.byref(d), ssm.SSM_TRUNCATED, 32, ctypes.byref(n)) == 0
    assert n.value > 0
    assert lib.ssm_adjoint_grad_pairs_workspace_size(ctypes.byref(d), ssm.SSM_TRUNCATED, 0, ctypes.byref(n)) == 2
    assert lib.ssm_proj_grad_workspace_size(8192, 1536, 1568, 0, ctypes.byref(n)) == 0
    assert lib.ssm_proj_grad_workspace_size(0, 1, 1, 0, ctypes.byref(n)) == 2
    # the channel limit: chunk byte offsets stay 32-bit
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(desc(channels=1 << 20)), ssm.SSM_FULL, 0,
                                               ctypes.byref(n)) == 0
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(desc(channels=(1 << 20) + 1)), ssm.SSM_FULL, 0,
                                               ctypes.byref(n)) == 2
    ld = desc(batch=2, seqlen=4096, channels=1536, in_dtype=ssm.SSM_BF16)
    assert lib.ssm_layer_grad_workspace_size(ctypes.byref(ld), ssm.SSM_FULL, 0, 768, ctypes.byref(n)) == 0
    assert n.value > 0


def test_proj_errors(lib):
    call = lambda M, K, N, X=FAKE, dZ=FAKE, W=None, dW=FAKE, dX=None, ldx=None: lib.ssm_proj_grad(
        M, K, N, X, ldx if ldx is not None else K, dZ, N, W, N, dW, dX, 0, FAKE, 1 << 40, None)
    assert call(0, 8, 8) == 2
    assert call(16, 12, 8) == 4          # K must be a multiple of 8
    assert call(16, 8, 8, dZ=None) == 1
    assert call(16, 8, 8, dX=FAKE) == 1  # dX needs W
    assert call(16, 8, 8, ldx=4) == 2
    assert call(16, 8, 8, ldx=(1 << 21) + 8) == 2  # strides past the 32-bit tile offsets


def test_layer_rejects_fp32(lib):
    d = desc()
    rc = lib.ssm_layer_grad(ctypes.byref(d), 0, 0, 64, *([FAKE] * 13), *([None] * 7), FAKE, 1 << 40, None)
    assert rc == 4


def test_stack_errors(lib):
    d = desc(in_dtype=ssm.SSM_BF16)
    arr = (ctypes.c_void_p * 2)(FAKE.value, FAKE.value)

    def call(dsc=d, K=2, grad=ssm.SSM_STACK_ADJOINT, mode=ssm.SSM_FULL, tbar=0, y0=FAKE, ws_bytes=1 << 40, W=arr):
        return lib.ssm_stack_grad(ctypes.byref(dsc), K, grad, mode, tbar, y0, W, arr, arr, FAKE, arr, arr, arr,
                                  None, FAKE, ws_bytes, None)
    assert call(K=0) == 2
    assert call(grad=5) == 2
    assert call(dsc=desc()) == 4                                     # fp32 activations
    assert call(dsc=desc(in_dtype=ssm.SSM_BF16, flags=ssm.SSM_A_SCALAR)) == 4
    assert call(dsc=desc(in_dtype=ssm.SSM_BF16, dstate=3)) == 4      # D + 2N not a multiple of 8
    assert call(mode=ssm.SSM_TRUNCATED, tbar=0) == 2
    assert call(y0=None) == 1
    assert call(W=None) == 1
    assert call(ws_bytes=16) == 5
    # the forward alone needs yK (the call above passes NULL) and nothing of the gradients
    assert call(grad=ssm.SSM_STACK_FORWARD) == 1 and "yK" in ssm.last_error()
    assert lib.ssm_stack_grad(ctypes.byref(d), 2, ssm.SSM_STACK_FORWARD, ssm.SSM_FULL, 0, FAKE, arr, arr, arr, None,
                              None, None, None, FAKE, FAKE, 16, None) == 5
    n = ctypes.c_size_t()
    assert lib.ssm_stack_grad_workspace_size(ctypes.byref(d), 3, ssm.SSM_STACK_EXACT, ssm.SSM_FULL, 0,
                                             ctypes.byref(n)) == 0
    three = n.value
    assert lib.ssm_stack_grad_workspace_size(ctypes.byref(d), 1, ssm.SSM_STACK_EXACT, ssm.SSM_FULL, 0,
                                             ctypes.byref(n)) == 0
    assert 0 < n.value < three


def noalloc_call(lib, dsc, mode=ssm.SSM_FULL, tbar=0, x=FAKE):
    return lib.ssm_adjoint_grad_noalloc(ctypes.byref(dsc) if dsc is not None else None, mode, tbar, x, FAKE, FAKE,
                                        FAKE, FAKE, None, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None,
                                        None)


def test_noalloc_host_errors(lib):
    """The entry point without a workspace validates like ssm_adjoint_grad and
    rejects problems whose scratch exceeds its fixed array, all before any HIP
    call (these run without a GPU)."""
    assert noalloc_call(lib, None) == 1
    assert noalloc_call(lib, desc(batch=0)) == 2
    assert noalloc_call(lib, desc(), x=None) == 1
    assert noalloc_call(lib, desc(), x=MISALIGNED) == 6
    assert noalloc_call(lib, desc(), mode=ssm.SSM_TRUNCATED, tbar=0) == 2
    big = desc(batch=8, seqlen=65536, channels=4096, in_dtype=ssm.SSM_BF16)
    n = ctypes.c_size_t()
    assert lib.ssm_adjoint_grad_workspace_size(ctypes.byref(big), ssm.SSM_FULL, 0, ctypes.byref(n)) == 0
    assert n.value > (64 << 20)
    assert noalloc_call(lib, big) == 5
    assert "no-allocation" in ssm.last_error()


def test_head_errors(lib):
    n = ctypes.c_size_t()
    ok = lambda M, P, V, flags=ssm.SSM_HEAD_NORM, rows=0: lib.ssm_lm_head_grad_workspace_size(
        M, P, V, flags, rows, ctypes.byref(n))
    assert ok(4096, 1536, 32000) == 0 and n.value > 1536 * 32000 * 2 + 4096 * 32000 * 6
    assert ok(4096, 1536, 32000, rows=512) == 0 and n.value < 1536 * 32000 * 2 + 1024 * 32000 * 6
    assert ok(4096, 64, 64, rows=100) == 2
    assert ok(0, 64, 64) == 2
    assert ok(64, 64, 64, flags=2) == 2
    assert ok(64, 60, 64) == 4 and "multiples of 8" in ssm.last_error()
    assert ok(64, 64, 1001) == 4
    assert lib.ssm_lm_head_grad_workspace_size(64, 64, 64, 0, 0, None) == 1
    call = lambda y=FAKE, om=FAKE, t=FAKE, loss=FAKE, dy=FAKE, dom=None, ws=FAKE, wsb=1 << 40: lib.ssm_lm_head_grad(
        256, 64, 128, ssm.SSM_HEAD_NORM, 0, y, om, t, loss, dy, dom, ws, wsb, None)
    assert call(y=None) == 1 and "y is NULL" in ssm.last_error()
    assert call(t=None) == 1
    assert call(dy=None) == 1
    assert call(dom=MISALIGNED) == 6
    assert call(ws=None) == 5
    assert call(wsb=1024) == 5


def test_unstructured_errors(lib):
    """The unstructured SSM (Table 1's N x N row) validates on the host: 16
    states, channels a multiple of 16 up to 4,096, fp32 tensors, no flags, a
    supported chunk, a known mode, tbar >= 1 when truncated, dh0 for the full
    gradient only, required and aligned pointers and the workspace, all before any
    HIP call (every call below fails validation, so nothing is enqueued)."""
    n = ctypes.c_size_t()
    ud = lambda **kw: desc(**{"channels": 64, **kw})
    size = lambda d, mode=ssm.SSM_FULL, tbar=0: lib.ssm_unstructured_grad_workspace_size(
        ctypes.byref(d) if d is not None else None, mode, tbar, ctypes.byref(n))
    assert size(ud()) == 0 and n.value > 0
    full = n.value
    assert size(ud(), ssm.SSM_TRUNCATED, 16) == 0 and n.value >= full
    assert size(None) == 1
    assert size(ud(batch=0)) == 2
    assert size(ud(dstate=8)) == 4 and "dstate = 16" in ssm.last_error()
    assert size(ud(channels=24)) == 4
    assert size(ud(channels=4112)) == 4
    assert size(ud(in_dtype=ssm.SSM_BF16)) == 4 and "fp32" in ssm.last_error()
    assert size(ud(flags=ssm.SSM_GATE_SILU)) == 4
    assert size(ud(chunk=48)) == 4
    assert size(ud(), mode=5) == 2
    assert size(ud(), ssm.SSM_TRUNCATED, 0) == 2
    assert lib.ssm_unstructured_grad_workspace_size(ctypes.byref(ud()), ssm.SSM_FULL, 0, None) == 1

    def call(d=None, mode=ssm.SSM_FULL, tbar=0, A=FAKE, x=FAKE, dh0=None, ws=FAKE, wsb=1 << 40):
        d = d if d is not None else ud()
        return lib.ssm_unstructured_grad(ctypes.byref(d), mode, tbar, A, FAKE, FAKE, x, None, FAKE, FAKE, FAKE,
                                         FAKE, FAKE, dh0, ws, wsb, None)

    assert call(d=ud(dstate=4)) == 4
    assert call(A=None) == 1 and "A is NULL" in ssm.last_error()
    assert call(x=MISALIGNED) == 6
    assert call(dh0=MISALIGNED) == 6
    assert call(mode=ssm.SSM_TRUNCATED, tbar=16, dh0=FAKE) == 4 and "full gradient" in ssm.last_error()
    assert call(ws=None) == 5
    assert call(wsb=16) == 5
