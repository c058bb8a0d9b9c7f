"""Host-side checks of the C ABI (no GPU needed, nothing is launched).

The library loads, exports every symbol the public header declares, and rejects
invalid arguments with the documented status before touching the device.
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hqlss.h")

import torch  # noqa: E402

# Host-only: these calls pass fake device pointers that must be rejected by validation.
# Never run them where a GPU is visible, so that a validation slip cannot launch.
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="host-only ABI validation checks (fake pointers)")

H = pytest.importorskip("paper_2306_11987_amd", reason="libhqlss.so not built")
lib = H.lib

OK, NULL, SHAPE, BLOCK, ALIGN, DTYPE, WS, OVF, HIP, ARG, SCRATCH = range(11)


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    names = re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", txt)
    skip = {"if", "sizeof", "defined"}
    return sorted({n for n in names if n not in skip and (n.startswith("hq") or n.startswith("lss"))})


def test_exports_every_declared_symbol():
    fns = declared_functions()
    assert len(fns) >= 13
    raw = ctypes.CDLL(H._binding.LIB_PATH)
    for name in fns:
        assert hasattr(raw, name), f"missing export {name}"


def test_status_strings():
    for s in range(11):
        assert H.status_string(s) and H.status_string(s) != "unknown status"
    assert H.status_string(99) == "unknown status"


def test_backward_workspace_shares_the_int8_operand():
    """dX and dW read one int8 operand A_T (dW reads it k-major): the combined backward needs
    at least round_up(N, 128) x C bytes less than the two single-gradient calls together
    (each of which also carries the sample's own buffers)."""
    for N, D, C in ((128, 256, 256), (16384, 768, 3072), (16384, 4096, 11008), (300, 1024, 384)):
        kp = (N + 127) // 128 * 128
        dx = H.workspace_bytes(H.WS_BWD_DX, N, D, C)
        dw = H.workspace_bytes(H.WS_BWD_DW, N, D, C)
        both = H.workspace_bytes(H.WS_BWD, N, D, C)
        assert max(dx, dw) <= both < dx + dw
        assert dx + dw - both >= kp * C


def test_workspace_sizes_monotone():
    for which in range(5):
        a = H.workspace_bytes(which, 128, 256, 256)
        b = H.workspace_bytes(which, 16384, 768, 3072)
        assert b >= a >= 0
    assert H.workspace_bytes(H.WS_FWD, 128, 256, 256) == H.workspace_bytes(H.WS_FWD, 16384, 768, 3072) > 0
    assert H.workspace_bytes(H.WS_PLAN, 128, 256, 256) > 0
    assert H.workspace_bytes(H.WS_BWD, 128, 256, 256) >= H.workspace_bytes(H.WS_BWD_DX, 128, 256, 256)
    assert H.workspace_bytes(H.WS_BWD, 0, 256, 256) == 0


def test_philox_offset_advance():
    assert H.lss_philox_offset_advance(128, 256) == 128 * 256 // 8
    assert H.lss_philox_offset_advance(3, 64) == 24
    assert H.lss_philox_offset_advance(1, 72) == 9


_Saved = H._binding._SavedC  # the hqlss_saved_t mirror of the binding


FAKE = 0x10000  # never dereferenced: every call below must fail validation first


def _saved(**over):
    s = _Saved(FAKE, FAKE, FAKE, FAKE, FAKE)
    for k, v in over.items():
        setattr(s, k, v)
    return s


def fwd(X=FAKE, W=FAKE, Y=FAKE, N=128, D=256, C=256, dt=0, k=5, saved=None):
    s = saved if saved is not None else _saved()
    return lib.hq_linear_fwd(X, W, Y, N, D, C, dt, k, ctypes.byref(s), FAKE, 1 << 40, None)


def test_fwd_argument_errors():
    assert fwd(X=None) == NULL
    assert fwd(saved=_saved(wqT=None)) == NULL
    assert fwd(N=0) == SHAPE
    assert fwd(D=100) == SHAPE
    assert fwd(C=32) == SHAPE
    assert fwd(k=8) == BLOCK
    assert fwd(k=-1) == BLOCK
    assert fwd(D=192, k=7) == BLOCK  # 192 % 128 != 0
    assert fwd(dt=3) == DTYPE
    assert fwd(X=FAKE + 4) == ALIGN
    assert fwd(saved=_saved(xq=FAKE + 8)) == ALIGN
    assert fwd(D=1 << 20, C=64, N=1) == OVF  # 256 * 49 * D >= 2^31
    s = _saved()
    assert lib.hq_linear_fwd(FAKE, FAKE, FAKE, 128, 256, 256, 0, 5, ctypes.byref(s), None, 0, None) == WS
    assert lib.hq_linear_fwd(FAKE, FAKE, FAKE, 128, 256, 256, 0, 5, ctypes.byref(s), FAKE, 16, None) == WS


def fwd_noalloc(X=FAKE, W=FAKE, Y=FAKE, N=128, D=256, C=256, dt=0, k=5, saved=None):
    s = saved if saved is not None else _saved()
    return lib.hq_linear_fwd_noalloc(X, W, Y, N, D, C, dt, k, ctypes.byref(s), None)


def test_fwd_noalloc_argument_errors():
    """The allocation-free forward validates as hq_linear_fwd does, and rejects shapes whose
    forward scratch exceeds the static array, before any HIP call."""
    txt = open(HEADER).read()
    m = re.search(r"#define HQLSS_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", txt)
    assert m and int(m.group(1)) << int(m.group(2)) == H.STATIC_SCRATCH_BYTES
    assert fwd_noalloc(X=None) == NULL
    assert fwd_noalloc(saved=_saved(wqT=None)) == NULL
    assert fwd_noalloc(N=0) == SHAPE
    assert fwd_noalloc(D=100) == SHAPE
    assert fwd_noalloc(k=8) == BLOCK
    assert fwd_noalloc(dt=3) == DTYPE
    assert fwd_noalloc(Y=FAKE + 4) == ALIGN
    assert fwd_noalloc(D=1 << 20, C=64, N=1) == OVF
    # small outputs over a long K split along K: their partials exceed the static array
    N, D, C = 2048, 16384, 2048
    assert H.workspace_bytes(H.WS_FWD, N, D, C) > H.STATIC_SCRATCH_BYTES
    assert fwd_noalloc(N=N, D=D, C=C) == SCRATCH
    assert H.workspace_bytes(H.WS_FWD, 16384, 4096, 4096) <= H.STATIC_SCRATCH_BYTES


def bwd(dY=FAKE, dX=FAKE, dW=FAKE, N=128, D=256, C=256, dt=0, k=5, budget=0, ws=FAKE, nbytes=1 << 40):
    s = _saved()
    return lib.lss_linear_bwd(dY, ctypes.byref(s), dX, dW, N, D, C, dt, k, budget, 0, 0, ws, nbytes, None)


def test_bwd_argument_errors():
    assert bwd(dX=None, dW=None) == NULL
    assert bwd(dY=None) == NULL
    assert bwd(N=-1) == SHAPE
    assert bwd(C=100) == SHAPE
    assert bwd(k=9) == BLOCK
    assert bwd(dt=7) == DTYPE
    assert bwd(dX=FAKE + 2) == ALIGN
    assert bwd(budget=1000) == ARG  # budget > 2N
    assert bwd(budget=-2) == ARG  # below HQLSS_BUDGET_KEEP_NONZERO
    assert bwd(ws=None) == WS
    assert bwd(nbytes=100) == WS
    assert bwd(N=70000) == SHAPE  # sampler limit
    assert bwd(N=1, C=1 << 20, D=64, k=0) == OVF  # 16 * 882 * C >= 2^31
    assert bwd(N=16384 + 8192, C=256, D=256, k=7) == OVF  # 128 * 882 * N >= 2^31
    assert lib.lss_linear_bwd_dx(FAKE, ctypes.byref(_saved()), None, 128, 256, 256, 0, 5, 0, 0, 0,
                                 FAKE, 1 << 40, None) == NULL
    assert lib.lss_linear_bwd_dw(FAKE, ctypes.byref(_saved()), None, 128, 256, 256, 0, 5, 0, 0, 0,
                                 FAKE, 1 << 40, None) == NULL


def test_budget_keep_nonzero_constant():
    txt = open(HEADER).read()
    m = re.search(r"#define HQLSS_BUDGET_KEEP_NONZERO \((-?\d+)\)", txt)
    assert m and int(m.group(1)) == H.BUDGET_KEEP_NONZERO == -1


def hsize(X=FAKE, W=FAKE, N=128, D=256, C=256, dt=0, kmax=7, k_out=FAKE, mse=FAKE, ws=FAKE,
          nbytes=1 << 40):
    return lib.hq_choose_hadamard_size(X, W, N, D, C, dt, kmax, k_out, mse, ws, nbytes, None)


def test_choose_hadamard_size_argument_errors():
    assert H.workspace_bytes(H.WS_HSIZE, 128, 256, 256) == H.workspace_bytes(H.WS_HSIZE, 1 << 20, 4096, 4096) > 0
    assert hsize(X=None) == NULL
    assert hsize(mse=None) == NULL
    assert hsize(k_out=None) == NULL
    assert hsize(N=0) == SHAPE
    assert hsize(D=96) == SHAPE
    assert hsize(kmax=8) == BLOCK
    assert hsize(kmax=-1) == BLOCK
    assert hsize(dt=3) == DTYPE
    assert hsize(W=FAKE + 4) == ALIGN
    assert hsize(mse=FAKE + 4) == ALIGN
    assert hsize(ws=None) == WS
    assert hsize(nbytes=1024) == WS


def test_debug_acc_errors():
    s = _saved()
    assert lib.hqlss_debug_gemm_acc(0, None, ctypes.byref(s), None, 128, 256, 256, None, 0, None) == NULL
    assert lib.hqlss_debug_gemm_acc(5, None, ctypes.byref(s), FAKE, 128, 256, 256, None, 0, None) == ARG
    assert lib.hqlss_debug_gemm_acc(1, None, ctypes.byref(s), FAKE, 128, 256, 256, None, 0, None) == NULL


def test_binding_rejects_cpu_tensors():
    import torch
    X = torch.zeros(128, 256)
    sv = H.Saved(*(torch.zeros(2) for _ in range(5)))
    with pytest.raises(ValueError):
        H.hq_linear_fwd(X, X, X, sv, 5)


_Lsq = H._binding._LsqC
_BmmLsq = H._binding._BmmLsqC


def fwd_lsq(N=128, D=256, C=256, k=5, lsq=None, saved=None, X=FAKE):
    s = saved if saved is not None else _saved(amax=None)  # amax is not used by this mode
    lq = lsq if lsq is not None else _Lsq(FAKE, FAKE, FAKE)
    return lib.hq_linear_fwd_lsq(X, FAKE, FAKE, N, D, C, 0, k, ctypes.byref(s), ctypes.byref(lq),
                                 FAKE, 1 << 40, None)


def bwd_lsq(dX=FAKE, dW=FAKE, lsq=None, budget=0, nbytes=1 << 40, N=128):
    lq = lsq if lsq is not None else _Lsq(FAKE, FAKE, FAKE)
    return lib.lss_linear_bwd_lsq(FAKE, ctypes.byref(_saved(amax=None)), ctypes.byref(lq), dX, dW, FAKE,
                                  N, 256, 256, 0, 5, budget, 0, 0, FAKE, nbytes, None)


def test_lsq_argument_errors():
    assert fwd_lsq(X=None) == NULL
    assert fwd_lsq(lsq=_Lsq(None, FAKE, FAKE)) == NULL
    assert fwd_lsq(lsq=_Lsq(FAKE, FAKE, None)) == NULL
    assert fwd_lsq(lsq=_Lsq(FAKE + 2, FAKE, FAKE)) == ALIGN  # steps need 4-byte alignment
    assert fwd_lsq(lsq=_Lsq(FAKE, FAKE + 8, FAKE)) == ALIGN
    assert fwd_lsq(saved=_saved(amax=None, xq=None)) == NULL
    assert fwd_lsq(N=0) == SHAPE
    assert fwd_lsq(k=8) == BLOCK
    assert bwd_lsq(dX=None, dW=None) == NULL
    assert bwd_lsq(dW=None, lsq=_Lsq(FAKE, None, FAKE)) == NULL  # dX reads delta_x
    assert bwd_lsq(budget=1000) == ARG
    assert bwd_lsq(nbytes=64) == WS
    assert bwd_lsq(N=70000) == SHAPE


def bmm_fwd(B=2, N=128, M=64, P=128, k=5, lsq=None, Q=FAKE):
    lq = lsq if lsq is not None else _BmmLsq(FAKE, FAKE, FAKE, FAKE)
    return lib.hq_bmm_fwd_lsq(Q, FAKE, FAKE, B, N, M, P, 0, k, ctypes.byref(_saved(amax=None)),
                              ctypes.byref(lq), None, 0, None)


def bmm_bwd(B=2, N=128, M=64, P=128, k=5, dQ=FAKE, dK=FAKE, nbytes=1 << 40, budget=0):
    lq = _BmmLsq(FAKE, FAKE, FAKE, FAKE)
    return lib.lss_bmm_bwd_lsq(FAKE, ctypes.byref(_saved(amax=None)), ctypes.byref(lq), dQ, dK, FAKE, FAKE,
                               B, N, M, P, 0, k, budget, 0, 0, FAKE, nbytes, None)


def test_bmm_argument_errors():
    assert bmm_fwd(Q=None) == NULL
    assert bmm_fwd(lsq=_BmmLsq(FAKE, None, FAKE, FAKE)) == NULL
    assert bmm_fwd(B=0) == SHAPE
    assert bmm_fwd(B=70000) == SHAPE  # grid z limit
    assert bmm_fwd(B=1 << 14, N=1 << 17) == SHAPE  # B N > 2^30
    assert bmm_fwd(M=96) == SHAPE
    assert bmm_fwd(k=7) == BLOCK  # M = 64 < 128
    assert bmm_bwd(dQ=None, dK=None) == NULL
    assert bmm_bwd(nbytes=1024) == WS
    assert bmm_bwd(budget=257) == ARG  # budget > 2N
    assert bmm_bwd(N=70000, B=2) == SHAPE


def test_bmm_workspace_sizes():
    a = H.bmm_workspace_bytes(H.WS_BMM_BWD, 2, 128, 64, 128)
    b = H.bmm_workspace_bytes(H.WS_BMM_BWD, 384, 512, 64, 512)
    assert 0 < a < b
    assert H.bmm_workspace_bytes(H.WS_BMM_FWD, 384, 512, 64, 512) == 0
    assert H.bmm_workspace_bytes(H.WS_BMM_BWD, 0, 512, 64, 512) == 0
