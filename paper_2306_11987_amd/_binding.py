"""ctypes binding of libhqlss.so: argument marshalling only (see include/hqlss.h)."""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhqlss.so")

WS_FWD, WS_BWD_DX, WS_BWD_DW, WS_BWD, WS_FROM_PLAN, WS_PLAN, WS_HSIZE = 0, 1, 2, 3, 4, 5, 6
WS_FWD_LSQ, WS_BWD_LSQ, WS_FWD_FP6, WS_BWD_FP6, WS_FROM_PLAN_FP6 = 7, 8, 9, 10, 11
WS_BMM_FWD, WS_BMM_BWD = 0, 1
BUDGET_KEEP_NONZERO = -1  # HQLSS_BUDGET_KEEP_NONZERO: keep every non-zero gradient row
STATIC_SCRATCH_BYTES = 8 << 20  # HQLSS_STATIC_SCRATCH_BYTES: the allocation-free forward's scratch
DTYPE_CODES = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}

_vp, _i64, _u64, _int, _sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ctypes.c_int, ctypes.c_size_t


class _SavedC(ctypes.Structure):
    _fields_ = [("xq", _vp), ("wq", _vp), ("wqT", _vp), ("x_sumsq", _vp), ("amax", _vp)]


class _PlanC(ctypes.Structure):
    _fields_ = [("qup", _vp), ("qdn", _vp), ("sumsq_up", _vp), ("sumsq_dn", _vp), ("w_up", _vp),
                ("w_dn", _vp), ("kept", _vp), ("n_kept", _vp), ("amax_g", _vp)]


class _LsqC(ctypes.Structure):
    _fields_ = [("step", _vp), ("delta_x", _vp), ("delta_w", _vp)]


class _BmmLsqC(ctypes.Structure):
    _fields_ = [("step_q", _vp), ("step_k", _vp), ("delta_q", _vp), ("delta_k", _vp)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    L = ctypes.CDLL(LIB_PATH)
    st = ctypes.c_int
    sig = {
        "hqlss_workspace_bytes": (_sz, [_int, _i64, _i64, _i64]),
        "hq_linear_fwd": (st, [_vp, _vp, _vp, _i64, _i64, _i64, _int, _int, ctypes.POINTER(_SavedC),
                               _vp, _sz, _vp]),
        "hq_linear_fwd_noalloc": (st, [_vp, _vp, _vp, _i64, _i64, _i64, _int, _int,
                                       ctypes.POINTER(_SavedC), _vp]),
        "hq_linear_fwd_fp6": (st, [_vp, _vp, _vp, _i64, _i64, _i64, _int, _int, ctypes.POINTER(_SavedC),
                                   _vp, _sz, _vp]),
        "lss_linear_bwd_fp6": (st, [_vp, ctypes.POINTER(_SavedC), _vp, _vp, _i64, _i64, _i64, _int, _int,
                                    _i64, _u64, _u64, _vp, _sz, _vp]),
        "hq_linear_fwd_lsq": (st, [_vp, _vp, _vp, _i64, _i64, _i64, _int, _int, ctypes.POINTER(_SavedC),
                                   ctypes.POINTER(_LsqC), _vp, _sz, _vp]),
        "lss_linear_bwd_lsq": (st, [_vp, ctypes.POINTER(_SavedC), ctypes.POINTER(_LsqC), _vp, _vp, _vp,
                                    _i64, _i64, _i64, _int, _int, _i64, _u64, _u64, _vp, _sz, _vp]),
        "hq_bmm_fwd_lsq": (st, [_vp, _vp, _vp, _i64, _i64, _i64, _i64, _int, _int, ctypes.POINTER(_SavedC),
                                ctypes.POINTER(_BmmLsqC), _vp, _sz, _vp]),
        "hqlss_bmm_workspace_bytes": (_sz, [_int, _i64, _i64, _i64, _i64]),
        "lss_bmm_bwd_lsq": (st, [_vp, ctypes.POINTER(_SavedC), ctypes.POINTER(_BmmLsqC), _vp, _vp, _vp, _vp,
                                 _i64, _i64, _i64, _i64, _int, _int, _i64, _u64, _u64, _vp, _sz, _vp]),
        "lss_grad_plan": (st, [_vp, ctypes.POINTER(_SavedC), ctypes.POINTER(_PlanC), _i64, _i64, _i64,
                               _int, _i64, _u64, _u64, _vp, _sz, _vp]),
        "lss_linear_bwd_from_plan": (st, [ctypes.POINTER(_PlanC), ctypes.POINTER(_SavedC), _vp, _vp,
                                          _i64, _i64, _i64, _int, _int, _vp, _sz, _vp]),
        "lss_linear_bwd": (st, [_vp, ctypes.POINTER(_SavedC), _vp, _vp, _i64, _i64, _i64, _int, _int,
                                _i64, _u64, _u64, _vp, _sz, _vp]),
        "lss_linear_bwd_dx": (st, [_vp, ctypes.POINTER(_SavedC), _vp, _i64, _i64, _i64, _int, _int,
                                   _i64, _u64, _u64, _vp, _sz, _vp]),
        "lss_linear_bwd_dw": (st, [_vp, ctypes.POINTER(_SavedC), _vp, _i64, _i64, _i64, _int, _int,
                                   _i64, _u64, _u64, _vp, _sz, _vp]),
        "hq_choose_hadamard_size": (st, [_vp, _vp, _i64, _i64, _i64, _int, _int, _vp, _vp, _vp, _sz,
                                         _vp]),
        "lss_philox_offset_advance": (_u64, [_i64, _i64]),
        "hqlss_status_string": (ctypes.c_char_p, [_int]),
        "hqlss_debug_gemm_acc": (st, [_int, ctypes.POINTER(_PlanC), ctypes.POINTER(_SavedC), _vp, _i64,
                                      _i64, _i64, _vp, _sz, _vp]),
        "hqlss_timing_enable": (st, [_int]),
        "hqlss_timing_read": (_int, [ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_float), _int]),
        "hqlss_kernel_name": (ctypes.c_char_p, [_int]),
        "hqlss_debug_set_gemm_splits": (None, [_int]),
        "hqlss_debug_set_gemm_tile_n": (None, [_int]),
        "hqlss_debug_set_fwd_fp6": (None, [_int]),
        "hqlss_debug_copy": (st, [_vp, _vp, _sz, _vp]),
        "hqlss_debug_plan_scores_offset": (_sz, [_i64, ctypes.POINTER(_i64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    return L


lib = _load()


class HQLSSError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} (status {status})")
        self.status = status


def status_string(status: int) -> str:
    return lib.hqlss_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != 0:
        raise HQLSSError(status, where)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors handed to libhqlss must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors handed to libhqlss must be contiguous")
    return t.data_ptr()


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _dt(t: torch.Tensor) -> int:
    if t.dtype not in DTYPE_CODES:
        raise ValueError(f"unsupported dtype {t.dtype}")
    return DTYPE_CODES[t.dtype]


@dataclass
class Saved:
    """Forward-to-backward state (hqlss_saved_t): codes of X H_u and W H_u and friends."""

    xq: torch.Tensor  # uint8 [N, D/2]
    wq: torch.Tensor  # uint8 [C, D/2]
    wqT: torch.Tensor  # uint8 [D, C/2]
    x_sumsq: torch.Tensor  # int32 [N]
    amax: torch.Tensor  # float32 [2]

    @staticmethod
    def empty(N: int, D: int, C: int, device="cuda") -> "Saved":
        u8 = dict(dtype=torch.uint8, device=device)
        return Saved(torch.empty(N, D // 2, **u8), torch.empty(C, D // 2, **u8),
                     torch.empty(D, C // 2, **u8), torch.empty(N, dtype=torch.int32, device=device),
                     torch.empty(2, dtype=torch.float32, device=device))

    def c(self) -> _SavedC:
        return _SavedC(_ptr(self.xq), _ptr(self.wq), _ptr(self.wqT), _ptr(self.x_sumsq), _ptr(self.amax))


@dataclass
class Plan:
    """Quantised gradient and its sample (lss_plan_t)."""

    qup: torch.Tensor  # uint8 [N, C/2]
    qdn: torch.Tensor  # uint8 [N, C/2]
    sumsq_up: torch.Tensor  # int32 [N]
    sumsq_dn: torch.Tensor  # int32 [N]
    w_up: torch.Tensor  # uint8 [N]
    w_dn: torch.Tensor  # uint8 [N]
    kept: torch.Tensor  # int32 [N]
    n_kept: torch.Tensor  # int32 [1]
    amax_g: torch.Tensor  # float32 [1]

    @staticmethod
    def empty(N: int, C: int, device="cuda") -> "Plan":
        u8 = dict(dtype=torch.uint8, device=device)
        i32 = dict(dtype=torch.int32, device=device)
        return Plan(torch.empty(N, C // 2, **u8), torch.empty(N, C // 2, **u8), torch.empty(N, **i32),
                    torch.empty(N, **i32), torch.empty(N, **u8), torch.empty(N, **u8),
                    torch.empty(N, **i32), torch.empty(1, **i32),
                    torch.empty(1, dtype=torch.float32, device=device))

    def c(self) -> _PlanC:
        return _PlanC(*[_ptr(getattr(self, f)) for f, _ in _PlanC._fields_])


@dataclass
class LSQ:
    """Learned-step-size state (hqlss_lsq_t): the steps and the forward's fp16 deltas."""

    step: torch.Tensor  # float32 [2]: s_X, s_W
    delta_x: torch.Tensor  # float16 [N, D]
    delta_w: torch.Tensor  # float16 [C, D]

    @staticmethod
    def empty(step: torch.Tensor, N: int, D: int, C: int) -> "LSQ":
        if step.dtype != torch.float32 or step.numel() != 2:
            raise ValueError("step must be a float32 tensor of two elements (s_X, s_W)")
        f16 = dict(dtype=torch.float16, device=step.device)
        return LSQ(step, torch.empty(N, D, **f16), torch.empty(C, D, **f16))

    def c(self) -> _LsqC:
        return _LsqC(_ptr(self.step), _ptr(self.delta_x), _ptr(self.delta_w))


@dataclass
class BmmLSQ:
    """Per-batch steps and fp16 deltas of the attention BMM (hqlss_bmm_lsq_t)."""

    step_q: torch.Tensor  # float32 [B]
    step_k: torch.Tensor  # float32 [B]
    delta_q: torch.Tensor  # float16 [B, N, M]
    delta_k: torch.Tensor  # float16 [B, P, M]

    @staticmethod
    def empty(step_q: torch.Tensor, step_k: torch.Tensor, N: int, M: int, P: int) -> "BmmLSQ":
        B = step_q.numel()
        if step_q.dtype != torch.float32 or step_k.dtype != torch.float32 or step_k.numel() != B:
            raise ValueError("step_q and step_k must be float32 tensors of B elements")
        f16 = dict(dtype=torch.float16, device=step_q.device)
        return BmmLSQ(step_q, step_k, torch.empty(B, N, M, **f16), torch.empty(B, P, M, **f16))

    def c(self) -> _BmmLsqC:
        return _BmmLsqC(_ptr(self.step_q), _ptr(self.step_k), _ptr(self.delta_q), _ptr(self.delta_k))


def bmm_saved_empty(B: int, N: int, M: int, P: int, device="cuda") -> "Saved":
    """Saved state of a batched call: the linear operator's, batch after batch."""
    u8 = dict(dtype=torch.uint8, device=device)
    return Saved(torch.empty(B, N, M // 2, **u8), torch.empty(B, P, M // 2, **u8),
                 torch.empty(B, M, P // 2, **u8), torch.empty(B, N, dtype=torch.int32, device=device),
                 torch.empty(2, dtype=torch.float32, device=device))


def bmm_workspace_bytes(which: int, B: int, N: int, M: int, P: int) -> int:
    return int(lib.hqlss_bmm_workspace_bytes(int(which), int(B), int(N), int(M), int(P)))


def bmm_workspace(which: int, B: int, N: int, M: int, P: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(bmm_workspace_bytes(which, B, N, M, P), 256), dtype=torch.uint8, device=device)


def hq_bmm_fwd_lsq(Q: torch.Tensor, K: torch.Tensor, T: torch.Tensor, saved: "Saved", lsq: BmmLSQ,
                   log2_block: int, ws: Optional[torch.Tensor] = None) -> None:
    B, N, M = Q.shape
    P = K.shape[1]
    p, n = _ws(ws)
    sv, lq = saved.c(), lsq.c()
    _check(lib.hq_bmm_fwd_lsq(_ptr(Q), _ptr(K), _ptr(T), B, N, M, P, _dt(Q), int(log2_block),
                              ctypes.byref(sv), ctypes.byref(lq), p, n, _stream(Q)), "hq_bmm_fwd_lsq")


def lss_bmm_bwd_lsq(dT: torch.Tensor, saved: "Saved", lsq: BmmLSQ, dQ: Optional[torch.Tensor],
                    dK: Optional[torch.Tensor], dstep_q: Optional[torch.Tensor],
                    dstep_k: Optional[torch.Tensor], M: int, log2_block: int, budget: int = 0,
                    seed: int = 0, offset: int = 0, ws: Optional[torch.Tensor] = None) -> None:
    B, N, P = dT.shape
    if ws is None:
        ws = bmm_workspace(WS_BMM_BWD, B, N, M, P, dT.device)
    p, n = _ws(ws)
    sv, lq = saved.c(), lsq.c()
    _check(lib.lss_bmm_bwd_lsq(_ptr(dT), ctypes.byref(sv), ctypes.byref(lq), _ptr(dQ), _ptr(dK),
                               _ptr(dstep_q), _ptr(dstep_k), B, N, int(M), P, _dt(dT), int(log2_block),
                               int(budget), int(seed), int(offset), p, n, _stream(dT)), "lss_bmm_bwd_lsq")


def workspace_bytes(which: int, N: int, D: int, C: int) -> int:
    return int(lib.hqlss_workspace_bytes(int(which), int(N), int(D), int(C)))


def workspace(which: int, N: int, D: int, C: int, device="cuda") -> torch.Tensor:
    return torch.empty(max(workspace_bytes(which, N, D, C), 256), dtype=torch.uint8, device=device)


def lss_philox_offset_advance(N: int, C: int) -> int:
    return int(lib.lss_philox_offset_advance(int(N), int(C)))


def _ws(ws: Optional[torch.Tensor]):
    return (None, 0) if ws is None else (_ptr(ws), ws.numel())


def hq_linear_fwd(X: torch.Tensor, W: torch.Tensor, Y: torch.Tensor, saved: Saved, log2_block: int,
                  ws: Optional[torch.Tensor] = None) -> None:
    N, D = X.shape
    C = W.shape[0]
    if ws is None:
        ws = workspace(WS_FWD, N, D, C, X.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.hq_linear_fwd(_ptr(X), _ptr(W), _ptr(Y), N, D, C, _dt(X), int(log2_block),
                             ctypes.byref(sv), p, n, _stream(X)), "hq_linear_fwd")


def hq_linear_fwd_noalloc(X: torch.Tensor, W: torch.Tensor, Y: torch.Tensor, saved: Saved,
                          log2_block: int) -> None:
    """hq_linear_fwd without a workspace: the library's static device scratch is used."""
    N, D = X.shape
    C = W.shape[0]
    sv = saved.c()
    _check(lib.hq_linear_fwd_noalloc(_ptr(X), _ptr(W), _ptr(Y), N, D, C, _dt(X), int(log2_block),
                                     ctypes.byref(sv), _stream(X)), "hq_linear_fwd_noalloc")


def saved_fp6_empty(N: int, D: int, C: int, device="cuda") -> "Saved":
    """Saved state of the FP6 route: one byte per code (padded FP6 layout)."""
    u8 = dict(dtype=torch.uint8, device=device)
    return Saved(torch.empty(N, D, **u8), torch.empty(C, D, **u8), torch.empty(D, C, **u8),
                 torch.empty(N, dtype=torch.int32, device=device),
                 torch.empty(2, dtype=torch.float32, device=device))


def hq_linear_fwd_fp6(X: torch.Tensor, W: torch.Tensor, Y: torch.Tensor, saved: Saved, log2_block: int,
                      ws: Optional[torch.Tensor] = None) -> None:
    N, D = X.shape
    C = W.shape[0]
    if ws is None:
        ws = workspace(WS_FWD_FP6, N, D, C, X.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.hq_linear_fwd_fp6(_ptr(X), _ptr(W), _ptr(Y), N, D, C, _dt(X), int(log2_block),
                                 ctypes.byref(sv), p, n, _stream(X)), "hq_linear_fwd_fp6")


def lss_linear_bwd_fp6(dY: torch.Tensor, saved: Saved, dX: Optional[torch.Tensor], dW: Optional[torch.Tensor],
                       D: int, log2_block: int, budget: int = 0, seed: int = 0, offset: int = 0,
                       ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    if ws is None:
        ws = workspace(WS_BWD_FP6, N, D, C, dY.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.lss_linear_bwd_fp6(_ptr(dY), ctypes.byref(sv), _ptr(dX), _ptr(dW), N, D, C, _dt(dY),
                                  int(log2_block), int(budget), int(seed), int(offset), p, n, _stream(dY)),
           "lss_linear_bwd_fp6")


def hq_linear_fwd_lsq(X: torch.Tensor, W: torch.Tensor, Y: torch.Tensor, saved: Saved, lsq: LSQ,
                      log2_block: int, ws: Optional[torch.Tensor] = None) -> None:
    N, D = X.shape
    C = W.shape[0]
    if ws is None:
        ws = workspace(WS_FWD_LSQ, N, D, C, X.device)
    p, n = _ws(ws)
    sv, lq = saved.c(), lsq.c()
    _check(lib.hq_linear_fwd_lsq(_ptr(X), _ptr(W), _ptr(Y), N, D, C, _dt(X), int(log2_block),
                                 ctypes.byref(sv), ctypes.byref(lq), p, n, _stream(X)),
           "hq_linear_fwd_lsq")


def lss_linear_bwd_lsq(dY: torch.Tensor, saved: Saved, lsq: LSQ, dX: Optional[torch.Tensor],
                       dW: Optional[torch.Tensor], dstep: Optional[torch.Tensor], D: int, log2_block: int,
                       budget: int = 0, seed: int = 0, offset: int = 0,
                       ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    if ws is None:
        ws = workspace(WS_BWD_LSQ, N, D, C, dY.device)
    p, n = _ws(ws)
    sv, lq = saved.c(), lsq.c()
    _check(lib.lss_linear_bwd_lsq(_ptr(dY), ctypes.byref(sv), ctypes.byref(lq), _ptr(dX), _ptr(dW),
                                  _ptr(dstep), N, int(D), C, _dt(dY), int(log2_block), int(budget),
                                  int(seed), int(offset), p, n, _stream(dY)), "lss_linear_bwd_lsq")


def hq_choose_hadamard_size(X: torch.Tensor, W: torch.Tensor, max_log2_block: int = 7,
                            log2_block_out: Optional[torch.Tensor] = None,
                            mse_out: Optional[torch.Tensor] = None,
                            ws: Optional[torch.Tensor] = None):
    """Enqueues the block-size search; returns (log2_block int32 [1], mse float64 [16]) on
    the device: MSE_X(k) at [k], MSE_W(k) at [8 + k], NaN where k is no candidate."""
    N, D = X.shape
    C = W.shape[0]
    if log2_block_out is None:
        log2_block_out = torch.empty(1, dtype=torch.int32, device=X.device)
    if mse_out is None:
        mse_out = torch.empty(16, dtype=torch.float64, device=X.device)
    if ws is None:
        ws = workspace(WS_HSIZE, N, D, C, X.device)
    p, n = _ws(ws)
    _check(lib.hq_choose_hadamard_size(_ptr(X), _ptr(W), N, D, C, _dt(X), int(max_log2_block),
                                       _ptr(log2_block_out), _ptr(mse_out), p, n, _stream(X)),
           "hq_choose_hadamard_size")
    return log2_block_out, mse_out


def lss_grad_plan(dY: torch.Tensor, saved: Saved, plan: Plan, D: int, budget: int = 0, seed: int = 0,
                  offset: int = 0, ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    if ws is None:
        ws = workspace(WS_PLAN, N, D, C, dY.device)
    p, n = _ws(ws)
    sv, pl = saved.c(), plan.c()
    _check(lib.lss_grad_plan(_ptr(dY), ctypes.byref(sv), ctypes.byref(pl), N, int(D), C, _dt(dY),
                             int(budget), int(seed), int(offset), p, n, _stream(dY)), "lss_grad_plan")


def lss_linear_bwd_from_plan(plan: Plan, saved: Saved, dX: Optional[torch.Tensor],
                             dW: Optional[torch.Tensor], N: int, D: int, C: int, log2_block: int,
                             ws: torch.Tensor) -> None:
    ref = dX if dX is not None else dW
    p, n = _ws(ws)
    sv, pl = saved.c(), plan.c()
    _check(lib.lss_linear_bwd_from_plan(ctypes.byref(pl), ctypes.byref(sv), _ptr(dX), _ptr(dW), N, D, C,
                                        _dt(ref), int(log2_block), p, n, _stream(ref)),
           "lss_linear_bwd_from_plan")


def lss_linear_bwd(dY: torch.Tensor, saved: Saved, dX: Optional[torch.Tensor], dW: Optional[torch.Tensor],
                   D: int, log2_block: int, budget: int = 0, seed: int = 0, offset: int = 0,
                   ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    if ws is None:
        ws = workspace(WS_BWD, N, D, C, dY.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.lss_linear_bwd(_ptr(dY), ctypes.byref(sv), _ptr(dX), _ptr(dW), N, int(D), C, _dt(dY),
                              int(log2_block), int(budget), int(seed), int(offset), p, n, _stream(dY)),
           "lss_linear_bwd")


def lss_linear_bwd_dx(dY: torch.Tensor, saved: Saved, dX: torch.Tensor, log2_block: int, budget: int = 0,
                      seed: int = 0, offset: int = 0, ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    D = dX.shape[1]
    if ws is None:
        ws = workspace(WS_BWD_DX, N, D, C, dY.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.lss_linear_bwd_dx(_ptr(dY), ctypes.byref(sv), _ptr(dX), N, D, C, _dt(dY), int(log2_block),
                                 int(budget), int(seed), int(offset), p, n, _stream(dY)), "lss_linear_bwd_dx")


def lss_linear_bwd_dw(dY: torch.Tensor, saved: Saved, dW: torch.Tensor, log2_block: int, budget: int = 0,
                      seed: int = 0, offset: int = 0, ws: Optional[torch.Tensor] = None) -> None:
    N, C = dY.shape
    D = dW.shape[1]
    if ws is None:
        ws = workspace(WS_BWD_DW, N, D, C, dY.device)
    p, n = _ws(ws)
    sv = saved.c()
    _check(lib.lss_linear_bwd_dw(_ptr(dY), ctypes.byref(sv), _ptr(dW), N, D, C, _dt(dY), int(log2_block),
                                 int(budget), int(seed), int(offset), p, n, _stream(dY)), "lss_linear_bwd_dw")


def debug_gemm_acc(which: int, plan: Optional[Plan], saved: Saved, acc: torch.Tensor, N: int, D: int, C: int,
                   ws: Optional[torch.Tensor] = None) -> None:
    p, n = _ws(ws)
    sv = saved.c()
    pl = plan.c() if plan is not None else None
    _check(lib.hqlss_debug_gemm_acc(int(which), ctypes.byref(pl) if pl is not None else None,
                                    ctypes.byref(sv), _ptr(acc), N, D, C, p, n, _stream(acc)),
           "hqlss_debug_gemm_acc")


def timing_enable(on: bool) -> None:
    _check(lib.hqlss_timing_enable(1 if on else 0), "hqlss_timing_enable")


def timing_read(cap: int = 4096):
    ids = (ctypes.c_int * cap)()
    ms = (ctypes.c_float * cap)()
    n = lib.hqlss_timing_read(ids, ms, cap)
    if n < 0:
        raise HQLSSError(8, "hqlss_timing_read")
    return [(int(ids[i]), float(ms[i])) for i in range(n)]


def debug_set_gemm_splits(splits: int) -> None:
    lib.hqlss_debug_set_gemm_splits(int(splits))


def debug_set_gemm_tile_n(bn: int) -> None:
    lib.hqlss_debug_set_gemm_tile_n(int(bn))


def debug_set_fwd_fp6(mode: int) -> None:
    """Test hook: hq_linear_fwd's product on FP6 (mode > 0), int8 (< 0) or by size (0)."""
    lib.hqlss_debug_set_fwd_fp6(int(mode))


def debug_plan_scores_offset(N: int):
    """Test hook: (byte offset, pitch) of the leverage scores in lss_grad_plan's workspace."""
    pitch = ctypes.c_int64(0)
    off = lib.hqlss_debug_plan_scores_offset(int(N), ctypes.byref(pitch))
    return int(off), int(pitch.value)


def debug_copy(src: torch.Tensor, dst: torch.Tensor) -> None:
    """Plain device copy kernel of src's bytes into dst (traffic-counter calibration)."""
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < n:
        raise ValueError("debug_copy: destination smaller than source")
    _check(lib.hqlss_debug_copy(_ptr(src), _ptr(dst), n, _stream(src)), "hqlss_debug_copy")


def kernel_name(i: int) -> str:
    return lib.hqlss_kernel_name(int(i)).decode()
