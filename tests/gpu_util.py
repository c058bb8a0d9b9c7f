"""Helpers of the GPU parity tests: run the HIP path through the C ABI, compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle as O

TORCH_DT = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def need_gpu():
    assert torch.cuda.is_available(), "GPU test run without a GPU"
    import paper_2306_11987_amd as H  # fails loudly when the library is missing

    return H


def dev_tensor(a: np.ndarray, dt: str) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(TORCH_DT[dt])


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").numpy()


def ulp(x: np.ndarray, dt: str) -> np.ndarray:
    ax = np.abs(x)
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    if dt == "f16":
        return 2.0 ** (np.maximum(e, -14) - 10)
    if dt == "bf16":
        return 2.0 ** (np.maximum(e, -126) - 7)
    return 2.0 ** (np.maximum(e, -126) - 23)


def check_float_output(name: str, got: torch.Tensor, ref: np.ndarray, dt: str) -> float:
    """fp32: elementwise relative error <= 1e-5.  fp16/bf16: the output cast is part of the
    operator, so every element must be within one unit in the last place of the dtype
    around the fp64 oracle value (plus the same 1e-5 relative allowance)."""
    g = got.detach().float().cpu().numpy().astype(np.float64)
    assert g.shape == ref.shape, (name, g.shape, ref.shape)
    assert np.all(np.isfinite(g)), f"{name}: non-finite output"
    err = np.abs(g - ref)
    allow = 1e-5 * np.abs(ref) + (0.0 if dt == "f32" else ulp(ref, dt))
    bad = err > allow
    if bad.any():
        i = np.unravel_index(np.argmax(err - allow), err.shape)
        raise AssertionError(f"{name}: {bad.sum()} elements out of tolerance, worst at {i}: "
                             f"got {g[i]!r} ref {ref[i]!r}")
    nrm = np.linalg.norm(ref)
    return float(np.linalg.norm(g - ref) / nrm) if nrm > 0 else float(np.linalg.norm(g))


def run_forward(H, X, W, k, dt):
    N, D = X.shape
    C = W.shape[0]
    tX, tW = dev_tensor(X, dt), dev_tensor(W, dt)
    Y = torch.empty(N, C, device="cuda", dtype=TORCH_DT[dt])
    saved = H.Saved.empty(N, D, C)
    H.hq_linear_fwd(tX, tW, Y, saved, k)
    return saved, Y


def check_forward(H, X, W, k, dt, saved, Y, f=None):
    N, D = X.shape
    C = W.shape[0]
    if f is None:
        f = O.hq_forward(X, W, k)
    torch.cuda.synchronize()
    am = to_np(saved.amax)
    assert am[0] == f.amax_x and am[1] == f.amax_w, (am, f.amax_x, f.amax_w)
    assert np.array_equal(to_np(saved.xq), O.pack_int4(f.xq)), "X codes"
    assert np.array_equal(to_np(saved.wq), O.pack_int4(f.wq)), "W codes"
    assert np.array_equal(to_np(saved.wqT), O.pack_int4(f.wq.T.copy())), "W^T codes"
    assert np.array_equal(to_np(saved.x_sumsq), f.x_sumsq.astype(np.int32)), "x_sumsq"
    acc = torch.empty(N, C, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(0, None, saved, acc, N, D, C, H.workspace(H.WS_FWD, N, D, C))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(acc), f.acc.astype(np.int32)), "forward int32 accumulators"
    return check_float_output("Y", Y, f.Y, dt)


def run_backward(H, G, saved, N, D, C, k, dt, budget, seed, offset):
    tG = dev_tensor(G, dt)
    plan = H.Plan.empty(N, C)
    H.lss_grad_plan(tG, saved, plan, D, budget, seed, offset)
    dX = torch.empty(N, D, device="cuda", dtype=TORCH_DT[dt])
    dW = torch.empty(C, D, device="cuda", dtype=TORCH_DT[dt])
    ws = H.workspace(H.WS_FROM_PLAN, N, D, C)
    H.lss_linear_bwd_from_plan(plan, saved, dX, dW, N, D, C, k, ws)
    return tG, plan, dX, dW


def check_plan(plan, b: "O.LSSBackward"):
    torch.cuda.synchronize()
    N = b.plan.w_up.shape[0]
    assert to_np(plan.amax_g)[0] == b.bs.amax
    assert np.array_equal(to_np(plan.qup), O.pack_int4(b.bs.q_up)), "upper codes"
    assert np.array_equal(to_np(plan.qdn), O.pack_int4(b.bs.q_dn)), "lower codes"
    su = (b.bs.q_up.astype(np.int64) ** 2).sum(1)
    sd = (b.bs.q_dn.astype(np.int64) ** 2).sum(1)
    assert np.array_equal(to_np(plan.sumsq_up), su.astype(np.int32))
    assert np.array_equal(to_np(plan.sumsq_dn), sd.astype(np.int32))
    assert np.array_equal(to_np(plan.w_up), b.plan.w_up.astype(np.uint8)), "upper weights"
    assert np.array_equal(to_np(plan.w_dn), b.plan.w_dn.astype(np.uint8)), "lower weights"
    nk = int(to_np(plan.n_kept)[0])
    assert nk == len(b.plan.kept), (nk, len(b.plan.kept))
    assert np.array_equal(to_np(plan.kept)[:nk], b.plan.kept.astype(np.int32)), "kept list"
    return nk


def check_backward_acc(H, plan, saved, b, N, D, C):
    nk = len(b.plan.kept)
    ws = H.workspace(H.WS_FROM_PLAN, N, D, C)
    acc = torch.zeros(N, D, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(1, plan, saved, acc, N, D, C, ws)
    accw = torch.empty(C, D, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(2, plan, saved, accw, N, D, C, ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_np(acc)[:nk], b.acc_dx.astype(np.int32)), "dX int32 accumulators"
    assert np.array_equal(to_np(accw), b.acc_dw.astype(np.int32)), "dW int32 accumulators"


# ---------------------------------------------------------------- FP6 route (test side)
# e2m3 (OCP Microscaling Formats): sign bit, 2 exponent bits with bias 1, 3 mantissa bits;
# exponent 0 is subnormal (value m / 8).
def e2m3_value(f: int) -> float:
    s, e, m = (f >> 5) & 1, (f >> 3) & 3, f & 7
    v = m / 8.0 if e == 0 else 2.0 ** (e - 1) * (1.0 + m / 8.0)
    return -v if s else v


E2M3_TABLE = np.array([e2m3_value(f) for f in range(64)])


def decode_fp6_rows(b: np.ndarray) -> np.ndarray:
    """Padded FP6 rows [R][K] (uint8) -> values [R][K]: every 32 codes are 24 bytes of 6-bit
    fields (code i at bits 6i..6i+5 of the little-endian group) and 8 bytes that must be 0."""
    b = np.asarray(b, dtype=np.uint8)
    R, K = b.shape
    g = b.reshape(R, K // 32, 32)
    assert not g[:, :, 24:].any(), "pad bytes of the FP6 layout are not zero"
    bits = np.unpackbits(g[:, :, :24], axis=-1, bitorder="little")  # [R][G][192]
    f = bits.reshape(R, K // 32, 32, 6) @ (1 << np.arange(6))
    return E2M3_TABLE[f].reshape(R, K)
