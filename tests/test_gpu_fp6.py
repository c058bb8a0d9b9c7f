"""GPU parity of the FP6 MFMA route (through the C ABI).

The route keeps the int8 route's codes, sample and integer results and only changes the
matrix instruction (INT4 codes are exact in e2m3, and the fp32 accumulation of their
products is exact), so every output must equal the int8 route's bit for bit and the oracle
to the same bar: saved codes decode to the oracle's codes, int32 accumulators equal the
oracle's, float outputs equal the int8 route's bits.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import (TORCH_DT, check_float_output, decode_fp6_rows, dev_tensor, need_gpu, say, to_np)

pytestmark = pytest.mark.gpu

SHAPES = [
    (128, 256, 256, 5, "f32", "sparse_rows"),
    (1, 64, 64, 0, "f32", "lognormal"),
    (200, 192, 320, 6, "f16", "lognormal"),
    (333, 256, 128, 7, "bf16", "pareto"),
    (77, 512, 576, 3, "f16", "pareto"),
    (300, 1024, 384, 5, "bf16", "lognormal"),
    (517, 128, 704, 1, "f32", "pareto"),
    (2048, 256, 256, 5, "f16", "lognormal"),
    (600, 4096, 256, 7, "bf16", "pareto"),  # long K: the forward splits along K
]


def _case(shape, seed=0):
    N, D, C, k, dt, kind = shape
    lin = synth.Linear(f"f6_{N}x{D}x{C}", N, D, C, k, dt, max(1, D // 100), 20.0, kind, N)
    X, W, G = synth.linear_inputs(lin, seed)
    return lin, X, W, G


def _bits(t):
    return t.contiguous().view(torch.uint8)


def _forward_both(H, X, W, k, dt):
    N, D = X.shape
    C = W.shape[0]
    tX, tW = dev_tensor(X, dt), dev_tensor(W, dt)
    Y4 = torch.empty(N, C, device="cuda", dtype=TORCH_DT[dt])
    sv4 = H.Saved.empty(N, D, C)
    H.hq_linear_fwd(tX, tW, Y4, sv4, k)
    Y6 = torch.full((N, C), float("nan"), device="cuda", dtype=TORCH_DT[dt])
    sv6 = H.saved_fp6_empty(N, D, C)
    H.hq_linear_fwd_fp6(tX, tW, Y6, sv6, k)
    torch.cuda.synchronize()
    return sv4, Y4, sv6, Y6


def _check_fp6_forward(H, X, W, k, dt, f, sv6, Y6, Y4, sv4):
    N, D = X.shape
    C = W.shape[0]
    assert np.array_equal(decode_fp6_rows(to_np(sv6.xq)), f.xq.astype(np.float64)), "X codes (FP6)"
    assert np.array_equal(decode_fp6_rows(to_np(sv6.wq)), f.wq.astype(np.float64)), "W codes (FP6)"
    assert np.array_equal(decode_fp6_rows(to_np(sv6.wqT)), f.wq.T.astype(np.float64)), "W^T codes (FP6)"
    assert np.array_equal(to_np(sv6.x_sumsq), f.x_sumsq.astype(np.int32))
    assert torch.equal(_bits(sv6.amax), _bits(sv4.amax))
    acc = torch.empty(N, C, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(10, None, sv6, acc, N, D, C, H.workspace(H.WS_FWD_FP6, N, D, C))
    torch.cuda.synchronize()
    assert np.array_equal(to_np(acc), f.acc.astype(np.int32)), "FP6 forward int32 accumulators"
    assert torch.equal(_bits(Y6), _bits(Y4)), "FP6 Y differs from the int8 route's"
    return check_float_output("Y", Y6, f.Y, dt)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}")
def test_fp6_forward_parity(shape):
    H = need_gpu()
    lin, X, W, _ = _case(shape)
    say(f"FP6 forward parity {shape}")
    sv4, Y4, sv6, Y6 = _forward_both(H, X, W, lin.log2_block, lin.dtype)
    f = O.hq_forward(X, W, lin.log2_block)
    _check_fp6_forward(H, X, W, lin.log2_block, lin.dtype, f, sv6, Y6, Y4, sv4)


@pytest.mark.parametrize("bn", [128, 256])
def test_fp6_forward_forced_tile_width(bn):
    H = need_gpu()
    lin, X, W, _ = _case((600, 448, 320, 5, "f16", "lognormal"), seed=8)
    say(f"FP6 forward, forced tile width {bn}")
    H.debug_set_gemm_tile_n(bn)
    try:
        sv4, Y4, sv6, Y6 = _forward_both(H, X, W, lin.log2_block, lin.dtype)
        f = O.hq_forward(X, W, lin.log2_block)
        _check_fp6_forward(H, X, W, lin.log2_block, lin.dtype, f, sv6, Y6, Y4, sv4)
    finally:
        H.debug_set_gemm_tile_n(0)


@pytest.mark.parametrize("splits", [2, 3])
def test_fp6_forward_forced_split_k(splits):
    H = need_gpu()
    lin, X, W, _ = _case((600, 1024, 512, 7, "bf16", "pareto"), seed=4)
    say(f"FP6 forward, forced split-K {splits}")
    H.debug_set_gemm_splits(splits)
    try:
        sv4, Y4, sv6, Y6 = _forward_both(H, X, W, lin.log2_block, lin.dtype)
        f = O.hq_forward(X, W, lin.log2_block)
        _check_fp6_forward(H, X, W, lin.log2_block, lin.dtype, f, sv6, Y6, Y4, sv4)
    finally:
        H.debug_set_gemm_splits(0)


@pytest.mark.parametrize("li", range(4))
def test_fp6_forward_full_size_sweep(li):
    """The GEMM sweep's linears at full size: Y bit for bit equal to the int8 route's, and
    sampled rows against the oracle."""
    H = need_gpu()
    lin = synth.workload(3).linears[li]
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"FP6 forward full size {lin.name}")
    X, W, _ = synth.linear_inputs(lin, 3, li, with_grad=False)
    sv4, Y4, sv6, Y6 = _forward_both(H, X, W, k, dt)
    assert torch.equal(_bits(Y6), _bits(Y4)), "FP6 Y differs from the int8 route's"
    assert torch.equal(sv6.x_sumsq, sv4.x_sumsq)
    f = O.hq_forward(X, W, k, compute_output=False)
    rng = np.random.default_rng(li)
    rows = np.sort(rng.choice(N, 64, replace=False))
    assert np.array_equal(decode_fp6_rows(to_np(sv6.xq[torch.from_numpy(rows).cuda()])),
                          f.xq[rows].astype(np.float64))
    ref = float(f.s_x) * float(f.s_w) * 2.0 ** -k * (f.xq[rows].astype(np.float64) @ f.wq.T.astype(np.float64))
    check_float_output("Y rows", Y6[torch.from_numpy(rows).cuda()], ref, dt)


def test_fp6_forward_argument_errors():
    H = need_gpu()
    X = torch.zeros(64, 100, device="cuda", dtype=torch.float16)
    W = torch.zeros(64, 100, device="cuda", dtype=torch.float16)
    Y = torch.empty(64, 64, device="cuda", dtype=torch.float16)
    with pytest.raises(H.HQLSSError):
        H.hq_linear_fwd_fp6(X, W, Y, H.saved_fp6_empty(64, 128, 64), 0)


# ---------------------------------------------------------------- backward (Sec. 4.2)
BWD_SHAPES = SHAPES + [
    (4096, 256, 192, 5, "f16", "sparse_rows"),  # ~10 % upper tokens: several two-pass dX tiles
    (3000, 128, 320, 4, "bf16", "sparse_rows"),
]


def _backward_both(H, G, sv4, sv6, N, D, C, k, dt, budget, seed, offset):
    tG = dev_tensor(G, dt)
    dX4 = torch.empty(N, D, device="cuda", dtype=TORCH_DT[dt])
    dW4 = torch.empty(C, D, device="cuda", dtype=TORCH_DT[dt])
    H.lss_linear_bwd(tG, sv4, dX4, dW4, D, k, budget, seed, offset)
    dX6 = torch.full((N, D), float("nan"), device="cuda", dtype=TORCH_DT[dt])
    dW6 = torch.full((C, D), float("nan"), device="cuda", dtype=TORCH_DT[dt])
    H.lss_linear_bwd_fp6(tG, sv6, dX6, dW6, D, k, budget, seed, offset)
    torch.cuda.synchronize()
    return tG, dX4, dW4, dX6, dW6


def _plan(H, tG, sv6, N, D, C, budget, seed, offset):
    plan = H.Plan.empty(N, C)
    H.lss_grad_plan(tG, sv6, plan, D, budget, seed, offset)
    return plan


@pytest.mark.parametrize("budget_div", [1, 4])
@pytest.mark.parametrize("shape", BWD_SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}")
def test_fp6_backward_parity(shape, budget_div):
    """dX, dW of the FP6 route equal the int8 route's bit for bit and the oracle's to the
    float bar; both int32 accumulators equal the oracle's."""
    H = need_gpu()
    lin, X, W, G = _case(shape, seed=1)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    budget = max(1, N // budget_div)
    seed, offset = 1234, 77
    say(f"FP6 backward parity {shape} budget={budget}")
    sv4, _, sv6, _ = _forward_both(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    b = O.lss_backward(G, f, budget, seed, offset)
    tG, dX4, dW4, dX6, dW6 = _backward_both(H, G, sv4, sv6, N, D, C, k, dt, budget, seed, offset)
    assert torch.equal(_bits(dX6), _bits(dX4)), "FP6 dX differs from the int8 route's"
    assert torch.equal(_bits(dW6), _bits(dW4)), "FP6 dW differs from the int8 route's"
    check_float_output("dX", dX6, b.dX, dt)
    check_float_output("dW", dW6, b.dW, dt)
    plan = _plan(H, tG, sv6, N, D, C, budget, seed, offset)
    nk = len(b.plan.kept)
    ws = H.workspace(H.WS_FROM_PLAN_FP6, N, D, C)
    acc = torch.zeros(N, D, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(11, plan, sv6, acc, N, D, C, ws)
    accw = torch.empty(C, D, dtype=torch.int32, device="cuda")
    H.debug_gemm_acc(12, plan, sv6, accw, N, D, C, ws)
    torch.cuda.synchronize()
    # FP6 dX rows come upper tokens first: compare by token
    order = np.concatenate([b.plan.kept[b.plan.w_up[b.plan.kept] > 0], b.plan.kept[b.plan.w_up[b.plan.kept] == 0]])
    pos = {int(t): i for i, t in enumerate(b.plan.kept)}
    ref_rows = b.acc_dx[[pos[int(t)] for t in order]] if nk else b.acc_dx
    assert np.array_equal(to_np(acc)[:nk], ref_rows.astype(np.int32)), "FP6 dX int32 accumulators"
    assert np.array_equal(to_np(accw), b.acc_dw.astype(np.int32)), "FP6 dW int32 accumulators"


def test_fp6_backward_keep_nonzero_and_live_sampling():
    """The keep-non-zero budget and a small budget (lower rows sampled with weights up to 16:
    every dW weight class in use) give the int8 route's bits."""
    H = need_gpu()
    lin, X, W, G = _case((2048, 512, 384, 7, "bf16", "sparse_rows"), seed=3)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sv4, _, sv6, _ = _forward_both(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    for budget in (H.BUDGET_KEEP_NONZERO, N // 8, N // 16):
        say(f"FP6 backward budget {budget}")
        b = O.lss_backward(G, f, budget, 9, 5)
        if budget > 0:
            assert (b.plan.w_dn >= 8).any(), "test must exercise the heavy weight classes"
        _, dX4, dW4, dX6, dW6 = _backward_both(H, G, sv4, sv6, N, D, C, k, dt, budget, 9, 5)
        assert torch.equal(_bits(dX6), _bits(dX4)) and torch.equal(_bits(dW6), _bits(dW4))
        check_float_output("dX", dX6, b.dX, dt)
        check_float_output("dW", dW6, b.dW, dt)


@pytest.mark.parametrize("splits", [2, 3])
def test_fp6_backward_forced_split_k(splits):
    """Split along K, each split applying the weights due in its own range: still the bits."""
    H = need_gpu()
    lin, X, W, G = _case((1500, 640, 448, 6, "f16", "sparse_rows"), seed=4)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sv4, _, sv6, _ = _forward_both(H, X, W, k, dt)
    H.debug_set_gemm_splits(splits)
    try:
        say(f"FP6 backward forced split-K {splits}")
        _, dX4, dW4, dX6, dW6 = _backward_both(H, G, sv4, sv6, N, D, C, k, dt, N // 6, 2, 3)
    finally:
        H.debug_set_gemm_splits(0)
    assert torch.equal(_bits(dX6), _bits(dX4)) and torch.equal(_bits(dW6), _bits(dW4))


@pytest.mark.parametrize("li", range(4))
def test_fp6_backward_full_size_sweep(li):
    """The GEMM sweep's linears at full size: dX and dW bit for bit equal to the int8 route's."""
    H = need_gpu()
    lin = synth.workload(3).linears[li]
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"FP6 backward full size {lin.name}")
    X, W, G = synth.linear_inputs(lin, 3, li)
    sv4, _, sv6, _ = _forward_both(H, X, W, k, dt)
    del X, W
    _, dX4, dW4, dX6, dW6 = _backward_both(H, G, sv4, sv6, N, D, C, k, dt, N, 42, 1000)
    assert torch.equal(_bits(dX6), _bits(dX4)), "FP6 dX differs from the int8 route's"
    assert torch.equal(_bits(dW6), _bits(dW4)), "FP6 dW differs from the int8 route's"


def test_fp6_backward_argument_errors():
    H = need_gpu()
    G = torch.zeros(64, 11520, device="cuda", dtype=torch.float16)
    dX = torch.empty(64, 64, device="cuda", dtype=torch.float16)
    with pytest.raises(H.HQLSSError) as e:  # C = 11520 > 11412
        H.lss_linear_bwd_fp6(G, H.saved_fp6_empty(64, 64, 11520), dX, None, 64, 0, 0, 0, 0,
                             torch.empty(16, dtype=torch.uint8, device="cuda"))
    assert "overflow" in str(e.value)
