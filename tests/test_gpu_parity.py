"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Bit-exact: codes, scales, row sums, sample weights, kept lists and every int32 GEMM
accumulator.  Float outputs: within 1e-5 relative (fp32) or one unit in the last place of
the output dtype around the fp64 oracle value (fp16, bf16).
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import (check_backward_acc, check_float_output, check_forward, check_plan,
                      dev_tensor, need_gpu, run_backward, run_forward, say, to_np, TORCH_DT)

pytestmark = pytest.mark.gpu

# (N, D, C, log2_block, dtype, grad_kind): several tiles, ragged N, every dtype and block size
SHAPES = [
    (128, 256, 256, 5, "f32", "sparse_rows"),
    (1, 64, 64, 0, "f32", "lognormal"),
    (200, 192, 320, 6, "f16", "lognormal"),
    (333, 256, 128, 7, "bf16", "pareto"),
    (77, 512, 576, 3, "f16", "pareto"),
    (300, 1024, 384, 5, "bf16", "lognormal"),
    (517, 128, 704, 1, "f32", "pareto"),
    (2048, 256, 256, 5, "f16", "lognormal"),  # dW over 2048 tokens: split-K by default
]


def _case(shape, seed=0):
    N, D, C, k, dt, kind = shape
    lin = synth.Linear(f"t{N}x{D}x{C}", N, D, C, k, dt, max(1, D // 100), 20.0, kind, N)
    X, W, G = synth.linear_inputs(lin, seed)
    return lin, X, W, G


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}")
def test_forward_parity(shape):
    H = need_gpu()
    lin, X, W, _ = _case(shape)
    say(f"forward parity {shape}")
    saved, Y = run_forward(H, X, W, lin.log2_block, lin.dtype)
    rel = check_forward(H, X, W, lin.log2_block, lin.dtype, saved, Y)
    assert rel <= (1e-5 if lin.dtype == "f32" else 2e-3)


@pytest.mark.parametrize("budget_div", [1, 4])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}")
def test_backward_parity(shape, budget_div):
    H = need_gpu()
    lin, X, W, G = _case(shape, seed=1)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    budget = max(1, N // budget_div)
    seed, offset = 1234, 77
    say(f"backward parity {shape} budget={budget}")
    saved, _ = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    b = O.lss_backward(G, f, budget, seed, offset)
    tG, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, budget, seed, offset)
    check_plan(plan, b)
    check_backward_acc(H, plan, saved, b, N, D, C)
    check_float_output("dX", dX, b.dX, dt)
    check_float_output("dW", dW, b.dW, dt)

    # the one-call entry points reproduce the same sample and outputs bit for bit
    ws = H.workspace(H.WS_BWD, N, D, C)
    dX2 = torch.empty_like(dX)
    dW2 = torch.empty_like(dW)
    H.lss_linear_bwd(tG, saved, dX2, dW2, D, k, budget, seed, offset, ws)
    dX3 = torch.empty_like(dX)
    dW3 = torch.empty_like(dW)
    H.lss_linear_bwd_dx(tG, saved, dX3, k, budget, seed, offset, ws)
    H.lss_linear_bwd_dw(tG, saved, dW3, k, budget, seed, offset, ws)
    # the single-gradient calls with workspaces of exactly their queried sizes
    dX4 = torch.empty_like(dX)
    dW4 = torch.empty_like(dW)
    H.lss_linear_bwd_dx(tG, saved, dX4, k, budget, seed, offset, H.workspace(H.WS_BWD_DX, N, D, C))
    H.lss_linear_bwd_dw(tG, saved, dW4, k, budget, seed, offset, H.workspace(H.WS_BWD_DW, N, D, C))
    torch.cuda.synchronize()
    for t in (dX2, dX3, dX4):
        assert torch.equal(t, dX)
    for t in (dW2, dW3, dW4):
        assert torch.equal(t, dW)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_{s[5]}")
def test_leverage_scores(shape):
    """The integer leverage scores the bit split writes (both stacked rows of every token)
    equal the oracle's, bit for bit (Sec. 4.2)."""
    H = need_gpu()
    lin, X, W, G = _case(shape, seed=3)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"leverage scores {shape}")
    saved, _ = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    b = O.lss_backward(G, f, N, 5, 9, need_dx=False, need_dw=False)
    plan = H.Plan.empty(N, C)
    ws = H.workspace(H.WS_PLAN, N, D, C)
    H.lss_grad_plan(dev_tensor(G, dt), saved, plan, D, N, 5, 9, ws)
    torch.cuda.synchronize()
    off, pitch = H.debug_plan_scores_offset(N)
    raw = to_np(ws)[off:off + 8 * pitch].view(np.uint32)
    got = np.concatenate([raw[:N], raw[pitch:pitch + N]]).astype(np.int64)
    su = (b.bs.q_up.astype(np.int64) ** 2).sum(1)
    sd = (b.bs.q_dn.astype(np.int64) ** 2).sum(1)
    ref = O.leverage_scores(su, sd, f.x_sumsq)
    assert np.array_equal(got, ref), "leverage scores"


def test_sampling_exercised_and_deterministic():
    """A small budget makes the Bernoulli path live; equal (seed, offset) give identical
    samples, a different offset a different one."""
    H = need_gpu()
    lin, X, W, G = _case((512, 256, 256, 5, "f16", "pareto"), seed=3)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    saved, _ = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    outs = []
    for off in (5, 5, 6):
        say(f"determinism offset={off}")
        b = O.lss_backward(G, f, N // 8, 9, off)
        assert (b.plan.e_dn > 0).any() and len(b.plan.kept) < N
        _, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N // 8, 9, off)
        check_plan(plan, b)
        outs.append((to_np(plan.w_dn).copy(), to_np(dW).copy()))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    assert not np.array_equal(outs[0][0], outs[2][0])


def test_zero_gradient_and_zero_input():
    """dY = 0: nothing is kept, both gradients are exactly zero.  X = 0: Y = 0."""
    H = need_gpu()
    lin, X, W, G = _case((130, 128, 192, 4, "bf16", "lognormal"))
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    saved, Y = run_forward(H, np.zeros_like(X), W, k, dt)
    torch.cuda.synchronize()
    assert not Y.float().abs().sum().item()
    saved, _ = run_forward(H, X, W, k, dt)
    _, plan, dX, dW = run_backward(H, np.zeros_like(G), saved, N, D, C, k, dt, N, 0, 0)
    torch.cuda.synchronize()
    assert int(to_np(plan.n_kept)[0]) == 0
    assert not dX.float().abs().sum().item() and not dW.float().abs().sum().item()


def test_exact_reconstruction_on_gpu():
    """X = 2^m Q H_u / b: the GPU codes equal Q and Y equals X W^T exactly (Sec. 3.3)."""
    import scipy.linalg
    H = need_gpu()
    k, b = 4, 16
    rng = np.random.default_rng(11)
    N, D, C = 70, 128, 64
    Qx = rng.integers(-7, 8, size=(N, D)); Qx[0, 0] = 7
    Qw = rng.integers(-7, 8, size=(C, D)); Qw[0, 1] = -7
    Hb = np.kron(np.eye(D // b), scipy.linalg.hadamard(b))
    X = (2.0 ** 2 * Qx @ Hb / b).astype(np.float32)
    W = (2.0 ** -3 * Qw @ Hb / b).astype(np.float32)
    saved, Y = run_forward(H, X, W, k, "f32")
    torch.cuda.synchronize()
    assert np.array_equal(O.unpack_int4(to_np(saved.xq)), Qx)
    exact = X.astype(np.float64) @ W.astype(np.float64).T
    assert np.array_equal(to_np(Y).astype(np.float64), exact)


# (workload id, linear index) at full size: every distinct linear of the named workloads
# (the BERT-large block's Q, K, V and O share one shape; Q stands for them)
FULL_SIZE = [(1, 0), (1, 1), (2, 0), (2, 1), (2, 2), (2, 3), (3, 0), (3, 1), (3, 2), (3, 3),
             (4, 0), (4, 4), (4, 5)]
N_Y_ROWS, N_DX_TOKENS, N_DW_ROWS = 256, 256, 64


def _acc_rows(H, which, plan, saved, N, D, C, rows, shape):
    """Whole rows of one GEMM's int32 accumulators (hqlss_debug_gemm_acc), copied back."""
    acc = torch.empty(*shape, dtype=torch.int32, device="cuda")
    ws = H.workspace(H.WS_FWD if which == 0 else H.WS_FROM_PLAN, N, D, C)
    H.debug_gemm_acc(which, plan, saved, acc, N, D, C, ws)
    out = to_np(acc[torch.from_numpy(rows).cuda()])
    del acc, ws
    return out


@pytest.mark.parametrize("case", FULL_SIZE, ids=lambda c: f"w{c[0]}_{synth.workload(c[0]).linears[c[1]].name}")
def test_full_size_sampled(case):
    """A linear of a named workload at full size, in the configuration the benchmark uses
    (budget N): the codes of every row, the leverage scores and the whole sample bit for
    bit; whole int32
    accumulator rows of all three GEMMs (sampled tokens and channels) bit for bit; sampled
    output rows of Y, dX and dW against the oracle computing them one by one."""
    H = need_gpu()
    cid, li = case
    lin = synth.workload(cid).linears[li]
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"full-size sampled parity {lin.name} N={N} D={D} C={C} b={1 << k} {dt}")
    X, W, G = synth.linear_inputs(lin, cid, li)
    saved, Y = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)  # codes of every row
    torch.cuda.synchronize()
    assert to_np(saved.amax)[0] == f.amax_x and to_np(saved.amax)[1] == f.amax_w
    assert np.array_equal(to_np(saved.xq), O.pack_int4(f.xq))
    assert np.array_equal(to_np(saved.wq), O.pack_int4(f.wq))
    assert np.array_equal(to_np(saved.wqT), O.pack_int4(f.wq.T.copy()))
    assert np.array_equal(to_np(saved.x_sumsq), f.x_sumsq.astype(np.int32))
    rng = np.random.default_rng(cid * 10 + li)
    rows = np.sort(rng.choice(N, N_Y_ROWS, replace=False))
    accf = f.xq[rows].astype(np.float64) @ f.wq.T.astype(np.float64)
    got = _acc_rows(H, 0, None, saved, N, D, C, rows, (N, C))
    assert np.array_equal(got, accf.astype(np.int32)), "forward int32 accumulator rows"
    ref = float(f.s_x) * float(f.s_w) * 2.0 ** -k * accf
    check_float_output("Y rows", Y[torch.from_numpy(rows).cuda()], ref, dt)
    del X, W

    seed, offset = 42, 1000
    b = O.lss_backward(G, f, N, seed, offset, need_dx=False, need_dw=False)
    tG, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N, seed, offset)
    nk = check_plan(plan, b)
    say(f"  kept {nk}/{N}")
    # the leverage scores of every stacked row, bit for bit
    ws = H.workspace(H.WS_PLAN, N, D, C)
    H.lss_grad_plan(tG, saved, H.Plan.empty(N, C), D, N, seed, offset, ws)
    torch.cuda.synchronize()
    off, pitch = H.debug_plan_scores_offset(N)
    raw = to_np(ws)[off:off + 8 * pitch].view(np.uint32)
    su = (b.bs.q_up.astype(np.int64) ** 2).sum(1)
    sd = (b.bs.q_dn.astype(np.int64) ** 2).sum(1)
    assert np.array_equal(np.concatenate([raw[:N], raw[pitch:pitch + N]]).astype(np.int64),
                          O.leverage_scores(su, sd, f.x_sumsq)), "leverage scores"
    del ws, tG
    A = b.A.astype(np.float64)
    kept = b.plan.kept
    a_dx, a_dw = b.alpha_dx, b.alpha_dw
    # dX: sampled kept tokens (accumulator rows sit at the tokens' positions in the kept list)
    pos = np.sort(rng.choice(len(kept), min(N_DX_TOKENS, len(kept)), replace=False))
    toks = kept[pos]
    accx = A[toks] @ f.wq.astype(np.float64)
    got = _acc_rows(H, 1, plan, saved, N, D, C, pos, (N, D))
    assert np.array_equal(got, accx.astype(np.int32)), "dX int32 accumulator rows"
    refx = a_dx * O.fwht_rows(accx.astype(np.int64), k).astype(np.float64)
    check_float_output("dX rows", dX[torch.from_numpy(toks).cuda()], refx, dt)
    dropped = np.setdiff1d(np.arange(N), kept)
    if len(dropped):
        assert not dX[torch.from_numpy(dropped[:N_DX_TOKENS]).cuda()].float().abs().sum().item()
    # dW: sampled rows c (all D columns, so whole Hadamard blocks)
    cs = np.sort(rng.choice(C, N_DW_ROWS, replace=False))
    accw = A[kept][:, cs].T @ f.xq[kept].astype(np.float64)
    got = _acc_rows(H, 2, plan, saved, N, D, C, cs, (C, D))
    assert np.array_equal(got, accw.astype(np.int32)), "dW int32 accumulator rows"
    refw = a_dw * O.fwht_rows(accw.astype(np.int64), k).astype(np.float64)
    check_float_output("dW rows", dW[torch.from_numpy(cs).cuda()], refw, dt)


def test_sampler_max_tokens():
    """The largest admitted token count (N = 65536, eight rounds of the one-workgroup
    sampler) with the clamp-and-rescale loop and the Bernoulli draws live (budget N/8):
    plan and both gradients against the oracle."""
    H = need_gpu()
    lin, X, W, G = _case((65536, 64, 128, 5, "bf16", "lognormal"), seed=6)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"sampler at N={N}")
    saved, _ = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    b = O.lss_backward(G, f, N // 8, 3, 11)
    assert b.plan.R > 0 and (b.plan.e_dn > 0).any()
    _, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N // 8, 3, 11)
    check_plan(plan, b)
    check_backward_acc(H, plan, saved, b, N, D, C)
    check_float_output("dX", dX, b.dX, dt)
    check_float_output("dW", dW, b.dW, dt)


@pytest.mark.parametrize("N,kind", [(3000, "lognormal"), (6000, "lognormal"), (12000, "lognormal"),
                                    (16384, "lognormal"), (16384, "pareto"), (12000, "sparse_rows")])
def test_sampler_clamp_sizes(N, kind):
    """The clamp-and-rescale loop live (budget N/4) on both sides of the sampler's size
    limits: the 256-thread build (N <= 4096, full passes over the scores) and the
    1024-thread one (binned scores); one or two compaction rounds (N > 8192); up to the
    largest N whose scores the clamp rounds hold in registers (2N = 32768;
    test_sampler_max_tokens covers the memory path).  Heavy-tailed and sparse rows put many
    scores in few bins.  Plan and both gradients against the oracle."""
    H = need_gpu()
    lin, X, W, G = _case((N, 64, 128, 5, "f16", kind), seed=N)
    D, C, k, dt = lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"sampler clamp at N={N}")
    saved, _ = run_forward(H, X, W, k, dt)
    f = O.hq_forward(X, W, k, compute_output=False)
    b = O.lss_backward(G, f, N // 4, 5, 7)
    assert (b.plan.e_dn > 0).any()
    _, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N // 4, 5, 7)
    check_plan(plan, b)
    check_float_output("dX", dX, b.dX, dt)
    check_float_output("dW", dW, b.dW, dt)


@pytest.mark.parametrize("splits", [2, 3])
@pytest.mark.parametrize("shape", [(600, 1024, 512, 7, "bf16", "pareto"), (300, 256, 320, 5, "f16", "lognormal")],
                         ids=["C512", "C320"])
def test_forced_split_k_parity(splits, shape):
    """Every GEMM split along K into int32 partials and re-summed: still bit-exact (C = 320
    leaves the last 128-row tile of the dW product half outside C)."""
    H = need_gpu()
    lin, X, W, G = _case(shape, seed=4)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"forced split-K {splits} {shape}")
    H.debug_set_gemm_splits(splits)
    try:
        saved, Y = run_forward(H, X, W, k, dt)
        check_forward(H, X, W, k, dt, saved, Y)
        f = O.hq_forward(X, W, k, compute_output=False)
        b = O.lss_backward(G, f, N // 2, 5, 0)
        _, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N // 2, 5, 0)
        check_plan(plan, b)
        check_backward_acc(H, plan, saved, b, N, D, C)
        check_float_output("dX", dX, b.dX, dt)
        check_float_output("dW", dW, b.dW, dt)
    finally:
        H.debug_set_gemm_splits(0)


@pytest.mark.parametrize("bn", [128, 256])
def test_forced_gemm_tile_width(bn):
    """Forward and gradient GEMMs with 128- or 256-wide workgroup tiles on a shape that
    fills neither width (C = 320 and D = 448 output columns, 600 tokens): bit-exact against
    the oracle under both widths."""
    H = need_gpu()
    lin, X, W, G = _case((600, 448, 320, 5, "f16", "lognormal"), seed=8)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    say(f"forced GEMM tile width {bn}")
    H.debug_set_gemm_tile_n(bn)
    try:
        saved, Y = run_forward(H, X, W, k, dt)
        check_forward(H, X, W, k, dt, saved, Y)
        f = O.hq_forward(X, W, k, compute_output=False)
        b = O.lss_backward(G, f, N // 2, 6, 0)
        _, plan, dX, dW = run_backward(H, G, saved, N, D, C, k, dt, N // 2, 6, 0)
        check_plan(plan, b)
        check_float_output("dX", dX, b.dX, dt)
        check_float_output("dW", dW, b.dW, dt)
    finally:
        H.debug_set_gemm_tile_n(0)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}")
def test_forward_fp6_product(shape):
    """hq_linear_fwd with its product forced onto the FP6 MFMA (the quantizer then also
    writes the codes as FP6): codes, scales and row sums bit-exact against the oracle, Y
    within the forward tolerance, and Y bit for bit the int8 product's."""
    H = need_gpu()
    lin, X, W, _ = _case(shape, seed=3)
    k, dt = lin.log2_block, lin.dtype
    say(f"forward, FP6 product {shape}")
    try:
        H.debug_set_fwd_fp6(1)
        saved6, Y6 = run_forward(H, X, W, k, dt)
        rel = check_forward(H, X, W, k, dt, saved6, Y6)
        assert rel <= (1e-5 if dt == "f32" else 2e-3)
        H.debug_set_fwd_fp6(-1)
        saved8, Y8 = run_forward(H, X, W, k, dt)
    finally:
        H.debug_set_fwd_fp6(0)
    assert torch.equal(Y6.view(torch.int16 if Y6.dtype != torch.float32 else torch.int32),
                       Y8.view(torch.int16 if Y8.dtype != torch.float32 else torch.int32))
    for name in ("xq", "wq", "wqT", "x_sumsq", "amax"):
        assert torch.equal(getattr(saved6, name), getattr(saved8, name)), name
