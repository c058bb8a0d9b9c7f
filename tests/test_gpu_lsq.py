"""GPU parity of the learned-step-size mode (Eq. 2 with Sec. 3.3; App. A.3) through the C ABI.

Bit-exact: codes, row sums, fp16 deltas, the sample.  Float outputs (Y, dX, dW): as in
the dynamic mode, 1e-5 relative (fp32) or one unit in the last place of the output dtype
around the fp64 oracle value.  Step-size gradients: both sides form the same exact fp64
products acc * delta and differ only in the order of the fp64 sum and in the final fp32
rounding, so |got - ref| <= 2^-24 |ref| + 2 (n - 1) 2^-53 g a sum|acc * delta| for n terms.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import check_float_output, dev_tensor, need_gpu, say, to_np, TORCH_DT

pytestmark = pytest.mark.gpu

# (N, D, C, log2_block, dtype, grad_kind): several tiles, ragged N, every dtype and block
SHAPES = [
    (128, 256, 256, 5, "f32", "sparse_rows"),
    (1, 64, 64, 0, "f32", "lognormal"),
    (200, 192, 320, 6, "f16", "lognormal"),
    (333, 256, 128, 7, "bf16", "pareto"),
    (77, 512, 576, 3, "f16", "pareto"),
    (517, 128, 704, 1, "f32", "pareto"),
    (2048, 256, 256, 5, "bf16", "lognormal"),  # dW over 2048 tokens: split-K by default
]
IDS = [f"N{s[0]}_D{s[1]}_C{s[2]}_k{s[3]}_{s[4]}" for s in SHAPES]


def _case(shape, seed=0):
    N, D, C, k, dt, kind = shape
    lin = synth.Linear(f"t{N}x{D}x{C}", N, D, C, k, dt, max(1, D // 100), 20.0, kind, N)
    X, W, G = synth.linear_inputs(lin, seed)
    return lin, X, W, G


def _steps(X, W, k, clip_frac=0.02):
    """fp32 steps that clip about clip_frac of the transformed entries (not powers of two,
    so that fl(1/s) rounds)."""
    out = []
    for V in (X, W):
        v = np.abs(O.fwht_rows(np.asarray(V, dtype=np.float32), k)).ravel()
        out.append(np.float32(np.quantile(v, 1.0 - clip_frac) / 7.0 * 1.0173))
    return out


def run_forward_lsq(H, X, W, k, dt, sx, sw):
    N, D = X.shape
    C = W.shape[0]
    tX, tW = dev_tensor(X, dt), dev_tensor(W, dt)
    Y = torch.empty(N, C, device="cuda", dtype=TORCH_DT[dt])
    saved = H.Saved.empty(N, D, C)
    step = torch.tensor([sx, sw], dtype=torch.float32, device="cuda")
    lsq = H.LSQ.empty(step, N, D, C)
    H.hq_linear_fwd_lsq(tX, tW, Y, saved, lsq, k)
    return saved, lsq, Y


def check_forward_codes(saved, lsq, f):
    torch.cuda.synchronize()
    assert np.array_equal(to_np(saved.xq), O.pack_int4(f.xq)), "X codes"
    assert np.array_equal(to_np(saved.wq), O.pack_int4(f.wq)), "W codes"
    assert np.array_equal(to_np(saved.wqT), O.pack_int4(f.wq.T.copy())), "W^T codes"
    assert np.array_equal(to_np(saved.x_sumsq), f.x_sumsq.astype(np.int32)), "x_sumsq"
    assert np.array_equal(to_np(lsq.delta_x).view(np.uint16), f.dx16.view(np.uint16)), "delta_X"
    assert np.array_equal(to_np(lsq.delta_w).view(np.uint16), f.dw16.view(np.uint16)), "delta_W"


def check_step_grad(got, ref, g, a, acc, delta):
    terms = np.abs(acc.astype(np.float64) * delta.astype(np.float64))
    n = max(terms.size, 1)
    tol = 2.0 ** -24 * abs(ref) + 2 * n * 2.0 ** -53 * g * abs(a) * float(terms.sum())
    assert abs(got - ref) <= tol, (got, ref, tol)


def run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, budget, seed, offset, want=(True, True)):
    tG = dev_tensor(G, dt)
    dX = torch.empty(N, D, device="cuda", dtype=TORCH_DT[dt]) if want[0] else None
    dW = torch.empty(C, D, device="cuda", dtype=TORCH_DT[dt]) if want[1] else None
    dstep = torch.full((2,), float("nan"), dtype=torch.float32, device="cuda")
    H.lss_linear_bwd_lsq(tG, saved, lsq, dX, dW, dstep, D, k, budget, seed, offset)
    return dX, dW, dstep


def check_backward(dX, dW, dstep, f, b, N, D, C, dt):
    torch.cuda.synchronize()
    check_float_output("dX", dX, b.dX, dt)
    check_float_output("dW", dW, b.dW, dt)
    ds = to_np(dstep).astype(np.float64)
    check_step_grad(ds[0], b.ds_x, O.lsq_grad_scale(N * D), b.alpha_dx, b.acc_dx,
                    f.dx16[b.plan.kept])
    check_step_grad(ds[1], b.ds_w, O.lsq_grad_scale(C * D), b.alpha_dw, b.acc_dw, f.dw16)


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_lsq_forward_parity(shape):
    H = need_gpu()
    lin, X, W, _ = _case(shape)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sx, sw = _steps(X, W, k)
    say(f"lsq forward parity {shape} s=({sx!r}, {sw!r})")
    saved, lsq, Y = run_forward_lsq(H, X, W, k, dt, sx, sw)
    f = O.lsq_forward(X, W, k, sx, sw)
    check_forward_codes(saved, lsq, f)
    assert np.abs(f.dx16.astype(np.float64)).max() > 0.5 or N * D < 2000, "no entry clipped"
    check_float_output("Y", Y, f.Y, dt)


@pytest.mark.parametrize("budget", [0, 3, -1], ids=["budgetN", "budget3", "keepnz"])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_lsq_backward_parity(shape, budget):
    H = need_gpu()
    lin, X, W, G = _case(shape, seed=1)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sx, sw = _steps(X, W, k)
    bud = {0: N, 3: max(1, N // 3), -1: H.BUDGET_KEEP_NONZERO}[budget]
    seed, offset = 4321, 19
    say(f"lsq backward parity {shape} budget={bud}")
    saved, lsq, _ = run_forward_lsq(H, X, W, k, dt, sx, sw)
    f = O.lsq_forward(X, W, k, sx, sw, compute_output=False)
    b = O.lsq_backward(G, f, O.KEEP_NONZERO if bud == H.BUDGET_KEEP_NONZERO else bud, seed, offset)
    dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, bud, seed, offset)
    check_backward(dX, dW, dstep, f, b, N, D, C, dt)

    # one gradient at a time: the same sample, the same outputs and step gradient, and the
    # other step gradient left unwritten
    dX1, _, ds1 = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, bud, seed, offset, (True, False))
    _, dW2, ds2 = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, bud, seed, offset, (False, True))
    torch.cuda.synchronize()
    assert torch.equal(dX1, dX) and torch.equal(dW2, dW)
    assert ds1[0].item() == dstep[0].item() and np.isnan(ds1[1].item())
    assert ds2[1].item() == dstep[1].item() and np.isnan(ds2[0].item())


@pytest.mark.parametrize("splits", [2, 3])
def test_lsq_forced_split_k(splits):
    """Every GEMM split along K: the reduction kernel then applies the masks and forms the
    partial sums of the step gradients."""
    H = need_gpu()
    lin, X, W, G = _case((600, 1024, 512, 7, "bf16", "pareto"), seed=4)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sx, sw = _steps(X, W, k, 0.05)
    say(f"lsq forced split-K {splits}")
    H.debug_set_gemm_splits(splits)
    try:
        saved, lsq, Y = run_forward_lsq(H, X, W, k, dt, sx, sw)
        f = O.lsq_forward(X, W, k, sx, sw)
        check_forward_codes(saved, lsq, f)
        check_float_output("Y", Y, f.Y, dt)
        b = O.lsq_backward(G, f, N // 2, 5, 0)
        dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N // 2, 5, 0)
        check_backward(dX, dW, dstep, f, b, N, D, C, dt)
    finally:
        H.debug_set_gemm_splits(0)


@pytest.mark.parametrize("bn", [128, 256])
def test_lsq_forced_gemm_tile_width(bn):
    """The learned-step forward and the masked gradient epilogues with their step-gradient
    partial sums (one per workgroup, as many as the tile width gives) under 128- and
    256-wide tiles."""
    H = need_gpu()
    lin, X, W, G = _case((600, 448, 320, 5, "f16", "lognormal"), seed=8)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sx, sw = _steps(X, W, k, 0.05)
    say(f"lsq forced gradient tile width {bn}")
    H.debug_set_gemm_tile_n(bn)
    try:
        saved, lsq, Y = run_forward_lsq(H, X, W, k, dt, sx, sw)
        f = O.lsq_forward(X, W, k, sx, sw)
        check_forward_codes(saved, lsq, f)
        check_float_output("Y", Y, f.Y, dt)
        b = O.lsq_backward(G, f, N // 2, 6, 0)
        dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N // 2, 6, 0)
        check_backward(dX, dW, dstep, f, b, N, D, C, dt)
    finally:
        H.debug_set_gemm_tile_n(0)


def test_lsq_deterministic():
    """Equal inputs give bit-identical gradients and step gradients (fixed-order sums)."""
    H = need_gpu()
    lin, X, W, G = _case((1000, 512, 384, 5, "f16", "lognormal"), seed=8)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    sx, sw = _steps(X, W, k)
    saved, lsq, _ = run_forward_lsq(H, X, W, k, dt, sx, sw)
    outs = [run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N // 2, 3, 3) for _ in range(2)]
    torch.cuda.synchronize()
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)


def test_lsq_all_clipped_and_all_zero():
    """A tiny step clips every entry (k = 0 and strictly positive inputs, so no transformed
    entry is 0): codes are 7, the masks are 0, so dX = dW = 0 exactly while the step
    gradients carry delta = 7.  A huge step gives all-zero codes: Y = 0, x_sumsq = 0, and
    every gradient and step gradient is 0."""
    H = need_gpu()
    lin, X, W, G = _case((130, 128, 192, 0, "bf16", "lognormal"), seed=2)
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    X = synth.round_to_dtype(np.abs(X) + np.float32(1.0), dt)
    W = synth.round_to_dtype(np.abs(W) + np.float32(0.01), dt)
    say("lsq all clipped")
    s = np.float32(2.0 ** -20)
    saved, lsq, _ = run_forward_lsq(H, X, W, k, dt, s, s)
    f = O.lsq_forward(X, W, k, s, s, compute_output=False)
    check_forward_codes(saved, lsq, f)
    assert np.all(f.dx16.astype(np.float64) == 7) and np.all(f.dw16.astype(np.float64) == 7)
    b = O.lsq_backward(G, f, N, 7, 0)
    dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N, 7, 0)
    torch.cuda.synchronize()
    assert not dX.float().abs().sum().item() and not dW.float().abs().sum().item()
    assert b.ds_x != 0 and b.ds_w != 0
    check_backward(dX, dW, dstep, f, b, N, D, C, dt)

    say("lsq all zero codes")
    big = np.float32(2.0 ** 40)
    saved, lsq, Y = run_forward_lsq(H, X, W, k, dt, big, big)
    dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N, 7, 0)
    torch.cuda.synchronize()
    assert not Y.float().abs().sum().item()
    assert not np.any(to_np(saved.x_sumsq))
    assert not dX.float().abs().sum().item() and not dW.float().abs().sum().item()
    assert np.array_equal(to_np(dstep), np.zeros(2, dtype=np.float32))


def test_lsq_exact_reconstruction():
    """X = s Q H_u / b with |Q| <= 7 and power-of-two steps: codes Q, deltas 0, and Y equals
    X W^T exactly."""
    import scipy.linalg
    H = need_gpu()
    k, bsz = 4, 16
    rng = np.random.default_rng(12)
    N, D, C = 70, 128, 64
    Qx = rng.integers(-7, 8, size=(N, D))
    Qw = rng.integers(-7, 8, size=(C, D))
    Hb = np.kron(np.eye(D // bsz), scipy.linalg.hadamard(bsz))
    sx, sw = np.float32(0.25), np.float32(2.0 ** -5)
    X = (float(sx) * Qx @ Hb / bsz).astype(np.float32)
    W = (float(sw) * Qw @ Hb / bsz).astype(np.float32)
    saved, lsq, Y = run_forward_lsq(H, X, W, k, "f32", sx, sw)
    torch.cuda.synchronize()
    assert np.array_equal(O.unpack_int4(to_np(saved.xq)), Qx)
    assert np.array_equal(O.unpack_int4(to_np(saved.wq)), Qw)
    assert not to_np(lsq.delta_x).any() and not to_np(lsq.delta_w).any()
    assert np.array_equal(to_np(Y).astype(np.float64), X.astype(np.float64) @ W.astype(np.float64).T)


def test_lsq_errors():
    """Argument errors are reported before anything is launched."""
    H = need_gpu()
    N, D, C = 64, 64, 64
    X = torch.zeros(N, D, device="cuda")
    W = torch.zeros(C, D, device="cuda")
    Y = torch.empty(N, C, device="cuda")
    saved = H.Saved.empty(N, D, C)
    step = torch.ones(2, dtype=torch.float32, device="cuda")
    lsq = H.LSQ.empty(step, N, D, C)
    bad = H.LSQ(step, None, lsq.delta_w)
    with pytest.raises(H.HQLSSError, match="NULL"):
        H.hq_linear_fwd_lsq(X, W, Y, saved, bad, 0)
    with pytest.raises(H.HQLSSError, match="block"):
        H.hq_linear_fwd_lsq(X, W, Y, saved, lsq, 7)
    H.hq_linear_fwd_lsq(X, W, Y, saved, lsq, 0)
    G = torch.zeros(N, C, device="cuda")
    with pytest.raises(H.HQLSSError, match="NULL"):
        H.lss_linear_bwd_lsq(G, saved, lsq, None, None, None, D, 0)
    small = torch.empty(256, dtype=torch.uint8, device="cuda")
    dX = torch.empty(N, D, device="cuda")
    with pytest.raises(H.HQLSSError, match="workspace"):
        H.lss_linear_bwd_lsq(G, saved, lsq, dX, None, None, D, 0, ws=small)


# (workload id, linear index) at full size: the BERT-base FFN pair and the GPT-2-medium
# b = 128 linear
FULL_SIZE = [(1, 0), (1, 1), (2, 0)]


@pytest.mark.parametrize("case", FULL_SIZE, ids=lambda c: f"w{c[0]}_{synth.workload(c[0]).linears[c[1]].name}")
def test_lsq_full_size(case):
    """A linear of a named workload at full size (budget N): every code and delta, sampled
    rows of Y, dX and dW, and both step gradients against their definitions (the full
    accumulators in exact fp64 matrix products)."""
    H = need_gpu()
    cid, li = case
    lin = synth.workload(cid).linears[li]
    N, D, C, k, dt = lin.N, lin.D, lin.C, lin.log2_block, lin.dtype
    X, W, G = synth.linear_inputs(lin, cid, li)
    sx, sw = _steps(X, W, k, 0.01)
    say(f"lsq full size {lin.name} N={N} D={D} C={C} b={1 << k} {dt}")
    saved, lsq, Y = run_forward_lsq(H, X, W, k, dt, sx, sw)
    f = O.lsq_forward(X, W, k, sx, sw, compute_output=False)
    check_forward_codes(saved, lsq, f)
    rng = np.random.default_rng(cid * 10 + li + 5)
    rows = rng.choice(N, 64, replace=False)
    ref = float(sx) * float(sw) * 2.0 ** -k * (f.xq[rows].astype(np.float64) @ f.wq.T.astype(np.float64))
    check_float_output("Y rows", Y[torch.from_numpy(rows).cuda()], ref, dt)

    seed, offset = 42, 1000
    b = O.lsq_backward(G, f, N, seed, offset, need_dx=False, need_dw=False)
    dX, dW, dstep = run_backward_lsq(H, G, saved, lsq, N, D, C, k, dt, N, seed, offset)
    kept = b.plan.kept
    say(f"  kept {len(kept)}/{N}")
    A = b.A.astype(np.float64)
    # whole accumulators: integers below 2^53, so the fp64 products are exact
    acc_dx = A[kept] @ f.wq.astype(np.float64)
    acc_dw = A[kept].T @ f.xq[kept].astype(np.float64)
    dlx = f.dx16[kept].astype(np.float64)
    dlw = f.dw16.astype(np.float64)
    a_dx, a_dw = b.alpha_dx, b.alpha_dw
    toks = rng.choice(len(kept), 32, replace=False)
    mx = np.where(np.abs(dlx[toks]) <= 0.5, acc_dx[toks], 0).astype(np.int64)
    check_float_output("dX rows", dX[torch.from_numpy(kept[toks]).cuda()],
                       a_dx * O.fwht_rows(mx, k).astype(np.float64), dt)
    cs = rng.choice(C, 16, replace=False)
    mw = np.where(np.abs(dlw[cs]) <= 0.5, acc_dw[cs], 0).astype(np.int64)
    check_float_output("dW rows", dW[torch.from_numpy(cs).cuda()],
                       a_dw * O.fwht_rows(mw, k).astype(np.float64), dt)
    torch.cuda.synchronize()
    ds = to_np(dstep).astype(np.float64)
    gx, gw = O.lsq_grad_scale(N * D), O.lsq_grad_scale(C * D)
    check_step_grad(ds[0], gx * a_dx * float(np.sum(acc_dx * dlx)), gx, a_dx, acc_dx, dlx)
    check_step_grad(ds[1], gw * a_dw * float(np.sum(acc_dw * dlw)), gw, a_dw, acc_dw, dlw)
