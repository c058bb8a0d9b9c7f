"""GPU parity of the attention BMM T = BMM(Q, K^T) with per-batch learned steps (App. A.1).

Every batch is checked against the oracle's batched functions: codes, row sums and fp16
deltas bit-exact, T to the float bound of the linear operator (1e-5 relative for fp32, one
unit in the last place of fp16 / bf16).
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import check_float_output, dev_tensor, need_gpu, say, to_np, TORCH_DT

pytestmark = pytest.mark.gpu

# (B, N, M, P, log2_block, dtype): ragged N, every dtype, attention-like head sizes
SHAPES = [
    (3, 100, 64, 128, 3, "f16"),
    (2, 7, 64, 64, 6, "f32"),
    (5, 300, 128, 192, 5, "bf16"),
    (24, 512, 64, 512, 6, "f16"),
]
IDS = [f"B{s[0]}_N{s[1]}_M{s[2]}_P{s[3]}_k{s[4]}_{s[5]}" for s in SHAPES]


def _inputs(shape, seed=0):
    B, N, M, P, k, dt = shape
    Qs, Ks, Gs = [], [], []
    for b in range(B):
        lin = synth.Linear(f"bmm{b}", N, M, P, k, dt, max(1, M // 32), 20.0, "lognormal", N)
        X, W, G = synth.linear_inputs(lin, seed * 1000 + b)
        Qs.append(X), Ks.append(W), Gs.append(G)
    return np.stack(Qs), np.stack(Ks), np.stack(Gs)


def _steps(V, k, clip_frac=0.02):
    """Per-batch fp32 steps clipping about clip_frac of each batch's transformed entries."""
    return np.array([np.quantile(np.abs(O.fwht_rows(V[b], k)), 1.0 - clip_frac) / 7.0 * 1.0173
                     for b in range(V.shape[0])], dtype=np.float32)


def run_bmm_forward(H, Q, K, k, dt, s_q, s_k):
    B, N, M = Q.shape
    P = K.shape[1]
    tQ, tK = dev_tensor(Q.reshape(B * N, M), dt).view(B, N, M), dev_tensor(K.reshape(B * P, M), dt).view(B, P, M)
    T = torch.empty(B, N, P, device="cuda", dtype=TORCH_DT[dt])
    saved = H.bmm_saved_empty(B, N, M, P)
    lsq = H.BmmLSQ.empty(torch.from_numpy(s_q).cuda(), torch.from_numpy(s_k).cuda(), N, M, P)
    H.hq_bmm_fwd_lsq(tQ, tK, T, saved, lsq, k)
    return saved, lsq, T


def check_bmm_codes(saved, lsq, fw):
    torch.cuda.synchronize()
    xq, wq, wqT, xs = (to_np(t) for t in (saved.xq, saved.wq, saved.wqT, saved.x_sumsq))
    dq, dk = to_np(lsq.delta_q).view(np.uint16), to_np(lsq.delta_k).view(np.uint16)
    for b, f in enumerate(fw):
        assert np.array_equal(xq[b], O.pack_int4(f.xq)), f"Q codes, batch {b}"
        assert np.array_equal(wq[b], O.pack_int4(f.wq)), f"K codes, batch {b}"
        assert np.array_equal(wqT[b], O.pack_int4(f.wq.T.copy())), f"K^T codes, batch {b}"
        assert np.array_equal(xs[b], f.x_sumsq.astype(np.int32)), f"row sums, batch {b}"
        assert np.array_equal(dq[b], f.dx16.view(np.uint16)), f"delta_Q, batch {b}"
        assert np.array_equal(dk[b], f.dw16.view(np.uint16)), f"delta_K, batch {b}"


@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_bmm_forward_parity(shape):
    H = need_gpu()
    B, N, M, P, k, dt = shape
    Q, K, _ = _inputs(shape)
    s_q, s_k = _steps(Q, k), _steps(K, k)
    say(f"bmm forward parity {shape}")
    saved, lsq, T = run_bmm_forward(H, Q, K, k, dt, s_q, s_k)
    fw = O.bmm_lsq_forward(Q, K, k, s_q, s_k)
    check_bmm_codes(saved, lsq, fw)
    check_float_output("T", T, np.stack([f.Y for f in fw]), dt)


def test_bmm_forward_errors():
    H = need_gpu()
    B, N, M, P = 2, 64, 64, 64
    Q = torch.zeros(B, N, M, device="cuda")
    K = torch.zeros(B, P, M, device="cuda")
    T = torch.empty(B, N, P, device="cuda")
    saved = H.bmm_saved_empty(B, N, M, P)
    s = torch.ones(B, dtype=torch.float32, device="cuda")
    lsq = H.BmmLSQ.empty(s, s, N, M, P)
    with pytest.raises(H.HQLSSError, match="block"):
        H.hq_bmm_fwd_lsq(Q, K, T, saved, lsq, 7)
    bad = H.BmmLSQ(s, None, lsq.delta_q, lsq.delta_k)
    with pytest.raises(H.HQLSSError, match="NULL"):
        H.hq_bmm_fwd_lsq(Q, K, T, saved, bad, 0)
    H.hq_bmm_fwd_lsq(Q, K, T, saved, lsq, 0)
    torch.cuda.synchronize()
    assert not T.abs().sum().item()


def _check_step_grad(got, ref, g, a, acc, delta):
    terms = np.abs(acc.astype(np.float64) * delta.astype(np.float64))
    n = max(terms.size, 1)
    tol = 2.0 ** -24 * abs(ref) + 2 * n * 2.0 ** -53 * g * abs(a) * float(terms.sum())
    assert abs(got - ref) <= tol, (got, ref, tol)


def run_bmm_backward(H, G, saved, lsq, M, k, dt, budget, seed, offset, want=(True, True)):
    B, N, P = G.shape
    tG = dev_tensor(G.reshape(B * N, P), dt).view(B, N, P)
    dQ = torch.empty(B, N, M, device="cuda", dtype=TORCH_DT[dt]) if want[0] else None
    dK = torch.empty(B, P, M, device="cuda", dtype=TORCH_DT[dt]) if want[1] else None
    nan = dict(dtype=torch.float32, device="cuda")
    ds_q, ds_k = torch.full((B,), float("nan"), **nan), torch.full((B,), float("nan"), **nan)
    H.lss_bmm_bwd_lsq(tG, saved, lsq, dQ, dK, ds_q, ds_k, M, k, budget, seed, offset)
    return dQ, dK, ds_q, ds_k


@pytest.mark.parametrize("budget", ["N", "N/3", "keepnz"])
@pytest.mark.parametrize("shape", SHAPES, ids=IDS)
def test_bmm_backward_parity(shape, budget):
    H = need_gpu()
    B, N, M, P, k, dt = shape
    Q, K, G = _inputs(shape, seed=1)
    s_q, s_k = _steps(Q, k), _steps(K, k)
    bud = {"N": N, "N/3": max(1, N // 3), "keepnz": H.BUDGET_KEEP_NONZERO}[budget]
    seed, offset = 77, 5
    say(f"bmm backward parity {shape} budget={bud}")
    saved, lsq, _ = run_bmm_forward(H, Q, K, k, dt, s_q, s_k)
    fw = O.bmm_lsq_forward(Q, K, k, s_q, s_k, compute_output=False)
    bw = O.bmm_lsq_backward(G, fw, O.KEEP_NONZERO if bud == H.BUDGET_KEEP_NONZERO else bud, seed, offset)
    dQ, dK, ds_q, ds_k = run_bmm_backward(H, G, saved, lsq, M, k, dt, bud, seed, offset)
    torch.cuda.synchronize()
    check_float_output("dQ", dQ, np.stack([b.dX for b in bw]), dt)
    check_float_output("dK", dK, np.stack([b.dW for b in bw]), dt)
    dsq, dsk = to_np(ds_q).astype(np.float64), to_np(ds_k).astype(np.float64)
    for b in range(B):
        _check_step_grad(dsq[b], bw[b].ds_x, O.lsq_grad_scale(N * M), bw[b].alpha_dx, bw[b].acc_dx,
                         fw[b].dx16[bw[b].plan.kept])
        _check_step_grad(dsk[b], bw[b].ds_w, O.lsq_grad_scale(P * M), bw[b].alpha_dw, bw[b].acc_dw,
                         fw[b].dw16)
    # one gradient at a time: identical outputs, the other step gradient left unwritten
    dQ1, _, q1, k1 = run_bmm_backward(H, G, saved, lsq, M, k, dt, bud, seed, offset, (True, False))
    _, dK2, q2, k2 = run_bmm_backward(H, G, saved, lsq, M, k, dt, bud, seed, offset, (False, True))
    torch.cuda.synchronize()
    assert torch.equal(dQ1, dQ) and torch.equal(dK2, dK)
    assert torch.equal(q1, ds_q) and torch.isnan(k1).all()
    assert torch.equal(k2, ds_k) and torch.isnan(q2).all()


def test_bmm_batches_match_single_instances():
    """Batch b of the batched backward equals the linear learned-step backward of that
    batch alone at counter offset + b * lss_philox_offset_advance(N, P) (bit for bit)."""
    H = need_gpu()
    shape = (4, 192, 64, 128, 4, "f16")
    B, N, M, P, k, dt = shape
    Q, K, G = _inputs(shape, seed=2)
    s_q, s_k = _steps(Q, k), _steps(K, k)
    saved, lsq, T = run_bmm_forward(H, Q, K, k, dt, s_q, s_k)
    dQ, dK, ds_q, ds_k = run_bmm_backward(H, G, saved, lsq, M, k, dt, N // 4, 9, 123)
    adv = H.lss_philox_offset_advance(N, P)
    for b in range(B):
        Y1 = torch.empty(N, P, device="cuda", dtype=TORCH_DT[dt])
        sv1 = H.Saved.empty(N, M, P)
        l1 = H.LSQ.empty(torch.tensor([s_q[b], s_k[b]], dtype=torch.float32, device="cuda"), N, M, P)
        H.hq_linear_fwd_lsq(dev_tensor(Q[b], dt), dev_tensor(K[b], dt), Y1, sv1, l1, k)
        dX1 = torch.empty(N, M, device="cuda", dtype=TORCH_DT[dt])
        dW1 = torch.empty(P, M, device="cuda", dtype=TORCH_DT[dt])
        st1 = torch.empty(2, dtype=torch.float32, device="cuda")
        H.lss_linear_bwd_lsq(dev_tensor(G[b], dt), sv1, l1, dX1, dW1, st1, M, k, N // 4, 9, 123 + b * adv)
        torch.cuda.synchronize()
        assert torch.equal(Y1, T[b]) and torch.equal(dX1, dQ[b]) and torch.equal(dW1, dK[b])
        assert st1[0].item() == ds_q[b].item() and st1[1].item() == ds_k[b].item()
