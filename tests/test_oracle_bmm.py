"""Pins of the oracle's attention BMM T = BMM(Q, K^T) (App. A.1) with per-batch learned steps.

The batched gradients, including every per-batch step-size gradient, are pinned against
torch float64 autograd of the batched straight-through forward; the per-batch random
streams against single-instance calls at their documented counters.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O


def _hadamard_block(D, k):
    H = O.hadamard_matrix_sylvester(k).astype(np.float64)
    return np.kron(np.eye(D >> k), H)


@pytest.mark.parametrize("k", [0, 3])
def test_bmm_gradients_equal_autograd(k):
    # integer inputs and power-of-two steps keep the float32 transform and v / s exact;
    # the keep-non-zero sample makes the LSS estimate the bit-split product itself
    rng = np.random.default_rng(200 + k)
    B, N, P, M = 3, 16, 24, 32
    Q = rng.integers(-20, 21, (B, N, M)).astype(np.float32)
    K = rng.integers(-9, 10, (B, P, M)).astype(np.float32)
    G = (rng.standard_normal((B, N, P)) * 1e-2).astype(np.float32)
    s_q = np.array([2.0, 4.0, 1.0], dtype=np.float32)
    s_k = np.array([1.0, 0.5, 2.0], dtype=np.float32)
    fw = O.bmm_lsq_forward(Q, K, k, s_q, s_k)
    exact = []
    for b in range(B):
        vq, vk = O.fwht_rows(Q[b], k), O.fwht_rows(K[b], k)
        dq = fw[b].xq.astype(np.float64) - np.where(np.abs(vq / s_q[b]) <= 7, vq / s_q[b], 0.0)
        dk = fw[b].wq.astype(np.float64) - np.where(np.abs(vk / s_k[b]) <= 7, vk / s_k[b], 0.0)
        exact.append((dq, dk))
    bw = [O.lsq_backward(G[b], fw[b], O.KEEP_NONZERO, 5, b * O.bmm_counter_stride(N, P),
                         delta_x=exact[b][0], delta_w=exact[b][1]) for b in range(B)]
    gY = torch.from_numpy(np.stack([bw[b].bs.s_dn * O.weighted_rows(bw[b].bs, bw[b].plan)
                                    .astype(np.float64) for b in range(B)]))

    H = torch.from_numpy(_hadamard_block(M, k))
    tQ = torch.from_numpy(Q.astype(np.float64)).requires_grad_()
    tK = torch.from_numpy(K.astype(np.float64)).requires_grad_()
    tsq = torch.from_numpy(s_q.astype(np.float64)).requires_grad_()
    tsk = torch.from_numpy(s_k.astype(np.float64)).requires_grad_()

    def lsq(v, s):  # s: [B] -> per-batch step
        s = s.view(-1, 1, 1)
        c = torch.clamp(v / s, -7, 7)
        return s * (c + (torch.round(c) - c).detach())

    T = torch.bmm(lsq(tQ @ H, tsq), lsq(tK @ H, tsk).transpose(1, 2).contiguous()) / (1 << k)
    (gY * T).sum().backward()
    for b in range(B):
        assert np.all(np.abs(fw[b].Y - T[b].detach().numpy()) <= 1e-12 * np.abs(fw[b].Y).max())
        assert np.allclose(bw[b].dX, tQ.grad[b].numpy(), rtol=1e-12, atol=1e-15)
        assert np.allclose(bw[b].dW, tK.grad[b].numpy(), rtol=1e-12, atol=1e-15)
        assert bw[b].ds_x == pytest.approx(tsq.grad[b].item() / math.sqrt(7 * N * M), rel=1e-12)
        assert bw[b].ds_w == pytest.approx(tsk.grad[b].item() / math.sqrt(7 * P * M), rel=1e-12)
    assert 0 < sum(float((np.abs(e[0]) > 0.5).mean()) for e in exact) < B  # some entries clip


def test_bmm_batches_use_their_own_counters():
    # with the Bernoulli draws live, batch b of the batched backward is the single-instance
    # backward at counter offset + b * bmm_counter_stride(N, P); equal batches therefore draw
    # different (independent) samples
    rng = np.random.default_rng(7)
    B, N, P, M = 3, 64, 64, 64
    Q1 = rng.standard_normal((N, M)).astype(np.float32)
    K1 = rng.standard_normal((P, M)).astype(np.float32)
    G1 = (rng.standard_normal((N, P)) * np.exp(rng.standard_normal((N, 1)) * 2)).astype(np.float32)
    Q, K, G = (np.repeat(a[None], B, 0) for a in (Q1, K1, G1))
    s = np.full(B, 0.2, dtype=np.float32)
    fw = O.bmm_lsq_forward(Q, K, 2, s, s, compute_output=False)
    seed, off, budget = 3, 11, N // 4
    bw = O.bmm_lsq_backward(G, fw, budget, seed, off)
    adv = O.bmm_counter_stride(N, P)
    assert adv == (N * P) // 8
    for b in range(B):
        ref = O.lsq_backward(G1, fw[b], budget, seed, off + b * adv)
        assert np.array_equal(bw[b].plan.kept, ref.plan.kept)
        assert np.array_equal(bw[b].dX, ref.dX) and np.array_equal(bw[b].dW, ref.dW)
    assert (bw[0].plan.e_dn > 0).any()
    assert not np.array_equal(bw[0].plan.w_dn, bw[1].plan.w_dn)
    # the streams of consecutive batches do not overlap: batch 1's first stochastic-rounding
    # uniforms are the ones a single instance would draw right after its last
    u = O.uniforms16(seed, off, O.STREAM_SR, 2 * N * P)
    assert np.array_equal(u[N * P:], O.uniforms16(seed, off + adv, O.STREAM_SR, N * P))
