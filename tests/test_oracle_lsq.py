"""Pins of the oracle's learned-step-size mode (Sec. 3.1 Eq. 2, Sec. 4, App. A.3).

Each pin ties the oracle to something other than itself: a textbook quantiser, the
dynamic mode where the two must agree, the straight-through-estimator derivatives that
torch's autograd computes in float64, special inputs with known results, and an exact
reconstruction.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O


def _hadamard_block(D, k):
    H = O.hadamard_matrix_sylvester(k).astype(np.float64)
    return np.kron(np.eye(D >> k), H)


def test_lsq_codes_textbook_k0():
    # k = 0 (no transform), power-of-two steps: v / s is exact, so the oracle's codes,
    # mask and delta equal the textbook quantiser computed with exact division
    rng = np.random.default_rng(3)
    v = (rng.standard_normal((40, 64)) * 3).astype(np.float32)
    for s in (0.25, 0.5, 1.0):
        q, inside, d16 = O.quantize_lsq(v, s)
        r = v.astype(np.float64) / s
        q_ref = np.clip(np.round(r), -7, 7)  # numpy rounds half to even
        assert np.array_equal(q.astype(np.float64), q_ref)
        assert np.array_equal(inside, np.abs(r) <= 7)
        d_ref = (q_ref - np.where(np.abs(r) <= 7, r, 0.0)).astype(np.float16)
        assert np.array_equal(d16, d_ref)


def test_lsq_mask_recovered_from_delta():
    # |delta| <= 1/2 exactly inside [-7, 7] and |delta| = 7 outside, including the edges
    s = np.float32(0.5)
    r = np.array([-7.5, -7.0, -6.5, -0.25, 0.0, 0.5, 6.75, 7.0, 7.0 + 2 ** -20, 7.25, 100.0],
                 dtype=np.float32)
    q, inside, d16 = O.quantize_lsq(r * s, s)
    assert np.array_equal(inside, (r >= -7) & (r <= 7))
    assert np.array_equal(np.abs(d16.astype(np.float64)) <= 0.5, inside)
    assert np.all(np.abs(d16[~inside]) == 7)


def test_lsq_no_clipping_matches_dynamic_backward():
    # with every value inside the range the masks are 1 and the LSQ gradients are the
    # dynamic mode's formula on the same codes and steps
    rng = np.random.default_rng(5)
    X = rng.standard_normal((48, 64)).astype(np.float32)
    W = (rng.standard_normal((32, 64)) * 0.02).astype(np.float32)
    G = (rng.standard_normal((48, 32)) * 1e-3).astype(np.float32)
    k = 3
    vx, vw = O.fwht_rows(X, k), O.fwht_rows(W, k)
    sx = np.float32(2.0 ** math.ceil(math.log2(float(O.absmax(vx)) / 7)))
    sw = np.float32(2.0 ** math.ceil(math.log2(float(O.absmax(vw)) / 7)))
    f = O.lsq_forward(X, W, k, sx, sw)
    assert np.all(np.abs(f.dx16.astype(np.float64)) <= 0.5) and np.all(np.abs(f.dw16.astype(np.float64)) <= 0.5)
    hq = O.HQForward(k, np.float32(0), np.float32(0), sx, sw, f.xq, f.wq, f.x_sumsq)
    b_lsq = O.lsq_backward(G, f, 0, 11, 7)
    b_dyn = O.lss_backward(G, hq, 0, 11, 7)
    assert np.array_equal(b_lsq.plan.kept, b_dyn.plan.kept)
    assert np.allclose(b_lsq.dX, b_dyn.dX, rtol=0, atol=0)
    assert np.allclose(b_lsq.dW, b_dyn.dW, rtol=0, atol=0)


def test_lsq_all_clipped():
    # a tiny step clips everything: codes are the signs times 7, masks are 0, so dX = dW =
    # 0, and delta = +-7 carries the whole step-size gradient
    rng = np.random.default_rng(6)
    X = rng.standard_normal((32, 64)).astype(np.float32) + 3.0
    W = rng.standard_normal((16, 64)).astype(np.float32) + 3.0
    G = rng.standard_normal((32, 16)).astype(np.float32)
    f = O.lsq_forward(X, W, 0, 2 ** -12, 2 ** -12)
    assert np.all(np.abs(f.xq) == 7) and np.all(f.xq == 7 * np.sign(X).astype(np.int8))
    b = O.lsq_backward(G, f, O.KEEP_NONZERO, 1, 0)
    assert not np.any(b.dX) and not np.any(b.dW)
    ref = O.lsq_grad_scale(32 * 64) * b.alpha_dx * float(np.sum(b.acc_dx * 7.0 * np.sign(X)[b.plan.kept]))
    assert b.ds_x == pytest.approx(ref, rel=1e-12)


def test_lsq_exact_reconstruction():
    # X = s Q H_u / b with integer |Q| <= 7: the transform returns s Q exactly, the codes
    # are Q, delta is 0 and Y is s_x s_w Q_x Q_w^T / b exactly
    rng = np.random.default_rng(7)
    k, D = 4, 64
    H = _hadamard_block(D, k)
    Qx = rng.integers(-7, 8, (24, D))
    Qw = rng.integers(-7, 8, (16, D))
    sx, sw = 0.125, 0.5
    X = (sx * Qx @ H / (1 << k)).astype(np.float32)
    W = (sw * Qw @ H / (1 << k)).astype(np.float32)
    f = O.lsq_forward(X, W, k, sx, sw)
    assert np.array_equal(f.xq, Qx) and np.array_equal(f.wq, Qw)
    assert not np.any(f.dx16) and not np.any(f.dw16)
    assert np.array_equal(f.Y, sx * sw * (Qx @ Qw.T) / (1 << k))


@pytest.mark.parametrize("k", [0, 2, 3])
def test_lsq_gradients_equal_autograd(k):
    # torch float64 autograd of L = sum(gY o Y) through the straight-through LSQ forward
    # (clamp derivative = mask, rounding derivative = 1) gives dX, dW and the step-size
    # gradients.  Inputs are small integers and the steps powers of two so that the
    # oracle's float32 transform and v / s are exact; with the keep-non-zero sample the
    # LSS estimate of grad_Y is the bit-split product exactly, which is what gY is here.
    rng = np.random.default_rng(100 + k)
    N, D, C = 24, 32, 16
    X = rng.integers(-20, 21, (N, D)).astype(np.float32)
    W = rng.integers(-9, 10, (C, D)).astype(np.float32)
    G = (rng.standard_normal((N, C)) * 1e-2).astype(np.float32)
    sx, sw = 2.0 ** 1, 2.0 ** 0  # a share of the entries clip
    f = O.lsq_forward(X, W, k, sx, sw)
    vx, vw = O.fwht_rows(X, k), O.fwht_rows(W, k)
    dx_exact = f.xq.astype(np.float64) - np.where(np.abs(vx / sx) <= 7, vx / sx, 0.0)
    dw_exact = f.wq.astype(np.float64) - np.where(np.abs(vw / sw) <= 7, vw / sw, 0.0)
    b = O.lsq_backward(G, f, O.KEEP_NONZERO, 3, 0, delta_x=dx_exact, delta_w=dw_exact)
    assert 0 < (np.abs(vx / sx) > 7).mean() < 1 and 0 < (np.abs(vw / sw) > 7).mean() < 1
    gY = torch.from_numpy(b.bs.s_dn * O.weighted_rows(b.bs, b.plan).astype(np.float64))

    H = torch.from_numpy(_hadamard_block(D, k))
    tX = torch.from_numpy(X.astype(np.float64)).requires_grad_()
    tW = torch.from_numpy(W.astype(np.float64)).requires_grad_()
    tsx = torch.tensor(sx, dtype=torch.float64, requires_grad=True)
    tsw = torch.tensor(sw, dtype=torch.float64, requires_grad=True)

    def lsq(v, s):
        c = torch.clamp(v / s, -7, 7)
        return s * (c + (torch.round(c) - c).detach())

    Y = lsq(tX @ H, tsx) @ lsq(tW @ H, tsw).T / (1 << k)
    (gY * Y).sum().backward()
    assert np.allclose(b.dX, tX.grad.numpy(), rtol=1e-12, atol=1e-15)
    assert np.allclose(b.dW, tW.grad.numpy(), rtol=1e-12, atol=1e-15)
    assert b.ds_x == pytest.approx(tsx.grad.item() / math.sqrt(7 * N * D), rel=1e-12)
    assert b.ds_w == pytest.approx(tsw.grad.item() / math.sqrt(7 * C * D), rel=1e-12)
    # the stored float16 deltas move the step gradients by at most 2^-11 relative per term
    b16 = O.lsq_backward(G, f, O.KEEP_NONZERO, 3, 0)
    assert np.array_equal(b16.dX, b.dX) and np.array_equal(b16.dW, b.dW)
    bound_x = O.lsq_grad_scale(N * D) * b.alpha_dx * float(np.sum(np.abs(b.acc_dx) * np.abs(dx_exact)[b.plan.kept])) * 2 ** -11
    assert abs(b16.ds_x - b.ds_x) <= bound_x


def test_lsq_grad_scale_values():
    # g(s) = 1 / sqrt(Q_P * numel) with Q_P = 7 (App. A.3): 7 * 448 = 56^2, 7 * 28 = 14^2
    assert O.lsq_grad_scale(448) == 1 / 56
    assert O.lsq_grad_scale(28) == 1 / 14
    # the autograd pin's shapes: 7 * 24 * 32 and 7 * 16 * 32
    assert O.lsq_grad_scale(24 * 32) == pytest.approx(1 / math.sqrt(5376), rel=1e-15)
    assert O.lsq_grad_scale(16 * 32) == pytest.approx(1 / math.sqrt(3584), rel=1e-15)
