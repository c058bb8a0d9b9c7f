"""Pins of the oracle's leverage scores against their definition in Sec. 4.2.

The weight-gradient product is the sum of 2N rank-one terms
grad_W_i = (stacked gradient row i)^T (stacked X row i), with the stacked gradient
rows [s_up q_up; s_dn q_dn] and the stacked X rows [X^; X^] (Sec. 4.2, Eq. 5).
The leverage score is c_i = ||stacked gradient row i|| * ||stacked X row i||
(Sec. 4.2, Prop. 4.1), and the variance is smallest at p proportional to c
(the Cauchy inequality of Sec. 4.2).

Here every c_i is computed in float64 from the dequantised rows, as the Frobenius
norm of its rank-one term, with none of the oracle's score arithmetic.  The oracle's
integer scores must be one common multiple of them (up to the floor of its integer
square root), and its inclusion probabilities must reach the Cauchy optimum with
these independent scores.  Planted mistakes (a wrong upper-row weight, a dropped X
factor, swapped halves) each fail the pins.
"""
import math

import numpy as np
import pytest

import oracle as O
import synth


def _case(N, D, C, k, seed, grad_kind="pareto", gseed=11):
    lin = synth.small_linear(N, D, C, k, grad_kind=grad_kind)
    X, W, G = synth.linear_inputs(lin, seed)
    f = O.hq_forward(X, W, k, compute_output=False)
    bs = O.bit_split(G, gseed, 0)
    return G, f, bs


def _reference_scores(G, f, bs):
    """c_i = ||grad_W_i||_F for the 2N rank-one terms, in float64.

    The lower step is the one that makes s_up q_up + s_dn q_dn a bit split of G:
    it is checked here to bound the reconstruction error by one lower step (the
    residual quantiser's own error), so that the rows used are those of Eq. 4."""
    s_up = float(bs.s_up)
    s_dn = s_up / 14.0
    g_up = s_up * bs.q_up.astype(np.float64)
    g_dn = s_dn * bs.q_dn.astype(np.float64)
    err = np.abs(G.astype(np.float64) - g_up - g_dn).max()
    assert err < s_dn, "rows used are not a bit split of G"
    x_rows = float(f.s_x) * f.xq.astype(np.float64)
    grad_stacked = np.vstack([g_up, g_dn])
    x_stacked = np.vstack([x_rows, x_rows])
    c = np.empty(grad_stacked.shape[0])
    for i in range(grad_stacked.shape[0]):
        c[i] = np.linalg.norm(np.outer(grad_stacked[i], x_stacked[i]))  # Frobenius norm
    return c


def _sums(bs):
    su = (bs.q_up.astype(np.int64) ** 2).sum(1)
    sd = (bs.q_dn.astype(np.int64) ** 2).sum(1)
    return su, sd


def _proportionality_error(c_int, c_ref):
    """Largest deviation of c_int from kappa * c_ref, in units of one integer step,
    with kappa taken from the largest reference score.  Zero scores must match
    exactly (returned as inf otherwise)."""
    c_int = np.asarray(c_int, dtype=np.float64)
    zero_ref = c_ref == 0
    if np.any(c_int[zero_ref] != 0) or np.any(c_int[~zero_ref] == 0):
        return math.inf
    j = int(np.argmax(c_ref))
    kappa = c_int[j] / c_ref[j]
    dev = np.abs(c_int[~zero_ref] - kappa * c_ref[~zero_ref])
    # the integer square root floors: c_int lies in (kappa c - 1, kappa c]; kappa itself
    # carries the same floor of the largest score, relative 1 / c_int[j]
    slack = 1.0 + kappa * c_ref[~zero_ref] / c_int[j] + 1e-9 * kappa * c_ref[~zero_ref]
    return float(np.max(dev / slack))


CASES = [
    (48, 64, 32, 3, 0, "pareto"),
    (64, 32, 64, 5, 1, "lognormal"),
    (40, 128, 16, 7, 2, "sparse_rows"),
    (33, 64, 48, 0, 3, "pareto"),
]


@pytest.mark.parametrize("N,D,C,k,seed,kind", CASES)
def test_scores_proportional_to_rank_one_norms(N, D, C, k, seed, kind):
    """The oracle's integer scores are kappa * ||grad_W_i||_F for one kappa over all 2N
    stacked rows (Sec. 4.2 defines c_i up to the common factor nothing depends on)."""
    G, f, bs = _case(N, D, C, k, seed, kind)
    su, sd = _sums(bs)
    assert (su > 0).any() and (sd > 0).any(), "both halves must carry non-zero rows"
    c_ref = _reference_scores(G, f, bs)
    c = O.leverage_scores(su, sd, f.x_sumsq)
    assert c.shape == (2 * N,)
    assert _proportionality_error(c, c_ref) <= 1.0
    # the common factor is the one the integer form drops: 2^8 / (s_dn s_x)
    kappa = 256.0 / ((float(bs.s_up) / 14.0) * float(f.s_x))
    j = int(np.argmax(c_ref))
    assert abs(c[j] - kappa * c_ref[j]) <= 1.0 + 1e-9 * kappa * c_ref[j]


def _unclamped_budget(c):
    """A budget at which no row clamps: B * max(c) < sum(c)."""
    c = np.asarray(c, dtype=np.float64)
    B = int(np.sum(c) / np.max(c)) - 1
    return max(B, 1)


@pytest.mark.parametrize("N,D,C,k,seed,kind", CASES[:3])
def test_probabilities_reach_cauchy_optimum(N, D, C, k, seed, kind):
    """With no clamped row, sum_i c_i^2 / p_i equals (sum_i c_i)^2 / B at the oracle's p,
    with the independently computed c (the equality case of the Cauchy inequality,
    Sec. 4.2), and any other distribution with the same budget does no better."""
    G, f, bs = _case(N, D, C, k, seed, kind)
    su, sd = _sums(bs)
    c_ref = _reference_scores(G, f, bs)
    c_int = O.leverage_scores(su, sd, f.x_sumsq)
    B = _unclamped_budget(c_int)
    clamped, R, S = O.clamp_rescale(c_int, B)
    assert not clamped.any() and R == B
    live = c_ref > 0
    p = R * c_int[live].astype(np.float64) / float(S)
    assert abs(p.sum() - B) < 1e-9 * B
    var_term = float(np.sum(c_ref[live] ** 2 / p))
    optimum = float(np.sum(c_ref[live])) ** 2 / B
    # isqrt floors each score by < 1 unit: relative slack 2 / min score
    tol = 4.0 / float(c_int[live].min()) + 1e-12
    assert abs(var_term / optimum - 1.0) <= tol
    rng = np.random.default_rng(seed)
    for _ in range(20):
        q = p * np.exp(rng.normal(0, 0.3, size=p.shape))
        q *= B / q.sum()
        if q.max() > 1:
            continue
        assert float(np.sum(c_ref[live] ** 2 / q)) >= optimum * (1 - tol)


# ------------------------------------------------------------ planted mistakes
def _wrong_up_weight(weight_sq):
    def scores(su, sd, xs):
        up = [math.isqrt(weight_sq * int(a) * int(x) << 16) for a, x in zip(su, xs)]
        dn = [math.isqrt(int(a) * int(x) << 16) for a, x in zip(sd, xs)]
        return np.array(up + dn, dtype=np.int64)
    return scores


def _dropped_x(su, sd, xs):
    return O.leverage_scores(su, sd, np.ones_like(np.asarray(xs)))


def _swapped_halves(su, sd, xs):
    c = O.leverage_scores(su, sd, xs)
    n = len(su)
    return np.concatenate([c[n:], c[:n]])


def _dx_score(su, sd, xs):
    # the activation-gradient score ||grad_i|| alone (no X factor), weight kept
    return O.leverage_scores(su, sd, np.full(len(su), 1, dtype=np.int64))


MUTANTS = {
    "up weight 196": _wrong_up_weight(196 * 196),
    "up weight sqrt(14)": _wrong_up_weight(14),
    "up weight 1": _wrong_up_weight(1),
    "dropped x_sumsq": _dropped_x,
    "swapped halves": _swapped_halves,
    "activation score": _dx_score,
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_score_mistakes_fail_the_pin(name):
    """Each plausible slip in the score formula breaks proportionality on some case."""
    mutant = MUTANTS[name]
    worst = 0.0
    for (N, D, C, k, seed, kind) in CASES:
        G, f, bs = _case(N, D, C, k, seed, kind)
        su, sd = _sums(bs)
        c_ref = _reference_scores(G, f, bs)
        assert _proportionality_error(O.leverage_scores(su, sd, f.x_sumsq), c_ref) <= 1.0
        worst = max(worst, _proportionality_error(mutant(su, sd, f.x_sumsq), c_ref))
    assert worst > 1.0, f"planted mistake '{name}' passes the score pin"


def test_plan_uses_the_pinned_scores():
    """lss_plan's scores are leverage_scores' (so the pin above covers the sample)."""
    G, f, bs = _case(48, 64, 32, 3, 0)
    su, sd = _sums(bs)
    plan = O.lss_plan(su, sd, f.x_sumsq, 12, 0, 0)
    assert np.array_equal(plan.c, O.leverage_scores(su, sd, f.x_sumsq))
