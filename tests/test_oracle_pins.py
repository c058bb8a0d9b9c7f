"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a library
routine, a closed form, an invariant, brute force or an exhaustive
enumeration, chosen so that a plausible slip (a dropped term, a wrong sign or
index, a swapped nibble, a wrong scale) fails at least one of them.
"""
import math
import os
from fractions import Fraction
from itertools import product

import numpy as np
import pytest
import scipy.linalg

import oracle as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- Hadamard (Sec. 3.3)
@pytest.mark.parametrize("k", range(0, 8))
def test_fwht_matches_library_hadamard(k):
    """FWHT(x) == x @ H_u with H_u from scipy's Sylvester construction (exact on ints)."""
    b = 1 << k
    rng = np.random.default_rng(k)
    x = rng.integers(-1000, 1000, size=(5, 3 * b))
    H = scipy.linalg.hadamard(b).astype(np.int64)
    ref = (x.reshape(5, 3, b) @ H).reshape(5, 3 * b)
    assert np.array_equal(O.fwht_rows(x, k), ref)


@pytest.mark.parametrize("k", range(0, 8))
def test_hadamard_orthogonal_symmetric(k):
    """H_u H_u^T = 2^k I and H_u = H_u^T (Sec. 3.3: H_k orthogonal and symmetric)."""
    b = 1 << k
    Hf = O.fwht_rows(np.eye(b, dtype=np.int64), k)  # rows e_i^T H_u
    assert np.array_equal(Hf, O.hadamard_matrix_sylvester(k))
    assert np.array_equal(Hf, Hf.T)
    assert np.array_equal(Hf @ Hf.T, b * np.eye(b, dtype=np.int64))
    # involution up to scale: FWHT(FWHT(x)) = b x
    x = np.random.default_rng(1).integers(-50, 50, size=(4, 2 * b))
    assert np.array_equal(O.fwht_rows(O.fwht_rows(x, k), k), b * x)


def test_one_hot_row_becomes_flat():
    """e_i^T H_k = 2^{-k/2} 1 (Sec. 3.3): an outlier spreads to all +-1; quantised: all +-7."""
    k, b = 5, 32
    for i in range(b):
        x = np.zeros((1, b), dtype=np.float32)
        x[0, i] = 123.25
        v = O.fwht_rows(x, k)
        assert np.all(np.abs(v) == np.float32(123.25))
        q, s = O.quantize_int4(v, O.absmax(v))
        assert np.all(np.abs(q) == 7)


def test_fwht_float_is_float32_stage_order():
    """Float transform is the radix-2 butterfly in float32, strides ascending."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((3, 16)) * 1e3).astype(np.float32)
    y = x.copy()
    h = 1
    while h < 16:
        for j in range(16):
            if j & h == 0:
                a, c = y[:, j].copy(), y[:, j + h].copy()
                y[:, j], y[:, j + h] = a + c, a - c
        h *= 2
    assert np.array_equal(O.fwht_rows(x, 4), y)


# ---------------------------------------------------------------- quantiser (Sec. 3.1)
def test_k0_is_textbook_absmax_int4():
    """With H_0 = [1] (Sec. 3.3) the quantiser is plain per-tensor absmax INT4."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal((64, 96)).astype(np.float32)
    f = O.hq_forward(x, x[:8], 0, compute_output=False)
    s = np.max(np.abs(x.astype(np.float64))) / 7.0
    t = x.astype(np.float64) / s
    ref = np.clip(np.round(t), -7, 7)  # numpy round = half-to-even
    near_tie = np.abs(np.abs(t - np.floor(t)) - 0.5) < 1e-5
    assert not np.any((f.xq != ref) & ~near_tie)
    assert f.xq.min() >= -7 and f.xq.max() <= 7
    assert abs(float(f.s_x) - s) <= 1e-7 * s


def test_exact_reconstruction_tiny():
    """X = 2^m Q H_u / b with integer |Q| <= 7 (max 7) is quantised exactly to Q and
    Y == X W^T exactly: H_u H_u^T = b I makes every scale a power of two."""
    k, b = 3, 8
    rng = np.random.default_rng(7)
    N, C, D = 5, 6, 16
    Qx = rng.integers(-7, 8, size=(N, D)); Qx[0, 0] = 7
    Qw = rng.integers(-7, 8, size=(C, D)); Qw[1, 3] = -7
    H = scipy.linalg.hadamard(b).astype(np.float64)
    Hb = np.kron(np.eye(D // b), H)
    X = (2.0 ** 3 * Qx @ Hb / b).astype(np.float32)
    W = (2.0 ** -4 * Qw @ Hb / b).astype(np.float32)
    f = O.hq_forward(X, W, k)
    assert np.array_equal(f.xq, Qx) and np.array_equal(f.wq, Qw)
    assert f.s_x == np.float32(8.0) and f.s_w == np.float32(2.0 ** -4)
    exact = X.astype(np.float64) @ W.astype(np.float64).T
    assert np.array_equal(f.Y, exact)


def test_pack_nibble_order_and_roundtrip():
    """(data[1] << 4) | (data[0] & 15) (App. A.6): even column in the low nibble."""
    q = np.array([[1, -1, -7, 7, 0, -8 + 1]], dtype=np.int8)
    p = O.pack_int4(q)
    assert list(p[0]) == [0xF1, 0x79, 0x90]
    rng = np.random.default_rng(0)
    q = rng.integers(-7, 8, size=(9, 32)).astype(np.int8)
    assert np.array_equal(O.unpack_int4(O.pack_int4(q)), q)


def test_forward_error_vs_dequantised_operands():
    """Y equals the fp64 product of the dequantised operands s x^ H_u^T / b."""
    lin = synth.workload(0).linears[0]
    X, W, _ = synth.linear_inputs(lin, 0)
    f = O.hq_forward(X, W, lin.log2_block)
    b = 1 << lin.log2_block
    H = scipy.linalg.hadamard(b).astype(np.float64)
    Hb = np.kron(np.eye(lin.D // b), H)
    Xd = float(f.s_x) * f.xq.astype(np.float64) @ Hb.T / b
    Wd = float(f.s_w) * f.wq.astype(np.float64) @ Hb.T / b
    ref = Xd @ Wd.T
    assert np.linalg.norm(f.Y - ref) <= 1e-12 * np.linalg.norm(ref)
    # and the HQ error against the unquantised product is the expected INT4 level
    exact = X.astype(np.float64) @ W.astype(np.float64).T
    rel = np.linalg.norm(f.Y - exact) / np.linalg.norm(exact)
    assert 0.05 < rel < 0.5


# ---------------------------------------------------------------- Philox (counter-based RNG)
def test_philox_known_answers():
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as fh:
        rows = [ln.split() for ln in fh if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 3
    for r in rows:
        v = [int(x, 16) for x in r]
        out = O.philox4x32_10(v[0], v[1], v[2], v[3], v[4], v[5])
        assert [int(o) for o in out] == v[6:10]


def test_uniforms16_layout():
    """element i uses half (i & 1) of word ((i >> 1) & 3) of block offset + (i >> 3)."""
    seed, off = (5 << 32) | 17, 123
    u = O.uniforms16(seed, off, 1, 40)
    for i in [0, 1, 2, 7, 8, 13, 39]:
        blk = off + (i >> 3)
        w = O.philox4x32_10(blk & 0xFFFFFFFF, blk >> 32, 1, 0, 17, 5)
        word = int(w[(i >> 1) & 3])
        assert int(u[i]) == (word >> (16 * (i & 1))) & 0xFFFF


def test_uniforms16_chi2():
    u = O.uniforms16(1, 0, 0, 1 << 16)
    h = np.bincount(u >> 12, minlength=16)
    chi2 = float(((h - 4096.0) ** 2 / 4096.0).sum())
    assert chi2 < 45.0  # 15 dof, p ~ 1e-4


# ---------------------------------------------------------------- bit splitting (Sec. 4.2)
def test_bitsplit_error_bound():
    """|g - s_up q_up - s_dn q_dn| < s_dn: the residual quantiser keeps one lower step."""
    lin = synth.workload(0).linears[0]
    _, _, G = synth.linear_inputs(lin, 0)
    bs = O.bit_split(G, 0, 0)
    assert bs.q_up.min() >= -7 and bs.q_up.max() <= 7
    assert bs.q_dn.min() >= -7 and bs.q_dn.max() <= 7
    rec = float(bs.s_up) * bs.q_up + bs.s_dn * bs.q_dn
    err = np.abs(G.astype(np.float64) - rec)
    assert err.max() < bs.s_dn * (1 + 1e-5)


def test_bitsplit_exact_on_grid():
    """dY = s_up U on the upper grid: the lower half is identically 0, reconstruction exact."""
    rng = np.random.default_rng(2)
    U = rng.integers(-7, 8, size=(16, 32)); U[0, 0] = 7
    G = (2.0 ** -5 * U).astype(np.float32)
    bs = O.bit_split(G, 9, 0)
    assert np.array_equal(bs.q_up, U) and not bs.q_dn.any()
    assert bs.s_up == np.float32(2.0 ** -5)


def test_stochastic_round_exhaustive_expectation():
    """Over all 2^16 uniforms, E[SR(w)] = floor(w) + ceil(frac*2^16)/2^16: bias in [0, 2^-16)."""
    u = np.arange(65536, dtype=np.uint16)
    for w in [-6.9, -3.25, -0.001, 0.0, 0.3, 2.5, 6.99999, 7.0, -7.0]:
        wf = np.float32(w)
        q = O.stochastic_round(np.full(65536, wf, dtype=np.float32), u).astype(np.float64)
        mean = q.mean()
        assert wf - 1e-12 <= mean < wf + 2.0 ** -16 + 1e-12
        assert set(np.unique(q)) <= {math.floor(wf), math.floor(wf) + 1}


def test_bitsplit_unbiased_monte_carlo():
    """E[s_up q_up + s_dn q_dn] = dY: the exact expectation of the implemented rounding
    (floor + ceil(frac 2^16)/2^16) reconstructs dY within 2^-16 s_dn plus float32 scale
    rounding, and Philox draws over offsets match that Bernoulli law (z-test with the
    exact variance p(1-p))."""
    rng = np.random.default_rng(4)
    G = (rng.standard_normal((8, 64)) * 0.3).astype(np.float32)
    bs0 = O.bit_split(G, 11, 0)
    inv = np.float32(7) / bs0.amax
    v = G * inv
    w = np.float32(14) * (v - np.rint(v))
    fl = np.floor(w)
    p = np.ceil((w - fl) * np.float32(65536.0)).astype(np.float64) / 65536.0
    expect = 14.0 * np.rint(v) + fl + p  # E[14 q_up + q_dn]
    err = np.abs(bs0.s_dn * expect - G.astype(np.float64))
    assert np.all(err <= bs0.s_dn * 2.0 ** -16 + np.abs(G) * 2.0 ** -21)
    T = 600
    acc = np.zeros(G.shape)
    for off in range(T):
        acc += O.bit_split(G, 11, off * 64).combined()
    mean = acc / T
    sd = np.sqrt(np.maximum(p * (1 - p), 1e-12) / T)
    z = (mean - expect) / sd
    assert np.all(np.abs(z) < 6.0)
    assert abs(float(np.mean(z))) < 6.0 / np.sqrt(z.size) * 2


# ---------------------------------------------------------------- clamp-rescale (App. A.2)
def _waterfill_sorted(c, B):
    """Closed form: sort c descending, k* = min{k : (B-k) c_(k+1) < sum_{i>k} c_(i)}."""
    cs = sorted((int(v) for v in c if v > 0), reverse=True)
    if len(cs) <= B:
        return len(cs), None
    tail = sum(cs)
    k = 0
    while k < len(cs) and (B - k) * cs[k] >= tail:
        tail -= cs[k]
        k += 1
    return k, tail


def _paper_loop_float(c, B):
    """App. A.2 exactly as worded, in float64: clamp to 1, rescale the rest to sum B."""
    c = np.asarray(c, dtype=np.float64)
    p = B * c / c.sum()
    for _ in range(len(c) + 1):
        big = p >= 1.0
        p = np.where(big, 1.0, p)
        rest = B - big.sum()
        small = ~big
        p[small] = rest * c[small] / c[small].sum()
        if not np.any(p[small] > 1.0):
            break
    return p


@pytest.mark.parametrize("seed", range(6))
def test_clamp_rescale_matches_closed_form_and_paper_loop(seed):
    rng = np.random.default_rng(seed)
    n = 200
    c = np.floor(rng.pareto(1.2, size=n) * 1000).astype(np.int64)
    c[rng.choice(n, 20, replace=False)] = 0
    B = int(rng.integers(10, 120))
    clamped, R, S = O.clamp_rescale(c, B)
    k_ref, tail = _waterfill_sorted(c, B)
    assert clamped.sum() == k_ref
    if tail is not None:
        assert R == B - k_ref and S == tail
        p = np.where(clamped, 1.0, R * c / S)
        assert abs(p.sum() - B) < 1e-9 and p.max() <= 1.0 + 1e-12
        assert np.allclose(p, _paper_loop_float(c, B), atol=1e-9)
        # clamped rows dominate every unclamped one
        if clamped.any() and (~clamped & (c > 0)).any():
            assert c[clamped].min() >= c[~clamped].max()


def test_clamp_rescale_brute_force_tiny():
    """Exhaustive: the loop of App. A.2 (clamp when p >= 1, rescale the rest) stops at
    the smallest clamped upper set K (top scores) leaving every other p < 1."""
    rng = np.random.default_rng(8)
    checked = 0
    for _ in range(300):
        n = int(rng.integers(3, 9))
        c = rng.integers(0, 50, size=n)
        B = int(rng.integers(1, n))
        if (c > 0).sum() <= B:
            continue
        clamped, R, S = O.clamp_rescale(c, B)
        fixpoints = []
        for mask in product([0, 1], repeat=n):
            m = np.array(mask, dtype=bool)
            if np.any(m & (c == 0)):
                continue
            if m.any() and (~m).any() and c[m].min() < c[~m].max():
                continue  # only upper sets: a clamped row never has a smaller score
            k = int(m.sum())
            rest = int(c[~m].sum())
            if k > B or rest == 0:
                continue
            if all(Fraction((B - k) * int(c[j]), rest) < 1 for j in range(n) if not m[j]):
                fixpoints.append(m)
        kmin = min(int(m.sum()) for m in fixpoints)
        least = [m for m in fixpoints if int(m.sum()) == kmin]
        assert len(least) == 1 and np.array_equal(least[0], clamped)
        checked += 1
    assert checked > 100


def test_keep_nonzero_special_case():
    """#nonzero rows <= B: every nonzero row kept with weight 1 (App. A.6, keep norm > 0);
    the estimate equals the bit-split product exactly, for every seed."""
    lin = synth.small_linear(24, 32, 16, 3, grad_kind="lognormal")
    X, W, G = synth.linear_inputs(lin, 3)
    f = O.hq_forward(X, W, 3, compute_output=False)
    assert O.resolve_budget(O.KEEP_NONZERO, 24) == 48 and O.resolve_budget(0, 24) == 24
    for seed in range(3):
        bw = O.lss_backward(G, f, budget=O.KEEP_NONZERO, seed=seed, offset=0)
        assert bw.plan.budget == 48
        assert (bw.plan.e_dn == 0).all()
        assert (f.x_sumsq > 0).all()
        nzdn = np.abs(bw.bs.q_dn).sum(1) > 0
        assert np.array_equal(bw.plan.w_dn, nzdn.astype(int))
        assert np.array_equal(bw.A, bw.bs.combined())  # exactly the bit-split product
        # a deterministic rule: for fixed codes the masks' uniforms play no part
        su = (bw.bs.q_up.astype(np.int64) ** 2).sum(1)
        sd = (bw.bs.q_dn.astype(np.int64) ** 2).sum(1)
        for mseed in range(1, 4):
            p2 = O.lss_plan(su, sd, f.x_sumsq, O.KEEP_NONZERO, mseed, 7)
            assert np.array_equal(p2.kept, bw.plan.kept) and np.array_equal(p2.w_dn, bw.plan.w_dn)


# ---------------------------------------------------------------- LSS estimator (Sec. 4.2)
def _small_case(budget_div=4, seed=0, N=24, D=32, C=16):
    lin = synth.small_linear(N, D, C, 3, grad_kind="pareto")
    X, W, G = synth.linear_inputs(lin, seed)
    f = O.hq_forward(X, W, 3, compute_output=False)
    bs = O.bit_split(G, 1, 0)
    su = (bs.q_up.astype(np.int64) ** 2).sum(1)
    sd = (bs.q_dn.astype(np.int64) ** 2).sum(1)
    return f, bs, su, sd, max(1, N // budget_div)


def test_lss_mask_rule_exhaustive_unbiased():
    """Over all 2^16 stream-1 uniforms, each down row is kept with probability exactly
    p~ = 2^-e and weighted 2^e: E[w_dn] = 1 for every row with c > 0 (unbiased)."""
    f, bs, su, sd, B = _small_case()
    N = len(su)
    tot = np.zeros(N)
    kept_cnt = np.zeros(N)
    for u in range(0, 65536, 1):
        plan = O.lss_plan(su, sd, f.x_sumsq, B, 0, 0, u16_masks=np.full(N, u, dtype=np.uint16))
        tot += plan.w_dn
        kept_cnt += plan.w_dn > 0
    plan = O.lss_plan(su, sd, f.x_sumsq, B, 0, 0)
    live = plan.c[N:] > 0
    assert np.array_equal(tot[live] / 65536.0, np.ones(live.sum()))
    assert np.array_equal(kept_cnt[live] / 65536.0, 2.0 ** -plan.e_dn[live])
    assert (plan.e_dn > 0).any(), "test must exercise sampling"
    # p~ rounds p* up to a power of two: p* <= p~ < 2 p* (below the cap)
    R, S = plan.R, plan.S
    for t in np.nonzero(live & ~plan.clamped[N:])[0]:
        p_star = Fraction(R * int(plan.c[N + t]), S)
        p_t = Fraction(1, 1 << int(plan.e_dn[t]))
        cap = 2 if su[t] > 0 else 4
        assert p_star <= p_t and (p_t < 2 * p_star or plan.e_dn[t] == cap)


def test_lss_expectation_by_enumeration_equals_bitsplit_product():
    """Enumerating every mask pattern of the sampled rows (with their probabilities)
    gives E[A^T X^] == (14 q_up + q_dn)^T X^ exactly (the estimator of Sec. 4.2)."""
    f, bs, su, sd, B = _small_case(N=10, D=16, C=8)
    plan = O.lss_plan(su, sd, f.x_sumsq, B, 0, 0)
    N = len(su)
    sampled = [t for t in range(N) if plan.c[N + t] > 0 and plan.e_dn[t] > 0]
    assert 0 < len(sampled) <= 10
    xq = f.xq.astype(np.int64)
    qd = bs.q_dn.astype(np.int64)
    exp = np.zeros((bs.q_up.shape[1], xq.shape[1]), dtype=object)
    base_w = np.where(plan.c[N:] > 0, 1, 0)
    for bits in product([0, 1], repeat=len(sampled)):
        prob = Fraction(1)
        w_dn = base_w.astype(object).copy()
        for t, bit in zip(sampled, bits):
            p = Fraction(1, 1 << int(plan.e_dn[t]))
            prob *= p if bit else (1 - p)
            w_dn[t] = (1 << int(plan.e_dn[t])) if bit else 0
        A = 14 * plan.w_up[:, None] * bs.q_up.astype(np.int64) + np.array(w_dn, dtype=np.int64)[:, None] * qd
        exp = exp + (A.T @ xq).astype(object) * prob
    live = (plan.c[N:] > 0)
    ref = (14 * bs.q_up.astype(np.int64) + live[:, None] * qd).T @ xq
    assert np.array_equal(np.array(exp, dtype=object), ref.astype(object))


def test_lss_variance_matches_proposition_4_1():
    """Monte-Carlo variance of the sampled weight gradient equals
    sum_i (1 - p_i)/p_i ||grad_i||^2 ||X_i||^2 (Prop. 4.1) with the plan's p~."""
    f, bs, su, sd, B = _small_case(budget_div=4, N=48, D=32, C=16)
    N = len(su)
    plan0 = O.lss_plan(su, sd, f.x_sumsq, B, 0, 0)
    xq = f.xq.astype(np.int64)
    p = plan0.p_dn()
    live = p > 0
    theory = float(np.sum(((1 - p[live]) / p[live]) * sd[live] * f.x_sumsq[live]))
    assert theory > 0
    T = 3000
    s1 = None; s2 = 0.0
    ests = []
    for off in range(T):
        plan = O.lss_plan(su, sd, f.x_sumsq, B, 0, off)
        A = O.weighted_rows(bs, plan)
        ests.append((A.T @ xq).astype(np.float64))
    E = np.stack(ests)
    var = float(((E - E.mean(0)) ** 2).sum(axis=(1, 2)).mean())
    assert abs(var / theory - 1) < 0.1


def test_lss_backward_unbiased_vs_exact_gradients():
    """Over offsets (both streams), mean dW and dX approach the fp64 gradients of the
    quantised forward: G^T X^ H_u s_x / b and G W^ H_u s_w / b (Sec. 4, STE)."""
    lin = synth.small_linear(32, 32, 16, 3, grad_kind="pareto")
    X, W, G = synth.linear_inputs(lin, 5)
    f = O.hq_forward(X, W, 3, compute_output=False)
    b = 8
    Hb = np.kron(np.eye(lin.D // b), scipy.linalg.hadamard(b))
    dW_ref = G.astype(np.float64).T @ (float(f.s_x) * f.xq @ Hb / b)
    dX_ref = G.astype(np.float64) @ (float(f.s_w) * f.wq @ Hb / b)
    T = 400
    mW = np.zeros_like(dW_ref); mX = np.zeros_like(dX_ref)
    for off in range(T):
        bw = O.lss_backward(G, f, budget=8, seed=2, offset=off * 4096)
        mW += bw.dW; mX += bw.dX
    mW /= T; mX /= T
    assert np.linalg.norm(mW - dW_ref) / np.linalg.norm(dW_ref) < 0.03
    assert np.linalg.norm(mX - dX_ref) / np.linalg.norm(dX_ref) < 0.03
    # a single draw is a useful estimate too (BS + LSS error), not a bit-identical one
    one = O.lss_backward(G, f, budget=8, seed=2, offset=0)
    assert np.linalg.norm(one.dW - dW_ref) / np.linalg.norm(dW_ref) < 1.0


def test_lss_deterministic_and_offset_sensitive():
    f, bs, su, sd, B = _small_case()
    a = O.lss_plan(su, sd, f.x_sumsq, B, 3, 100)
    b = O.lss_plan(su, sd, f.x_sumsq, B, 3, 100)
    c = O.lss_plan(su, sd, f.x_sumsq, B, 3, 101)
    assert np.array_equal(a.w_dn, b.w_dn) and np.array_equal(a.kept, b.kept)
    assert not np.array_equal(a.w_dn, c.w_dn)


def test_weighted_rows_fit_int8():
    """|14 q_up + 2^e q_dn| <= 126 under the exponent caps (one int8 GEMM operand)."""
    f, bs, su, sd, B = _small_case(budget_div=8, N=64)
    for off in range(20):
        plan = O.lss_plan(su, sd, f.x_sumsq, B, 0, off)
        A = O.weighted_rows(bs, plan)
        assert np.abs(A).max() <= 126


# ---------------------------------------------------------------- Hadamard size (App. A.5)
def test_hadamard_mse_closed_form():
    """x = [1, 1/2, 0, ..., 0] (D = 8), worked by hand.  k = 0: a = 1, codes (7, 4) (rint
    of 3.5 is 4), error 4/7 - 1/2 = 1/14 on one entry: MSE = 1/14^2/8 = 1/1568.  k >= 1:
    the first block of x H_u is (3/2, 1/2) repeated, a = 3/2, codes (7, 2), error
    3/7 - 1/2 = -1/14 on half of the block's entries; back in the x domain the squared
    error is divided by 2^k (H_u H_u^T = 2^k I): MSE = 1/3136 for k = 1, 2, 3."""
    x = np.zeros((1, 8), dtype=np.float32)
    x[0, :2] = (1.0, 0.5)
    want = [1 / 1568, 1 / 3136, 1 / 3136, 1 / 3136]
    for k, m in enumerate(want):
        assert O.hadamard_mse(x, k) == pytest.approx(m, rel=1e-6)  # s = fl(a/7): ~1e-7
    # X = W = x: objectives 1/1568^2 > 1/3136^2 (k = 1, 2, 3 tie): the smallest tied k wins
    c = O.choose_hadamard_size(x, x, 3)
    assert c.log2_block == 1
    assert np.all(np.isnan(c.mse_x[4:]))


@pytest.mark.parametrize("k", range(0, 8))
def test_hadamard_reconstruction_matches_dense_matrices(k):
    """V_bar = s q H^T with H the orthonormal block-diagonal matrix built from scipy's
    Hadamard matrix (normalised, explicit dense product, codes from V H)."""
    b, D = 1 << k, 256
    rng = np.random.default_rng(40 + k)
    V = rng.standard_normal((6, D)).astype(np.float32)
    V[:, 7] *= 30
    Hn = np.kron(np.eye(D // b), scipy.linalg.hadamard(b) / math.sqrt(b))
    VH = V.astype(np.float64) @ Hn
    a = np.abs(VH).max()
    q = np.clip(np.round(VH / (a / 7)), -7, 7)
    ref = (a / 7) * q @ Hn.T
    got = O.hadamard_reconstruction(V, k)
    # codes agree (no value of VH sits within rounding of a half-integer step here)
    assert np.abs(got - ref).max() <= 1e-5 * np.abs(ref).max()
    assert O.hadamard_mse(V, k) == pytest.approx(np.mean((ref - V) ** 2), rel=1e-5)


@pytest.mark.parametrize("k", [0, 3, 5, 7])
def test_hadamard_mse_parseval(k):
    """Parseval: ||V_bar - V||^2 = ||s q - V H_u||^2 / 2^k (H_u / 2^{k/2} orthogonal), the
    transform-domain form of the error."""
    rng = np.random.default_rng(k)
    V = (rng.standard_normal((16, 384)) * rng.lognormal(0, 1, size=384)).astype(np.float32)
    v = O.fwht_rows(V, k).astype(np.float64)
    a = np.abs(v).max()
    q = np.rint(v * np.float32(7.0) / np.float32(a))  # only the codes matter; ties absent
    e = (a / 7) * q - v
    assert O.hadamard_mse(V, k) == pytest.approx(np.sum(e * e) / (1 << k) / V.size, rel=1e-5)


def test_hadamard_mse_k0_textbook():
    """k = 0 is plain per-tensor absmax RTN to [-7, 7]: mean((s round(x/s) - x)^2)."""
    rng = np.random.default_rng(5)
    V = rng.standard_normal((32, 64)).astype(np.float32)
    s = float(np.abs(V).max()) / 7
    ref = np.mean((s * np.round(V / s) - V) ** 2)
    assert O.hadamard_mse(V, 0) == pytest.approx(ref, rel=1e-6)


def test_choose_hadamard_size_exact_grid_picks_zero():
    """X on the INT4 grid of its own absmax is exact at k = 0 (MSE 0, objective 0), and a
    transform can only keep or lose that: k = 0 wins, ties included."""
    rng = np.random.default_rng(6)
    X = (rng.integers(-7, 8, size=(16, 128)) * 0.375).astype(np.float32)
    X[0, 0] = 7 * 0.375
    W = rng.standard_normal((32, 128)).astype(np.float32)
    c = O.choose_hadamard_size(X, W)
    assert c.mse_x[0] == 0.0 and c.log2_block == 0


def test_choose_hadamard_size_outlier_channel_prefers_large_blocks():
    """One input channel 100x the rest (the outlier structure of Sec. 3.2): a larger block
    spreads it over more entries (Sec. 3.3), MSE_X falls with every k, and k = 7 wins."""
    rng = np.random.default_rng(0)
    X = rng.standard_normal((64, 128), dtype=np.float32)
    X[:, 5] *= 100
    W = rng.standard_normal((96, 128), dtype=np.float32) * np.float32(0.02)
    c = O.choose_hadamard_size(X, W)
    assert np.all(np.diff(c.mse_x) < 0)
    assert c.log2_block == 7


def test_choose_hadamard_size_candidates_and_scale_invariance():
    """Only 2^k dividing D are candidates (D = 96: k <= 5), max_log2_block caps the search,
    and scaling X by 2^j (exact) scales MSE_X by 4^j without moving the choice."""
    rng = np.random.default_rng(8)
    X = rng.standard_normal((8, 96), dtype=np.float32)
    X[:, 3] *= 40
    W = rng.standard_normal((16, 96), dtype=np.float32)
    c = O.choose_hadamard_size(X, W)
    assert c.log2_block <= 5 and np.all(np.isnan(c.mse_x[6:])) and not np.isnan(c.mse_x[5])
    c2 = O.choose_hadamard_size(X, W, 2)
    assert c2.log2_block <= 2 and np.all(np.isnan(c2.mse_x[3:]))
    c4 = O.choose_hadamard_size(X * np.float32(8), W)
    assert np.allclose(c4.mse_x[:6], 64 * c.mse_x[:6], rtol=1e-12)
    assert c4.log2_block == c.log2_block
