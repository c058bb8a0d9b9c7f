"""Plain CPU oracle of HQ-MM (forward) and LSS-MM (backward) of one linear layer.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may use this module.  It shares no code with the GPU library
and imports nothing from it.

Notation follows the paper ("Training Transformers with 4-bit Integers",
arXiv 2306.11987): Y = X W^T with X: N x D, W: C x D (Sec. 3, Eq. 1); H_k the
2^k x 2^k Hadamard matrix, H = BlockDiag(H_k, ..., H_k) (Sec. 3.3); INT4 codes
in [-7, 7] (Sec. 3.1, Eq. 2, Q_N = Q_P = 7).

Readings of the paper taken here (each is listed with its reason in the design
notes of the repository):

* H_u = 2^{k/2} H_k, the unnormalised +-1 Sylvester matrix, is applied by the
  radix-2 fast transform, strides ascending, in float32 (the paper computes XH
  in FP16 on its GPU).  The factor 2^{-k} is folded into the dequantisation
  scale (H_u H_u^T = 2^k I).
* Step sizes are dynamic per-tensor absmax scales s = max|v| / 7 (gradients are
  quantised dynamically in Sec. 4; the learned static step size of Sec. 3.1 is
  a separate mode).  Codes are round-half-even(v * fl(7/a)), clamped to +-7.
* Bit splitting (Sec. 4.2, Eq. 4): upper codes round to nearest with
  s_up = a/7; the residual is scaled by 14 and rounded stochastically, so that
  s_dn = s_up / 14 and the pair is the integer 14*q_up + q_dn (the paper's
  "INT8 representation").
* Leverage scores (Sec. 4.2) are taken on the codes; one shared sample serves
  both gradients (App. A.6: the activation gradient reuses the weight
  gradient's quantisation and scores).  Inclusion probabilities follow the
  clamp-and-rescale loop of App. A.2 in exact integers, then are rounded up to
  powers of two (p~ = 2^-e >= p*), which keeps the estimator unbiased and lets
  the weights 2^e enter one exact integer GEMM operand.
* The gradients carry H^T along D (Sec. 4, the STE gradients): it is applied to
  the integer GEMM results, before dequantisation.

Everything that decides an integer (codes, stochastic rounding, samples) runs in
float32 or exact integers exactly as the GPU must; the float outputs are
formed in float64.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from .philox_ref import philox_blocks, uniforms16

QMAX = 7  # Q_N = Q_P = 7 (Sec. 3.1)
BS_RATIO = 14  # s_up / s_dn (bit-split reading)
STREAM_SR = 0  # Philox stream of the lower-half stochastic rounding
STREAM_MASK = 1  # Philox stream of the LSS Bernoulli masks
MAX_LOG2_BLOCK = 7  # largest Hadamard block 2^k searched (App. A.5)
KEEP_NONZERO = -1  # budget value selecting the keep-every-non-zero-row rule (App. A.6)

__all__ = [
    "QMAX", "BS_RATIO", "fwht_rows", "hadamard_matrix_sylvester", "absmax", "quantize_int4",
    "pack_int4", "unpack_int4", "HQForward", "hq_forward", "BitSplit", "bit_split",
    "leverage_scores", "clamp_rescale", "LSSPlan", "lss_plan", "LSSBackward",
    "lss_backward", "weighted_rows", "stochastic_round", "MAX_LOG2_BLOCK", "KEEP_NONZERO",
    "resolve_budget", "hadamard_reconstruction", "hadamard_mse", "HadamardChoice",
    "choose_hadamard_size", "quantize_lsq", "LSQForward", "lsq_forward", "LSQBackward",
    "lsq_backward", "lsq_grad_scale", "bmm_counter_stride", "bmm_lsq_forward",
    "bmm_lsq_backward", "STREAM_SR", "STREAM_MASK",
]


# --------------------------------------------------------------------------
# Hadamard transform (Sec. 3.3)
# --------------------------------------------------------------------------
def fwht_rows(v: np.ndarray, log2_block: int) -> np.ndarray:
    """Block-diagonal unnormalised Hadamard transform of every row: v @ BlockDiag(H_u).

    H_k is defined by the Sylvester recursion H_k = [[H, H], [H, -H]] (Sec. 3.3,
    here without the 1/sqrt(2) per level).  Applying the recursion level by
    level gives the radix-2 butterfly (x[j], x[j+h]) <- (x[j]+x[j+h], x[j]-x[j+h])
    for h = 1, 2, ..., b/2.  Float inputs are transformed in float32, integer
    inputs in exact int64.
    """
    b = 1 << int(log2_block)
    v = np.asarray(v)
    R, D = v.shape
    assert D % b == 0, "D must be a multiple of the block size (Sec. 3.3)"
    x = v.astype(np.int64 if np.issubdtype(v.dtype, np.integer) else np.float32, copy=True)
    h = 1
    while h < b:
        y = x.reshape(R, D // (2 * h), 2, h)
        lo = y[:, :, 0, :].copy()
        hi = y[:, :, 1, :].copy()
        y[:, :, 0, :] = lo + hi
        y[:, :, 1, :] = lo - hi
        h *= 2
    return x


def hadamard_matrix_sylvester(log2_block: int) -> np.ndarray:
    """H_u by the Sylvester recursion itself (used to check the fast transform)."""
    H = np.ones((1, 1), dtype=np.int64)
    for _ in range(int(log2_block)):
        H = np.block([[H, H], [H, -H]])
    return H


# --------------------------------------------------------------------------
# Quantiser (Sec. 3.1, Eq. 2)
# --------------------------------------------------------------------------
def absmax(v: np.ndarray) -> np.float32:
    v = np.asarray(v, dtype=np.float32)
    return np.float32(np.max(np.abs(v))) if v.size else np.float32(0.0)


def quantize_int4(v: np.ndarray, a: np.float32):
    """int_s(v) = round(clamp(v / s, -7, 7)) with s = a / 7 (Eq. 2).

    The division by s is taken as a multiplication by inv = fl(7 / a), computed
    once; rounding is half-to-even.  Returns (codes int8, s float32)."""
    v = np.asarray(v, dtype=np.float32)
    a = np.float32(a)
    if a == 0:
        return np.zeros(v.shape, dtype=np.int8), np.float32(0.0)
    inv = np.float32(QMAX) / a
    q = np.clip(np.rint(v * inv), -QMAX, QMAX).astype(np.int8)
    s = a / np.float32(QMAX)
    return q, s


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Two codes per byte: (q[2i+1] << 4) | (q[2i] & 15) (App. A.6, data pack)."""
    q = np.asarray(q).astype(np.int16)
    assert q.shape[-1] % 2 == 0
    lo = q[..., 0::2] & 15
    hi = q[..., 1::2] & 15
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(p: np.ndarray) -> np.ndarray:
    p = np.asarray(p, dtype=np.uint8).astype(np.int16)
    lo = p & 15
    hi = (p >> 4) & 15
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


def _int_matmul(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Exact integer product a @ b.  float64 BLAS is exact here because every
    partial sum stays far below 2^53 (|a|,|b| <= 126, K <= 2^20)."""
    assert a.shape[1] < (1 << 20)
    r = a.astype(np.float64) @ b.astype(np.float64)
    return r.astype(np.int64)


# --------------------------------------------------------------------------
# HQ-MM forward (Sec. 3.3, Procedure HQ-MM)
# --------------------------------------------------------------------------
@dataclass
class HQForward:
    log2_block: int
    amax_x: np.float32
    amax_w: np.float32
    s_x: np.float32
    s_w: np.float32
    xq: np.ndarray  # int8 [N][D] codes of X H_u
    wq: np.ndarray  # int8 [C][D] codes of W H_u
    x_sumsq: np.ndarray  # int64 [N]  sum_d xq^2
    acc: np.ndarray = field(default=None)  # int64 [N][C]
    Y: np.ndarray = field(default=None)  # float64 [N][C]


def hq_forward(X: np.ndarray, W: np.ndarray, log2_block: int, compute_output: bool = True) -> HQForward:
    """Steps of HQ-MM: (1) X H and H^T W^T; (2) quantise both to INT4;
    (3) integer product; (4) dequantise by s_X s_W (and 2^-k, see module notes)."""
    vx = fwht_rows(np.asarray(X, dtype=np.float32), log2_block)
    vw = fwht_rows(np.asarray(W, dtype=np.float32), log2_block)
    ax, aw = absmax(vx), absmax(vw)
    xq, sx = quantize_int4(vx, ax)
    wq, sw = quantize_int4(vw, aw)
    x_sumsq = np.sum(xq.astype(np.int64) ** 2, axis=1)
    out = HQForward(int(log2_block), ax, aw, sx, sw, xq, wq, x_sumsq)
    if compute_output:
        out.acc = _int_matmul(xq, wq.T)
        out.Y = float(sx) * float(sw) * 2.0 ** (-int(log2_block)) * out.acc.astype(np.float64)
    return out


# --------------------------------------------------------------------------
# Choice of the Hadamard block size (App. A.5)
# --------------------------------------------------------------------------
def hadamard_reconstruction(V: np.ndarray, log2_block: int) -> np.ndarray:
    """V_bar = s int_s(V H) H^T (App. A.5) in float64.

    The codes and the step are those of the forward quantiser (module notes: V H_u in
    float32, s = a/7, codes rint(v * fl(7/a))).  With H_u = 2^{k/2} H the normalised
    form gives the same codes, and V_bar = s q H_u^T / 2^k; H_u is symmetric, so the
    product with H_u^T is the transform of the code rows, taken exactly in int64."""
    k = int(log2_block)
    v = fwht_rows(np.asarray(V, dtype=np.float32), k)
    q, s = quantize_int4(v, absmax(v))
    back = fwht_rows(q.astype(np.int64), k).astype(np.float64)
    return float(s) * back / float(1 << k)


def hadamard_mse(V: np.ndarray, log2_block: int) -> float:
    """MSE(V_bar, V): mean of the squared entries of V_bar - V (0 for an empty tensor)."""
    V = np.asarray(V, dtype=np.float32)
    if V.size == 0:
        return 0.0
    d = hadamard_reconstruction(V, log2_block) - V.astype(np.float64)
    return float(np.mean(d * d))


@dataclass
class HadamardChoice:
    log2_block: int
    mse_x: np.ndarray  # float64 [MAX_LOG2_BLOCK + 1]; nan where 2^k is not a candidate
    mse_w: np.ndarray

    @property
    def objective(self) -> np.ndarray:
        return self.mse_x * self.mse_w


def choose_hadamard_size(X: np.ndarray, W: np.ndarray,
                         max_log2_block: int = MAX_LOG2_BLOCK) -> HadamardChoice:
    """The k minimising MSE(X_bar, X) x MSE(W_bar, W) (App. A.5).

    Candidates are 0 <= k <= min(max_log2_block, 7) with D a multiple of 2^k (Sec. 3.3:
    H is block-diagonal in 2^k blocks).  Equal objectives go to the smaller k, the
    cheaper transform (Sec. 3.3 trade-off)."""
    X = np.asarray(X, dtype=np.float32)
    W = np.asarray(W, dtype=np.float32)
    D = X.shape[1]
    assert W.shape[1] == D
    n = MAX_LOG2_BLOCK + 1
    mse_x = np.full(n, np.nan)
    mse_w = np.full(n, np.nan)
    best, best_obj = None, None
    for k in range(0, min(int(max_log2_block), MAX_LOG2_BLOCK) + 1):
        if D % (1 << k):
            continue
        mse_x[k] = hadamard_mse(X, k)
        mse_w[k] = hadamard_mse(W, k)
        obj = mse_x[k] * mse_w[k]
        if best is None or obj < best_obj:
            best, best_obj = k, obj
    assert best is not None
    return HadamardChoice(best, mse_x, mse_w)


# --------------------------------------------------------------------------
# Bit splitting (Sec. 4.2, Eq. 4)
# --------------------------------------------------------------------------
@dataclass
class BitSplit:
    amax: np.float32
    s_up: np.float32
    q_up: np.ndarray  # int8 [N][C]
    q_dn: np.ndarray  # int8 [N][C]

    @property
    def s_dn(self) -> float:
        return float(self.s_up) / BS_RATIO

    def combined(self) -> np.ndarray:
        """The integer 14 q_up + q_dn, i.e. dY / s_dn (the INT8 view)."""
        return BS_RATIO * self.q_up.astype(np.int32) + self.q_dn.astype(np.int32)


def stochastic_round(w: np.ndarray, u16: np.ndarray) -> np.ndarray:
    """floor(w) + [u < frac(w) * 2^16] in float32, u uniform on 0..65535."""
    w = np.asarray(w, dtype=np.float32)
    fl = np.floor(w)
    thr = (w - fl) * np.float32(65536.0)
    return (fl + (u16.astype(np.float32) < thr)).astype(np.int8)


def bit_split(G: np.ndarray, seed: int, offset: int) -> BitSplit:
    """dY ~ s_up q_up + s_dn q_dn: quantise dY to INT4, then the residual (Sec. 4.2)."""
    G = np.asarray(G, dtype=np.float32)
    N, C = G.shape
    a = absmax(G)
    if a == 0:
        z = np.zeros((N, C), dtype=np.int8)
        return BitSplit(a, np.float32(0.0), z, z.copy())
    inv = np.float32(QMAX) / a
    v = G * inv
    q_up = np.rint(v)  # |v| <= 7(1+2^-23): no clamp needed
    r = v - q_up  # exact: |r| <= 1/2
    w = np.float32(BS_RATIO) * r  # |w| <= 7
    u = uniforms16(seed, offset, STREAM_SR, N * C).reshape(N, C)
    q_dn = stochastic_round(w, u)
    return BitSplit(a, a / np.float32(QMAX), q_up.astype(np.int8), q_dn)


# --------------------------------------------------------------------------
# Leverage score sampling (Sec. 4.2, App. A.2)
# --------------------------------------------------------------------------
def leverage_scores(sumsq_up: np.ndarray, sumsq_dn: np.ndarray, x_sumsq: np.ndarray) -> np.ndarray:
    """Integer leverage scores of the 2N stacked rows [up rows; down rows].

    c_i = ||grad_i|| ||X_i|| (Sec. 4.2) with grad rows s_up q_up and s_dn q_dn =
    s_dn (14 q_up) and s_dn q_dn, and X rows taken as codes.  Dropping the common
    factor s_dn s_x: c^2 = w^2 * sum q^2 * x_sumsq, w = 14 (up) or 1 (down).
    Returned as isqrt(c^2 * 2^16), an exact integer (< 2^31 for the shapes here)."""
    su = [int(v) for v in np.asarray(sumsq_up)]
    sd = [int(v) for v in np.asarray(sumsq_dn)]
    sx = [int(v) for v in np.asarray(x_sumsq)]
    up = [math.isqrt(BS_RATIO * BS_RATIO * a * x << 16) for a, x in zip(su, sx)]
    dn = [math.isqrt(a * x << 16) for a, x in zip(sd, sx)]
    return np.array(up + dn, dtype=np.int64)


def clamp_rescale(c: np.ndarray, budget: int):
    """Inclusion probabilities p_i proportional to c_i with sum p_i = budget and
    p_i <= 1, by the clamp-and-rescale loop of App. A.2, in exact integers.

    Returns (clamped bool[2N], R, S) where rows with clamped=True have p = 1
    and every other row has p = R * c_i / S (0 if c_i = 0).  When no more rows
    than the budget have c_i > 0, every such row gets p = 1 (S = 0)."""
    c = [int(v) for v in c]
    nz = [v > 0 for v in c]
    if sum(nz) <= budget:
        return np.array(nz, dtype=bool), 0, 0
    clamped = [False] * len(c)
    k = 0
    S = sum(c)
    while True:
        R = budget - k
        new = [j for j, v in enumerate(c) if not clamped[j] and v > 0 and R * v >= S]
        if not new:
            break
        for j in new:
            clamped[j] = True
        k += len(new)
        S -= sum(c[j] for j in new)
    return np.array(clamped, dtype=bool), budget - k, S


def resolve_budget(budget: int, N: int) -> int:
    """0 selects B = N (Sec. 4.2: sum p_i = N).  KEEP_NONZERO selects B = 2N: no more than
    2N rows are non-zero, so every non-zero row gets p = 1 and the sample is the
    deterministic rule of the paper's implementation, keep the rows of non-zero norm
    (App. A.6)."""
    if budget == 0:
        return N
    if budget == KEEP_NONZERO:
        return 2 * N
    assert 0 < budget <= 2 * N
    return int(budget)


@dataclass
class LSSPlan:
    budget: int
    c: np.ndarray  # int64 [2N] scores
    clamped: np.ndarray  # bool [2N]
    R: int
    S: int
    e_dn: np.ndarray  # int [N] exponent of each down row (p~ = 2^-e)
    w_up: np.ndarray  # int [N] in {0, 1}
    w_dn: np.ndarray  # int [N] in {0, 1, 2, 4, 8, 16}
    kept: np.ndarray  # int64 [T] ascending token indices with w_up + w_dn > 0

    def p_dn(self) -> np.ndarray:
        """Inclusion probability p~ of every down row (0 for rows never kept)."""
        N = self.w_up.shape[0]
        p = np.where(self.c[N:] > 0, 2.0 ** (-self.e_dn.astype(np.float64)), 0.0)
        return p


def lss_plan(sumsq_up, sumsq_dn, x_sumsq, budget: int, seed: int, offset: int,
             u16_masks: np.ndarray = None) -> LSSPlan:
    """Masks and weights of the shared sample (Sec. 4.2, App. A.2, App. A.6).

    * up rows are always kept when non-zero (weight 1, p~ = 1);
    * down rows get p~ = 2^-e, the smallest power of two >= p*, with e capped at 4
      (at 2 when the token's up row is non-zero so |14 q_up + 2^e q_dn| <= 126);
    * m ~ Bern(p~) from Philox stream 1 as [u16 < 2^(16-e)]; the weight m/p~ = m 2^e."""
    N = len(sumsq_up)
    budget = resolve_budget(budget, N)
    c = leverage_scores(sumsq_up, sumsq_dn, x_sumsq)
    clamped, R, S = clamp_rescale(c, budget)
    su = np.asarray(sumsq_up, dtype=np.int64)
    w_up = (su > 0).astype(np.int64)
    e_dn = np.zeros(N, dtype=np.int64)
    for t in range(N):
        j = N + t
        cj = int(c[j])
        if cj == 0 or clamped[j]:
            continue
        cap = 2 if su[t] > 0 else 4
        e = 0
        while e < cap and (R * cj) << (e + 1) <= S:
            e += 1
        e_dn[t] = e
    if u16_masks is None:
        u16_masks = uniforms16(seed, offset, STREAM_MASK, N)
    u = np.asarray(u16_masks).astype(np.int64)
    m = u < (1 << (16 - e_dn))
    w_dn = np.where((c[N:] > 0) & m, 1 << e_dn, 0).astype(np.int64)
    kept = np.nonzero((w_up + w_dn) > 0)[0].astype(np.int64)
    return LSSPlan(int(budget), c, clamped, int(R), int(S), e_dn, w_up, w_dn, kept)


# --------------------------------------------------------------------------
# LSS-MM backward (Sec. 4.2, App. A.3)
# --------------------------------------------------------------------------
@dataclass
class LSSBackward:
    bs: BitSplit
    plan: LSSPlan
    A: np.ndarray  # int32 [N][C] weighted integer gradient rows (0 for dropped tokens)
    acc_dx: np.ndarray  # int64 [T][D]  A[kept] @ wq
    acc_dw: np.ndarray  # int64 [C][D]  A[kept]^T @ xq[kept]
    dX: np.ndarray  # float64 [N][D]
    dW: np.ndarray  # float64 [C][D]
    alpha_dx: float
    alpha_dw: float


def weighted_rows(bs: BitSplit, plan: LSSPlan) -> np.ndarray:
    """Rows of (I~ M~ grad) in units of s_dn: 14 w_up q_up + w_dn q_dn per token."""
    return (BS_RATIO * plan.w_up[:, None] * bs.q_up.astype(np.int64)
            + plan.w_dn[:, None] * bs.q_dn.astype(np.int64))


def _sample(G: np.ndarray, x_sumsq: np.ndarray, budget: int, seed: int, offset: int):
    """Steps 1-4 of LSS-MM shared by both gradients (App. A.6): bit split, leverage
    scores on the codes, the sample, and the weighted integer rows A."""
    bs = bit_split(G, seed, offset)
    su = np.sum(bs.q_up.astype(np.int64) ** 2, axis=1)
    sd = np.sum(bs.q_dn.astype(np.int64) ** 2, axis=1)
    plan = lss_plan(su, sd, x_sumsq, budget, seed, offset)
    A = weighted_rows(bs, plan)
    assert np.abs(A).max(initial=0) <= 126
    return bs, plan, A


def lss_backward(G: np.ndarray, fwd: HQForward, budget: int, seed: int, offset: int,
                 need_dx: bool = True, need_dw: bool = True) -> LSSBackward:
    """Activation and weight gradients of HQ-MM by LSS-MM.

    grad_X = s_W (grad_Y W^) H^T and grad_W = s_X (grad_Y^T X^) H^T (Sec. 4; the
    clip masks are identically 1 under absmax scales), with grad_Y replaced by
    the sampled bit-split estimate s_dn * A (Sec. 4.2, App. A.3)."""
    k = fwd.log2_block
    bs, plan, A = _sample(G, fwd.x_sumsq, budget, seed, offset)
    N, C = A.shape
    D = fwd.xq.shape[1]
    s_dn = float(bs.s_up) / BS_RATIO
    a_dx = s_dn * float(fwd.s_w) * 2.0 ** (-k)
    a_dw = s_dn * float(fwd.s_x) * 2.0 ** (-k)
    At = A[plan.kept]
    acc_dx = acc_dw = dX = dW = None
    if need_dx:
        acc_dx = _int_matmul(At, fwd.wq.astype(np.int64))
        dX = np.zeros((N, D), dtype=np.float64)
        dX[plan.kept] = a_dx * fwht_rows(acc_dx, k).astype(np.float64)
    if need_dw:
        acc_dw = _int_matmul(At.T, fwd.xq[plan.kept].astype(np.int64))
        dW = a_dw * fwht_rows(acc_dw, k).astype(np.float64)
    return LSSBackward(bs, plan, A, acc_dx, acc_dw, dX, dW, a_dx, a_dw)


# --------------------------------------------------------------------------
# Learned step size mode (Sec. 3.1 Eq. 2, Sec. 4, App. A.3)
# --------------------------------------------------------------------------
# Readings (listed with their reasons in the design notes):
# * the caller's step sizes s_x, s_w belong to the unnormalised transform v = V H_u
#   (the paper's s for the orthonormal H times 2^{k/2}), so Y = s_x s_w x^ w^^T / 2^k
#   exactly as in the dynamic mode;
# * v / s is taken as r = fl(v * fl(1/s)) in float32, codes clamp(rint(r), -7, 7);
# * the clip mask of Sec. 4 is taken on r: I = [-7 <= r <= 7] (Hadamard domain);
# * delta(s) = int_s(v) - I o (v / s) of App. A.3 is formed as q - I r (exact in float32)
#   and kept as float16, in place of the fp16 copy of the input that the paper's
#   implementation keeps for the LSQ backward (App. A.6); |delta| <= 1/2 inside the range
#   and |delta| = 7 where clipped,
#   so the backward reads the mask back as I = [|delta| <= 1/2];
# * the STE gradients mask the integer accumulators in the Hadamard domain, then apply
#   H^T (mask first: chain rule), and the step-size gradients are
#   grad s = g(s) (s_other s_dn / 2^k) sum(acc o delta), g(s) = 1 / sqrt(Q_P numel),
#   the chain rule through s q (App. A.3), with grad_Y replaced by the LSS estimate.


def quantize_lsq(v: np.ndarray, s: float):
    """int_s(v) = round(clamp(v / s, -7, 7)) with a given step s > 0 (Eq. 2).

    Returns (codes int8, mask bool, delta float16): the clip mask I of Sec. 4 and
    delta = q - I o (v / s) of App. A.3 (see the readings above)."""
    v = np.asarray(v, dtype=np.float32)
    s = np.float32(s)
    assert s > 0 and np.isfinite(s)
    inv = np.float32(1.0) / s
    r = (v * inv).astype(np.float32)
    inside = (r >= -QMAX) & (r <= QMAX)
    q = np.clip(np.rint(r), -QMAX, QMAX).astype(np.int8)
    delta = q.astype(np.float32) - np.where(inside, r, np.float32(0.0))
    return q, inside, delta.astype(np.float16)


def lsq_grad_scale(numel: int) -> float:
    """g(s) = 1 / sqrt(Q_P numel), the step-size gradient scale of App. A.3."""
    return 1.0 / math.sqrt(QMAX * int(numel))


@dataclass
class LSQForward:
    log2_block: int
    s_x: np.float32
    s_w: np.float32
    xq: np.ndarray  # int8 [N][D]
    wq: np.ndarray  # int8 [C][D]
    x_sumsq: np.ndarray  # int64 [N]
    dx16: np.ndarray  # float16 [N][D]  delta of X (clip mask |delta| <= 1/2)
    dw16: np.ndarray  # float16 [C][D]
    acc: np.ndarray = field(default=None)
    Y: np.ndarray = field(default=None)


def lsq_forward(X: np.ndarray, W: np.ndarray, log2_block: int, s_x: float, s_w: float,
                compute_output: bool = True) -> LSQForward:
    """HQ-MM with learned step sizes: (1) X H and W H; (2) LSQ to INT4 (Eq. 2, Sec. 3.3
    step 2); (3) integer product; (4) dequantise by s_X s_W (and 2^-k)."""
    k = int(log2_block)
    s_x, s_w = np.float32(s_x), np.float32(s_w)
    vx = fwht_rows(np.asarray(X, dtype=np.float32), k)
    vw = fwht_rows(np.asarray(W, dtype=np.float32), k)
    xq, _, dx16 = quantize_lsq(vx, s_x)
    wq, _, dw16 = quantize_lsq(vw, s_w)
    out = LSQForward(k, s_x, s_w, xq, wq, np.sum(xq.astype(np.int64) ** 2, axis=1), dx16, dw16)
    if compute_output:
        out.acc = _int_matmul(xq, wq.T)
        out.Y = float(s_x) * float(s_w) * 2.0 ** (-k) * out.acc.astype(np.float64)
    return out


@dataclass
class LSQBackward:
    bs: BitSplit
    plan: LSSPlan
    A: np.ndarray
    acc_dx: np.ndarray  # int64 [T][D] unmasked
    acc_dw: np.ndarray  # int64 [C][D] unmasked
    dX: np.ndarray
    dW: np.ndarray
    ds_x: float
    ds_w: float
    alpha_dx: float
    alpha_dw: float


def lsq_backward(G: np.ndarray, fwd: LSQForward, budget: int, seed: int, offset: int,
                 need_dx: bool = True, need_dw: bool = True,
                 delta_x: np.ndarray = None, delta_w: np.ndarray = None) -> LSQBackward:
    """Gradients of HQ-MM with learned step sizes by LSS-MM (Sec. 4, App. A.3).

    grad_X = s_W (I_X o grad_Y W^) H^T, grad_W = s_X (grad_Y^T X^ o I_W) H^T, and the
    step-size gradients g(s) s_other sum(grad_Y W^ o delta_X) (resp. grad_Y^T X^ o
    delta_W), with grad_Y the sampled bit-split estimate s_dn A.  delta_x / delta_w
    replace the stored float16 deltas (tests pass exact ones)."""
    k = fwd.log2_block
    bs, plan, A = _sample(G, fwd.x_sumsq, budget, seed, offset)
    N, C = A.shape
    D = fwd.xq.shape[1]
    s_dn = float(bs.s_up) / BS_RATIO
    a_dx = s_dn * float(fwd.s_w) * 2.0 ** (-k)
    a_dw = s_dn * float(fwd.s_x) * 2.0 ** (-k)
    dlx = np.asarray(fwd.dx16 if delta_x is None else delta_x, dtype=np.float64)
    dlw = np.asarray(fwd.dw16 if delta_w is None else delta_w, dtype=np.float64)
    At = A[plan.kept]
    acc_dx = acc_dw = dX = dW = None
    ds_x = ds_w = 0.0
    if need_dx:
        acc_dx = _int_matmul(At, fwd.wq.astype(np.int64))
        d = dlx[plan.kept]
        masked = np.where(np.abs(d) <= 0.5, acc_dx, 0)
        dX = np.zeros((N, D), dtype=np.float64)
        dX[plan.kept] = a_dx * fwht_rows(masked, k).astype(np.float64)
        ds_x = lsq_grad_scale(N * D) * a_dx * float(np.sum(acc_dx.astype(np.float64) * d))
    if need_dw:
        acc_dw = _int_matmul(At.T, fwd.xq[plan.kept].astype(np.int64))
        masked = np.where(np.abs(dlw) <= 0.5, acc_dw, 0)
        dW = a_dw * fwht_rows(masked, k).astype(np.float64)
        ds_w = lsq_grad_scale(C * D) * a_dw * float(np.sum(acc_dw.astype(np.float64) * dlw))
    return LSQBackward(bs, plan, A, acc_dx, acc_dw, dX, dW, ds_x, ds_w, a_dx, a_dw)


# --------------------------------------------------------------------------
# Attention BMM, T = BMM(Q, K^T) (App. A.1)
# --------------------------------------------------------------------------
# Readings:
# * the batch is B independent instances of the learned-step-size linear operator above,
#   X = Q_b [N][M], W = K_b [P][M], Y = T_b [N][P], with the per-batch steps s_Q[b],
#   s_K[b] of App. A.1 and one Hadamard block size for all batches (H^ repeats H);
# * the backward bit-splits and samples every batch on its own (per-batch scales s_up,b
#   and leverage scores c_{b,i}, as for the linear operator), one shared sample per
#   batch for grad Q and grad K;
# * the random numbers of batch b are those of a single-instance backward at counter
#   offset + b * bmm_counter_stride(N, P): disjoint Philox ranges for every batch;
# * grad s_Q[b] and grad s_K[b] scale by g = 1 / sqrt(Q_P N_s) with N_s the elements
#   quantised with that step (N M and P M).


def bmm_counter_stride(N: int, P: int) -> int:
    """Counter blocks between consecutive batches: those one backward over an N x P
    gradient draws on its stochastic-rounding stream (8 uniforms per block)."""
    return philox_blocks(int(N) * int(P))


def bmm_lsq_forward(Q: np.ndarray, K: np.ndarray, log2_block: int, s_q, s_k,
                    compute_output: bool = True):
    """HQ-MM of every batch (App. A.1): Q [B][N][M], K [B][P][M], steps s_q, s_k [B]."""
    Q = np.asarray(Q, dtype=np.float32)
    K = np.asarray(K, dtype=np.float32)
    assert Q.ndim == 3 and K.ndim == 3 and Q.shape[0] == K.shape[0] and Q.shape[2] == K.shape[2]
    return [lsq_forward(Q[b], K[b], log2_block, np.float32(s_q[b]), np.float32(s_k[b]),
                        compute_output) for b in range(Q.shape[0])]


def bmm_lsq_backward(G: np.ndarray, fwds, budget: int, seed: int, offset: int,
                     need_dq: bool = True, need_dk: bool = True):
    """LSS-MM of every batch (App. A.1): G = grad T [B][N][P]; batch b draws its random
    numbers at counter offset + b * bmm_counter_stride(N, P)."""
    G = np.asarray(G, dtype=np.float32)
    B, N, P = G.shape
    adv = bmm_counter_stride(N, P)
    return [lsq_backward(G[b], fwds[b], budget, seed, offset + b * adv, need_dq, need_dk)
            for b in range(B)]
