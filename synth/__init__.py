"""Seeded synthetic workloads for the INT4 HQ-MM / LSS-MM linear operator.

This module only draws random inputs.  It holds none of the method's
arithmetic (no transform, no quantiser, no sampling), so that both the CPU
oracle and the GPU path can consume the very same inputs without sharing any
code that computes a result.

The paper's workloads are transformer linears fed by datasets and pretrained
checkpoints that are not available here.  The generators below stand in for
them, reproducing the structure the paper describes:

* activations with a few outlier channels (Sec. 3.2 and Fig. 1: outliers are
  concentrated on a few feature dimensions);
* row-sparse output gradients whose per-token norms are heavy-tailed
  (Sec. 4.1 and Fig. 2: a few tokens carry large gradients, most are ~0).

Every array is returned as float32 holding values that are exactly
representable in the workload dtype ("f32", "f16" or "bf16"), i.e. the
*cast* tensor is the input seen by every consumer.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Tuple

import numpy as np

DTYPES = ("f32", "f16", "bf16")


def round_to_dtype(a: np.ndarray, dtype: str) -> np.ndarray:
    """Return float32 values rounded (RNE) to `dtype` and widened back."""
    a = np.asarray(a, dtype=np.float32)
    if dtype == "f32":
        return a.copy()
    if dtype == "f16":
        return a.astype(np.float16).astype(np.float32)
    if dtype == "bf16":
        import torch  # CPU-only use: numpy has no bfloat16

        return torch.from_numpy(a.copy()).to(torch.bfloat16).to(torch.float32).numpy()
    raise ValueError(dtype)


@dataclasses.dataclass(frozen=True)
class Linear:
    """One linear layer Y = X W^T with X: N x D, W: C x D (Eq. 1)."""

    name: str
    N: int
    D: int  # C_in
    C: int  # C_out
    log2_block: int
    dtype: str
    x_outlier_channels: int  # number of outlier input channels
    x_outlier_scale: float
    grad_kind: str  # "sparse_rows" | "lognormal" | "pareto"
    budget: int  # LSS budget B (sum of inclusion probabilities)


@dataclasses.dataclass(frozen=True)
class Workload:
    cfg_id: int
    name: str
    linears: Tuple[Linear, ...]


def _pct_channels(D: int) -> int:
    return int(math.ceil(0.01 * D))


def workload(cfg_id: int) -> Workload:
    """The five transformer-shaped workloads (sizes from the paper's setting:
    typical Hadamard block 2^5, hidden sizes 768..4096; Sec. 3.3)."""
    if cfg_id == 0:
        N, D, C = 128, 256, 256
        return Workload(0, "single linear N=128 256->256 b=32 fp32", (
            Linear("single", N, D, C, 5, "f32", 4, 50.0, "sparse_rows", N),))
    if cfg_id == 1:
        N = 16384
        mk = lambda nm, d, c: Linear(nm, N, d, c, 5, "f16", _pct_channels(d), 20.0, "lognormal", N)
        return Workload(1, "BERT-base FFN pair N=16384 768->3072->768 b=32 fp16",
                        (mk("ffn1", 768, 3072), mk("ffn2", 3072, 768)))
    if cfg_id == 2:
        N = 8192
        mk = lambda nm, d, c: Linear(nm, N, d, c, 7, "f16", _pct_channels(d), 20.0, "lognormal", N)
        return Workload(2, "GPT-2-medium linears N=8192 b=128 fp16",
                        (mk("qkv", 1024, 3072), mk("attn_out", 1024, 1024),
                         mk("ffn1", 1024, 4096), mk("ffn2", 4096, 1024)))
    if cfg_id == 3:
        N = 16384
        mk = lambda nm, d, c: Linear(nm, N, d, c, 7, "bf16", _pct_channels(d), 50.0, "pareto", N)
        return Workload(3, "GEMM sweep N=16384 b=128 bf16",
                        (mk("4096x4096", 4096, 4096), mk("4096x11008", 4096, 11008),
                         mk("11008x4096", 11008, 4096), mk("8192x8192", 8192, 8192)))
    if cfg_id == 4:
        N = 16384
        mk = lambda nm, d, c: Linear(nm, N, d, c, 5, "f16", _pct_channels(d), 20.0, "lognormal", N)
        return Workload(4, "BERT-large encoder block linears N=16384 b=32 fp16",
                        (mk("q", 1024, 1024), mk("k", 1024, 1024), mk("v", 1024, 1024),
                         mk("o", 1024, 1024), mk("ffn1", 1024, 4096), mk("ffn2", 4096, 1024)))
    raise ValueError(cfg_id)


def _rngs(seed: int, index: int, n: int) -> List[np.random.Generator]:
    ss = np.random.SeedSequence([seed, index])
    return [np.random.default_rng(s) for s in ss.spawn(n)]


def gen_x(N: int, D: int, n_outlier: int, scale: float, rng_x, rng_sel) -> np.ndarray:
    x = rng_x.standard_normal((N, D), dtype=np.float32)
    if n_outlier > 0:
        ch = rng_sel.choice(D, size=n_outlier, replace=False)
        x[:, ch] *= np.float32(scale)
    return x


def gen_w(C: int, D: int, rng) -> np.ndarray:
    return rng.standard_normal((C, D), dtype=np.float32) * np.float32(0.02)


def gen_grad(N: int, C: int, kind: str, rng_g, rng_rows) -> np.ndarray:
    g = rng_g.standard_normal((N, C), dtype=np.float32)
    if kind == "sparse_rows":
        # N(0, 1e-3) entries; 90 % of the rows shrunk by a further 1e-3
        g *= np.float32(1e-3)
        rows = rng_rows.choice(N, size=int(round(0.9 * N)), replace=False)
        g[rows] *= np.float32(1e-3)
        return g
    # unit-norm Gaussian row direction times a heavy-tailed row norm rho
    nrm = np.sqrt(np.einsum("ij,ij->i", g, g, dtype=np.float64)).astype(np.float32)
    nrm[nrm == 0] = 1
    g /= nrm[:, None]
    if kind == "lognormal":
        rho = rng_rows.lognormal(0.0, 2.0, size=N)
    elif kind == "pareto":
        rho = rng_rows.pareto(1.5, size=N) + 1.0
    else:
        raise ValueError(kind)
    g *= rho.astype(np.float32)[:, None]
    return g


def linear_inputs(lin: Linear, seed: int, index: int = 0, with_grad: bool = True):
    """(X, W, dY) float32 arrays holding exact `lin.dtype` values."""
    r_x, r_w, r_g, r_ch, r_rows = _rngs(seed, index, 5)
    X = round_to_dtype(gen_x(lin.N, lin.D, lin.x_outlier_channels, lin.x_outlier_scale, r_x, r_ch),
                       lin.dtype)
    W = round_to_dtype(gen_w(lin.C, lin.D, r_w), lin.dtype)
    G = None
    if with_grad:
        G = round_to_dtype(gen_grad(lin.N, lin.C, lin.grad_kind, r_g, r_rows), lin.dtype)
    return X, W, G


def small_linear(N: int, D: int, C: int, log2_block: int, dtype: str = "f32",
                 grad_kind: str = "lognormal", n_outlier: int = 2, budget: int = 0) -> Linear:
    """A small ad-hoc linear for parity tests (same generators, any shape)."""
    return Linear(f"small_{N}x{D}x{C}", N, D, C, log2_block, dtype, n_outlier, 20.0, grad_kind,
                  budget if budget > 0 else N)
