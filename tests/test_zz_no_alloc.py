"""GPU test of the allocation-free forward, hq_linear_fwd_noalloc, through the C ABI.

It must give the same bits as hq_linear_fwd with a caller workspace (codes, row sums,
maxima, Y), and meet the oracle, on consecutive calls that share the library's static
scratch array: a shape that splits its GEMM along K (partials in the scratch), then a
smaller one, then a smaller split shape again (stale partials from the first call must
not leak into it).
"""
import numpy as np
import pytest
import torch

import synth
from gpu_util import TORCH_DT, check_forward, dev_tensor, need_gpu, say, to_np

pytestmark = pytest.mark.gpu

# (N, D, C, log2_block, dtype): the first and third split along K
CALLS = [
    (300, 4096, 256, 7, "bf16"),
    (77, 512, 192, 5, "f16"),
    (64, 2048, 64, 3, "f32"),
]


def _inputs(shape, seed):
    N, D, C, k, dt = shape
    lin = synth.Linear(f"na{N}x{D}x{C}", N, D, C, k, dt, max(1, D // 100), 20.0, "lognormal", N)
    X, W, _ = synth.linear_inputs(lin, seed, with_grad=False)
    return X, W


def _bits(t):
    return t.contiguous().view(torch.uint8) if t.dtype != torch.uint8 else t


def test_noalloc_forward_matches_workspace_forward():
    H = need_gpu()
    assert H.workspace_bytes(H.WS_FWD, *CALLS[0][:3]) > H.workspace_bytes(H.WS_FWD, *CALLS[1][:3])
    assert H.workspace_bytes(H.WS_FWD, *CALLS[2][:3]) > H.workspace_bytes(H.WS_FWD, *CALLS[1][:3])
    for i, shape in enumerate(CALLS):
        N, D, C, k, dt = shape
        say(f"noalloc forward call {i}: N={N} D={D} C={C} k={k} {dt} "
            f"(scratch {H.workspace_bytes(H.WS_FWD, N, D, C)} of {H.STATIC_SCRATCH_BYTES} bytes)")
        X, W = _inputs(shape, 40 + i)
        tX, tW = dev_tensor(X, dt), dev_tensor(W, dt)
        Y_ref = torch.empty(N, C, device="cuda", dtype=TORCH_DT[dt])
        sv_ref = H.Saved.empty(N, D, C)
        H.hq_linear_fwd(tX, tW, Y_ref, sv_ref, k, H.workspace(H.WS_FWD, N, D, C))
        Y = torch.full((N, C), float("nan"), device="cuda", dtype=TORCH_DT[dt])
        sv = H.Saved.empty(N, D, C)
        H.hq_linear_fwd_noalloc(tX, tW, Y, sv, k)
        torch.cuda.synchronize()
        for name in ("xq", "wq", "wqT", "x_sumsq", "amax"):
            assert torch.equal(_bits(getattr(sv, name)), _bits(getattr(sv_ref, name))), name
        assert torch.equal(_bits(Y), _bits(Y_ref)), "Y differs from hq_linear_fwd"
        rel = check_forward(H, X, W, k, dt, sv, Y)
        assert np.isfinite(rel)


def test_noalloc_forward_rejects_oversized_shape():
    """A shape whose forward scratch exceeds the static array returns HQLSS_ERR_SCRATCH from
    host validation (nothing is launched)."""
    H = need_gpu()
    N, D, C = 2048, 16384, 2048
    assert H.workspace_bytes(H.WS_FWD, N, D, C) > H.STATIC_SCRATCH_BYTES
    X = torch.zeros(N, D, device="cuda", dtype=torch.bfloat16)
    W = torch.zeros(C, D, device="cuda", dtype=torch.bfloat16)
    Y = torch.empty(N, C, device="cuda", dtype=torch.bfloat16)
    sv = H.Saved.empty(N, D, C)
    with pytest.raises(H.HQLSSError) as e:
        H.hq_linear_fwd_noalloc(X, W, Y, sv, 7)
    assert "scratch" in str(e.value)
    torch.cuda.synchronize()
