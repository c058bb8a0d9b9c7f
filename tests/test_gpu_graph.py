"""The hot path captured in one HIP graph, through torch's graph capture on the current
stream.  The library's launches allocate nothing and never synchronise, so a whole forward
and backward step (quantizers, bit split, sampler, operand builder, the three GEMMs)
captures as it is.  Every replay, with eager steps and synchronisations between replays,
must reproduce the eager step bit for bit (the Philox offset is a kernel argument, so each
replay draws the sample it captured), and the eager step matches the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from gpu_util import TORCH_DT, check_float_output, dev_tensor, need_gpu, say, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape", [(600, 256, 320, 5, "f16", "pareto"), (1024, 512, 256, 7, "bf16", "lognormal")],
                         ids=["N600_b32_f16", "N1024_b128_bf16"])
def test_graph_replay_matches_eager(shape):
    H = need_gpu()
    N, D, C, k, dt, kind = shape
    lin = synth.Linear(f"t{N}x{D}x{C}", N, D, C, k, dt, max(1, D // 100), 20.0, kind, N)
    X, W, G = synth.linear_inputs(lin, 7)
    budget, seed, offset = N // 2, 3, 5
    say(f"graph replay {shape}")
    tX, tW, tG = dev_tensor(X, dt), dev_tensor(W, dt), dev_tensor(G, dt)
    Y = torch.empty(N, C, device="cuda", dtype=TORCH_DT[dt])
    dX = torch.empty(N, D, device="cuda", dtype=TORCH_DT[dt])
    dW = torch.empty(C, D, device="cuda", dtype=TORCH_DT[dt])
    saved = H.Saved.empty(N, D, C)
    wsf = H.workspace(H.WS_FWD, N, D, C)
    ws = H.workspace(H.WS_BWD, N, D, C)
    outs = (Y, dX, dW, saved.xq, saved.wq, saved.wqT)

    def step():
        H.hq_linear_fwd(tX, tW, Y, saved, k, wsf)
        H.lss_linear_bwd(tG, saved, dX, dW, D, k, budget, seed, offset, ws)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    f = O.hq_forward(X, W, k)
    b = O.lss_backward(G, f, budget, seed, offset)
    check_float_output("Y", Y, f.Y, dt)
    check_float_output("dX", dX, b.dX, dt)
    check_float_output("dW", dW, b.dW, dt)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        for t in (Y, dX, dW):
            t.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("Y", "dX", "dW", "X codes", "W codes", "W^T codes"), outs, ref):
            assert torch.equal(got, want), f"replay {rep}: {name}"
        step()  # eager work between replays
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(outs, ref)), f"eager step after replay {rep}"
    del g
