"""Benchmark: INT4 HQ-MM / LSS-MM linear fwd+bwd on one MI355X.

One step = forward (HQ-MM) and backward (LSS-MM: dX and dW from one shared sample) of
every linear of the workload.  The default workload is the square and rectangular GEMM
sweep: N = 16384 tokens, (D, C) = (4096, 4096), (4096, 11008), (11008, 4096),
(8192, 8192), bf16 inputs, Hadamard block 128, LSS budget N.  Inputs are seeded
synthetic tensors with the paper's structure (outlier channels in X, heavy-tailed row
norms in dY), resident in HBM before timing starts; the steps cycle over enough copies
of them that no step reads inputs a previous step left in the 256 MB MALL.

Timing: W warm-up steps, then K timed steps with one HIP event pair per step; the step
time is the median over the K steps (the wall-clock mean is printed beside it).

Metric: effective TOPS = sum over linears of 6 N C D / step time (the dense-equivalent
work of fwd + dX + dW), also as a fraction of the int8 MFMA peak, beside the same three
GEMMs per linear in bf16 through torch (hipBLASLt) and the CPU oracle on a token slice.
Each linear is also timed alone (`per_linear`), and the error of its outputs against
the unquantised fp64 products is reported (`quant_error_vs_fp64`, untimed).

--workload 1, 2 or 4 runs the same step on the other linear-layer workloads instead
(the BERT-base FFN pair N = 16384; GPT-2-medium linears N = 8192; the BERT-large
encoder block linears).

--mode bmm times the attention BMM T = BMM(Q, K^T) of App. A.1 instead (per-batch learned
steps, per-batch sampling): BERT-base attention scores, 32 sequences x 12 heads = 384
batches of 512 x 512 x 64, fp16, Hadamard block 32, steps half of each batch's dynamic
step; effective TOPS = 6 B N P M / step time, beside the same three products per step as
bf16 torch.bmm.

--mode lsq times the learned-step-size variant instead (Eq. 2 with caller-given steps,
App. A.3 gradients including the step-size gradients), on the same workload with steps set
before timing to half of each tensor's dynamic step (s = max|V H| / 14, so the largest
entries clip).

Prints ONE JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0  # MI355X dense int8 MFMA
FP6_PEAK_TOPS = 10100.0  # MI355X dense FP6 MFMA
HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20  # MI355X last-level (Infinity) cache
# vector ALU: 256 CUs x 4 SIMDs x 16 lanes per clock x 2.4 GHz (the fp32 vector peak of
# 157.3 TFLOP/s counts a packed FMA, 4 flops, per slot)
VALU_PEAK_TSLOTS = 256 * 4 * 16 * 2.4e9 / 1e12
# bit split, per gradient element: one Philox4x32-10 block per 8 elements (10 rounds of two
# 32x32->64 multiplies, 4 slots each, and two 3-input xors) = 12.5, plus 11 full-rate
# operations (widen and scale, round, residual x 14, floor, fraction, x 2^16, uniform to
# float, compare, add, pack, sum of squares)
BS_VALU_SLOTS_PER_ELEM = 23.5
METRIC = "INT4 linear fwd+bwd effective TOPS (fraction of int8-MFMA peak) vs bf16"
# workloads: id -> key of the committed counter summaries under profiles/
WORKLOAD_KEYS = {1: "bert_base_ffn", 2: "gpt2_medium", 3: "gemm_sweep", 4: "bert_large_block"}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-bf16", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU-oracle sample time")
    p.add_argument("--mode", choices=("dynamic", "lsq", "bmm", "fp6"), default="dynamic",
                   help="dynamic: per-tensor maxima on the int8 MFMA route (default); fp6: the same "
                        "operator on the FP6 MFMA route; lsq: learned step sizes; bmm: attention BMM")
    p.add_argument("--workload", type=int, choices=sorted(WORKLOAD_KEYS), default=3,
                   help="1: BERT-base FFN pair; 2: GPT-2-medium linears; "
                        "3: GEMM sweep N=16384 (4096..11008, bf16; default); 4: BERT-large encoder block linears")
    p.add_argument("--rotate", type=int, default=0, metavar="K",
                   help="cycle the steps over K copies of the inputs at different addresses "
                        "(no cross-step cache reuse; the bf16 comparison cycles likewise); "
                        "0 (default): enough copies that one cycle exceeds twice the 256 MB MALL")
    p.add_argument("--no-per-linear", action="store_true",
                   help="skip timing each linear alone (profiling runs)")
    p.add_argument("--no-error", action="store_true",
                   help="skip the (untimed) error of the outputs against the unquantised fp64 products")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="before the steps, run the library's plain copy kernel once over MIB MiB "
                        "(reference for hardware traffic counters)")
    return p.parse_args()


def gemm_source_digest() -> str:
    h = hashlib.sha256()
    for f in ("gemm.hip", "gemm_kernel.h", "gemm6.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2306_11987_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` measured by rocprofv3 counters, if the committed
    summary was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_pmc.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_src = re.search(r"kernel_source_digest:\s*([0-9a-f]+)", txt)
    m_b = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", txt)
    if not (m_src and m_b) or m_src.group(1) != gemm_source_digest():
        return None
    return float(m_b.group(1))


def progress(msg):
    """One progress line on stderr per finished stage (the JSON line stays alone on stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def _median(xs):
    s = sorted(xs)
    n = len(s)
    return 0.5 * (s[(n - 1) // 2] + s[n // 2]) if n else float("nan")


def _timed_steps(torch, fn, steps):
    """Run fn `steps` times with a HIP event pair around each call on the current stream
    (the stream every library launch and torch op here is issued on).  Returns the wall
    time of the whole bracket (synchronised on both sides) and the per-step event times."""
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3
    return wall_ms, [a.elapsed_time(b) for a, b in evs]


def _auto_rotation(L, eb):
    """Copies of the inputs such that one cycle of them exceeds twice the 256 MB MALL:
    a step then never reads inputs the previous steps left in the cache."""
    set_bytes = sum(eb * (e["lin"].N * e["lin"].D + e["lin"].C * e["lin"].D + e["lin"].N * e["lin"].C)
                    for e in L)
    return max(1, -(-(2 * MALL_BYTES) // set_bytes))


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the operator runs on exactly one GPU (asked for {args.gpus}); "
              "multi-GPU runs are not supported", file=sys.stderr)
        sys.exit(3)

    import numpy as np
    import torch

    import paper_2306_11987_amd as H
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    if args.mode == "bmm":
        return main_bmm(args, np, torch, H, synth, dev)
    cfg_id = args.workload
    wl = synth.workload(cfg_id)
    lins = wl.linears
    N = lins[0].N
    tdt = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}[lins[0].dtype]
    eb = {"f16": 2, "bf16": 2, "f32": 4}[lins[0].dtype]

    # ---- inputs resident in HBM, state and workspaces preallocated
    L = []
    for li, lin in enumerate(lins):
        X, W, G = synth.linear_inputs(lin, cfg_id, li)
        e = dict(lin=lin,
                 X=torch.from_numpy(X).to(dev, tdt), W=torch.from_numpy(W).to(dev, tdt),
                 G=torch.from_numpy(G).to(dev, tdt),
                 Y=torch.empty(lin.N, lin.C, device=dev, dtype=tdt),
                 dX=torch.empty(lin.N, lin.D, device=dev, dtype=tdt),
                 dW=torch.empty(lin.C, lin.D, device=dev, dtype=tdt),
                 saved=(H.saved_fp6_empty if args.mode == "fp6" else H.Saved.empty)(lin.N, lin.D, lin.C, dev),
                 ws=H.workspace(H.WS_BWD_FP6 if args.mode == "fp6" else H.WS_BWD, lin.N, lin.D, lin.C, dev),
                 wsf=H.workspace(H.WS_FWD_FP6 if args.mode == "fp6" else H.WS_FWD, lin.N, lin.D, lin.C, dev),
                 adv=H.lss_philox_offset_advance(lin.N, lin.C))
        L.append(e)
    del X, W, G
    progress(f"inputs resident: {wl.name}")
    seed = 0
    offsets = [0] * len(L)
    lsq_mode = args.mode == "lsq"
    fp6_mode = args.mode == "fp6"
    if lsq_mode:
        # steps (untimed): half of the dynamic step a / 7 of each tensor, a from the library
        for e in L:
            lin = e["lin"]
            H.hq_linear_fwd(e["X"], e["W"], e["Y"], e["saved"], lin.log2_block, e["wsf"])
            step_t = (e["saved"].amax / 14.0).contiguous()
            e["lsq"] = H.LSQ.empty(step_t, lin.N, lin.D, lin.C)
            e["dstep"] = torch.empty(2, dtype=torch.float32, device=dev)
            e["ws"] = H.workspace(H.WS_BWD_LSQ, lin.N, lin.D, lin.C, dev)
            e["wsf"] = H.workspace(H.WS_FWD_LSQ, lin.N, lin.D, lin.C, dev)
        torch.cuda.synchronize()

    def fwd_one(e):
        if lsq_mode:
            H.hq_linear_fwd_lsq(e["X"], e["W"], e["Y"], e["saved"], e["lsq"], e["lin"].log2_block,
                                e["wsf"])
        elif fp6_mode:
            H.hq_linear_fwd_fp6(e["X"], e["W"], e["Y"], e["saved"], e["lin"].log2_block, e["wsf"])
        else:
            H.hq_linear_fwd(e["X"], e["W"], e["Y"], e["saved"], e["lin"].log2_block, e["wsf"])

    def bwd_one(i):
        e = L[i]
        lin = e["lin"]
        if lsq_mode:
            H.lss_linear_bwd_lsq(e["G"], e["saved"], e["lsq"], e["dX"], e["dW"], e["dstep"], lin.D,
                                 lin.log2_block, lin.budget, seed, offsets[i], e["ws"])
        elif fp6_mode:
            H.lss_linear_bwd_fp6(e["G"], e["saved"], e["dX"], e["dW"], lin.D, lin.log2_block,
                                 lin.budget, seed, offsets[i], e["ws"])
        else:
            H.lss_linear_bwd(e["G"], e["saved"], e["dX"], e["dW"], lin.D, lin.log2_block,
                             lin.budget, seed, offsets[i], e["ws"])
        offsets[i] += e["adv"]

    def fwd():
        for e in L:
            fwd_one(e)

    def bwd():
        for i in reversed(range(len(L))):
            bwd_one(i)

    # --rotate K: K copies of every input; step s reads copy s % K
    rot = args.rotate if args.rotate > 0 else _auto_rotation(L, eb)
    for e in L:
        e["sets"] = [(e["X"], e["W"], e["G"])] + [
            (e["X"].clone(), e["W"].clone(), e["G"].clone()) for _ in range(rot - 1)]
    cur = [0]

    def select(e, k):
        e["X"], e["W"], e["G"] = e["sets"][k % rot]

    def step():
        if rot > 1:
            for e in L:
                select(e, cur[0])
            cur[0] += 1
        fwd()
        bwd()

    if args.copy_calibration > 0:
        nb = args.copy_calibration << 20
        src = torch.ones(nb // 4, device=dev, dtype=torch.int32)
        dst = torch.empty_like(src)
        H.debug_copy(src, dst)
        torch.cuda.synchronize()
        assert torch.equal(src, dst)
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # launches of the forwards of one step (splits the per-launch log into fwd and bwd)
    H.timing_enable(True)
    H.timing_read()  # clear
    fwd()
    torch.cuda.synchronize()
    n_fwd = len(H.timing_read(1 << 16))
    H.timing_enable(False)
    step_offsets = list(offsets)
    H.timing_enable(True)
    H.timing_read()  # clear
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    log = H.timing_read(1 << 16)
    H.timing_enable(False)
    ms_step_events = (t1 - t0) * 1e3 / args.steps

    # ---- the headline: the same steps again without per-kernel events; one event pair
    # per step, the median step time reported (the wall time of all steps beside it)
    offsets[:] = step_offsets
    wall_ms, step_ms = _timed_steps(torch, step, args.steps)
    ms_step = _median(step_ms)
    ms_step_wall = wall_ms / args.steps
    progress(f"timed steps done: median {ms_step:.4f} ms per step")

    ops_step = sum(6.0 * e["lin"].N * e["lin"].C * e["lin"].D for e in L)
    tops = ops_step / (ms_step * 1e-3) / 1e12

    # ---- per-kernel times (HIP events on the launch stream, over the timed region)
    per = {}
    for kid, ms in log:
        nm = H.kernel_name(kid)
        c = per.setdefault(nm, [0, 0.0])
        c[0] += 1
        c[1] += ms
    kernels = {nm: {"launches_per_step": c[0] / args.steps, "avg_us": 1e3 * c[1] / c[0],
                    "us_per_step": 1e3 * c[1] / args.steps} for nm, c in per.items()}

    # forward and backward time per step: the log is in launch order, and each step
    # launches the forwards of all linears (n_fwd kernels) before the backwards
    per_step = len(log) // args.steps
    fwd_us = bwd_us = 0.0
    if per_step * args.steps == len(log) and per_step > n_fwd:
        for st in range(args.steps):
            chunk = log[st * per_step:(st + 1) * per_step]
            fwd_us += 1e3 * sum(ms for _, ms in chunk[:n_fwd])
            bwd_us += 1e3 * sum(ms for _, ms in chunk[n_fwd:])
        fwd_us /= args.steps
        bwd_us /= args.steps

    # kept tokens of the timed steps (replayed plans; needed for algorithmic GEMM ops)
    kept = []
    for i, e in enumerate(L):
        lin = e["lin"]
        plan = H.Plan.empty(lin.N, lin.C, dev)
        wsp = H.workspace(H.WS_PLAN, lin.N, lin.D, lin.C, dev)
        off = step_offsets[i]
        ks = []
        for _ in range(args.steps):
            H.lss_grad_plan(e["G"], e["saved"], plan, lin.D, lin.budget, seed, off, wsp)
            ks.append(int(plan.n_kept.item()))
            off += e["adv"]
        kept.append(float(np.mean(ks)))
        del plan, wsp

    # dominant kernel and its roofline
    dom = max(kernels, key=lambda k: kernels[k]["us_per_step"])
    algo = None
    if dom == "gemm_fwd":
        algo = float(np.mean([2.0 * e["lin"].N * e["lin"].C * e["lin"].D for e in L]))
    elif dom in ("gemm_dx", "gemm_dw"):
        algo = float(np.mean([2.0 * k * e["lin"].C * e["lin"].D for k, e in zip(kept, L)]))
    roof = None
    peak = FP6_PEAK_TOPS if fp6_mode else INT8_PEAK_TOPS
    if algo is not None:
        ach = algo / (kernels[dom]["avg_us"] * 1e-6) / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                "traffic": committed_traffic(dom, WORKLOAD_KEYS[cfg_id] + ("_lsq" if lsq_mode else "_fp6" if fp6_mode else "")),
                "algorithmic_ops_per_launch": algo,
                "note": ("FP6" if fp6_mode else "int8") + " MFMA ops (multiply-adds x 2) of the kept-token GEMM, averaged over "
                        "the workload's linears; traffic: HBM bytes per launch from rocprofv3 "
                        "FETCH_SIZE + WRITE_SIZE, calibrated on a copy kernel"}
    gemms = {}
    for nm in ("gemm_fwd", "gemm_dx", "gemm_dw"):
        if nm not in kernels:
            continue
        if nm == "gemm_fwd":
            ops = sum(2.0 * e["lin"].N * e["lin"].C * e["lin"].D for e in L)
        else:
            ops = sum(2.0 * k * e["lin"].C * e["lin"].D for k, e in zip(kept, L))
        us = kernels[nm]["us_per_step"] + (kernels["gemm_reduce"]["us_per_step"]
                                           if nm == "gemm_dw" and "gemm_reduce" in kernels else 0.0)
        gemms[nm] = {"frac": round(ops / (us * 1e-6) / 1e12 / peak, 4),
                     "us_per_step": round(us, 1)}

    # ---- memory-bound stages against the HBM peak, with algorithmic bytes of one read
    # of each input and one write of each result (the second read of a dynamic per-tensor
    # scale is implementation cost): F2+F3 (maximum + quantiser of X and W) and B1+B2
    # (maximum + bit split of dY), each over the summed time of its kernels
    stages = {}
    # linears whose forward product runs on the FP6 MFMA (hq_linear_fwd's size rule): their
    # forward workspace holds the FP6 copies of the codes
    fwd_fp6 = []
    if not (fp6_mode or lsq_mode):
        for e in L:
            lin = e["lin"]
            auto = H.workspace_bytes(H.WS_FWD, lin.N, lin.D, lin.C)
            H.debug_set_fwd_fp6(-1)
            int8 = H.workspace_bytes(H.WS_FWD, lin.N, lin.D, lin.C)
            H.debug_set_fwd_fp6(0)
            if auto > int8:
                fwd_fp6.append([lin.D, lin.C])
    # bytes of the FP6 copies of the codes that the quantizer writes: X and W of every
    # linear on the FP6 route, of the FP6-product linears otherwise
    copies6 = sum(e["lin"].N * e["lin"].D + e["lin"].C * e["lin"].D for e in L
                  if fp6_mode or [e["lin"].D, e["lin"].C] in fwd_fp6)
    if lsq_mode:
        b_q = sum((eb + 2.5) * (e["lin"].N + e["lin"].C) * e["lin"].D + 0.5 * e["lin"].C * e["lin"].D
                  + 4 * (e["lin"].N + e["lin"].C) for e in L)
        stages["F2+F3 lsq_quant"] = (b_q, ["lsq_quant"])
    else:
        b_q = sum((eb + 0.5) * (e["lin"].N + e["lin"].C) * e["lin"].D + 0.5 * e["lin"].C * e["lin"].D
                  + 4 * (e["lin"].N + e["lin"].C) for e in L)
        stages["F2+F3 absmax+quant"] = (b_q, ["fwht_absmax:fwd", "fwht_quant"])
    b_g = sum((eb + 1.0) * e["lin"].N * e["lin"].C + 8 * e["lin"].N for e in L)
    stages["B1+B2 absmax+bit_split"] = (b_g, ["fwht_absmax:bwd", "bit_split"])
    # the maximum kernel serves both F2 and B1: split its time by launch position
    absmax_fwd = absmax_bwd = 0.0
    if per_step * args.steps == len(log):
        for st in range(args.steps):
            chunk = log[st * per_step:(st + 1) * per_step]
            for j, (kid, ms) in enumerate(chunk):
                if H.kernel_name(kid) == "fwht_absmax":
                    if j < n_fwd:
                        absmax_fwd += 1e3 * ms
                    else:
                        absmax_bwd += 1e3 * ms
        absmax_fwd /= args.steps
        absmax_bwd /= args.steps
    part_us = {"fwht_absmax:fwd": absmax_fwd, "fwht_absmax:bwd": absmax_bwd}
    hbm = {}
    for stage, (b, ks) in stages.items():
        us = sum(part_us[k] if k in part_us else kernels.get(k, {}).get("us_per_step", 0.0) for k in ks)
        if us > 0:
            gbs = b / (us * 1e-6) / 1e9
            hbm[stage] = {"algorithmic_MB_per_step": round(b / 1e6, 2), "us_per_step": round(us, 1),
                          "achieved_GBps": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
            if stage.startswith("F2+F3") and copies6 > 0:
                # the quantizer also writes FP6 copies of the codes for the FP6 products
                gbs6 = (b + copies6) / (us * 1e-6) / 1e9
                hbm[stage].update({"fp6_copies_MB_per_step": round(copies6 / 1e6, 2),
                                   "frac_with_fp6_copies": round(gbs6 / HBM_PEAK_GBS, 4)})
    overhead = {k: round(kernels[k]["us_per_step"], 1)
                for k in ("build_operands", "lss_plan", "gemm_reduce", "lsq_step_grad", "fp6_convert",
                          "fp6_plan", "fp6_build") if k in kernels}

    # ---- per linear: that linear's fwd + bwd alone, median of per-step event times
    per_linear = []
    n_lin_steps = max(5, min(args.steps, 20))
    for i, e in (() if args.no_per_linear else enumerate(L)):
        lin = e["lin"]
        c = [0]

        def lstep(e=e, i=i, c=c):
            if rot > 1:
                select(e, c[0])
                c[0] += 1
            fwd_one(e)
            bwd_one(i)

        for _ in range(2):
            lstep()
        _, ts = _timed_steps(torch, lstep, n_lin_steps)
        ms_l = _median(ts)
        ops_l = 6.0 * lin.N * lin.C * lin.D
        per_linear.append({"D": lin.D, "C": lin.C, "ms": round(ms_l, 4),
                           "tops": round(ops_l / (ms_l * 1e-3) / 1e12, 1),
                           "frac_int8_peak": round(ops_l / (ms_l * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
                           "kept_tokens": round(kept[i], 1),
                           "kept_over_budget": round(kept[i] / (lin.budget or lin.N), 4)})

    progress("per-linear timings done")
    # ---- bf16 reference: the same three GEMMs per linear through torch (hipBLASLt)
    bf16 = None
    if not args.no_bf16:
        Bs = [[tuple(t.to(torch.bfloat16) for t in e["sets"][k]) for e in L] for k in range(rot)]
        bcur = [0]

        def bstep():
            for X, W, G in Bs[bcur[0] % rot]:
                torch.matmul(X, W.t())
                torch.matmul(G, W)
                torch.matmul(G.t(), X)
            bcur[0] += 1

        for _ in range(args.warmup):
            bstep()
        _, bts = _timed_steps(torch, bstep, args.steps)
        bms = _median(bts)
        bf16 = {"ms_per_step": round(bms, 4), "tops": round(ops_step / (bms * 1e-3) / 1e12, 2),
                "speedup_int4_over_bf16": round(bms / ms_step, 3)}
        for i, e in enumerate(L[:len(per_linear)]):
            c = [0]

            def bl(i=i, c=c):
                X, W, G = Bs[c[0] % rot][i]
                torch.matmul(X, W.t())
                torch.matmul(G, W)
                torch.matmul(G.t(), X)
                c[0] += 1

            for _ in range(2):
                bl()
            _, ts = _timed_steps(torch, bl, n_lin_steps)
            per_linear[i]["bf16_ms"] = round(_median(ts), 4)
            per_linear[i]["speedup_int4_over_bf16"] = round(per_linear[i]["bf16_ms"] / per_linear[i]["ms"], 3)
        del Bs

    # ---- error of the outputs against the unquantised fp64 products (untimed): relative
    # Frobenius norm of Y - X W^T, dX - dY W, dW - dY^T X for the last step's outputs
    qerr = None
    if not args.no_error:
        qerr = []
        for i, e in enumerate(L):
            select(e, 0)
            fwd_one(e)
            bwd_one(i)
            torch.cuda.synchronize()
            X64, W64, G64 = (t.to(torch.float64) for t in (e["X"], e["W"], e["G"]))

            def rel(got, ref):
                return float(torch.linalg.norm(got.to(torch.float64) - ref) / torch.linalg.norm(ref))

            r = {"D": e["lin"].D, "C": e["lin"].C,
                 "Y": round(rel(e["Y"], X64 @ W64.t()), 4),
                 "dX": round(rel(e["dX"], G64 @ W64), 4),
                 "dW": round(rel(e["dW"], G64.t() @ X64), 4)}
            qerr.append(r)
            del X64, W64, G64
            torch.cuda.empty_cache()

    progress("bf16 and error checks done")
    # ---- CPU oracle on a bounded token slice of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(lins, cfg_id, args.cpu_seconds, lsq_mode)
        progress("CPU baseline done")

    route = "FP6 MFMA (e2m3 codes)" if fp6_mode else "int8 MFMA"
    if fwd_fp6:
        route += "; forward products of the linears " + ", ".join(f"{d}x{c}" for d, c in fwd_fp6) + \
                 " on the FP6 MFMA (e2m3 copies of the codes)"
    out = {
        "metric": METRIC,
        "value": round(tops, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp6-e2m3" if fp6_mode else ("i8+fp6-e2m3" if fwd_fp6 else "i8"),
        "data": "synthetic",
        "config": {"workload": wl.name, "N": N, "linears": [[e["lin"].D, e["lin"].C] for e in L],
                   "log2_block": lins[0].log2_block, "io_dtype": lins[0].dtype, "budget": lins[0].budget,
                   "quantizer": "lsq (s = max|V H| / 14)" if lsq_mode else "per-tensor max",
                   "route": route,
                   "kept_tokens": [round(k, 1) for k in kept]},
        "frac_int8_peak": round(tops / INT8_PEAK_TOPS, 4),
        "timing": "median of per-step HIP-event times over the timed steps",
        "ms_per_step_wall_mean": round(ms_step_wall, 4),
        "ms_per_step_min_max": [round(min(step_ms), 4), round(max(step_ms), 4)],
        "ms_per_step_with_kernel_events": round(ms_step_events, 4),
        "us_per_step_fwd_bwd": [round(fwd_us, 1), round(bwd_us, 1)],
        "input_sets": rot,
        "roofline": roof,
        "cpu_baseline": cpu,
        "gemm_frac_of_peak": gemms,
        "gemm_peak_tops": peak,
        "hbm_stages": hbm,
        "overhead_us_per_step": overhead,
        "per_linear": per_linear,
        "quant_error_vs_fp64": qerr,
        "bf16": bf16,
        "kernels": {k: {kk: round(vv, 3) for kk, vv in v.items()} for k, v in sorted(kernels.items())},
    }
    print(json.dumps(out), flush=True)


BMM_B, BMM_N, BMM_P, BMM_M, BMM_K = 384, 512, 512, 64, 5
BMM_METRIC = "INT4 attention BMM fwd+bwd effective TOPS (fraction of int8-MFMA peak) vs bf16"


def bmm_inputs(np, synth, b, n_rows=BMM_N):
    """Q_b, K_b, dT_b of batch b: the linear workload generators at attention shapes."""
    lin = synth.Linear(f"attn{b}", n_rows, BMM_M, BMM_P, BMM_K, "f16", 2, 20.0, "lognormal", n_rows)
    return synth.linear_inputs(lin, 5000 + b)


def main_bmm(args, np, torch, H, synth, dev):
    B, N, P, M, k = BMM_B, BMM_N, BMM_P, BMM_M, BMM_K
    tdt = torch.float16
    Qh, Kh, Gh = (np.stack(a) for a in zip(*[bmm_inputs(np, synth, b) for b in range(B)]))
    Q = torch.from_numpy(Qh).to(dev, tdt)
    K = torch.from_numpy(Kh).to(dev, tdt)
    G = torch.from_numpy(Gh).to(dev, tdt)
    del Qh, Kh, Gh
    # per-batch steps (untimed): half of each batch's dynamic step, from the library's forward
    s_q = torch.empty(B, dtype=torch.float32, device=dev)
    s_k = torch.empty(B, dtype=torch.float32, device=dev)
    sv1 = H.Saved.empty(N, M, P, dev)
    Y1 = torch.empty(N, P, device=dev, dtype=tdt)
    ws1 = H.workspace(H.WS_FWD, N, M, P, dev)
    for b in range(B):
        H.hq_linear_fwd(Q[b], K[b], Y1, sv1, k, ws1)
        s_q[b:b + 1].copy_(sv1.amax[0:1] / 14.0)
        s_k[b:b + 1].copy_(sv1.amax[1:2] / 14.0)
    del sv1, Y1, ws1
    T = torch.empty(B, N, P, device=dev, dtype=tdt)
    dQ = torch.empty(B, N, M, device=dev, dtype=tdt)
    dK = torch.empty(B, P, M, device=dev, dtype=tdt)
    ds_q = torch.empty(B, dtype=torch.float32, device=dev)
    ds_k = torch.empty(B, dtype=torch.float32, device=dev)
    saved = H.bmm_saved_empty(B, N, M, P, dev)
    lsq = H.BmmLSQ.empty(s_q, s_k, N, M, P)
    ws = H.bmm_workspace(H.WS_BMM_BWD, B, N, M, P, dev)
    adv = B * H.lss_philox_offset_advance(N, P)
    off = [0]

    def step():
        H.hq_bmm_fwd_lsq(Q, K, T, saved, lsq, k)
        H.lss_bmm_bwd_lsq(G, saved, lsq, dQ, dK, ds_q, ds_k, M, k, N, 0, off[0], ws)
        off[0] += adv

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    H.timing_enable(True)
    H.timing_read()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    log = H.timing_read(1 << 16)
    H.timing_enable(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    ops_step = 6.0 * B * N * P * M
    tops = ops_step / (ms_step * 1e-3) / 1e12
    per = {}
    for kid, ms in log:
        c = per.setdefault(H.kernel_name(kid), [0, 0.0])
        c[0] += 1
        c[1] += ms
    kernels = {nm: {"launches_per_step": c[0] / args.steps, "avg_us": 1e3 * c[1] / c[0],
                    "us_per_step": 1e3 * c[1] / args.steps} for nm, c in per.items()}
    dom = max(kernels, key=lambda x: kernels[x]["us_per_step"])
    roof = None
    if dom == "gemm_fwd":
        algo = 2.0 * B * N * P * M
        ach = algo / (kernels[dom]["avg_us"] * 1e-6) / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 2), "peak": INT8_PEAK_TOPS,
                "unit": "TFLOP/s", "frac": round(ach / INT8_PEAK_TOPS, 4), "traffic": None,
                "algorithmic_ops_per_launch": algo}
    elif dom == "bit_split":  # bound by vector-ALU issue (Philox and the rounding)
        algo = BS_VALU_SLOTS_PER_ELEM * B * N * P
        ach = algo / (kernels[dom]["avg_us"] * 1e-6) / 1e12
        roof = {"kernel": dom, "bound": "alu", "achieved": round(ach, 2), "peak": VALU_PEAK_TSLOTS,
                "unit": "T VALU lane-slots/s", "frac": round(ach / VALU_PEAK_TSLOTS, 4), "traffic": None,
                "algorithmic_ops_per_launch": algo,
                "note": f"{BS_VALU_SLOTS_PER_ELEM} lane-slots per element of dT (Philox4x32-10 share "
                        "with 32x32->64 multiplies at quarter rate, plus the rounding and packing)"}
    bf16 = None
    if not args.no_bf16:
        Qb, Kb, Gb = (t.to(torch.bfloat16) for t in (Q, K, G))
        KbT = Kb.transpose(1, 2).contiguous()
        GbT = Gb.transpose(1, 2).contiguous()

        def bstep():
            torch.bmm(Qb, KbT)
            torch.bmm(Gb, Kb)
            torch.bmm(GbT, Qb)

        for _ in range(args.warmup):
            bstep()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            bstep()
        torch.cuda.synchronize()
        bms = (time.perf_counter() - t0) * 1e3 / args.steps
        bf16 = {"ms_per_step": round(bms, 4), "tops": round(ops_step / (bms * 1e-3) / 1e12, 2),
                "speedup_int4_over_bf16": round(bms / ms_step, 3)}
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline_bmm(np, synth, args.cpu_seconds)
    out = {
        "metric": BMM_METRIC, "value": round(tops, 2), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "i8",
        "data": "synthetic",
        "config": {"workload": "BERT-base attention scores BMM (App. A.1)", "B": B, "N": N, "P": P,
                   "M": M, "log2_block": k, "io_dtype": "f16", "budget": N,
                   "quantizer": "lsq, per-batch steps (s = max|V H| / 14)"},
        "frac_int8_peak": round(tops / INT8_PEAK_TOPS, 4),
        "roofline": roof, "cpu_baseline": cpu, "bf16": bf16,
        "kernels": {x: {kk: round(vv, 3) for kk, vv in v.items()} for x, v in sorted(kernels.items())},
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_bmm(np, synth, target_s: float):
    """The oracle, as it stands, on the first nb batches of the attention BMM (fwd + bwd)."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1

    def run(nb):
        Qh, Kh, Gh = (np.stack(a) for a in zip(*[bmm_inputs(np, synth, b) for b in range(nb)]))
        t0 = time.perf_counter()
        sq = np.array([O.absmax(O.fwht_rows(Qh[b], BMM_K)) / np.float32(14.0) for b in range(nb)])
        sk = np.array([O.absmax(O.fwht_rows(Kh[b], BMM_K)) / np.float32(14.0) for b in range(nb)])
        fw = O.bmm_lsq_forward(Qh, Kh, BMM_K, sq, sk)
        O.bmm_lsq_backward(Gh, fw, BMM_N, 0, 0)
        return time.perf_counter() - t0, 6.0 * nb * BMM_N * BMM_P * BMM_M

    nb = 2
    t, ops = run(nb)
    for _ in range(3):
        if t >= 0.7 * target_s or nb >= BMM_B:
            break
        nb = int(min(BMM_B, max(nb + 1, nb * target_s / max(t, 1e-3))))
        t, ops = run(nb)
    return {"value": round(ops / t / 1e12, 6), "unit": "TOPS", "cores": int(threads), "kind": "oracle",
            "sample": f"first {nb} of {BMM_B} batches, fwd + bwd (budget = {BMM_N}); {t:.1f} s",
            "seconds": round(t, 2)}


def _host_info():
    """CPU model and the cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        nproc = os.cpu_count() or 1
    return model, nproc


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        return 1


def cpu_baseline(lins, cfg_id: int, target_s: float, lsq_mode: bool = False):
    """The oracle, as it stands, on the first n tokens of the workload's linears: the
    forward, the dX backward and the dW backward each timed three times (median), linear
    after linear until about target_s of CPU work is spent (at least one linear)."""
    import numpy as np

    import oracle as O
    import synth

    def ops_of(n, lin):
        if lsq_mode:
            k = lin.log2_block
            sub = synth.Linear(lin.name, n, lin.D, lin.C, k, lin.dtype, lin.x_outlier_channels,
                               lin.x_outlier_scale, lin.grad_kind, n)
            X, W, G = synth.linear_inputs(sub, cfg_id, lins.index(lin))
            sx = O.absmax(O.fwht_rows(X, k)) / np.float32(14.0)
            sw = O.absmax(O.fwht_rows(W, k)) / np.float32(14.0)
            fw = lambda: O.lsq_forward(X, W, k, sx, sw)
            f = fw()
            dx = lambda: O.lsq_backward(G, f, n, 0, 0, need_dw=False)
            dw = lambda: O.lsq_backward(G, f, n, 0, 0, need_dx=False)
        else:
            sub = synth.Linear(lin.name, n, lin.D, lin.C, lin.log2_block, lin.dtype,
                               lin.x_outlier_channels, lin.x_outlier_scale, lin.grad_kind, n)
            X, W, G = synth.linear_inputs(sub, cfg_id, lins.index(lin))
            fw = lambda: O.hq_forward(X, W, lin.log2_block)
            f = fw()
            dx = lambda: O.lss_backward(G, f, n, 0, 0, need_dw=False)
            dw = lambda: O.lss_backward(G, f, n, 0, 0, need_dx=False)
        return fw, dx, dw

    def med3(fn):
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return _median(ts), sum(ts)

    def run(n):
        spent = 0.0
        per_op = {"fwd": 0.0, "dx": 0.0, "dw": 0.0}
        ops = 0.0
        used = []
        for lin in lins:
            if used and spent >= target_s:
                break
            for name, fn in zip(("fwd", "dx", "dw"), ops_of(n, lin)):
                m, t = med3(fn)
                per_op[name] += m
                spent += t
            ops += 6.0 * n * lin.C * lin.D
            used.append(f"{lin.D}x{lin.C}")
        return per_op, ops, used, spent

    n = min(256, lins[0].N)
    per_op, ops, used, spent = run(n)
    for _ in range(3):  # a larger token slice while the sample is well under target_s
        if spent >= 0.3 * target_s or n >= lins[0].N:
            break
        n = int(min(lins[0].N, max(2 * n, n * 0.7 * target_s / max(spent, 1e-3))) // 64 * 64)
        per_op, ops, used, spent = run(n)
    total = sum(per_op.values())
    model, nproc = _host_info()
    return {"value": round(ops / total / 1e12, 6), "unit": "TOPS", "cores": int(_blas_threads()),
            "kind": "oracle",
            "sample": f"first {n} of {lins[0].N} tokens of the linears {', '.join(used)} (of "
                      f"{len(lins)}), fwd, dX and dW each the median of 3 runs (budget = {n}"
                      f"{', learned step sizes' if lsq_mode else ''}); {spent:.1f} s of CPU work",
            "median_s_per_op": {k: round(v, 3) for k, v in per_op.items()},
            "cpu_model": model, "nproc": nproc,
            "threads_note": "cores = BLAS threads of the integer products; the oracle's "
                            "element-wise numpy steps run on one thread",
            "seconds": round(spent, 2)}


if __name__ == "__main__":
    main()
