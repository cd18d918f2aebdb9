#!/usr/bin/env python3
"""Throughput of the dense-layer training step on one MI355X.

One step = the whole hot path on one batch of synthetic inputs already in
HBM: Y = X W^T + b (mt_linear_fwd), then dX = dY W, dW = dY^T X and
db = 1^T dY (one mt_linear_bwd call). Events at every step boundary time
each step; `value` comes from the median step (the mean is reported
beside it). A second pass issues the same kernels with the backward split
into one call per output, so that HIP events bracket each kernel for the
roofline of the dominant one.

Prints ONE JSON line: TFLOP/s of the three products (6 M N K flop per step)
at the median step time, the dominant kernel's roofline, and the fp64 CPU
oracle timed on full row bands of the step as a baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak (256 CU x 256 flop/clk x 2.4 GHz)
BF16_MFMA_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 matrix peak
HBM_PEAK_GBS = 8000.0
METRIC = "TFLOP/s for linear fwd+bwd (3 GEMMs) at M=N=K=8192 fp32; % MFMA peak"

# sources whose text decides each measured kernel (counters taken on other
# sources are stale and not reported)
KERNEL_SOURCES = {
    "gemm": ["paper_2602_00125_amd/csrc/gemm_kernel.hpp", "paper_2602_00125_amd/csrc/gemm_dma.hpp",
             "paper_2602_00125_amd/csrc/gemm_dma_body.inc", "paper_2602_00125_amd/csrc/gemm_f32.hip",
             "paper_2602_00125_amd/csrc/gemm_params.hpp", "paper_2602_00125_amd/csrc/capi.cpp",
             "paper_2602_00125_amd/csrc/host.hpp"],
    "gemm_bf16": ["paper_2602_00125_amd/csrc/gemm_kernel.hpp", "paper_2602_00125_amd/csrc/gemm_dma.hpp",
                  "paper_2602_00125_amd/csrc/gemm_dma_body.inc", "paper_2602_00125_amd/csrc/gemm_bf16.hip",
                  "paper_2602_00125_amd/csrc/gemm_params.hpp", "paper_2602_00125_amd/csrc/capi.cpp",
                  "paper_2602_00125_amd/csrc/host.hpp"],
    "colsum": ["paper_2602_00125_amd/csrc/reduce.hip", "paper_2602_00125_amd/csrc/capi.cpp"],
}


def sources_hash(family: str) -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[family]:
        p = os.path.join(ROOT, rel)
        if os.path.exists(p):
            h.update(rel.encode())
            h.update(open(p, "rb").read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=-1,
                    help="untimed warm-up steps (default: as many as take about three seconds, at "
                         "least 5, so that the GPU clock has ramped up before timing starts)")
    ap.add_argument("--workload", default="linear_8192x8192x8192_f32")
    ap.add_argument("--graph", action="store_true",
                    help="linear workloads: replay the step from a captured HIP graph (one launch "
                         "per step instead of one per kernel; for launch-bound sizes)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target wall time of the CPU-oracle baseline sample (0 disables it)")
    ap.add_argument("--torch-reference", action="store_true",
                    help="linear workloads: also time torch's own products on the same device inputs "
                         "(context only; never part of value)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (calibrates HBM "
                         "byte counters against a kernel of known traffic) and exit")
    return ap.parse_args()


def copy_probe(mib: int) -> None:
    import torch

    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4}))


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, seconds: float):
    """Time the fp64 oracle on full row bands of the step: for each band of R
    rows, Y and dX for R rows of X / dY and dW for R rows of dW (R columns of
    dY), each through the oracle's row-major whole-matrix functions at full
    contraction length; bands are taken until about `seconds` have passed."""
    import numpy as np
    import torch

    import oracle

    def f64(t):
        if t.dtype == torch.bfloat16:
            return oracle.bf16_bits_to_f64(t.view(torch.int16).numpy())
        return t.double().numpy()

    X, W, dY = f64(inp["X"]), f64(inp["W"]), f64(inp["dY"])
    B = inp["b"].double().numpy()
    M, K = X.shape
    N = W.shape[0]
    R = 32
    macs = bands = 0
    t0 = time.perf_counter()
    while True:
        r0 = (bands * R) % max(M - R + 1, 1)
        n0 = (bands * R) % max(N - R + 1, 1)
        xb, gb = X[r0:r0 + R], dY[r0:r0 + R]
        oracle.linear_fwd(xb, W, B)
        oracle.linear_bwd_dx(gb, W)
        oracle.linear_bwd_dw(np.ascontiguousarray(dY[:, n0:n0 + R]), X)
        macs += len(xb) * N * K + len(gb) * N * K + R * M * K
        bands += 1
        if time.perf_counter() - t0 >= seconds:
            break
    el = time.perf_counter() - t0
    flops = 2.0 * macs / el
    return {"value": flops / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "gflops": round(flops / 1e9, 3), "cpu_model": cpu_model(),
            "sample": f"row band: {bands} bands of {R} rows, each {R} full rows of Y = X W^T + b "
                      f"and of dX = dY W and {R} full rows of dW = dY^T X (the oracle's row-major "
                      f"fp64 functions with the |a*b| bound, full contraction length) in {el:.1f} s; "
                      f"TFLOP/s = 2*MACs/s"}


def torch_reference(x, w, b, dy, steps: int):
    """torch's own products of the same layer on the same device inputs (the
    library it calls, for context): Y = X W^T + b, dX = dY W, dW = dY^T X,
    db = 1^T dY, each timed with events after a second of warm-up. bf16
    products return bf16 there (fp32 here)."""
    import torch

    ops = {"fwd": lambda: torch.addmm(b.to(x.dtype), x, w.t()),
           "dx": lambda: dy @ w,
           "dw": lambda: dy.t() @ x,
           "db": lambda: dy.sum(0, dtype=torch.float32)}
    M, K = x.shape
    N = w.shape[0]
    out = {}
    for name, fn in ops.items():
        t = time.perf_counter()
        while time.perf_counter() - t < 1.0:
            fn()
            torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        out[name] = {"ms": round(ms, 4)}
        if name != "db":
            out[name]["tflops"] = round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 1)
    return out


WARMUP_USED = [None]  # warm-up steps of the run's timed pass (reported as "warmup")


def timed_steps(step, n_events: int, steps: int, warmup: int):
    """Warm up, then time `steps` steps, bracketed by synchronisations, with an
    event at every step boundary (and events between a step's calls when
    n_events > 1). Returns (median ms per step, mean ms between each step's
    events, mean ms per step). warmup < 0: steps, each waited for, until
    about three seconds have passed (at least 5): the clock settles, and the
    run holds the GPU busy long enough for an outside sampler to see it."""
    import statistics

    import torch

    if warmup < 0:
        t = time.perf_counter()
        warmup = 0
        while warmup < 5 or (time.perf_counter() - t < 3.0 and warmup < 100000):
            step()
            torch.cuda.synchronize()
            warmup += 1
    else:
        for _ in range(warmup):
            step()
    if WARMUP_USED[0] is None:  # the first call is the timed pass of the run
        WARMUP_USED[0] = warmup
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(n_events)] for _ in range(steps)]
    if n_events < 2:
        events = [None] * steps
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    for i in range(steps):
        bounds[i].record()
        step(events[i])
    bounds[steps].record()
    torch.cuda.synchronize()
    per_step = [bounds[i].elapsed_time(bounds[i + 1]) for i in range(steps)]
    per = [0.0] * max(n_events - 1, 0)
    for ev in events:
        for j in range(n_events - 1):
            per[j] += ev[j].elapsed_time(ev[j + 1])
    mean = bounds[0].elapsed_time(bounds[steps]) / steps
    return statistics.median(per_step), [v / steps for v in per], mean


def bench_bmm(args, w, inp, dev):
    """Broadcasting batched matmul step: C = A @ B, then dA and dB with the
    broadcast-axis sums folded into the products (MT_REDUCE_INTO)."""
    import torch

    from paper_2602_00125_amd import binding as mt

    A, B, dC = (inp[k].to(dev) for k in ("A", "B", "dC"))
    C = torch.empty(w.cshape, device=dev)
    dA = torch.empty(w.ashape, device=dev)
    dB = torch.empty(w.bshape, device=dev)
    Bt, At = B.transpose(-1, -2), A.transpose(-1, -2)
    need = max(mt.matmul_workspace(A, B, C), mt.matmul_workspace(dC, Bt, dA, reduce_into=True),
               mt.matmul_workspace(At, dC, dB, reduce_into=True))
    ws = torch.empty(need // 4 + 64, device=dev) if need else None

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        mt.matmul(A, B, C, workspace=ws)
        if ev is not None:
            ev[1].record()
        mt.matmul(dC, Bt, dA, reduce_into=True, workspace=ws)
        if ev is not None:
            ev[2].record()
        mt.matmul(At, dC, dB, reduce_into=True, workspace=ws)
        if ev is not None:
            ev[3].record()

    # the step's time from events at step boundaries only (an event between
    # two calls holds the queue for a few microseconds), then a second pass
    # with events between the calls for the per-product breakdown
    ms, _, ms_mean = timed_steps(step, 1, args.steps, args.warmup)
    _, per, _ = timed_steps(step, 4, args.steps, 1)
    names = ["fwd_gemm", "dA_gemm_reduce_into", "dB_gemm_reduce_into"]
    per = dict(zip(names, per))
    value = w.flops() / (ms * 1e-3) / 1e12
    dominant = max(names, key=lambda k: per[k])
    achieved = (w.flops() / 3) / (per[dominant] * 1e-3) / 1e12
    out = {"metric": f"TFLOP/s for broadcast matmul fwd+bwd (3 products) on {args.workload}",
           "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": WARMUP_USED[0], "ms_per_step": round(ms, 4), "ms_per_step_mean": round(ms_mean, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": args.workload, "a": list(w.ashape), "b": list(w.bshape),
                      "pct_of_mfma_peak": round(100.0 * value / FP32_MFMA_PEAK_TFLOPS, 2)},
           "roofline": {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 3),
                        "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None},
           "kernels_ms": {k: round(v, 4) for k, v in per.items()}, "cpu_baseline": None}
    print(json.dumps(out), flush=True)


def cpu_baseline_mlp(inp, seconds: float):
    """Time the fp64 oracle on sampled rows of the perceptron's forward pass:
    each sampled row goes through both dense layers, the nonlinearity and the
    loss gradient, as the oracle computes them."""
    import numpy as np

    import oracle
    from oracle import nn as onn

    X, W1, b1, W2, b2, T = (inp[k].double().numpy() for k in ("X", "W1", "b1", "W2", "b2", "T"))
    M = X.shape[0]
    rng = np.random.default_rng(0)
    macs = rows = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        idx = rng.integers(0, M, 16)   # 16 rows: the oracle runs one thread per row
        Z, H, _ = onn.linear_act_fwd(X[idx], W1, b1, onn.GELU)
        P, _ = oracle.linear_fwd(H, W2, b2)
        onn.mse_loss(P, T[idx])
        macs += len(idx) * (W1.size + W2.size)
        rows += len(idx)
    el = time.perf_counter() - t0
    return {"value": 2.0 * macs / el / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{rows} random rows of X through both dense layers, GELU and the MSE "
                      f"gradient in fp64 (with the |a*b| bound) in {el:.1f} s; TFLOP/s = 2*MACs/s"}


def bench_mlp(args, w, inp, dev):
    """Two-layer perceptron training step: forward with the fused GELU
    epilogue, MSE, backward (dH1, dW2, db2, the GELU pullback with db1 folded
    in, dW1), and one Adam update of all four parameters."""
    import torch

    from paper_2602_00125_amd import binding as mt

    x, W1, b1, W2, b2, t = (inp[k].to(dev) for k in ("X", "W1", "b1", "W2", "b2", "T"))
    M, D1, D2 = w.M, w.D1, w.D2
    z1 = torch.empty(M, D1, device=dev)
    h1 = torch.empty(M, D1, device=dev)
    pr = torch.empty(M, D2, device=dev)
    loss = torch.empty(1, device=dev)
    dp = torch.empty(M, D2, device=dev)
    dh1 = torch.empty(M, D1, device=dev)
    dz1 = torch.empty(M, D1, device=dev)
    params = [W1, b1, W2, b2]
    grads = [torch.empty_like(p) for p in params]
    ms = [torch.zeros_like(p) for p in params]
    vs = [torch.zeros_like(p) for p in params]
    need = max(mt.linear_bwd_workspace(h1, W2, dp, dh1, grads[2], grads[3]),
               mt.act_bwd_workspace(w.act, z1, dh1, dz1, grads[1]),
               mt.linear_bwd_workspace(x, W1, dz1, None, grads[0], None),
               mt.mse_loss_workspace(pr, t))
    ws = torch.empty(need // 4 + 64, device=dev) if need else None
    counter = [0]

    def step(ev=None):
        counter[0] += 1
        marks = iter(ev) if ev is not None else None

        def mark():
            if marks is not None:
                next(marks).record()
        mark()
        mt.linear_act_fwd(x, W1, b1, w.act, h1, z=z1)
        mark()
        mt.linear_fwd(h1, W2, b2, pr)
        mark()
        mt.mse_loss(pr, t, loss, dp, workspace=ws)
        mark()
        if ev is None:
            mt.linear_bwd(h1, W2, dp, dh1, grads[2], grads[3], workspace=ws)
        else:
            mt.linear_bwd(h1, W2, dp, dh1, None, None, workspace=ws)
            mark()
            # db2 is summed inside the dW2 product
            mt.linear_bwd(h1, W2, dp, None, grads[2], grads[3], workspace=ws)
        mark()
        mt.act_bwd(w.act, z1, dh1, dz1, grads[1], workspace=ws)
        mark()
        mt.linear_bwd(x, W1, dz1, None, grads[0], None, workspace=ws)
        mark()
        mt.adam_step(params, grads, ms, vs, 1e-4, 0.9, 0.999, 1e-8, counter[0])
        mark()

    names = ["fwd1_nt_gemm_gelu", "fwd2_nt_gemm", "mse", "dh1_nn_gemm", "dw2_tn_gemm_db2",
             "act_bwd_db1", "dw1_tn_gemm", "adam"]
    ms_step, _, ms_mean = timed_steps(step, 1, args.steps, args.warmup)
    _, per, _ = timed_steps(step, len(names) + 1, args.steps, 1)
    per = dict(zip(names, per))
    value = w.flops() / (ms_step * 1e-3) / 1e12
    gemm_flops = {"fwd1_nt_gemm_gelu": 2.0 * M * w.D0 * D1, "fwd2_nt_gemm": 2.0 * M * D1 * D2,
                  "dh1_nn_gemm": 2.0 * M * D2 * D1, "dw2_tn_gemm_db2": 2.0 * M * D2 * D1,
                  "dw1_tn_gemm": 2.0 * M * D1 * w.D0}
    dominant = max(gemm_flops, key=lambda k: per[k])
    achieved = gemm_flops[dominant] / (per[dominant] * 1e-3) / 1e12
    nparam = sum(p.numel() for p in params)
    hbm_bytes = {"act_bwd_db1": 12.0 * M * D1 + 4 * D1, "mse": 12.0 * M * D2 + 4,
                 "adam": 28.0 * nparam}
    hbm = {k: {"ms": round(per[k], 4), "gbs": round(v / (per[k] * 1e-3) / 1e9, 1),
               "frac": round(v / (per[k] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4), "bytes": int(v)}
           for k, v in hbm_bytes.items()}
    out = {"metric": f"TFLOP/s for a two-layer perceptron training step (5 GEMMs + GELU, MSE, "
                     f"Adam) on {args.workload}",
           "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": WARMUP_USED[0], "ms_per_step": round(ms_step, 4), "ms_per_step_mean": round(ms_mean, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": args.workload, "M": M, "D0": w.D0, "D1": D1, "D2": D2,
                      "act": w.act, "optimizer": "adam",
                      "pct_of_mfma_peak": round(100.0 * value / FP32_MFMA_PEAK_TFLOPS, 2)},
           "roofline": {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 3),
                        "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": round(achieved / FP32_MFMA_PEAK_TFLOPS, 4), "traffic": None},
           "kernels_ms": {k: round(v, 4) for k, v in per.items()},
           "hbm_kernels": hbm,
           "loss_after_timed_steps": round(float(loss.item()), 6)}
    out["cpu_baseline"] = cpu_baseline_mlp(inp, args.cpu_seconds) if args.cpu_seconds > 0 else None
    print(json.dumps(out), flush=True)


def cpu_baseline_conv(w, inp, seconds: float):
    """Time the fp64 oracle on sampled output elements of the convolution's
    forward, dX and dW (each a full-length sum with the |a*b| bound)."""
    import numpy as np

    import oracle

    X, W, B, dY = (inp[k].double().numpy() for k in ("x", "w", "b", "dy"))
    st, pd = w.stride, w.pad
    rng = np.random.default_rng(0)
    macs = done = 0
    kc = w.C * w.KH * w.KW
    HO, WO = w.out_hw()
    chunk = 64
    t0 = time.perf_counter()
    while True:
        oracle.conv2d_fwd_at(X, W, B, rng.integers(0, dY.size, chunk), st, pd)
        oracle.conv2d_bwd_dx_at(dY, W, X.shape, rng.integers(0, X.size, chunk), st, pd)
        oracle.conv2d_bwd_dw_at(dY, X, W.shape, rng.integers(0, W.size, max(1, chunk // 64)), st, pd)
        macs += chunk * kc + chunk * w.CO * w.KH * w.KW + max(1, chunk // 64) * w.N * HO * WO
        done += chunk
        el = time.perf_counter() - t0
        if el >= seconds:
            break
        if el < seconds / 8:
            chunk *= 2
    el = time.perf_counter() - t0
    return {"value": 2.0 * macs / el / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{done} random elements of y and of dx and {max(1, done // 64)} of dw (full "
                      f"fp64 sums with the |a*b| bound) in {el:.1f} s; TFLOP/s = 2*MACs/s"}


def bench_conv(args, w, inp, dev):
    """Convolution step: forward (the product gathering the image in its
    loads, bias epilogue), then the backward call producing dx, dw and db
    (dW product gathering the image, column sum, dU product, fold). With
    layouts that cannot gather, the forward unfolds the input into the
    workspace and the backward's dW reuses it."""
    import torch

    from paper_2602_00125_amd import binding as mt

    cl = torch.channels_last
    x = inp["x"].to(dev).contiguous(memory_format=cl)
    wt = inp["w"].to(dev).contiguous(memory_format=cl)
    bias = inp["b"].to(dev)
    dy = inp["dy"].to(dev).contiguous(memory_format=cl)
    HO, WO = w.out_hw()
    y = torch.empty(w.N, w.CO, HO, WO, device=dev).contiguous(memory_format=cl)
    dx = torch.empty(w.N, w.C, w.H, w.W, device=dev).contiguous(memory_format=cl)
    dw = torch.empty_like(wt)
    db = torch.empty(w.CO, device=dev)
    st, pd = w.stride, w.pad
    need = max(mt.conv2d_fwd_workspace(x, wt, bias, y, st, pd),
               mt.conv2d_bwd_workspace(x, wt, dy, dx, dw, db, st, pd))
    ws = torch.empty(need // 4 + 64, device=dev)

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        mt.conv2d_fwd(x, wt, bias, y, st, pd, workspace=ws)
        if ev is not None:
            ev[1].record()
        # where the forward unfolded its input, the backward reuses it
        mt.conv2d_bwd(x, wt, dy, dx, dw, db, st, pd, workspace=ws, reuse_unfold=True)
        if ev is not None:
            ev[2].record()

    ms, _, ms_mean = timed_steps(step, 1, args.steps, args.warmup)
    _, per, _ = timed_steps(step, 3, args.steps, 1)
    per = dict(zip(["conv2d_fwd", "conv2d_bwd"], per))
    value = w.flops() / (ms * 1e-3) / 1e12
    out = {"metric": f"TFLOP/s for a 2-D convolution fwd+bwd (3 products) on {args.workload}",
           "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": WARMUP_USED[0], "ms_per_step": round(ms, 4), "ms_per_step_mean": round(ms_mean, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": args.workload, "x": [w.N, w.C, w.H, w.W],
                      "w": [w.CO, w.C, w.KH, w.KW], "stride": list(st), "pad": list(pd),
                      "layout": "channels-last",
                      "pct_of_mfma_peak": round(100.0 * value / FP32_MFMA_PEAK_TFLOPS, 2)},
           "roofline": {"bound": "mfma", "kernel": "whole step (per-kernel: rocprofv3 summary)",
                        "achieved": round(value, 3), "peak": FP32_MFMA_PEAK_TFLOPS,
                        "unit": "TFLOP/s", "frac": round(value / FP32_MFMA_PEAK_TFLOPS, 4),
                        "traffic": None},
           "calls_ms": {k: round(v, 4) for k, v in per.items()}}
    out["cpu_baseline"] = cpu_baseline_conv(w, inp, args.cpu_seconds) if args.cpu_seconds > 0 else None
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); this build has no "
              f"multi-GPU path", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2602_00125_amd import binding as mt
    from paper_2602_00125_amd import workloads as wl

    w = wl.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    inp = w.make()
    if isinstance(w, wl.BmmWorkload):
        return bench_bmm(args, w, inp, dev)
    if isinstance(w, wl.MlpWorkload):
        return bench_mlp(args, w, inp, dev)
    if isinstance(w, wl.ConvWorkload):
        return bench_conv(args, w, inp, dev)
    x, wt, bias, dy = (inp[k].to(dev) for k in ("X", "W", "b", "dY"))
    M, N, K = w.M, w.N, w.K
    y = torch.empty(M, N, device=dev)
    dx = torch.empty(M, K, device=dev)
    dw = torch.empty(N, K, device=dev)
    db = torch.empty(N, device=dev)
    ws_bytes = mt.linear_bwd_workspace(x, wt, dy, dx, dw, db)
    ws = torch.empty(max(ws_bytes, 256) // 4 + 64, device=dev) if ws_bytes else None

    def step(ev=None):
        # the path as a caller runs it: one forward call, one backward call
        mt.linear_fwd(x, wt, bias, y)
        mt.linear_bwd(x, wt, dy, dx, dw, db, workspace=ws)

    def step_per_kernel(ev=None):
        # the same kernels, the backward issued as two calls so that events
        # bracket each product (db is summed inside the dW product)
        if ev is not None:
            ev[0].record()
        mt.linear_fwd(x, wt, bias, y)
        if ev is not None:
            ev[1].record()
        mt.linear_bwd(x, wt, dy, dx, None, None, workspace=ws)
        if ev is not None:
            ev[2].record()
        mt.linear_bwd(x, wt, dy, None, dw, db, workspace=ws)
        if ev is not None:
            ev[3].record()

    # the stand-alone column sum (db without dw), for its HBM rate
    ws_db_bytes = mt.linear_bwd_workspace(x, wt, dy, None, None, db)
    ws_db = torch.empty(ws_db_bytes // 4 + 64, device=dev) if ws_db_bytes else None

    def colsum_alone(ev=None):
        if ev is not None:
            ev[0].record()
        mt.linear_bwd(x, wt, dy, None, None, db, workspace=ws_db)
        if ev is not None:
            ev[1].record()

    run = step
    if args.graph:
        # capture one step (its kernels, on the capture stream) and replay it
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()

        def run(ev=None):
            graph.replay()
    ms_per_step, _, ms_mean = timed_steps(run, 1, args.steps, args.warmup)
    _, per_list, _ = timed_steps(step_per_kernel, 4, args.steps, 1)
    per = dict(zip(["fwd_nt_gemm", "dx_nn_gemm", "dw_tn_gemm_db"], per_list))
    _, cs_list, _ = timed_steps(colsum_alone, 2, args.steps, 1)
    flops = w.flops()
    value = flops / (ms_per_step * 1e-3) / 1e12
    gemm_flops = 2.0 * M * N * K
    is_bf16 = w.dtype == "bf16"
    peak = BF16_MFMA_PEAK_TFLOPS if is_bf16 else FP32_MFMA_PEAK_TFLOPS
    dominant = max(("fwd_nt_gemm", "dx_nn_gemm", "dw_tn_gemm_db"), key=lambda k: per[k])
    achieved = gemm_flops / (per[dominant] * 1e-3) / 1e12
    # HBM traffic of the dominant kernel from committed rocprofv3 counters, if
    # they were taken on the current kernel sources
    traffic = None
    tfile = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tfile):
        try:
            rec = json.load(open(tfile)).get(args.workload, {}).get(dominant)
            fam = "gemm_bf16" if is_bf16 else "gemm"
            if rec and rec.get("sources_hash") == sources_hash(fam):
                traffic = rec["hbm_bytes_per_launch"]
        except (ValueError, OSError):
            traffic = None
    db_bytes = M * N * (2 if is_bf16 else 4) + N * 4
    out = {
        "metric": METRIC if args.workload == "linear_8192x8192x8192_f32" else
        f"TFLOP/s for linear fwd+bwd (3 GEMMs) on {args.workload}",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": WARMUP_USED[0],
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_mean": round(ms_mean, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if is_bf16 else "f32",
        "data": "synthetic",
        "config": {"workload": args.workload, "M": M, "N": N, "K": K,
                   "inputs": "seeded synthetic, resident in HBM before timing",
                   "hip_graph": bool(args.graph),
                   "pct_of_mfma_peak": round(100.0 * value / peak, 2)},
        "roofline": {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 3),
                     "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": traffic},
        "kernels_ms": {k: round(v, 4) for k, v in per.items()},
        "colsum_alone": {"ms": round(cs_list[0], 4),
                         "gbs": round(db_bytes / (cs_list[0] * 1e-3) / 1e9, 1), "bytes": db_bytes},
    }
    if args.torch_reference:
        out["torch_reference"] = torch_reference(x, wt, bias, dy, args.steps)
    if args.cpu_seconds > 0:
        out["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
