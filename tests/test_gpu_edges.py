"""Edge cases of the C-ABI path on the GPU against the fp64 oracle: extreme
aspect ratios, very long contractions (deep split-K), pitched outputs, large
batch grids, and the documented limits."""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, sample_positions, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"


def linear_all(inp, ypitch=None, xpitch_extra=0):
    x, w, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    M, K = x.shape
    N = w.shape[0]
    if ypitch:
        ybuf = torch.full((M, ypitch), float("nan"), device=DEV)
        y = ybuf[:, :N]
    else:
        y = torch.full((M, N), float("nan"), device=DEV)
    dx = torch.full((M, K), float("nan"), device=DEV)
    dw = torch.full((N, K), float("nan"), device=DEV)
    db = torch.full((N,), float("nan"), device=DEV)
    b.linear_fwd(x, w, bias, y)
    n = b.linear_bwd_workspace(x, w, dy, dx, dw, db)
    ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.linear_bwd(x, w, dy, dx, dw, db, workspace=ws)
    torch.cuda.synchronize()
    if ypitch:
        assert torch.isnan(ybuf[:, N:]).all(), "wrote outside the pitched output"
    return {"Y": y, "dX": dx, "dW": dw, "db": db}


def check_all(inp, out):
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    assert_close(to_f64(out["Y"]), *oracle.linear_fwd(X, W, B), what="Y")
    assert_close(to_f64(out["dX"]), *oracle.linear_bwd_dx(dY, W), what="dX")
    assert_close(to_f64(out["dW"]), *oracle.linear_bwd_dw(dY, X), what="dW")
    assert_close(to_f64(out["db"]), *oracle.linear_bwd_db(dY), what="db")


@pytest.mark.parametrize("M,N,K", [(1, 300, 257), (300, 1, 257), (1, 1, 4096), (2, 3, 100000),
                                   (64, 64, 1 << 20)])
def test_extreme_aspect_ratios_and_long_k(M, N, K):
    inp = wl.linear(M, N, K, seed=M + N).make()
    check_all(inp, linear_all(inp))


def test_long_k_deep_split_is_deterministic():
    inp = wl.linear(64, 64, 1 << 18, seed=3).make()
    a = linear_all(inp)
    c = linear_all(inp)
    for k in a:
        assert torch.equal(a[k], c[k]), k


def test_pitched_output_rows():
    inp = wl.linear(200, 120, 64, seed=4).make()
    out = linear_all(inp, ypitch=133)
    check_all(inp, out)


def test_many_batches_large_grid():
    # 4096 batch elements, one 64x64 output tile each: a grid of 4096 blocks
    A = wl.tensor((4096, 1, 40, 24), ("uniform", 1.0), seed=5)
    B = wl.tensor((1, 1, 24, 36), ("uniform", 1.0), seed=6)
    C = torch.empty(4096, 1, 40, 36, device=DEV)
    b.matmul(A.to(DEV), B.to(DEV), C)
    torch.cuda.synchronize()
    Cr, S = oracle.matmul(A.double().numpy(), B.double().numpy())
    assert_close(to_f64(C), Cr, S, what="C")
    # and the gradient of the broadcast B: a sum over 4096 batch elements
    G = wl.tensor((4096, 1, 40, 36), ("normal",), seed=7)
    dB = torch.empty(1, 1, 24, 36, device=DEV)
    n = b.matmul_workspace(A.to(DEV).transpose(-1, -2), G.to(DEV), dB, reduce_into=True)
    ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.matmul(A.to(DEV).transpose(-1, -2), G.to(DEV), dB, reduce_into=True, workspace=ws)
    torch.cuda.synchronize()
    _, _, dBr, SB = oracle.matmul_bwd(A.double().numpy(), B.double().numpy(), G.double().numpy(),
                                      need_a=False)
    assert_close(to_f64(dB), dBr, SB, what="dB (summed over 4096 batches)")


def test_long_row_pitch_few_rows():
    """Rows 2**21 floats apart (8 MiB): accepted while a tile's rows times the
    pitch stay within the kernels' 32-bit offsets; only in-range rows are read."""
    big = torch.empty(2, 1 << 21, device=DEV)
    x = big[:, :8]
    x.copy_(wl.tensor((2, 8), ("uniform", 1.0), seed=8).to(DEV))
    w = wl.tensor((300, 8), ("uniform", 1.0), seed=9).to(DEV)
    y = torch.full((2, 300), 7.0, device=DEV)
    b.linear_fwd(x, w, None, y)
    torch.cuda.synchronize()
    Yr, S = oracle.linear_fwd(to_f64(x), to_f64(w), None)
    assert_close(to_f64(y), Yr, S, what="Y (long pitch, few rows)")


@pytest.mark.parametrize("krot", [0, 1])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dma_tile_k_rotation_settings(krot, dtype):
    """4096^2 outputs (the 256x256 DMA tile) with K = 1000 (a K tail): every
    block starting at k = 0, and blocks starting at an XCD-dependent stage
    and wrapping around; sampled against the oracle, reruns bit-identical."""
    M = N = 4096
    K = 1000
    inp = wl.linear(M, N, K, dtype=dtype, seed=krot, dist={"X": ("normal",), "W": ("uniform", 1 / 32),
                                                           "dY": ("normal",)}).make()
    x, w, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    b.debug_set("krot", krot)
    try:
        outs = []
        for _ in range(2):
            y = torch.full((M, N), float("nan"), device=DEV)
            dw = torch.full((N, K), float("nan"), device=DEV)
            b.linear_fwd(x, w, bias, y)
            b.linear_bwd(x, w, dy, None, dw, None)
            torch.cuda.synchronize()
            outs.append((y, dw))
    finally:
        b.debug_set("krot", 1)
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    r, c = sample_positions(M, N, 2000, seed=krot)
    want, S = oracle.linear_fwd_at(X, W, B, r, c)
    assert_close(to_f64(outs[0][0])[r, c], want, S, what="Y")
    r, c = sample_positions(N, K, 2000, seed=krot + 7)
    want, S = oracle.linear_bwd_dw_at(dY, X, r, c)
    assert_close(to_f64(outs[0][1])[r, c], want, S, what="dW")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_few_tiles_long_contraction_dma_split(dtype):
    """dW of a 65536-row layer with 512 x 512 weights: four 256x256 output
    tiles over 65536 summed rows run on the DMA tile split into 64 runs (one
    wave of 256 blocks) with a fixed-order second pass. Sampled against the
    oracle; reruns bit-identical; the same without workspace (unsplit)."""
    M, N, K = 65536, 512, 512
    inp = wl.linear(M, N, K, dtype=dtype, seed=4, dist={"X": ("normal",), "dY": ("normal",)}).make()
    x, w, dy = (inp[k].to(DEV) for k in ("X", "W", "dY"))
    outs = []
    for use_ws in (True, True, False):
        dw = torch.full((N, K), float("nan"), device=DEV)
        ws = None
        if use_ws:
            n = b.linear_bwd_workspace(x, w, dy, None, dw, None)
            # fp32: 2048 K-stages of 32 -> 64 runs of 32 on the DMA tile; bf16
            # (stages of 64) stays below the run length and splits on 128x128
            assert n >= (64 if dtype == "f32" else 2) * N * K * 4, n
            ws = torch.empty(n // 4 + 64, device=DEV)
        b.linear_bwd(x, w, dy, None, dw, None, workspace=ws)
        torch.cuda.synchronize()
        outs.append(dw)
    assert torch.equal(outs[0], outs[1])
    X, dY = to_f64(inp["X"]), to_f64(inp["dY"])
    r, c = sample_positions(N, K, 1500, seed=3)
    want, S = oracle.linear_bwd_dw_at(dY, X, r, c)
    for o, what in ((outs[0], "split"), (outs[2], "unsplit")):
        assert_close(to_f64(o)[r, c], want, S, what=f"dW ({what})")
