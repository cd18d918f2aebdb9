"""GPU parity of the 2-D convolution (Sec. 3.3 Eq. (6)) and its pullbacks
against the fp64 oracle, through the C-ABI library: the unfolded input times
the flattened weights on the matrix cores (forward, dW, dU), the unfold and
the gather fold on the HBM side.

Bar: the dense-layer bar |gpu - oracle| <= 1e-4 S + 1e-6 with S the sum of
|terms| the oracle returns for each element (every output is a sum of
products of inputs, as in the dense layer; the fold adds up to KH KW
dot-product results, each within that bar, whose S add up).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"
CL = torch.channels_last

# (N, C, H, W, CO, KH, KW, stride, pad, weight layout, input layout)
CASES = [
    (2, 3, 7, 6, 4, 3, 3, (1, 1), (1, 1), "std", "nchw"),
    (2, 8, 9, 9, 12, 3, 3, (2, 2), (1, 1), "cl", "cl"),
    (1, 16, 16, 16, 32, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (2, 4, 8, 5, 8, 1, 1, (1, 1), (0, 0), "std", "cl"),
    (1, 3, 10, 7, 5, 5, 3, (2, 1), (2, 0), "std", "nchw"),
    (4, 32, 14, 14, 64, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (2, 64, 28, 28, 64, 3, 3, (2, 2), (1, 1), "cl", "cl"),
    (3, 12, 11, 13, 20, 2, 4, (3, 2), (0, 1), "std", "cl"),
    (1, 4, 5, 5, 4, 5, 5, (1, 1), (0, 0), "cl", "nchw"),
]


def make(case, seed=0):
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    x = wl.tensor((N, C, H, W), ("normal",), seed=seed)
    w = wl.tensor((CO, C, KH, KW), ("uniform", 1.0 / (C * KH * KW) ** 0.5), seed=seed + 1)
    bias = wl.tensor((CO,), ("uniform", 0.5), seed=seed + 2)
    HO, WO = oracle.conv2d_out_hw(H, W, KH, KW, st, pd)
    dy = wl.tensor((N, CO, HO, WO), ("normal",), seed=seed + 3)
    return x, w, bias, dy


def to_dev(t, layout):
    t = t.to(DEV)
    return t.contiguous(memory_format=CL) if layout == "cl" else t.contiguous()


def run(case, x, w, bias, dy, outputs=("dx", "dw", "db"), dx_layout="cl", accumulate=False,
        prior=None):
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    HO, WO = dy.shape[2:]
    xd, wd = to_dev(x, xlay), to_dev(w, wlay)
    bd, dyd = bias.to(DEV), to_dev(dy, "cl")
    y = torch.full((N, CO, HO, WO), float("nan"), device=DEV).contiguous(memory_format=CL)
    n = b.conv2d_fwd_workspace(xd, wd, bd, y, st, pd)
    ws = torch.empty(n // 4 + 64, device=DEV)
    b.conv2d_fwd(xd, wd, bd, y, st, pd, workspace=ws)
    dx = dw = db = None
    if "dx" in outputs:
        dx = torch.full((N, C, H, W), float("nan"), device=DEV)
        dx = dx.contiguous(memory_format=CL) if dx_layout == "cl" else dx
    if "dw" in outputs:
        dw = torch.full((CO, C, KH, KW), float("nan"), device=DEV)
        dw = dw.contiguous(memory_format=CL) if wlay == "cl" else dw
    if "db" in outputs:
        db = torch.full((CO,), float("nan"), device=DEV)
    if prior is not None:
        for t, p in zip((dx, dw, db), prior):
            if t is not None:
                t.copy_(p)
    n = b.conv2d_bwd_workspace(xd, wd, dyd, dx, dw, db, st, pd)
    ws2 = torch.empty(n // 4 + 64, device=DEV)
    b.conv2d_bwd(xd, wd, dyd, dx, dw, db, st, pd, accumulate=accumulate, workspace=ws2)
    torch.cuda.synchronize()
    return y, dx, dw, db


def check(case, x, w, bias, dy, y, dx, dw, db, prior=None):
    st, pd = case[7], case[8]
    X, Wt, B, dY = (to_f64(t) for t in (x, w, bias, dy))
    Y, SY = oracle.conv2d_fwd(X, Wt, B, st, pd)
    assert_close(to_f64(y.contiguous()), Y, SY, what="y")
    for got, (want, S), pr, name in (
            (dx, oracle.conv2d_bwd_dx(dY, Wt, X.shape, st, pd), 0, "dx"),
            (dw, oracle.conv2d_bwd_dw(dY, X, Wt.shape, st, pd), 1, "dw"),
            (db, oracle.conv2d_bwd_db(dY), 2, "db")):
        if got is None:
            continue
        if prior is not None:
            p = to_f64(prior[pr])
            want, S = want + p, S + np.abs(p)
        assert_close(to_f64(got.contiguous()), want, S, what=name)


@pytest.mark.parametrize("case", CASES, ids=[f"c{i}" for i in range(len(CASES))])
def test_conv2d_fwd_bwd(case):
    x, w, bias, dy = make(case)
    y, dx, dw, db = run(case, x, w, bias, dy)
    check(case, x, w, bias, dy, y, dx, dw, db)


def test_conv2d_optional_outputs_layouts_accumulate():
    case = CASES[1]
    x, w, bias, dy = make(case, seed=5)
    y, dx, _, _ = run(case, x, w, bias, dy, outputs=("dx",), dx_layout="nchw")
    check(case, x, w, bias, dy, y, dx, None, None)
    _, _, dw, _ = run(case, x, w, bias, dy, outputs=("dw",))
    check(case, x, w, bias, dy, y, None, dw, None)
    N, C, H, W, CO, KH, KW = case[:7]
    prior = (torch.randn(N, C, H, W, device=DEV), torch.randn(CO, C, KH, KW, device=DEV),
             torch.randn(CO, device=DEV))
    y, dx, dw, db = run(case, x, w, bias, dy, accumulate=True, prior=prior)
    check(case, x, w, bias, dy, y, dx, dw, db, prior=prior)


def test_conv2d_without_bias_and_deterministic():
    case = CASES[5]
    x, w, bias, dy = make(case, seed=9)
    outs = [run(case, x, w, torch.zeros_like(bias), dy) for _ in range(2)]
    for a, c in zip(outs[0], outs[1]):
        assert torch.equal(a, c), "reruns must be bit-identical"
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    xd, wd = to_dev(x, xlay), to_dev(w, wlay)
    y = torch.empty_like(outs[0][0])
    n = b.conv2d_fwd_workspace(xd, wd, None, y, st, pd)
    b.conv2d_fwd(xd, wd, None, y, st, pd, workspace=torch.empty(n // 4 + 64, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(y, outs[0][0]), "a zero bias and no bias give the same y"


def test_conv2d_missing_workspace_is_an_error():
    case = CASES[0]
    x, w, bias, dy = make(case)
    y = torch.empty(2, 4, 7, 6, device=DEV).contiguous(memory_format=CL)
    with pytest.raises(b.MtError) as e:
        b.conv2d_fwd(x.to(DEV), w.to(DEV), bias.to(DEV), y, 1, 1)
    assert e.value.status == 7


def test_conv2d_large_sampled():
    """32 x 256 x 56 x 56 input, 256 3x3 filters, stride 1, padding 1: the
    shape the bench times. Sampled y, dx, dw elements against the oracle,
    db in full."""
    case = (32, 256, 56, 56, 256, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=21)
    y, dx, dw, db = run(case, x, w, bias, dy)
    # every element written (the outputs start as NaN): tiles computed whole
    # and tiles summed from stream-K segments
    for t, name in ((y, "y"), (dx, "dx"), (dw, "dw")):
        assert not torch.isnan(t).any(), name
    X, Wt, B, dY = (to_f64(t) for t in (x, w, bias, dy))
    rng = np.random.default_rng(0)
    st, pd = case[7], case[8]
    yn = to_f64(y.contiguous())
    f = rng.integers(0, yn.size, 3000)
    want, S = oracle.conv2d_fwd_at(X, Wt, B, f, st, pd)
    assert_close(yn.flat[f], want, S, what="y sampled")
    dxn = to_f64(dx.contiguous())
    f = rng.integers(0, dxn.size, 3000)
    want, S = oracle.conv2d_bwd_dx_at(dY, Wt, X.shape, f, st, pd)
    assert_close(dxn.flat[f], want, S, what="dx sampled")
    dwn = to_f64(dw.contiguous())
    f = rng.integers(0, dwn.size, 300)
    want, S = oracle.conv2d_bwd_dw_at(dY, X, Wt.shape, f, st, pd)
    assert_close(dwn.flat[f], want, S, what="dw sampled")
    want, S = oracle.conv2d_bwd_db(dY)
    assert_close(to_f64(db), want, S, what="db")


def test_conv2d_backward_reuses_the_forward_unfold():
    case = CASES[6]
    x, w, bias, dy = make(case, seed=13)
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    HO, WO = dy.shape[2:]
    xd, wd, bd, dyd = to_dev(x, xlay), to_dev(w, wlay), bias.to(DEV), to_dev(dy, "cl")
    y = torch.empty(N, CO, HO, WO, device=DEV).contiguous(memory_format=CL)
    dx = torch.empty(N, C, H, W, device=DEV).contiguous(memory_format=CL)
    dw = torch.empty_like(wd)
    db = torch.empty(CO, device=DEV)
    need = max(b.conv2d_fwd_workspace(xd, wd, bd, y, st, pd),
               b.conv2d_bwd_workspace(xd, wd, dyd, dx, dw, db, st, pd))
    ws = torch.empty(need // 4 + 64, device=DEV)
    b.conv2d_fwd(xd, wd, bd, y, st, pd, workspace=ws)
    b.conv2d_bwd(xd, wd, dyd, dx, dw, db, st, pd, workspace=ws, reuse_unfold=True)
    torch.cuda.synchronize()
    check(case, x, w, bias, dy, y, dx, dw, db)


# Layouts where the products gather an operand in their loads (channels-last
# x and w; the forward needs C % 32 == 0, the weight gradient C % 4 == 0, the
# input gradient stride 1 and CO % 32 == 0): strides, paddings, 1x1 to 7x7
# windows, several images per 256-pixel tile, ragged last tiles, CO not a
# multiple of the tile.
GATHER_CASES = [
    (2, 32, 7, 6, 16, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (3, 64, 9, 11, 20, 3, 3, (2, 2), (1, 1), "cl", "cl"),
    (1, 32, 5, 5, 8, 5, 5, (1, 1), (0, 0), "cl", "cl"),
    (2, 96, 8, 8, 36, 1, 1, (1, 1), (0, 0), "cl", "cl"),
    (2, 32, 10, 7, 12, 5, 3, (2, 1), (2, 0), "cl", "cl"),
    (2, 64, 6, 6, 64, 7, 7, (3, 3), (3, 3), "cl", "cl"),
    (2, 12, 11, 13, 20, 2, 4, (3, 2), (0, 1), "cl", "cl"),
    (5, 32, 20, 20, 40, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (2, 32, 7, 6, 32, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (3, 8, 9, 11, 64, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (1, 12, 5, 5, 32, 5, 5, (1, 1), (0, 0), "cl", "cl"),
    (2, 64, 6, 6, 64, 7, 7, (1, 1), (3, 3), "cl", "cl"),
    (2, 4, 10, 7, 32, 5, 3, (1, 1), (2, 0), "cl", "cl"),
    (3, 36, 17, 19, 96, 3, 3, (1, 1), (1, 1), "cl", "cl"),
]


@pytest.mark.parametrize("cfg", [-1, 5, 6, 10, 11])
@pytest.mark.parametrize("case", GATHER_CASES, ids=[f"g{i}" for i in range(len(GATHER_CASES))])
def test_conv2d_gather_parity(case, cfg):
    """The gathering products against the oracle, and the unfolded path too;
    with one of their tiles forced (6: 256x256, 10 / 11: 128x128), y and dw
    also bit-identical to the same tile reading the unfolded input (the same
    values reach LDS in the same order; dx sums in another order when
    gathered: one product instead of dU and the fold). A forced tile outside
    that set (5) maps to 128x128."""
    x, w, bias, dy = make(case, seed=31)
    try:
        b.debug_set("cfg", cfg)
        got = run(case, x, w, bias, dy)
        check(case, x, w, bias, dy, *got)
        if cfg in (6, 10, 11):
            b.debug_set("conv_gather", 0)
            ref = run(case, x, w, bias, dy)
            check(case, x, w, bias, dy, *ref)
            for a, r, name in zip(got, ref, ("y", "dx", "dw", "db")):
                if name == "dx":
                    continue
                d = (a - r).abs()
                assert torch.equal(a, r), (f"{name}: gathered and unfolded products differ: max "
                                           f"{float(d.max())} at {int(d.argmax())}, "
                                           f"{int((d > 0).sum())} of {d.numel()}")
    finally:
        b.debug_set("conv_gather", 1)
        b.debug_set("cfg", -1)


def test_conv2d_gather_split_weight_gradient():
    """A long pixel contraction split into runs (dW), with the pixel count not
    a multiple of the 32-pixel stage."""
    case = (7, 32, 30, 29, 32, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=37)
    try:
        b.debug_set("splits", 5)
        got = run(case, x, w, bias, dy, outputs=("dw",))
    finally:
        b.debug_set("splits", 0)
    check(case, x, w, bias, dy, *got)


@pytest.mark.parametrize("co", [32, 44])
@pytest.mark.parametrize("splits", [0, 3, 5])
@pytest.mark.parametrize("acc", [False, True])
def test_conv2d_db_inside_weight_gradient(co, splits, acc):
    """db summed inside the gathered dW product (the column sums of dY^T, its
    first operand): whole or split into runs whose parts the finish adds,
    with and without accumulation, an output-channel count that leaves part
    of a tile, against the oracle."""
    case = (7, 32, 30, 29, co, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=41)
    prior = None
    if acc:
        prior = (None, wl.tensor((co, 32, 3, 3), ("normal",), seed=43).to(DEV),
                 wl.tensor((co,), ("normal",), seed=44).to(DEV))
    try:
        b.debug_set("splits", splits)
        got = run(case, x, w, bias, dy, outputs=("dw", "db"), accumulate=acc, prior=prior)
    finally:
        b.debug_set("splits", 0)
    check(case, x, w, bias, dy, *got, prior=prior)


def test_conv2d_reuse_flag_after_a_gathering_forward():
    """The forward gathered (no unfolded input left in the workspace) and the
    weight gradient cannot (dw 4 bytes off 16-byte alignment): the backward
    unfolds by itself although MT_CONV_REUSE_UNFOLD is passed."""
    case = (2, 32, 9, 9, 16, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=41)
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    xd, wd, bd, dyd = to_dev(x, xlay), to_dev(w, wlay), bias.to(DEV), to_dev(dy, "cl")
    y = torch.empty(N, CO, 9, 9, device=DEV).contiguous(memory_format=CL)
    assert b.conv2d_fwd_workspace(xd, wd, bd, y, st, pd) == 0
    b.conv2d_fwd(xd, wd, bd, y, st, pd)
    store = torch.full((CO * KH * KW * C + 1,), float("nan"), device=DEV)
    dw = store[1:].view(CO, KH, KW, C).permute(0, 3, 1, 2)
    n = b.conv2d_bwd_workspace(xd, wd, dyd, None, dw, None, st, pd)
    ws = torch.full((n // 4 + 64,), float("nan"), device=DEV)
    b.conv2d_bwd(xd, wd, dyd, None, dw, None, st, pd, workspace=ws, reuse_unfold=True)
    torch.cuda.synchronize()
    check(case, x, w, bias, dy, y, None, dw, None)


def test_conv2d_gathered_input_gradient_accumulates():
    """dx gathered from dy (stride 1, CO % 32 == 0) into channels-last dx with
    MT_ACCUMULATE; an [N][C][H][W] dx takes the dU + fold path instead."""
    case = (2, 16, 12, 10, 32, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=43)
    N, C, H, W, CO, KH, KW = case[:7]
    prior = (torch.randn(N, C, H, W, device=DEV), torch.randn(CO, C, KH, KW, device=DEV),
             torch.randn(CO, device=DEV))
    y, dx, dw, db = run(case, x, w, bias, dy, accumulate=True, prior=prior)
    check(case, x, w, bias, dy, y, dx, dw, db, prior=prior)
    y, dx, _, _ = run(case, x, w, bias, dy, outputs=("dx",), dx_layout="nchw")
    check(case, x, w, bias, dy, y, dx, None, None)


def test_conv2d_gathered_backward_needs_no_unfolded_workspace():
    """Every product of the step gathers: the backward's workspace holds only
    split partials, and the step runs with no workspace at all."""
    case = (4, 32, 14, 14, 64, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=47)
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    xd, wd, bd, dyd = to_dev(x, xlay), to_dev(w, wlay), bias.to(DEV), to_dev(dy, "cl")
    y = torch.empty(N, CO, H, W, device=DEV).contiguous(memory_format=CL)
    dx = torch.empty(N, C, H, W, device=DEV).contiguous(memory_format=CL)
    dw = torch.empty_like(wd)
    db = torch.empty(CO, device=DEV)
    col = N * H * W * C * KH * KW * 4
    assert b.conv2d_bwd_workspace(xd, wd, dyd, dx, dw, db, st, pd) < col
    b.conv2d_fwd(xd, wd, bd, y, st, pd)
    b.conv2d_bwd(xd, wd, dyd, dx, dw, db, st, pd)
    torch.cuda.synchronize()
    check(case, x, w, bias, dy, y, dx, dw, db)


SK_CASES = [
    (5, 32, 20, 20, 40, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (4, 64, 20, 20, 64, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (2, 32, 12, 12, 288, 3, 3, (1, 1), (1, 1), "cl", "cl"),
    (3, 36, 17, 19, 96, 3, 3, (1, 1), (1, 1), "cl", "cl"),
]


@pytest.mark.parametrize("blocks", [3, 5, 7, 13, 64])
@pytest.mark.parametrize("case", SK_CASES, ids=[f"s{i}" for i in range(len(SK_CASES))])
def test_conv2d_stream_k(case, blocks):
    """The gathered forward and input-gradient products in stream-K order over
    a forced number of blocks (tiles cut into 1-3 segments at arbitrary
    stages, several tile rows and columns, up to three tiles' stages per
    block): against the oracle, and bit-identical on a rerun (segments are
    summed in a fixed order)."""
    x, w, bias, dy = make(case, seed=53)
    try:
        b.debug_set("cfg", 6)
        b.debug_set("stream_k", 2)
        b.debug_set("sk_blocks", blocks)
        got = run(case, x, w, bias, dy)
        again = run(case, x, w, bias, dy)
    finally:
        b.debug_set("sk_blocks", 0)
        b.debug_set("stream_k", 1)
        b.debug_set("cfg", -1)
    check(case, x, w, bias, dy, *got)
    for a, c in zip(got, again):
        assert torch.equal(a, c), "stream-K reruns must be bit-identical"


def test_conv2d_stream_k_accumulates_and_needs_its_workspace():
    """Stream-K with MT_ACCUMULATE (the finish adds C for cut tiles, the
    product for whole ones); with no workspace the product runs one tile per
    block and gives the same values up to rounding."""
    case = SK_CASES[1]
    x, w, bias, dy = make(case, seed=59)
    N, C, H, W, CO, KH, KW = case[:7]
    prior = (torch.randn(N, C, H, W, device=DEV), torch.randn(CO, C, KH, KW, device=DEV),
             torch.randn(CO, device=DEV))
    try:
        b.debug_set("stream_k", 2)
        b.debug_set("sk_blocks", 13)
        y, dx, dw, db = run(case, x, w, bias, dy, accumulate=True, prior=prior)
        check(case, x, w, bias, dy, y, dx, dw, db, prior=prior)
        st, pd = case[7], case[8]
        xd, wd, bd = to_dev(x, "cl"), to_dev(w, "cl"), bias.to(DEV)
        assert b.conv2d_fwd_workspace(xd, wd, bd, y, st, pd) > 0
        y2 = torch.empty_like(y)
        b.conv2d_fwd(xd, wd, bd, y2, st, pd)        # no workspace: plain schedule
        torch.cuda.synchronize()
        check(case, x, w, bias, dy, y2, None, None, None)
    finally:
        b.debug_set("sk_blocks", 0)
        b.debug_set("stream_k", 1)


# Edge cases of the gathered path: one pixel, a window larger than the image
# (all taps but a few in the padding), a 1-row image, asymmetric strides and
# paddings, a batch whose pixels do not fill one 128-row tile.
GATHER_EDGES = [
    (1, 32, 1, 1, 32, 1, 1, (1, 1), (0, 0), "cl", "cl"),
    (2, 32, 3, 3, 32, 5, 5, (1, 1), (2, 2), "cl", "cl"),
    (3, 64, 1, 9, 32, 1, 3, (1, 1), (0, 1), "cl", "cl"),
    (1, 64, 7, 5, 36, 3, 3, (2, 1), (0, 1), "cl", "cl"),
    (2, 32, 4, 4, 32, 3, 3, (3, 3), (1, 1), "cl", "cl"),
    (1, 96, 2, 3, 64, 2, 2, (1, 1), (1, 1), "cl", "cl"),
]


@pytest.mark.parametrize("case", GATHER_EDGES, ids=[f"e{i}" for i in range(len(GATHER_EDGES))])
def test_conv2d_gather_edges(case):
    x, w, bias, dy = make(case, seed=67)
    got = run(case, x, w, bias, dy)
    check(case, x, w, bias, dy, *got)
    try:
        b.debug_set("stream_k", 2)
        b.debug_set("sk_blocks", 3)
        got = run(case, x, w, bias, dy)
    finally:
        b.debug_set("sk_blocks", 0)
        b.debug_set("stream_k", 1)
    check(case, x, w, bias, dy, *got)


# Strided convolutions whose input gradient runs as one gathered product per
# sub-pixel phase (CO % 32 == 0, KH >= sh, KW >= sw), and one (1x1 window,
# stride 2) that keeps dU and the fold.
PHASE_CASES = [
    (2, 8, 9, 9, 32, 3, 3, (2, 2), (1, 1), "cl", "cl"),
    (2, 16, 10, 7, 64, 5, 3, (2, 1), (2, 0), "cl", "cl"),
    (1, 12, 11, 13, 32, 3, 4, (3, 2), (1, 1), "cl", "cl"),
    (2, 32, 28, 28, 64, 3, 3, (2, 2), (1, 1), "cl", "cl"),
    (3, 4, 12, 12, 32, 4, 4, (2, 2), (0, 0), "cl", "cl"),
    (2, 8, 8, 8, 32, 1, 1, (2, 2), (0, 0), "cl", "cl"),
]


@pytest.mark.parametrize("grid", [0, 2])
@pytest.mark.parametrize("case", PHASE_CASES, ids=[f"p{i}" for i in range(len(PHASE_CASES))])
def test_conv2d_strided_input_gradient_by_phases(case, grid):
    """A launch per phase (grid 0) or every phase in one grid of 256x256 tiles
    (grid 2), with and without MT_ACCUMULATE."""
    x, w, bias, dy = make(case, seed=71)
    try:
        b.debug_set("phase_grid", grid)
        got = run(case, x, w, bias, dy)
        check(case, x, w, bias, dy, *got)
        N, C, H, W, CO, KH, KW = case[:7]
        prior = (torch.randn(N, C, H, W, device=DEV), torch.randn(CO, C, KH, KW, device=DEV),
                 torch.randn(CO, device=DEV))
        got = run(case, x, w, bias, dy, outputs=("dx",), accumulate=True, prior=prior)
        check(case, x, w, bias, dy, got[0], got[1], None, None, prior=prior)
    finally:
        b.debug_set("phase_grid", 1)


def test_conv2d_strided_phases_need_no_unfolded_workspace():
    case = PHASE_CASES[3]
    x, w, bias, dy = make(case, seed=73)
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    xd, wd, dyd = to_dev(x, xlay), to_dev(w, wlay), to_dev(dy, "cl")
    dx = torch.empty(N, C, H, W, device=DEV).contiguous(memory_format=CL)
    HO, WO = dy.shape[2:]
    col = N * HO * WO * C * KH * KW * 4
    assert b.conv2d_bwd_workspace(xd, wd, dyd, dx, None, None, st, pd) < col
