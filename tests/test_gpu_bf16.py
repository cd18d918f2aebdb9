"""GPU parity of the bf16-operand dense layer and matmul (exact bf16
products, fp32 accumulation, fp32 bias/outputs) against the fp64 oracle run
on the identical bf16 values.

Bar (reading R2 of the relative 2e-2 tolerance): elementwise
|gpu - oracle| <= 2e-2 * S + 1e-6 and normwise ||gpu - oracle|| / ||oracle||
<= 2e-2. Since bf16 x bf16 products are exact in fp32, the kernels should
also meet the fp32 bar (1e-4 * S + 1e-6); that is checked as well.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, sample_positions, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"


def check_bf16(got, want, S, what):
    assert_close(got, want, S, rel=2e-2, abs_=1e-6, what=what + " (bf16 bar)")
    nrm = np.linalg.norm(want)
    if nrm > 0:
        assert np.linalg.norm(got - want) / nrm <= 2e-2, what
    assert_close(got, want, S, what=what + " (fp32 bar)")


def make(M, N, K, seed, dist=None):
    return wl.linear(M, N, K, dtype="bf16", seed=seed, dist=dist).make()


def run(inp):
    x, w, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    M, K = x.shape
    N = w.shape[0]
    y = torch.full((M, N), float("nan"), device=DEV)
    dx = torch.full((M, K), float("nan"), device=DEV)
    dw = torch.full((N, K), float("nan"), device=DEV)
    db = torch.full((N,), float("nan"), device=DEV)
    b.linear_fwd(x, w, bias, y)
    n = b.linear_bwd_workspace(x, w, dy, dx, dw, db)
    ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.linear_bwd(x, w, dy, dx, dw, db, workspace=ws)
    torch.cuda.synchronize()
    return {"Y": y, "dX": dx, "dW": dw, "db": db}


def check_full(inp, out):
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    Y, SY = oracle.linear_fwd(X, W, B)
    check_bf16(to_f64(out["Y"]), Y, SY, "Y")
    dX, SX = oracle.linear_bwd_dx(dY, W)
    check_bf16(to_f64(out["dX"]), dX, SX, "dX")
    dW, SW = oracle.linear_bwd_dw(dY, X)
    check_bf16(to_f64(out["dW"]), dW, SW, "dW")
    db, Sb = oracle.linear_bwd_db(dY)
    check_bf16(to_f64(out["db"]), db, Sb, "db")


@pytest.mark.parametrize("M,N,K", [(64, 32, 128), (300, 200, 100), (520, 392, 264), (257, 129, 67),
                                   (1, 1, 1), (96, 1000, 40), (1000, 96, 40)])
def test_bf16_linear_small_and_ragged(M, N, K):
    inp = make(M, N, K, seed=M + N + K)
    check_full(inp, run(inp))


@pytest.mark.parametrize("cfg", list(range(b.NUM_GEMM_CFG)))
@pytest.mark.parametrize("vec1", [0, 1])
@pytest.mark.parametrize("shape", [(520, 392, 264), (576, 320, 256)])
def test_bf16_every_tile_config(cfg, vec1, shape):
    # K tails in every product, then none (see the fp32 test of the same name)
    inp = make(*shape, seed=17)
    b.debug_set("cfg", cfg)
    b.debug_set("vec1", vec1)
    try:
        out = run(inp)
    finally:
        b.debug_set("cfg", -1)
        b.debug_set("vec1", 0)
    check_full(inp, out)


def test_bf16_linear_16384x8192x8192_sampled():
    inp = wl.LINEAR_16384x8192x8192_BF16.make()
    out = run(inp)
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    M, K = X.shape
    N = W.shape[0]
    r, c = sample_positions(M, N, 3000, seed=1)
    v, S = oracle.linear_fwd_at(X, W, B, r, c)
    check_bf16(to_f64(out["Y"])[r, c], v, S, "Y (sampled)")
    r, c = sample_positions(M, K, 3000, seed=2)
    v, S = oracle.linear_bwd_dx_at(dY, W, r, c)
    check_bf16(to_f64(out["dX"])[r, c], v, S, "dX (sampled)")
    r, c = sample_positions(N, K, 3000, seed=3)
    v, S = oracle.linear_bwd_dw_at(dY, X, r, c)
    check_bf16(to_f64(out["dW"])[r, c], v, S, "dW (sampled)")
    db, Sb = oracle.linear_bwd_db(dY)
    check_bf16(to_f64(out["db"]), db, Sb, "db")
    for k in out:
        assert torch.isfinite(out[k]).all(), k
    # whole 256-row bands at full contraction length, crossing a tile boundary
    R, r0, n0 = 256, 8064, 2944
    Yb, SY = oracle.linear_fwd(X[r0:r0 + R], W, B)
    check_bf16(to_f64(out["Y"][r0:r0 + R]), Yb, SY, "Y (band)")
    dXb, SX = oracle.linear_bwd_dx(dY[r0:r0 + R], W)
    check_bf16(to_f64(out["dX"][r0:r0 + R]), dXb, SX, "dX (band)")
    dWb, SW = oracle.linear_bwd_dw(np.ascontiguousarray(dY[:, n0:n0 + R]), X)
    check_bf16(to_f64(out["dW"][n0:n0 + R]), dWb, SW, "dW (band)")


def test_bf16_integer_inputs_bit_exact_at_16384x8192x8192():
    """Integers in [-4, 4] are exact in bf16 and every partial sum stays below
    2**24, so the result is exact in any summation order."""
    inp = make(16384, 8192, 8192, seed=6, dist={k: wl.integers(-4, 4) for k in ("X", "W", "b", "dY")})
    out = run(inp)
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    for k in out:
        assert torch.equal(out[k], torch.round(out[k])), k
    r, c = sample_positions(16384, 8192, 2000, seed=7)
    assert np.array_equal(to_f64(out["Y"])[r, c], oracle.linear_fwd_at(X, W, B, r, c)[0])
    assert np.array_equal(to_f64(out["dX"])[r, c], oracle.linear_bwd_dx_at(dY, W, r, c)[0])
    r, c = sample_positions(8192, 8192, 2000, seed=8)
    assert np.array_equal(to_f64(out["dW"])[r, c], oracle.linear_bwd_dw_at(dY, X, r, c)[0])
    assert np.array_equal(to_f64(out["db"]), oracle.linear_bwd_db(dY)[0])


@pytest.mark.parametrize("seed", range(8))
def test_bf16_broadcast_matmul(seed):
    rng = np.random.default_rng(100 + seed)
    M, K, N = (int(rng.choice([5, 32, 77, 128, 200])) for _ in range(3))
    A = wl.tensor((3, 1, M, K), ("normal",), seed=seed).to(torch.bfloat16)
    B = wl.tensor((1, 2, K, N), ("normal",), seed=seed + 50).to(torch.bfloat16)
    dC = wl.tensor((3, 2, M, N), ("normal",), seed=seed + 99).to(torch.bfloat16)
    Ad, Bd, dCd = A.to(DEV), B.to(DEV), dC.to(DEV)
    C = torch.empty(3, 2, M, N, device=DEV)
    b.matmul(Ad, Bd, C)
    dA = torch.empty(3, 1, M, K, device=DEV)
    dB = torch.empty(1, 2, K, N, device=DEV)
    b.matmul(dCd, Bd.transpose(-1, -2), dA, reduce_into=True)
    b.matmul(Ad.transpose(-1, -2), dCd, dB, reduce_into=True)
    torch.cuda.synchronize()
    An, Bn, dCn = to_f64(A), to_f64(B), to_f64(dC)
    Cr, SC = oracle.matmul(An, Bn)
    check_bf16(to_f64(C), Cr, SC, "C")
    dAr, SA, dBr, SB = oracle.matmul_bwd(An, Bn, dCn)
    check_bf16(to_f64(dA), dAr, SA, "dA")
    check_bf16(to_f64(dB), dBr, SB, "dB")


@pytest.mark.parametrize("cfg", [6, 7, 8, 9, 10, 11])
@pytest.mark.parametrize("splits", [0, 3])
def test_bf16_db_folded_into_dw(cfg, splits):
    """bf16 dY: db summed inside the dW product (pairs of bf16 elements added
    by v_dot2_f32_bf16 against ones: exact products, fp32 sums), whole and
    split along the contraction."""
    M, N, K = 520, 392, 264
    inp = make(M, N, K, seed=41)
    x, w, dy = (inp[k].to(DEV) for k in ("X", "W", "dY"))
    dw = torch.full((N, K), float("nan"), device=DEV)
    db = torch.full((N,), float("nan"), device=DEV)
    b.debug_set("cfg", cfg)
    b.debug_set("splits", splits)
    try:
        need = b.linear_bwd_workspace(x, w, dy, None, dw, db)
        if splits:
            need_dw = b.linear_bwd_workspace(x, w, dy, None, dw, None)
            assert need == ((need_dw + 255) // 256) * 256 + splits * N * 4
        ws = torch.empty(need // 4 + 64, device=DEV) if need else None
        b.linear_bwd(x, w, dy, None, dw, db, workspace=ws)
        torch.cuda.synchronize()
    finally:
        b.debug_set("cfg", -1)
        b.debug_set("splits", 0)
    X, dY = to_f64(inp["X"]), to_f64(inp["dY"])
    check_bf16(to_f64(db), *oracle.linear_bwd_db(dY), "db")
    check_bf16(to_f64(dw), *oracle.linear_bwd_dw(dY, X), "dW")


def _three_products(inp):
    """Y, dX and dW as three calls (dW without db, so that no column sum
    rides on it), then dW with db (the column sum of dY inside the product)."""
    x, w, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    M, K = x.shape
    N = w.shape[0]
    y = torch.full((M, N), float("nan"), device=DEV)
    dx = torch.full((M, K), float("nan"), device=DEV)
    dw = torch.full((N, K), float("nan"), device=DEV)
    b.linear_fwd(x, w, bias, y)
    b.linear_bwd(x, w, dy, dx, None, None)
    b.linear_bwd(x, w, dy, None, dw, None)
    dw2 = torch.full((N, K), float("nan"), device=DEV)
    db = torch.full((N,), float("nan"), device=DEV)
    b.linear_bwd(x, w, dy, None, dw2, db)
    torch.cuda.synchronize()
    return {"Y": y, "dX": dx, "dW": dw, "dW+db": dw2, "db": db}


def _persist_on_off(inp):
    try:
        b.debug_set("persist", 1)
        got = _three_products(inp)
        b.debug_set("persist", 0)
        plain = _three_products(inp)
    finally:
        b.debug_set("persist", 1)
    return got, plain


# (M, N, K) with 17 x 16 = 272 whole output tiles of 256x256 (more than the
# CUs) for one product each: the forward (Y is M x N, with the bias), dX
# (M x K) and dW (N x K); three K-stages of 64 in the product that is
# persistent, or one (the forward and dX take the ring of half-slots, whose
# A loads run a stage ahead of the B loads: with one stage per tile they
# are a whole tile ahead)
PERSIST_SHAPES = {"Y": (4352, 4096, 192), "dX": (4352, 192, 4096), "dW": (192, 4352, 4096),
                  "Y1": (4352, 4096, 64), "dX1": (4352, 64, 4096)}


@pytest.mark.parametrize("cfg", [6, 7])
@pytest.mark.parametrize("which", ["Y", "dX", "dW", "Y1", "dX1"])
def test_bf16_persistent_grid(cfg, which):
    """A product with more 256x256 tiles than CUs runs on a persistent grid
    (one block per CU, the first 16 blocks taking two tiles): every element
    against the oracle, and bit for bit against the plain grid, whose block
    for each tile sums in the same order."""
    M, N, K = PERSIST_SHAPES[which]
    inp = make(M, N, K, seed=41)
    b.debug_set("cfg", cfg)
    try:
        got, plain = _persist_on_off(inp)
    finally:
        b.debug_set("cfg", -1)
    for k in got:
        assert torch.equal(got[k], plain[k]), k
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    out = which.rstrip("1")
    if out == "Y":
        want, S = oracle.linear_fwd(X, W, B)
    elif out == "dX":
        want, S = oracle.linear_bwd_dx(dY, W)
    else:
        want, S = oracle.linear_bwd_dw(dY, X)
    check_bf16(to_f64(got[out]), want, S, which + " (persistent grid)")
    if out == "dW":
        assert torch.equal(got["dW+db"], got["dW"])
        check_bf16(to_f64(got["db"]), *oracle.linear_bwd_db(dY), which + " db (persistent grid)")


def test_bf16_persistent_grid_bitwise_at_16384x8192x8192():
    """The bench's products on the persistent grid (2048 tiles, eight per
    block) equal the plain grid's bit for bit."""
    got, plain = _persist_on_off(wl.LINEAR_16384x8192x8192_BF16.make())
    for k in got:
        assert not torch.isnan(got[k]).any(), k
        assert torch.equal(got[k], plain[k]), k
