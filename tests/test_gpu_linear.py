"""GPU parity of the dense layer (Eq. (5)) and its gradients (Eq. (4) and
the add pullback) against the fp64 oracle, through the C-ABI library."""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, sample_positions, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)

DEV = "cuda:0"


def run_linear(inp, accumulate=False, prior=None, use_ws=True, outputs=("dx", "dw", "db")):
    x, w, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    M, K = x.shape
    N = w.shape[0]
    y = torch.full((M, N), float("nan"), device=DEV)
    dx = torch.full((M, K), float("nan"), device=DEV) if "dx" in outputs else None
    dw = torch.full((N, K), float("nan"), device=DEV) if "dw" in outputs else None
    db = torch.full((N,), float("nan"), device=DEV) if "db" in outputs else None
    if prior is not None:
        for t, p in ((dx, prior.get("dx")), (dw, prior.get("dw")), (db, prior.get("db"))):
            if t is not None:
                t.copy_(p)
    b.linear_fwd(x, w, bias, y)
    ws = None
    if use_ws:
        n = b.linear_bwd_workspace(x, w, dy, dx, dw, db)
        ws = torch.empty(max(n, 1) // 4 + 64, device=DEV, dtype=torch.float32) if n else None
    b.linear_bwd(x, w, dy, dx, dw, db, accumulate=accumulate, workspace=ws)
    torch.cuda.synchronize()
    return {"Y": y, "dX": dx, "dW": dw, "db": db}


def oracle_full(inp):
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    Y, SY = oracle.linear_fwd(X, W, B)
    dX, SX = oracle.linear_bwd_dx(dY, W)
    dW, SW = oracle.linear_bwd_dw(dY, X)
    db, Sb = oracle.linear_bwd_db(dY)
    return {"Y": (Y, SY), "dX": (dX, SX), "dW": (dW, SW), "db": (db, Sb)}


def check_full(out, ref, names=("Y", "dX", "dW", "db")):
    for k in names:
        assert_close(to_f64(out[k]), ref[k][0], ref[k][1], what=k)


SMALL = [(64, 32, 128), (300, 200, 100), (257, 129, 67), (1, 1, 1), (3, 5, 7), (520, 392, 264),
         (33, 65, 4), (1000, 8, 36), (8, 1000, 36)]


@pytest.mark.parametrize("M,N,K", SMALL)
def test_linear_small_and_ragged(M, N, K):
    inp = wl.linear(M, N, K, seed=M * 7 + N).make()
    out = run_linear(inp)
    check_full(out, oracle_full(inp))


def test_linear_64x32x128_workload():
    inp = wl.LINEAR_64x32x128_F32.make()
    out = run_linear(inp)
    check_full(out, oracle_full(inp))


@pytest.mark.parametrize("cfg", list(range(b.NUM_GEMM_CFG)))
@pytest.mark.parametrize("vec1", [0, 1])
@pytest.mark.parametrize("shape", [(520, 392, 264), (576, 320, 256)])
def test_linear_every_tile_config(cfg, vec1, shape):
    # (520, 392, 264): no product's K is a whole number of K-stages (K tails);
    # (576, 320, 256): every product's K is (the tail-free kernel builds),
    # with M and N still cutting the tiles
    inp = wl.linear(*shape, seed=11).make()
    b.debug_set("cfg", cfg)
    b.debug_set("vec1", vec1)
    try:
        out = run_linear(inp)
    finally:
        b.debug_set("cfg", -1)
        b.debug_set("vec1", 0)
    check_full(out, oracle_full(inp))


def test_linear_4096x1024x1024_full():
    inp = wl.LINEAR_4096x1024x1024_F32.make()
    out = run_linear(inp)
    check_full(out, oracle_full(inp))


def test_linear_determinism_and_splitk_agree():
    inp = wl.LINEAR_4096x1024x1024_F32.make()
    a = run_linear(inp)
    a2 = run_linear(inp)
    for k in a:
        assert torch.equal(a[k], a2[k]), k
    nows = run_linear(inp, use_ws=False)
    ref = oracle_full(inp)
    check_full(nows, ref)
    b.debug_set("splits", 3)
    b.debug_set("parts", 5)
    try:
        forced = run_linear(inp)
    finally:
        b.debug_set("splits", 0)
        b.debug_set("parts", 0)
    check_full(forced, ref)


def _sampled_check(inp, out, n_random=3000):
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    M, K = X.shape
    N = W.shape[0]
    Y, dX, dW = to_f64(out["Y"]), to_f64(out["dX"]), to_f64(out["dW"])
    r, c = sample_positions(M, N, n_random, seed=1)
    v, S = oracle.linear_fwd_at(X, W, B, r, c)
    assert_close(Y[r, c], v, S, what="Y (sampled)")
    r, c = sample_positions(M, K, n_random, seed=2)
    v, S = oracle.linear_bwd_dx_at(dY, W, r, c)
    assert_close(dX[r, c], v, S, what="dX (sampled)")
    r, c = sample_positions(N, K, n_random, seed=3)
    v, S = oracle.linear_bwd_dw_at(dY, X, r, c)
    assert_close(dW[r, c], v, S, what="dW (sampled)")
    db, Sb = oracle.linear_bwd_db(dY)
    assert_close(to_f64(out["db"]), db, Sb, what="db")
    for k in ("Y", "dX", "dW", "db"):
        assert torch.isfinite(out[k]).all(), f"{k}: unwritten (NaN) or non-finite elements"


def _band_check(inp, out, r0, n0, R=256):
    """Whole 256-row bands at full contraction length against the row-major
    oracle: rows r0..r0+R-1 of Y and dX (X and dY rows of the band) and rows
    n0..n0+R-1 of dW (dY columns of the band)."""
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    Y, SY = oracle.linear_fwd(X[r0:r0 + R], W, B)
    assert_close(to_f64(out["Y"][r0:r0 + R]), Y, SY, what=f"Y rows {r0}..{r0 + R - 1}")
    dX, SX = oracle.linear_bwd_dx(dY[r0:r0 + R], W)
    assert_close(to_f64(out["dX"][r0:r0 + R]), dX, SX, what=f"dX rows {r0}..{r0 + R - 1}")
    dW, SW = oracle.linear_bwd_dw(np.ascontiguousarray(dY[:, n0:n0 + R]), X)
    assert_close(to_f64(out["dW"][n0:n0 + R]), dW, SW, what=f"dW rows {n0}..{n0 + R - 1}")


def test_linear_8192_cubed_sampled():
    inp = wl.LINEAR_8192x8192x8192_F32.make()
    out = run_linear(inp)
    _sampled_check(inp, out)
    # one whole band each, crossing a 256-row tile boundary (rows 3968..4223
    # of Y and dX, rows 6016..6271 of dW)
    _band_check(inp, out, r0=3968, n0=6016)


def test_linear_8192_cubed_integer_inputs_bit_exact():
    """Integer inputs in [-2, 2]: every partial sum is an integer below 2**24,
    so fp32 accumulation is exact in any order and the GPU must equal the
    oracle bit for bit."""
    w = wl.linear(8192, 8192, 8192, seed=5,
                  dist={k: wl.integers(-2, 2) for k in ("X", "W", "b", "dY")})
    inp = w.make()
    out = run_linear(inp)
    X, W, B, dY = (to_f64(inp[k]) for k in ("X", "W", "b", "dY"))
    for k in ("Y", "dX", "dW", "db"):
        t = out[k]
        assert torch.equal(t, torch.round(t)), f"{k}: non-integer value"
    r, c = sample_positions(8192, 8192, 2000, seed=4)
    assert np.array_equal(to_f64(out["Y"])[r, c], oracle.linear_fwd_at(X, W, B, r, c)[0])
    assert np.array_equal(to_f64(out["dX"])[r, c], oracle.linear_bwd_dx_at(dY, W, r, c)[0])
    assert np.array_equal(to_f64(out["dW"])[r, c], oracle.linear_bwd_dw_at(dY, X, r, c)[0])
    assert np.array_equal(to_f64(out["db"]), oracle.linear_bwd_db(dY)[0])


def test_linear_identity_weight_bit_exact():
    M = K = N = 384
    x = wl.tensor((M, K), ("normal",), seed=9)
    dy = wl.tensor((M, N), ("normal",), seed=10)
    inp = {"X": x, "W": torch.eye(N), "b": torch.zeros(N), "dY": dy}
    out = run_linear(inp)
    assert torch.equal(out["Y"].cpu(), x)
    assert torch.equal(out["dX"].cpu(), dy)
    # X = I: dW = dY^T exactly
    inp2 = {"X": torch.eye(M), "W": torch.eye(N), "b": torch.zeros(N), "dY": dy}
    out2 = run_linear(inp2)
    assert torch.equal(out2["dW"].cpu(), dy.t())


def test_linear_accumulate():
    inp = wl.linear(300, 200, 100, seed=21).make()
    prior = {"dx": torch.randn(300, 100), "dw": torch.randn(200, 100), "db": torch.randn(200)}
    out = run_linear(inp, accumulate=True, prior=prior)
    ref = oracle_full(inp)
    assert_close(to_f64(out["dX"]), ref["dX"][0] + prior["dx"].double().numpy(), ref["dX"][1] + 1, what="dX+=")
    assert_close(to_f64(out["dW"]), ref["dW"][0] + prior["dw"].double().numpy(), ref["dW"][1] + 1, what="dW+=")
    assert_close(to_f64(out["db"]), ref["db"][0] + prior["db"].double().numpy(), ref["db"][1] + 1, what="db+=")


def test_linear_accumulate_on_whole_tiles():
    """dX += dY W on a product with more whole 256x256 tiles than CUs (the
    shape that runs on the persistent grid when it overwrites): the
    accumulating product takes the plain grid and adds to the prior."""
    M, N, K = 4352, 192, 4096
    inp = wl.linear(M, N, K, seed=23).make()
    prior = {"dx": torch.randn(M, K)}
    out = run_linear(inp, accumulate=True, prior=prior, outputs=("dx",))
    dY, W = to_f64(inp["dY"]), to_f64(inp["W"])
    dX, SX = oracle.linear_bwd_dx(dY, W)
    assert_close(to_f64(out["dX"]), dX + prior["dx"].double().numpy(), SX + 1, what="dX+= (whole tiles)")


@pytest.mark.parametrize("outputs", [("dx",), ("dw",), ("db",), ("dx", "db"), ()])
def test_linear_optional_outputs(outputs):
    inp = wl.linear(130, 70, 40, seed=3).make()
    out = run_linear(inp, outputs=outputs)
    ref = oracle_full(inp)
    names = ["Y"] + [{"dx": "dX", "dw": "dW", "db": "db"}[o] for o in outputs]
    check_full(out, ref, names)


def test_linear_unaligned_views():
    """Operands offset by one element and with odd row pitches take the
    4-byte-load kernels."""
    M, N, K = 200, 120, 88
    inp = wl.linear(M, N, K, seed=8).make()
    bufx = torch.zeros(M * (K + 3) + 1, device=DEV)
    x = bufx[1:].view(M, K + 3)[:, :K]
    x.copy_(inp["X"].to(DEV))
    w = inp["W"].to(DEV)
    bias = inp["b"].to(DEV)
    dy = inp["dY"].to(DEV)
    y = torch.empty(M, N, device=DEV)
    dx = torch.empty(M, K, device=DEV)
    dw = torch.empty(N, K, device=DEV)
    db = torch.empty(N, device=DEV)
    b.linear_fwd(x, w, bias, y)
    b.linear_bwd(x, w, dy, dx, dw, db)
    torch.cuda.synchronize()
    check_full({"Y": y, "dX": dx, "dW": dw, "db": db}, oracle_full(inp))


def test_linear_zero_k_and_empty():
    inp = {"X": torch.zeros(5, 0), "W": torch.zeros(3, 0), "b": torch.randn(3), "dY": torch.randn(5, 3)}
    out = run_linear(inp)
    assert torch.equal(out["Y"].cpu(), inp["b"].expand(5, 3))
    assert out["dX"].numel() == 0 and out["dW"].numel() == 0
    ref = oracle_full(inp)
    assert_close(to_f64(out["db"]), ref["db"][0], ref["db"][1], what="db")
    # M = 0: dw = 0 and db = 0
    inp0 = {"X": torch.zeros(0, 4), "W": torch.randn(3, 4), "b": torch.randn(3), "dY": torch.zeros(0, 3)}
    out0 = run_linear(inp0)
    assert torch.equal(out0["dW"].cpu(), torch.zeros(3, 4))
    assert torch.equal(out0["db"].cpu(), torch.zeros(3))


# DMA tiles (cfg, 4-byte lanes) whose weight-gradient product sums db itself
FOLD_CFGS = [(6, 0), (6, 1), (7, 0), (8, 0), (8, 1), (9, 0), (9, 1), (10, 0), (10, 1), (11, 0),
             (12, 0)]


@pytest.mark.parametrize("cfg,vec1", FOLD_CFGS)
@pytest.mark.parametrize("splits", [0, 3])
@pytest.mark.parametrize("shape", [(520, 392, 264), (576, 320, 256), (520, 391, 264)])
def test_linear_db_folded_into_dw(cfg, vec1, splits, shape):
    """db = 1^T dY summed inside the dW product from the dY tiles it already
    reads (no second pass over dY), on every DMA tile with 16- and 4-byte
    lanes, whole and split along the contraction (one sum per run, the runs
    added in order by the split-K finish, in its 16-byte form or, for an odd
    N, the element form and a pass of their own), overwriting and
    accumulating; (520, 392, 264) has a K tail in the product and ragged
    edge tiles."""
    M, N, K = shape
    inp = wl.linear(M, N, K, seed=31).make()
    x, w, dy = (inp[k].to(DEV) for k in ("X", "W", "dY"))
    prior = torch.randn(N, generator=torch.Generator().manual_seed(5)).to(DEV)
    X, dY = to_f64(inp["X"]), to_f64(inp["dY"])
    dW_ref, SW = oracle.linear_bwd_dw(dY, X)
    db_ref, Sb = oracle.linear_bwd_db(dY)
    for acc in (False, True):
        dw = torch.zeros(N, K, device=DEV) if acc else torch.full((N, K), float("nan"), device=DEV)
        db = prior.clone() if acc else torch.full((N,), float("nan"), device=DEV)
        b.debug_set("cfg", cfg)
        b.debug_set("vec1", vec1)
        b.debug_set("splits", splits)
        try:
            need = b.linear_bwd_workspace(x, w, dy, None, dw, db)
            need_dw = b.linear_bwd_workspace(x, w, dy, None, dw, None)
            # the 4-wave 256x256 tile (cfg 7) has 16-byte lanes only: an odd N
            # takes the register-staged tile there, which leaves db to the
            # column-sum pass
            if splits and not (N % 4 and cfg == 7):
                # the runs' db sums sit after the partial tiles: the fold is in use
                assert need == ((need_dw + 255) // 256) * 256 + splits * N * 4, (need, need_dw)
            ws = torch.empty(need // 4 + 64, device=DEV) if need else None
            b.linear_bwd(x, w, dy, None, dw, db, accumulate=acc, workspace=ws)
            torch.cuda.synchronize()
        finally:
            b.debug_set("cfg", -1)
            b.debug_set("vec1", 0)
            b.debug_set("splits", 0)
        base = prior.double().cpu().numpy() if acc else 0.0
        assert_close(to_f64(db), db_ref + base, Sb + (1 if acc else 0), what=f"db (acc={acc})")
        assert_close(to_f64(dw), dW_ref, SW, what="dW")


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
# (M x K) and dW (N x K); six K-stages of 32 in the product that is
# persistent, or one (the loaders move to the next tile at every stage).
# fp32 dW stays on the plain grid (the persistent one measured slower), so
# its case checks the plain grid against itself and the oracle
PERSIST_SHAPES = {"Y": (4352, 4096, 192), "dX": (4352, 192, 4096), "dW": (192, 4352, 4096),
                  "Y1": (4352, 4096, 32), "dX1": (4352, 32, 4096)}


@pytest.mark.parametrize("cfg", [6, 7])
@pytest.mark.parametrize("which", ["Y", "dX", "dW", "Y1", "dX1"])
def test_persistent_grid(cfg, which):
    """A product with more 256x256 tiles than CUs runs on a persistent grid
    (one block per CU, the first 16 blocks taking two tiles): every element
    against the oracle, and bit for bit against the plain grid, whose block
    for each tile sums in the same order."""
    M, N, K = PERSIST_SHAPES[which]
    inp = wl.linear(M, N, K, seed=43).make()
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
    assert_close(to_f64(got[out]), want, S, what=which + " (persistent grid)")
    if out == "dW":
        assert torch.equal(got["dW+db"], got["dW"])
        assert_close(to_f64(got["db"]), *oracle.linear_bwd_db(dY), what=which + " db (persistent grid)")


def test_persistent_grid_bitwise_at_8192_cubed():
    """The bench's products on the persistent grid (1024 tiles, four per
    block) equal the plain grid's bit for bit."""
    got, plain = _persist_on_off(wl.LINEAR_8192x8192x8192_F32.make())
    for k in got:
        assert not torch.isnan(got[k]).any(), k
        assert torch.equal(got[k], plain[k]), k
