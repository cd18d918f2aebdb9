"""GPU parity of the training-step kernels around the dense layer against the
fp64 oracle (oracle/nn.py), through the C-ABI library:

* mt_linear_act_fwd: the dense layer with a nonlinearity fused into the
  product's epilogue (Sec. 3.3 Eq. (5) and "Nonlinearities");
* mt_act_bwd: dZ = dH act'(Z) with the bias column sum in the same pass;
* mt_mse_loss: mean squared error and its gradient;
* mt_sgd_step / mt_adam_step / mt_rmsprop_step (Eq. (9), Eq. (10), RMSprop);
* a two-layer perceptron trained for a few hundred steps whose loss falls.

Bars (derived from fp32 arithmetic, u = 2^-24):
* pre-activation Z: the dense-layer bar |gpu - oracle| <= 1e-4 S + 1e-6;
* H = act(Z): L (1e-4 S + 1e-6) + 1e-6 |Z| + 1e-7, where L bounds |act'|
  (ReLU, Tanh 1; Sigmoid 1/4; GELU 1.13) and the last two terms cover the
  few-ulp evaluation of act in fp32 (GELU: |error| <= ~8 u |z|);
* dZ: 2e-6 |dH| (act' in fp32 is within ~16 u of its value, whose size is at
  most 1.13; one more rounding for the product), plus 2^-8 |dZ| when dZ is
  stored as bf16 (round to nearest even);
* db: 1e-4 S_db + 2e-6 sum |dH| + 1e-6 (the dense-layer bar over the summed
  terms plus the error carried by each term);
* loss: 1e-4 S (S = the loss, all terms non-negative); dP: 1e-6 |dP|;
* optimizer outputs: 1e-6 times the scale the oracle returns for each
  (the sum of magnitudes of the terms; a handful of fp32 roundings).
Each step's oracle runs on the very inputs that step's kernel consumed, so
decisions (ReLU's z > 0) and roundings never differ between the two sides.
"""
import math

import numpy as np
import pytest
import torch

from oracle import nn as onn
import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, sample_positions, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"
LIP = {onn.NONE: 1.0, onn.RELU: 1.0, onn.SIGMOID: 0.25, onn.TANH: 1.0, onn.GELU: 1.13}
ACTS = [onn.NONE, onn.RELU, onn.SIGMOID, onn.TANH, onn.GELU]


def check_act_out(got_z, got_h, Z, S, kind, what):
    assert_close(got_z, Z, S, what=what + " Z")
    H = onn.act(kind, Z)
    bound_S = LIP[kind] * (1e-4 * S + 1e-6) + 1e-6 * np.abs(Z) + 1e-7
    assert_close(got_h, H, bound_S, rel=1.0, abs_=0.0, what=what + " H")


def run_act_fwd(inp, kind, with_z=True):
    x, w, bias = (inp[k].to(DEV) for k in ("X", "W", "b"))
    M, N = x.shape[0], w.shape[0]
    y = torch.full((M, N), float("nan"), device=DEV)
    z = torch.full((M, N), float("nan"), device=DEV) if with_z else None
    b.linear_act_fwd(x, w, bias, kind, y, z=z)
    torch.cuda.synchronize()
    return z, y


SMALL = [(64, 32, 128), (300, 200, 100), (257, 129, 67), (1, 1, 1), (33, 65, 4), (520, 392, 264)]


@pytest.mark.parametrize("kind", ACTS)
@pytest.mark.parametrize("M,N,K", SMALL)
def test_linear_act_fwd_small(kind, M, N, K):
    inp = wl.linear(M, N, K, seed=M + N + K, dist={"X": ("normal",), "b": ("uniform", 1.0)}).make()
    z, y = run_act_fwd(inp, kind)
    X, W, B = (to_f64(inp[k]) for k in ("X", "W", "b"))
    Z, S = oracle.linear_fwd(X, W, B)
    check_act_out(to_f64(z), to_f64(y), Z, S, kind, f"{M}x{N}x{K}")


@pytest.mark.parametrize("kind", [onn.RELU, onn.GELU])
def test_linear_act_fwd_without_z_and_bf16(kind):
    for dtype in ("f32", "bf16"):
        inp = wl.linear(300, 260, 200, dtype=dtype, seed=5, dist={"X": ("normal",)}).make()
        z0, y0 = run_act_fwd(inp, kind, with_z=True)
        _, y1 = run_act_fwd(inp, kind, with_z=False)
        assert torch.equal(y0, y1), "storing z must not change y"
        X, W, B = (to_f64(inp[k]) for k in ("X", "W", "b"))
        Z, S = oracle.linear_fwd(X, W, B)
        check_act_out(to_f64(z0), to_f64(y0), Z, S, kind, dtype)


@pytest.mark.parametrize("cfg", [6, 10, 3, 4])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_linear_act_fwd_every_epilogue_tile(cfg, dtype):
    inp = wl.linear(520, 392, 264, dtype=dtype, seed=cfg, dist={"X": ("normal",)}).make()
    b.debug_set("cfg", cfg)
    try:
        z, y = run_act_fwd(inp, onn.GELU)
    finally:
        b.debug_set("cfg", -1)
    X, W, B = (to_f64(inp[k]) for k in ("X", "W", "b"))
    Z, S = oracle.linear_fwd(X, W, B)
    check_act_out(to_f64(z), to_f64(y), Z, S, onn.GELU, f"cfg {cfg}")


def test_linear_act_fwd_unaligned_operands():
    # odd row pitch: the element-load tiles carry the epilogue
    inp = wl.linear(130, 70, 45, seed=3, dist={"X": ("normal",)}).make()
    x = torch.zeros(130, 47, device=DEV)[:, :45]
    x.copy_(inp["X"])
    w, bias = inp["W"].to(DEV), inp["b"].to(DEV)
    y = torch.full((130, 70), float("nan"), device=DEV)
    z = torch.full((130, 71), float("nan"), device=DEV)[:, :70]
    b.linear_act_fwd(x, w, bias, "tanh", y, z=z)
    torch.cuda.synchronize()
    Z, S = oracle.linear_fwd(to_f64(inp["X"]), to_f64(inp["W"]), to_f64(inp["b"]))
    check_act_out(to_f64(z), to_f64(y), Z, S, onn.TANH, "unaligned")


def test_linear_act_fwd_zero_k_is_act_of_bias():
    x = torch.empty(5, 0, device=DEV)
    w = torch.empty(8, 0, device=DEV)
    bias = torch.linspace(-2, 2, 8, device=DEV)
    y = torch.full((5, 8), float("nan"), device=DEV)
    z = torch.full((5, 8), float("nan"), device=DEV)
    b.linear_act_fwd(x, w, bias, "sigmoid", y, z=z)
    torch.cuda.synchronize()
    B = to_f64(bias)
    assert np.array_equal(to_f64(z), np.tile(B, (5, 1)))
    assert np.max(np.abs(to_f64(y) - onn.act(onn.SIGMOID, np.tile(B, (5, 1))))) < 1e-6


@pytest.mark.parametrize("kind", [onn.RELU, onn.GELU])
def test_linear_act_fwd_large_sampled(kind):
    # 4096 x 4096 outputs: the 256x256 DMA tile, in the launch bench uses
    M = N = 4096
    K = 1024
    inp = wl.linear(M, N, K, seed=11, dist={"X": ("normal",), "W": ("uniform", 1 / 32),
                                            "b": ("uniform", 1 / 32)}).make()
    z, y = run_act_fwd(inp, kind)
    X, W, B = (to_f64(inp[k]) for k in ("X", "W", "b"))
    r, c = sample_positions(M, N, 3000, seed=2)
    Zs, Ss = oracle.linear_fwd_at(X, W, B, r, c)
    check_act_out(to_f64(z)[r, c], to_f64(y)[r, c], Zs, Ss, kind, "4096^2 sampled")


# ------------------------------------------------------------- act_bwd --

def run_act_bwd(kind, Z, dH, dtype="f32", db=True, prior=None, use_ws=True):
    z = Z.to(DEV)
    dh = dH.to(DEV)
    if dtype == "bf16":
        dh = dh.to(torch.bfloat16)
    M, N = z.shape
    dz = torch.full((M, N), float("nan"), device=DEV, dtype=dh.dtype)
    dbt = torch.full((N,), float("nan"), device=DEV) if db else None
    if prior is not None:
        dz.copy_(prior[0])
        if dbt is not None:
            dbt.copy_(prior[1])
    ws = None
    if use_ws:
        n = b.act_bwd_workspace(kind, z, dh, dz, dbt)
        ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.act_bwd(kind, z, dh, dz, dbt, accumulate=prior is not None, workspace=ws)
    torch.cuda.synchronize()
    return dh, dz, dbt


def check_act_bwd(kind, Z, dh, dz, dbt, bf16_dz, prior=None):
    Zd, dHd = to_f64(Z), to_f64(dh)
    dZ, db, Sdb = onn.act_bwd(kind, Zd, dHd)
    if prior is not None:
        dZ = dZ + to_f64(prior[0])
        db = db + to_f64(prior[1])
        Sdb = Sdb + np.abs(to_f64(prior[1]))
    bound = 2e-6 * np.abs(dHd) + (2.0 ** -8 * np.abs(dZ) if bf16_dz else 0.0) + 1e-30
    if prior is not None:
        bound = bound + 1e-7 * np.abs(dZ)
    assert_close(to_f64(dz), dZ, bound, rel=1.0, abs_=0.0, what="dZ")
    if dbt is not None:
        extra = 2e-6 * np.abs(dHd).sum(axis=0)
        assert_close(to_f64(dbt), db, 1e-4 * Sdb + extra, rel=1.0, abs_=1e-6, what="db")


@pytest.mark.parametrize("kind", ACTS)
@pytest.mark.parametrize("M,N", [(300, 200), (257, 129), (1, 1), (2048, 516), (7, 4096)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_act_bwd(kind, M, N, dtype):
    Z = wl.tensor((M, N), ("normal",), seed=M) * 2.0
    Z[0, 0] = 0.0   # ReLU's derivative at exactly 0 is 0
    dH = wl.tensor((M, N), ("normal",), seed=N + 1)
    dh, dz, dbt = run_act_bwd(kind, Z, dH, dtype)
    check_act_bwd(kind, Z, dh, dz, dbt, dtype == "bf16")
    if kind == onn.RELU:
        assert to_f64(dz)[0, 0] == 0.0


def test_act_bwd_accumulate_no_db_no_workspace():
    Z = wl.tensor((513, 264), ("normal",), seed=1)
    dH = wl.tensor((513, 264), ("normal",), seed=2)
    prior = (wl.tensor((513, 264), ("normal",), seed=3).to(DEV),
             wl.tensor((264,), ("normal",), seed=4).to(DEV))
    dh, dz, dbt = run_act_bwd(onn.GELU, Z, dH, prior=prior, use_ws=False)
    check_act_bwd(onn.GELU, Z, dh, dz, dbt, False, prior=prior)
    dh, dz, dbt = run_act_bwd(onn.TANH, Z, dH, db=False)
    check_act_bwd(onn.TANH, Z, dh, dz, None, False)


def test_act_bwd_large_deterministic():
    M, N = 8192, 8192
    Z = wl.tensor((M, N), ("normal",), seed=21)
    dH = wl.tensor((M, N), ("normal",), seed=22)
    dh, dz, dbt = run_act_bwd(onn.GELU, Z, dH)
    again = run_act_bwd(onn.GELU, Z, dH)
    assert torch.equal(dz, again[1]) and torch.equal(dbt, again[2])
    # every db element in full; dZ on sampled rows
    rows = np.random.default_rng(0).integers(0, M, 64)
    Zd, dHd = to_f64(Z), to_f64(dH)
    dZ, db, Sdb = onn.act_bwd(onn.GELU, Zd, dHd)
    assert_close(to_f64(dbt), db, 1e-4 * Sdb + 2e-6 * np.abs(dHd).sum(axis=0), rel=1.0, abs_=1e-6,
                 what="db")
    got = to_f64(dz)[rows]
    assert_close(got, dZ[rows], 2e-6 * np.abs(dHd[rows]) + 1e-30, rel=1.0, abs_=0.0, what="dZ rows")


# ----------------------------------------------------------------- mse --

@pytest.mark.parametrize("shape", [(7,), (300, 200), (1000, 1001), (4096, 4096), (1,)])
def test_mse(shape):
    P = wl.tensor(shape, ("normal",), seed=1).to(DEV)
    T = wl.tensor(shape, ("normal",), seed=2).to(DEV)
    loss = torch.full((1,), float("nan"), device=DEV)
    dp = torch.full(shape, float("nan"), device=DEV)
    n = b.mse_loss_workspace(P, T)
    ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.mse_loss(P, T, loss, dp, workspace=ws)
    torch.cuda.synchronize()
    L, dP, S = onn.mse_loss(to_f64(P), to_f64(T))
    assert abs(loss.item() - L) <= 1e-4 * S, (loss.item(), L)
    assert_close(to_f64(dp), dP, 1e-6 * np.abs(dP) + 1e-38, rel=1.0, abs_=0.0, what="dP")
    # the same without workspace (one block) and with one output at a time
    loss2 = torch.full((1,), float("nan"), device=DEV)
    b.mse_loss(P, T, loss2, None)
    dp2 = torch.full(shape, float("nan"), device=DEV)
    b.mse_loss(P, T, None, dp2)
    torch.cuda.synchronize()
    assert abs(loss2.item() - L) <= 1e-4 * S
    assert torch.equal(dp, dp2)


def test_mse_empty():
    P = torch.empty(0, device=DEV)
    loss = torch.full((1,), float("nan"), device=DEV)
    b.mse_loss(P, P.clone(), loss, None)
    torch.cuda.synchronize()
    assert loss.item() == 0.0


# ---------------------------------------------------------- optimizers --

SHAPES = [(1,), (7,), (4096,), (300, 257), (1024, 1024), (0,), (5, 3)]


def f32(*xs):
    """The fp32 values the C ABI receives for float hyperparameters; the
    oracle takes the same numbers (e.g. 1 - beta is then exact on both sides)."""
    return [float(np.float32(x)) for x in xs]


def _tensors(seed, unaligned=False):
    out = []
    for i, s in enumerate(SHAPES):
        t = wl.tensor(s, ("normal",), seed=seed + i)
        if unaligned and t.numel() > 1:
            buf = torch.empty(t.numel() + 1, device=DEV)[1:].view(s)   # 4-byte aligned only
            buf.copy_(t)
            out.append(buf)
        else:
            out.append(t.to(DEV))
    return out


@pytest.mark.parametrize("unaligned", [False, True])
def test_sgd_steps(unaligned):
    ps, vs = _tensors(0, unaligned), [t.abs() * 0.1 for t in _tensors(50)]
    lr, mu, wd = f32(0.05, 0.9, 1e-2)
    for step in range(3):
        gs = _tensors(100 + step)
        before = [(to_f64(p), to_f64(g), to_f64(v)) for p, g, v in zip(ps, gs, vs)]
        b.sgd_step(ps, gs, vs, lr, mu, wd)
        torch.cuda.synchronize()
        for (p0, g0, v0), p, v in zip(before, ps, vs):
            th, vn, St, Sv = onn.sgd_step(p0, g0, v0, lr, mu, wd)
            assert_close(to_f64(v), vn, 1e-6 * Sv + 1e-38, rel=1.0, abs_=0.0, what="velocity")
            assert_close(to_f64(p), th, 1e-6 * St + 1e-38, rel=1.0, abs_=0.0, what="param")


@pytest.mark.parametrize("unaligned", [False, True])
def test_adam_steps(unaligned):
    ps = _tensors(0, unaligned)
    ms = [torch.zeros_like(p) for p in ps]
    vs = [torch.zeros_like(p) for p in ps]
    lr, b1, b2, eps = f32(1e-2, 0.9, 0.999, 1e-8)
    for t in range(1, 5):
        gs = _tensors(200 + t)
        before = [tuple(to_f64(x) for x in q) for q in zip(ps, gs, ms, vs)]
        b.adam_step(ps, gs, ms, vs, lr, b1, b2, eps, t)
        torch.cuda.synchronize()
        for (p0, g0, m0, v0), p, m, v in zip(before, ps, ms, vs):
            th, mn, vn, St, Sm = onn.adam_step(p0, g0, m0, v0, lr, b1, b2, eps, t)
            assert_close(to_f64(m), mn, 1e-6 * Sm + 1e-38, rel=1.0, abs_=0.0, what="m")
            assert_close(to_f64(v), vn, 1e-6 * vn + 1e-38, rel=1.0, abs_=0.0, what="v")
            assert_close(to_f64(p), th, 1e-6 * St + 1e-38, rel=1.0, abs_=0.0, what="param")


def test_rmsprop_steps():
    ps = _tensors(0)
    vs = [torch.zeros_like(p) for p in ps]
    lr, alpha, eps = f32(1e-2, 0.99, 1e-8)
    for step in range(3):
        gs = _tensors(300 + step)
        before = [tuple(to_f64(x) for x in q) for q in zip(ps, gs, vs)]
        b.rmsprop_step(ps, gs, vs, lr, alpha, eps)
        torch.cuda.synchronize()
        for (p0, g0, v0), p, v in zip(before, ps, vs):
            th, vn, St = onn.rmsprop_step(p0, g0, v0, lr, alpha, eps)
            assert_close(to_f64(v), vn, 1e-6 * vn + 1e-38, rel=1.0, abs_=0.0, what="v")
            assert_close(to_f64(p), th, 1e-6 * St + 1e-38, rel=1.0, abs_=0.0, what="param")


def test_optimizer_many_tensors_one_call():
    # 70 tensors: three launches of up to 32
    shapes = [(int(n),) for n in np.random.default_rng(5).integers(1, 5000, 70)]
    ps = [wl.tensor(s, ("normal",), seed=i).to(DEV) for i, s in enumerate(shapes)]
    gs = [wl.tensor(s, ("normal",), seed=100 + i).to(DEV) for i, s in enumerate(shapes)]
    vs = [torch.zeros_like(p) for p in ps]
    before = [(to_f64(p), to_f64(g)) for p, g in zip(ps, gs)]
    lr = f32(0.1)[0]
    b.sgd_step(ps, gs, vs, lr, 0.0, 0.0)
    torch.cuda.synchronize()
    for (p0, g0), p in zip(before, ps):
        th, _, St, _ = onn.sgd_step(p0, g0, np.zeros_like(p0), lr, 0.0, 0.0)
        assert_close(to_f64(p), th, 1e-6 * St + 1e-38, rel=1.0, abs_=0.0, what="param")


# ------------------------------------------------- two-layer perceptron --

def test_mlp2_step_parity_and_training_descends():
    """P = Dense2(GELU(Dense1(X))) under MSE against a teacher's outputs,
    trained with Adam entirely through the library; each stage of the first
    step is checked against the oracle on that stage's inputs, and the loss
    must fall by 10x over 300 steps."""
    M, D0, D1, D2 = 256, 64, 128, 16
    g = torch.Generator().manual_seed(0)
    X = torch.randn(M, D0, generator=g)
    T = torch.tanh(X @ (torch.randn(D0, D2, generator=g) / 8.0))
    a1, a2 = 1 / math.sqrt(D0), 1 / math.sqrt(D1)
    params = [(torch.rand(D1, D0, generator=g) * 2 - 1) * a1, torch.zeros(D1),
              (torch.rand(D2, D1, generator=g) * 2 - 1) * a2, torch.zeros(D2)]
    x, t = X.to(DEV), T.to(DEV)
    W1, b1, W2, b2 = [p.to(DEV) for p in params]
    z1 = torch.empty(M, D1, device=DEV)
    h1 = torch.empty(M, D1, device=DEV)
    pr = torch.empty(M, D2, device=DEV)
    loss = torch.empty(1, device=DEV)
    dp = torch.empty(M, D2, device=DEV)
    dh1 = torch.empty(M, D1, device=DEV)
    dz1 = torch.empty(M, D1, device=DEV)
    grads = [torch.empty_like(p) for p in (W1, b1, W2, b2)]
    ms = [torch.zeros_like(p) for p in (W1, b1, W2, b2)]
    vs = [torch.zeros_like(p) for p in (W1, b1, W2, b2)]
    first = None
    for step in range(1, 301):
        b.linear_act_fwd(x, W1, b1, "gelu", h1, z=z1)
        b.linear_fwd(h1, W2, b2, pr)
        b.mse_loss(pr, t, loss, dp)
        b.linear_bwd(h1, W2, dp, dh1, grads[2], grads[3])
        b.act_bwd("gelu", z1, dh1, dz1, grads[1])
        b.linear_bwd(x, W1, dz1, None, grads[0], None)
        if step == 1:
            torch.cuda.synchronize()
            Xd, W1d, b1d, W2d, b2d = (to_f64(v) for v in (x, W1, b1, W2, b2))
            Z, S = oracle.linear_fwd(Xd, W1d, b1d)
            check_act_out(to_f64(z1), to_f64(h1), Z, S, onn.GELU, "layer 1")
            P, SP = oracle.linear_fwd(to_f64(h1), W2d, b2d)
            assert_close(to_f64(pr), P, SP, what="layer 2")
            L, dP, SL = onn.mse_loss(to_f64(pr), T.double().numpy())
            assert abs(loss.item() - L) <= 1e-4 * SL
            assert_close(to_f64(dp), dP, 1e-6 * np.abs(dP) + 1e-38, rel=1.0, abs_=0.0, what="dP")
            dH, SH = oracle.linear_bwd_dx(to_f64(dp), W2d)
            assert_close(to_f64(dh1), dH, SH, what="dH1")
            dW2, SW2 = oracle.linear_bwd_dw(to_f64(dp), to_f64(h1))
            assert_close(to_f64(grads[2]), dW2, SW2, what="dW2")
            check_act_bwd(onn.GELU, z1, dh1, dz1, grads[1], False)
            dW1, SW1 = oracle.linear_bwd_dw(to_f64(dz1), Xd)
            assert_close(to_f64(grads[0]), dW1, SW1, what="dW1")
            first = loss.item()
        b.adam_step([W1, b1, W2, b2], grads, ms, vs, 1e-2, 0.9, 0.999, 1e-8, step)
        if step % 50 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    last = loss.item()
    assert math.isfinite(last) and last < 0.1 * first, (first, last)
