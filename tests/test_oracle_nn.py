"""Pins of the fp64 oracle for activations, loss, optimizers and the
two-layer perceptron step (oracle/nn.py) against what the paper and
mathematics fix.

None of these compare the oracle with itself. Each check is a textbook value,
an identity, a closed form, a library routine (torch on the CPU in float64)
or central finite differences (Sec. 5, Eq. (11)).
"""
import importlib.util
import math
import os

import numpy as np
import pytest
import torch

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _load_nn():
    # a planted-mistake copy may stand in for the module (test_oracle_mutants.py)
    path = os.environ.get("MT_ORACLE_NN_OVERRIDE")
    if not path:
        from oracle import nn
        return nn
    spec = importlib.util.spec_from_file_location("oracle_nn_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


nn = _load_nn()
RNG = np.random.default_rng(4321)
ACT_KINDS = [nn.RELU, nn.SIGMOID, nn.TANH, nn.GELU]


def _central_diff(f, x, i, h):
    xp, xm = x.copy(), x.copy()
    xp.flat[i] += h
    xm.flat[i] -= h
    return (f(xp) - f(xm)) / (2 * h)


# ------------------------------------------------------------ activations --

def test_relu_values_and_indicator_derivative():
    z = np.array([-2.0, -1e-300, 0.0, 1e-300, 3.5])
    assert np.array_equal(nn.act(nn.RELU, z), [0.0, 0.0, 0.0, 1e-300, 3.5])
    # the paper's derivative: the indicator of z > 0 (0 at z = 0)
    assert np.array_equal(nn.act_grad(nn.RELU, z), [0.0, 0.0, 0.0, 1.0, 1.0])


def test_sigmoid_textbook_values_and_symmetry():
    assert nn.act(nn.SIGMOID, np.array([0.0]))[0] == 0.5
    # sigma(ln 3) = 3 / 4, sigma(-ln 3) = 1 / 4
    v = nn.act(nn.SIGMOID, np.array([math.log(3.0), -math.log(3.0)]))
    assert abs(v[0] - 0.75) < 1e-15 and abs(v[1] - 0.25) < 1e-15
    z = RNG.uniform(-30, 30, 1000)
    assert np.max(np.abs(nn.act(nn.SIGMOID, z) + nn.act(nn.SIGMOID, -z) - 1.0)) < 1e-15
    # no overflow in the far tails
    far = nn.act(nn.SIGMOID, np.array([-800.0, 800.0]))
    assert far[0] == 0.0 and far[1] == 1.0


def test_tanh_is_shifted_sigmoid():
    # tanh(z) = 2 sigma(2z) - 1 ties the two nonlinearities together
    z = RNG.uniform(-6, 6, 1000)
    got = nn.act(nn.TANH, z)
    want = 2.0 * nn.act(nn.SIGMOID, 2.0 * z) - 1.0
    assert np.max(np.abs(got - want)) < 1e-14
    assert abs(nn.act(nn.TANH, np.array([math.atanh(0.5)]))[0] - 0.5) < 1e-15


def test_gelu_textbook_quantiles_and_symmetry():
    # GELU(z) = z Phi(z); Phi at the standard normal quantiles of 0.95 and 0.975
    for z, p in ((1.6448536269514722, 0.95), (1.959963984540054, 0.975), (0.0, 0.5)):
        if z:
            assert abs(nn.act(nn.GELU, np.array([z]))[0] / z - p) < 1e-14
    assert nn.act_grad(nn.GELU, np.array([0.0]))[0] == 0.5
    # Phi(z) + Phi(-z) = 1  =>  GELU(z) - GELU(-z) = z
    z = RNG.uniform(-8, 8, 1000)
    assert np.max(np.abs(nn.act(nn.GELU, z) - nn.act(nn.GELU, -z) - z)) < 1e-14
    # large |z|: GELU(z) -> z for z -> +inf and -> 0 for z -> -inf
    big = nn.act(nn.GELU, np.array([40.0, -40.0]))
    assert big[0] == 40.0 and abs(big[1]) < 1e-300


def test_gelu_matches_torch_float64():
    z = torch.from_numpy(RNG.uniform(-7, 7, 4000))
    want = torch.nn.functional.gelu(z).numpy()
    assert np.max(np.abs(nn.act(nn.GELU, z.numpy()) - want)) < 1e-15
    zz = z.clone().requires_grad_(True)
    torch.nn.functional.gelu(zz).sum().backward()
    assert np.max(np.abs(nn.act_grad(nn.GELU, z.numpy()) - zz.grad.numpy())) < 1e-14


@pytest.mark.parametrize("kind", ACT_KINDS)
def test_activation_derivative_central_differences(kind):
    z = RNG.uniform(-4, 4, 200)
    z = z[np.abs(z) > 1e-3]   # keep away from the ReLU kink
    h = 1e-5
    fd = (nn.act(kind, z + h) - nn.act(kind, z - h)) / (2 * h)
    assert np.max(np.abs(fd - nn.act_grad(kind, z))) < 1e-8


def test_gelu_stationary_point():
    # GELU has one minimum; there Phi(z) + z phi(z) = 0 (z ~ -0.7518)
    lo, hi = -1.0, -0.5
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        if nn.act_grad(nn.GELU, np.array([mid]))[0] < 0:
            lo = mid   # still descending: the minimum lies to the right
        else:
            hi = mid
    z = 0.5 * (lo + hi)
    assert abs(z - (-0.7517916)) < 1e-6
    vals = nn.act(nn.GELU, np.linspace(-3, 3, 6001))
    assert abs(vals.min() - nn.act(nn.GELU, np.array([z]))[0]) < 1e-6


# ---------------------------------------------------- dense + activation --

@pytest.mark.parametrize("kind", ACT_KINDS)
def test_linear_act_gradients_central_differences(kind):
    M, N, K = 5, 4, 3
    X, W, b = RNG.uniform(-1, 1, (M, K)), RNG.uniform(-1, 1, (N, K)), RNG.uniform(-1, 1, N)
    G = RNG.uniform(-1, 1, (M, N))

    def L(X_, W_, b_):
        _, H, _ = nn.linear_act_fwd(X_, W_, b_, kind)
        return float(np.sum(G * H))

    Z, H, _ = nn.linear_act_fwd(X, W, b, kind)
    if kind == nn.RELU:
        assert np.min(np.abs(Z)) > 1e-4   # FD is valid away from the kink
    dZ, db, S = nn.act_bwd(kind, Z, G)
    dX, _ = oracle.linear_bwd_dx(dZ, W)
    dW, _ = oracle.linear_bwd_dw(dZ, X)
    h = 1e-6
    for i in range(X.size):
        assert abs(_central_diff(lambda v: L(v, W, b), X, i, h) - dX.flat[i]) < 1e-7
    for i in range(W.size):
        assert abs(_central_diff(lambda v: L(X, v, b), W, i, h) - dW.flat[i]) < 1e-7
    for i in range(N):
        assert abs(_central_diff(lambda v: L(X, W, v), b, i, h) - db[i]) < 1e-7
    assert np.allclose(S, np.abs(dZ).sum(axis=0), rtol=1e-15, atol=0)


def test_linear_act_relu_identity_weights():
    # W = I, b = 0: Z = X exactly and H = max(X, 0)
    X = RNG.uniform(-1, 1, (7, 6))
    Z, H, _ = nn.linear_act_fwd(X, np.eye(6), np.zeros(6), nn.RELU)
    assert np.array_equal(Z, X) and np.array_equal(H, np.maximum(X, 0.0))


# ------------------------------------------------------------------ loss --

def test_mse_by_hand():
    L, dP, S = nn.mse_loss(np.array([[1.0, 2.0, 3.0]]), np.zeros((1, 3)))
    assert L == 14.0 / 3.0 and S == L
    assert np.allclose(dP, [[2.0 / 3.0, 4.0 / 3.0, 2.0]], rtol=1e-15, atol=0)


def test_mse_gradient_central_differences_and_torch():
    P, T = RNG.normal(size=(4, 5)), RNG.normal(size=(4, 5))
    L, dP, _ = nn.mse_loss(P, T)
    for i in range(P.size):
        assert abs(_central_diff(lambda v: nn.mse_loss(v, T)[0], P, i, 1e-6) - dP.flat[i]) < 1e-9
    pt = torch.from_numpy(P).requires_grad_(True)
    lt = torch.nn.functional.mse_loss(pt, torch.from_numpy(T))
    lt.backward()
    assert abs(lt.item() - L) < 1e-15
    assert np.max(np.abs(pt.grad.numpy() - dP)) < 1e-16


# ------------------------------------------------------------ optimizers --

def test_sgd_constant_gradient_closed_form():
    # with lambda = 0 and a constant gradient, v_t = g (1 - mu^t) / (1 - mu)
    # and theta_t = theta_0 - eta g sum_{s<=t} (1 - mu^s) / (1 - mu)
    mu, eta = 0.9, 0.05
    theta0, g = RNG.normal(size=50), RNG.normal(size=50)
    theta, v = theta0.copy(), np.zeros(50)
    for t in range(1, 13):
        theta, v, _, _ = nn.sgd_step(theta, g, v, eta, mu, 0.0)
        assert np.allclose(v, g * (1 - mu ** t) / (1 - mu), rtol=1e-13, atol=0)
        coef = sum((1 - mu ** s) / (1 - mu) for s in range(1, t + 1))
        assert np.allclose(theta, theta0 - eta * g * coef, rtol=1e-12, atol=1e-14)


def test_sgd_matches_torch_optim_float64():
    theta0 = RNG.normal(size=(6, 7))
    grads = [RNG.normal(size=(6, 7)) for _ in range(6)]
    lr, mu, wd = 0.03, 0.8, 0.01
    p = torch.nn.Parameter(torch.from_numpy(theta0.copy()))
    opt = torch.optim.SGD([p], lr=lr, momentum=mu, weight_decay=wd)
    theta, v = theta0.copy(), np.zeros_like(theta0)
    for g in grads:
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        theta, v, S, _ = nn.sgd_step(theta, g, v, lr, mu, wd)
        assert np.max(np.abs(theta - p.detach().numpy())) < 1e-14
    assert (S >= np.abs(theta)).all()


def test_adam_constant_gradient_closed_form():
    # a constant gradient gives mhat_t = g and vhat_t = g^2 at every t, so each
    # step moves theta by eta g / (|g| + eps)
    eta, b1, b2, eps = 1e-2, 0.9, 0.999, 1e-8
    theta0, g = RNG.normal(size=40), RNG.normal(size=40)
    theta, m, v = theta0.copy(), np.zeros(40), np.zeros(40)
    for t in range(1, 9):
        theta, m, v, _, _ = nn.adam_step(theta, g, m, v, eta, b1, b2, eps, t)
        assert np.allclose(m, g * (1 - b1 ** t), rtol=1e-13, atol=0)
        assert np.allclose(v, g * g * (1 - b2 ** t), rtol=1e-12, atol=0)
        assert np.allclose(theta, theta0 - t * eta * g / (np.abs(g) + eps), rtol=1e-12, atol=1e-14)


def test_adam_matches_torch_optim_float64():
    theta0 = RNG.normal(size=(5, 9))
    grads = [RNG.normal(size=(5, 9)) for _ in range(7)]
    lr, b1, b2, eps = 3e-3, 0.85, 0.99, 1e-6
    p = torch.nn.Parameter(torch.from_numpy(theta0.copy()))
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps)
    theta, m, v = theta0.copy(), np.zeros_like(theta0), np.zeros_like(theta0)
    for t, g in enumerate(grads, start=1):
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        theta, m, v, _, _ = nn.adam_step(theta, g, m, v, lr, b1, b2, eps, t)
        assert np.max(np.abs(theta - p.detach().numpy())) < 1e-14


def test_rmsprop_constant_gradient_closed_form():
    # v_t = g^2 (1 - a^t); the step is eta g (v_t + eps)^(-1/2), eps inside the root
    eta, a, eps = 1e-2, 0.9, 1e-3
    theta0, g = RNG.normal(size=30), RNG.normal(size=30)
    theta, v = theta0.copy(), np.zeros(30)
    expect = theta0.copy()
    for t in range(1, 10):
        theta, v, _ = nn.rmsprop_step(theta, g, v, eta, a, eps)
        vt = g * g * (1 - a ** t)
        assert np.allclose(v, vt, rtol=1e-13, atol=0)
        expect = expect - eta * g / np.sqrt(vt + eps)
        assert np.allclose(theta, expect, rtol=1e-12, atol=1e-14)


def test_rmsprop_matches_torch_optim_without_eps():
    # torch adds eps outside the root; with eps = 0 the two forms coincide
    theta0 = RNG.normal(size=(4, 4))
    grads = [RNG.normal(size=(4, 4)) for _ in range(5)]
    p = torch.nn.Parameter(torch.from_numpy(theta0.copy()))
    opt = torch.optim.RMSprop([p], lr=1e-2, alpha=0.95, eps=0.0)
    theta, v = theta0.copy(), np.zeros_like(theta0)
    for g in grads:
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        theta, v, _ = nn.rmsprop_step(theta, g, v, 1e-2, 0.95, 0.0)
        assert np.max(np.abs(theta - p.detach().numpy())) < 1e-14


# ------------------------------------------------- two-layer perceptron --

@pytest.mark.parametrize("kind", [nn.GELU, nn.TANH])
def test_mlp2_gradients_central_differences(kind):
    X, T = RNG.normal(size=(6, 4)), RNG.normal(size=(6, 3))
    W1, b1 = RNG.uniform(-0.5, 0.5, (5, 4)), RNG.uniform(-0.5, 0.5, 5)
    W2, b2 = RNG.uniform(-0.5, 0.5, (3, 5)), RNG.uniform(-0.5, 0.5, 3)
    r = nn.mlp2_grads(X, W1, b1, W2, b2, T, kind)
    params = {"W1": W1, "b1": b1, "W2": W2, "b2": b2}

    def loss_with(name, val):
        q = dict(params, **{name: val})
        return nn.mlp2_grads(X, q["W1"], q["b1"], q["W2"], q["b2"], T, kind)["loss"]

    for name, val in params.items():
        for i in range(val.size):
            fd = _central_diff(lambda v: loss_with(name, v), val, i, 1e-6)
            assert abs(fd - r["d" + name].flat[i]) < 1e-8, (name, i)


def test_mlp2_matches_torch_autograd_float64():
    X, T = RNG.normal(size=(8, 6)), RNG.normal(size=(8, 2))
    ps = [RNG.uniform(-0.5, 0.5, s) for s in ((7, 6), (7,), (2, 7), (2,))]
    r = nn.mlp2_grads(X, *ps[:2], *ps[2:], T, nn.GELU)
    tp = [torch.from_numpy(p.copy()).requires_grad_(True) for p in ps]
    h = torch.nn.functional.gelu(torch.from_numpy(X) @ tp[0].T + tp[1])
    loss = torch.nn.functional.mse_loss(h @ tp[2].T + tp[3], torch.from_numpy(T))
    loss.backward()
    assert abs(loss.item() - r["loss"]) < 1e-15
    for name, t in zip(("dW1", "db1", "dW2", "db2"), tp):
        assert np.max(np.abs(t.grad.numpy() - r[name])) < 1e-14, name


def test_mlp2_training_descends():
    # a student of the teacher's shape fits the teacher's outputs with Adam
    rng = np.random.default_rng(7)
    X = rng.normal(size=(64, 8))
    T = np.tanh(X @ rng.normal(size=(8, 4)))
    W1, b1 = rng.uniform(-0.3, 0.3, (16, 8)), np.zeros(16)
    W2, b2 = rng.uniform(-0.3, 0.3, (4, 16)), np.zeros(4)
    params = [W1, b1, W2, b2]
    state = [(np.zeros_like(p), np.zeros_like(p)) for p in params]
    losses = []
    for t in range(1, 201):
        r = nn.mlp2_grads(X, *params, T, nn.GELU)
        losses.append(r["loss"])
        grads = [r["dW1"], r["db1"], r["dW2"], r["db2"]]
        new = [nn.adam_step(p, g, m, v, 1e-2, 0.9, 0.999, 1e-8, t)
               for p, g, (m, v) in zip(params, grads, state)]
        params = [n[0] for n in new]
        state = [(n[1], n[2]) for n in new]
    assert losses[-1] < 0.1 * losses[0]
