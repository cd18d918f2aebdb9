"""Plain fp64 oracle for the steps around the dense layer in a training loop.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
bench's CPU-baseline leg, never by the product path. It shares no code with
the HIP library and does not import it.

What it computes (MiniTensor paper):
  * Sec. 3.3, "Nonlinearities": ReLU, Sigmoid, Tanh and GELU and their
    derivatives (the ReLU derivative is the indicator of x > 0).
  * Sec. 3.3, Eq. (5) followed by a nonlinearity: H = act(X W^T + 1 b^T), and
    its pullback by the chain rule (Sec. 3.2, Eqs. (2)-(3)): the cotangent of
    the pre-activation is the upstream cotangent times act'(Z), elementwise
    (the Hadamard pullback of Sec. 3.2), and the bias cotangent is its column
    sum (the add pullback through the broadcast of Sec. 3.1).
  * Sec. 3.3, "Losses": mean squared error (1/N) sum_i (x_i - xhat_i)^2 and
    its gradient.
  * Sec. 3.3, "Optimizers": SGD with momentum and weight decay (Eq. (9)),
    Adam with debiased moments (Eq. (10)), RMSprop scaling the step by
    (v_t + eps)^(-1/2).
  * A two-layer perceptron step composed of the above and the dense-layer
    oracle (``oracle.linear_*``).

Every function takes and returns float64 numpy arrays and evaluates the
formula as written, elementwise, with no fusion or reordering beyond it.
Where a result feeds a tolerance, the function also returns the magnitude
scale that tolerance is stated against (documented per function).

The standard normal CDF of GELU uses ``scipy.special.erf`` as a library
primitive: Phi(z) = (1 + erf(z / sqrt 2)) / 2.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf as _erf

import oracle as _dense

# activation codes (same numbering as the library's MT_ACT_*)
NONE, RELU, SIGMOID, TANH, GELU = 0, 1, 2, 3, 4
ACTS = {"none": NONE, "relu": RELU, "sigmoid": SIGMOID, "tanh": TANH, "gelu": GELU}

_SQRT2 = math.sqrt(2.0)
_INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def normal_cdf(z):
    """Phi(z) = P(N(0,1) <= z) = (1 + erf(z / sqrt 2)) / 2."""
    return 0.5 * (1.0 + _erf(_f64(z) / _SQRT2))


def normal_pdf(z):
    """phi(z) = exp(-z^2 / 2) / sqrt(2 pi)."""
    z = _f64(z)
    return np.exp(-0.5 * z * z) * _INV_SQRT_2PI


def sigmoid(z):
    """1 / (1 + exp(-z)), written as exp(z) / (1 + exp(z)) for z < 0 so that
    exp never overflows."""
    z = _f64(z)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    e = np.exp(z[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def act(kind: int, z):
    """Sec. 3.3 nonlinearities, elementwise."""
    z = _f64(z)
    if kind == NONE:
        return z.copy()
    if kind == RELU:
        return np.where(z > 0, z, 0.0)
    if kind == SIGMOID:
        return sigmoid(z)
    if kind == TANH:
        return np.tanh(z)
    if kind == GELU:
        return z * normal_cdf(z)
    raise ValueError(f"unknown activation {kind}")


def act_grad(kind: int, z):
    """Derivative of act at z, elementwise (ReLU: the indicator of z > 0)."""
    z = _f64(z)
    if kind == NONE:
        return np.ones_like(z)
    if kind == RELU:
        return (z > 0).astype(np.float64)
    if kind == SIGMOID:
        s = sigmoid(z)
        return s * (1.0 - s)
    if kind == TANH:
        t = np.tanh(z)
        return 1.0 - t * t
    if kind == GELU:
        # d/dz [z Phi(z)] = Phi(z) + z phi(z)
        return normal_cdf(z) + z * normal_pdf(z)
    raise ValueError(f"unknown activation {kind}")


# ------------------------------------------------------ dense + activation --

def linear_act_fwd(X, W, b, kind: int):
    """H = act(Z), Z = X W^T + 1 b^T (Eq. (5) then a nonlinearity).

    Returns (Z, H, S) where S is the dense layer's sum |x_k w_k| + |b| of
    each pre-activation element (from ``oracle.linear_fwd``).
    """
    Z, S = _dense.linear_fwd(X, W, b)
    return Z, act(kind, Z), S


def act_bwd(kind: int, Z, dH):
    """Pullback of H = act(Z) with the bias column sum folded in.

    dZ = dH * act'(Z) (elementwise), db = sum over rows of dZ.
    Returns (dZ, db, S_db) with S_db[n] = sum_m |dZ[m, n]|.
    """
    Z, dH = _f64(Z), _f64(dH)
    assert Z.shape == dH.shape and Z.ndim == 2
    dZ = dH * act_grad(kind, Z)
    db = np.zeros(Z.shape[1])
    S = np.zeros(Z.shape[1])
    for m in range(Z.shape[0]):   # rows in ascending order
        db += dZ[m]
        S += np.abs(dZ[m])
    return dZ, db, S


# ------------------------------------------------------------------ loss --

def mse_loss(P, T):
    """L = (1/N) sum_i (P_i - T_i)^2 over all N elements, and dL/dP.

    Returns (L, dP, S) with S = L (every term is non-negative).
    """
    P, T = _f64(P), _f64(T)
    assert P.shape == T.shape
    N = P.size
    d = P - T
    L = float(np.sum(d * d)) / N if N else 0.0
    dP = 2.0 * d / N if N else d.copy()
    return L, dP, L


# ------------------------------------------------------------ optimizers --

def sgd_step(theta, g, v, lr, momentum, weight_decay):
    """Eq. (9): v_t = mu v_{t-1} + g_t + lambda theta_t; theta_{t+1} = theta_t - eta v_t.

    Returns (theta_new, v_new, S_theta, S_v): S_v = mu |v| + |g| + lambda |theta|,
    S_theta = |theta| + eta S_v (the magnitudes the rounding errors scale with).
    """
    theta, g, v = _f64(theta), _f64(g), _f64(v)
    v_new = momentum * v + g + weight_decay * theta
    theta_new = theta - lr * v_new
    S_v = abs(momentum) * np.abs(v) + np.abs(g) + abs(weight_decay) * np.abs(theta)
    S_theta = np.abs(theta) + abs(lr) * S_v
    return theta_new, v_new, S_theta, S_v


def adam_step(theta, g, m, v, lr, beta1, beta2, eps, t: int):
    """Eq. (10) at step t >= 1:

    m_t = b1 m + (1 - b1) g,  v_t = b2 v + (1 - b2) g^2,
    mhat = m_t / (1 - b1^t),  vhat = v_t / (1 - b2^t),
    theta_{t+1} = theta - eta mhat / (sqrt(vhat) + eps).

    Returns (theta_new, m_new, v_new, S_theta, S_m): S_m = b1 |m| + (1-b1) |g|,
    S_theta = |theta| + eta (S_m / (1 - b1^t)) / (sqrt(vhat) + eps); v_t is a
    sum of non-negative terms and is its own scale.
    """
    assert t >= 1
    theta, g, m, v = _f64(theta), _f64(g), _f64(m), _f64(v)
    m_new = beta1 * m + (1.0 - beta1) * g
    v_new = beta2 * v + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** t
    bc2 = 1.0 - beta2 ** t
    mhat = m_new / bc1
    vhat = v_new / bc2
    denom = np.sqrt(vhat) + eps
    theta_new = theta - lr * mhat / denom
    S_m = beta1 * np.abs(m) + (1.0 - beta1) * np.abs(g)
    S_theta = np.abs(theta) + abs(lr) * (S_m / bc1) / denom
    return theta_new, m_new, v_new, S_theta, S_m


def rmsprop_step(theta, g, v, lr, alpha, eps):
    """RMSprop as the paper states it: v_t = a v + (1 - a) g^2 (an exponential
    average of squared gradients) and theta_{t+1} = theta - eta g (v_t + eps)^(-1/2).

    Returns (theta_new, v_new, S_theta) with S_theta = |theta| + |eta g| (v_t + eps)^(-1/2).
    """
    theta, g, v = _f64(theta), _f64(g), _f64(v)
    v_new = alpha * v + (1.0 - alpha) * g * g
    scale = 1.0 / np.sqrt(v_new + eps)
    theta_new = theta - lr * g * scale
    S_theta = np.abs(theta) + np.abs(lr * g) * scale
    return theta_new, v_new, S_theta


# ------------------------------------------------- two-layer perceptron --

def mlp2_grads(X, W1, b1, W2, b2, T, kind: int):
    """One forward and backward pass of P = Dense2(act(Dense1(X))) under the
    mean squared error against T. Returns a dict with every intermediate:
    Z1, H1, P, loss, dP, dH1, dZ1, and the parameter gradients dW1, db1, dW2, db2.
    """
    Z1, H1, _ = linear_act_fwd(X, W1, b1, kind)
    P, _ = _dense.linear_fwd(H1, W2, b2)
    loss, dP, _ = mse_loss(P, T)
    dH1, _ = _dense.linear_bwd_dx(dP, W2)
    dW2, _ = _dense.linear_bwd_dw(dP, H1)
    db2, _ = _dense.linear_bwd_db(dP)
    dZ1, db1, _ = act_bwd(kind, Z1, dH1)
    dW1, _ = _dense.linear_bwd_dw(dZ1, X)
    return {"Z1": Z1, "H1": H1, "P": P, "loss": loss, "dP": dP, "dH1": dH1, "dZ1": dZ1,
            "dW1": dW1, "db1": db1, "dW2": dW2, "db2": db2}
