"""Host-side validation of the training-step entry points (dense layer with a
nonlinearity, its pullback, the loss and the optimizers): every bad argument
is reported with the documented status before any HIP call. No case here
passes validation, so nothing is ever launched and no GPU is needed."""
import ctypes

import pytest

from helpers import load_binding

b = load_binding()

from test_abi_host import BF16, D, F32, R  # noqa: E402


def act_fwd(x, w, bias, act, z, y):
    return b.lib.mt_linear_act_fwd(R(x), R(w), R(bias), act, R(z), R(y), None)


def test_linear_act_fwd_validation():
    X, W, B = D([8, 4], ptr=0x10000), D([6, 4], ptr=0x20000), D([6], ptr=0x30000)
    Z, Y = D([8, 6], ptr=0x40000), D([8, 6], ptr=0x50000)
    assert act_fwd(X, W, B, 5, Z, Y) == 9                         # unknown activation
    assert act_fwd(X, W, B, -1, Z, Y) == 9
    assert act_fwd(X, W, B, 4, D([8, 5], ptr=0x40000), Y) == 3     # z shape
    assert act_fwd(X, W, B, 4, D([8, 6], BF16, 0x40000), Y) == 4   # z must be f32
    assert act_fwd(X, W, B, 4, D([8, 6], ptr=0x50000 + 4), Y) == 6  # z overlaps y
    assert act_fwd(X, W, B, 4, D([8, 6], ptr=0x10000), Y) == 6     # z overlaps x
    assert act_fwd(X, W, B, 4, D([8, 6], ptr=0x40000, stride=[1, 8]), Y) == 5
    assert act_fwd(X, D([6, 5], ptr=0x20000), B, 1, Z, Y) == 3     # as mt_linear_fwd
    assert act_fwd(X, W, B, 1, Z, None) == 1


def act_bwd(act, z, dy, dz, db, flags=0):
    return b.lib.mt_act_bwd(act, R(z), R(dy), R(dz), R(db), flags, None, 0, None)


def test_act_bwd_validation():
    Z, dY, dZ, db = D([8, 6], ptr=0x10000), D([8, 6], ptr=0x20000), D([8, 6], ptr=0x30000), \
        D([6], ptr=0x40000)
    assert act_bwd(7, Z, dY, dZ, db) == 9
    assert act_bwd(4, Z, dY, dZ, db, flags=2) == 9                 # unknown flag
    assert act_bwd(4, None, dY, dZ, db) == 1
    assert act_bwd(4, Z, dY, D([8, 5], ptr=0x30000), db) == 3
    assert act_bwd(4, Z, D([7, 6], ptr=0x20000), dZ, db) == 3
    assert act_bwd(4, Z, dY, dZ, D([5], ptr=0x40000)) == 3
    assert act_bwd(4, D([8, 6], BF16, 0x10000), dY, dZ, db) == 4   # z must be f32
    assert act_bwd(4, Z, D([8, 6], BF16, 0x20000), dZ, db) == 4    # dz dtype must follow dy
    assert act_bwd(4, Z, dY, D([8, 6], ptr=0x20000 + 8), db) == 6  # dz overlaps dy
    assert act_bwd(4, Z, dY, dZ, D([6], ptr=0x30000 + 4)) == 6     # db overlaps dz
    assert act_bwd(4, Z, dY, D([8, 6], ptr=0x30000, stride=[1, 8]), db) == 5


def test_mse_validation():
    P, T = D([10, 3], ptr=0x10000), D([10, 3], ptr=0x20000)
    L, dP = D([1], ptr=0x30000), D([10, 3], ptr=0x40000)
    mse = lambda p, t, l, d: b.lib.mt_mse_loss(R(p), R(t), R(l), R(d), None, 0, None)
    assert mse(P, T, None, None) == 1                              # no output
    assert mse(P, D([10, 4], ptr=0x20000), L, dP) == 3
    assert mse(P, T, D([2], ptr=0x30000), dP) == 3                 # loss holds one value
    assert mse(P, T, L, D([30], ptr=0x40000)) == 3                 # dpred has pred's shape
    assert mse(P, T, L, D([10, 3], ptr=0x20000 + 4)) == 6          # dpred overlaps target
    assert mse(D([10, 3], BF16, 0x10000), T, L, dP) == 4
    assert mse(D([10, 3], ptr=0x10000, stride=[1, 10]), T, L, dP) == 5
    n = ctypes.c_size_t(0)
    assert b.lib.mt_mse_loss_workspace(R(D([4096, 4096], ptr=1 << 33)), R(D([4096, 4096], ptr=1 << 34)),
                                       ctypes.byref(n)) == 0
    assert n.value > 0


def _arr(ds):
    a = (b.MtTensor * len(ds))()
    for i, d in enumerate(ds):
        a[i] = d
    return a


def test_optimizer_validation():
    p = [D([4, 5], ptr=0x10000), D([7], ptr=0x20000)]
    g = [D([4, 5], ptr=0x30000), D([7], ptr=0x40000)]
    m = [D([4, 5], ptr=0x50000), D([7], ptr=0x60000)]
    v = [D([4, 5], ptr=0x70000), D([7], ptr=0x80000)]
    sgd = lambda pp, gg, vv, n=2, lr=0.1: b.lib.mt_sgd_step(n, _arr(pp), _arr(gg), _arr(vv), lr, 0.9,
                                                           0.0, None)
    assert sgd(p, g, m, n=-1) == 9
    assert sgd(p, g, m, lr=float("nan")) == 9
    assert sgd(p, [g[0], D([8], ptr=0x40000)], m) == 3                 # grad shape
    assert sgd(p, g, [m[0], D([7], ptr=0x10000 + 8)]) == 6             # state overlaps a param
    assert sgd(p, [g[0], D([7], ptr=0x50000 + 4)], m) == 6             # grad under a state
    assert sgd([p[0], D([7], BF16, 0x20000)], g, m) == 4
    assert sgd([D([4, 5], ptr=0x10000, stride=[1, 4]), p[1]], g, m) == 5
    adam = lambda step, b1=0.9, b2=0.999, eps=1e-8: b.lib.mt_adam_step(
        2, _arr(p), _arr(g), _arr(m), _arr(v), 1e-3, b1, b2, eps, step, None)
    assert adam(0) == 9                                                # steps count from 1
    assert adam(1, b1=1.0) == 9
    assert adam(1, b2=-0.1) == 9
    assert adam(1, eps=-1.0) == 9
    rms = lambda a, eps: b.lib.mt_rmsprop_step(2, _arr(p), _arr(g), _arr(m), 1e-3, a, eps, None)
    assert rms(1.5, 1e-8) == 9
    assert rms(0.9, float("inf")) == 9
    # no tensors: nothing to do, valid
    assert b.lib.mt_sgd_step(0, None, None, None, 0.1, 0.0, 0.0, None) == 0
