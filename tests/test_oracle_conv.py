"""Pins of the fp64 convolution oracle (Sec. 3.3 Eq. (6) and its pullbacks)
against what the paper and mathematics fix: torch float64 conv2d and its
autograd on the CPU (library routines), central finite differences (Sec. 5,
Eq. (11)), the identity kernel, the whole-image kernel that reduces Eq. (6)
to the dense layer of Eq. (5), a delta input, integer inputs summed exactly
in int64 by numpy, and the adjoint identity of a bilinear map."""
import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(99)

# (N, C, H, W, CO, KH, KW, stride, pad)
CASES = [(2, 3, 7, 6, 4, 3, 3, (1, 1), (1, 1)), (1, 2, 9, 9, 3, 3, 3, (2, 2), (1, 1)),
         (2, 4, 8, 5, 2, 1, 1, (1, 1), (0, 0)), (1, 3, 10, 7, 5, 5, 3, (2, 1), (2, 0)),
         (3, 1, 6, 6, 2, 2, 2, (2, 2), (0, 0)), (1, 2, 5, 5, 2, 3, 3, (3, 3), (2, 2))]


def _inputs(N, C, H, W, CO, KH, KW, stride, pad):
    x = RNG.uniform(-1, 1, (N, C, H, W))
    w = RNG.uniform(-1, 1, (CO, C, KH, KW))
    b = RNG.uniform(-1, 1, CO)
    HO, WO = oracle.conv2d_out_hw(H, W, KH, KW, stride, pad)
    dy = RNG.uniform(-1, 1, (N, CO, HO, WO))
    return x, w, b, dy


@pytest.mark.parametrize("case", CASES)
def test_conv_matches_torch_float64(case):
    N, C, H, W, CO, KH, KW, stride, pad = case
    x, w, b, dy = _inputs(*case)
    y, S = oracle.conv2d_fwd(x, w, b, stride, pad)
    tx, tw, tb = (torch.from_numpy(v.copy()).requires_grad_(True) for v in (x, w, b))
    ty = torch.nn.functional.conv2d(tx, tw, tb, stride=stride, padding=pad)
    assert ty.shape == y.shape
    assert np.max(np.abs(ty.detach().numpy() - y)) <= 1e-12 * np.max(S)
    ty.backward(torch.from_numpy(dy))
    dx, Sx = oracle.conv2d_bwd_dx(dy, w, x.shape, stride, pad)
    dw, Sw = oracle.conv2d_bwd_dw(dy, x, w.shape, stride, pad)
    db, Sb = oracle.conv2d_bwd_db(dy)
    assert np.max(np.abs(tx.grad.numpy() - dx)) <= 1e-12 * max(1.0, np.max(Sx))
    assert np.max(np.abs(tw.grad.numpy() - dw)) <= 1e-12 * max(1.0, np.max(Sw))
    assert np.max(np.abs(tb.grad.numpy() - db)) <= 1e-12 * max(1.0, np.max(Sb))
    # S is the sum of |terms|: at least |value|, and equal to it for all-positive inputs
    assert (S >= np.abs(y) - 1e-12).all() and (Sx >= np.abs(dx) - 1e-12).all()


def test_conv_S_of_positive_inputs_is_the_value():
    x, w, b, dy = (np.abs(v) for v in _inputs(*CASES[0]))
    y, S = oracle.conv2d_fwd(x, w, b, CASES[0][7], CASES[0][8])
    assert np.allclose(S, y, rtol=1e-14, atol=0)


@pytest.mark.parametrize("case", CASES[:3])
def test_conv_gradients_central_differences(case):
    N, C, H, W, CO, KH, KW, stride, pad = case
    x, w, b, G = _inputs(*case)

    def L(x_, w_, b_):
        return float(np.sum(G * oracle.conv2d_fwd(x_, w_, b_, stride, pad)[0]))

    dx, _ = oracle.conv2d_bwd_dx(G, w, x.shape, stride, pad)
    dw, _ = oracle.conv2d_bwd_dw(G, x, w.shape, stride, pad)
    db, _ = oracle.conv2d_bwd_db(G)
    h = 2.0 ** -10
    for arr, grad, f in ((x, dx, lambda v: L(v, w, b)), (w, dw, lambda v: L(x, v, b)),
                         (b, db, lambda v: L(x, w, v))):
        for i in RNG.choice(arr.size, size=min(arr.size, 25), replace=False):
            p, m = arr.copy(), arr.copy()
            p.flat[i] += h
            m.flat[i] -= h
            fd = (f(p) - f(m)) / (2 * h)
            assert abs(fd - grad.flat[i]) < 1e-9, (i, fd, grad.flat[i])


def test_identity_kernel_is_exact():
    x = RNG.uniform(-1, 1, (2, 4, 5, 6))
    w = np.eye(4).reshape(4, 4, 1, 1)
    y, _ = oracle.conv2d_fwd(x, w, None)
    assert np.array_equal(y, x)
    dy = RNG.uniform(-1, 1, x.shape)
    dx, _ = oracle.conv2d_bwd_dx(dy, w, x.shape)
    assert np.array_equal(dx, dy)


def test_whole_image_kernel_is_the_dense_layer():
    # KH = H, KW = W, no padding: one output pixel, y[n, co] = <w[co], x[n]> + b[co],
    # the dense layer of Eq. (5) on the flattened image; the same fp64 sum in the
    # same (c, u, v) order, so the two oracles agree bit for bit
    N, C, H, W, CO = 5, 3, 4, 6, 7
    x = RNG.uniform(-1, 1, (N, C, H, W))
    w = RNG.uniform(-1, 1, (CO, C, H, W))
    b = RNG.uniform(-1, 1, CO)
    y, S = oracle.conv2d_fwd(x, w, b)
    Y, SY = oracle.linear_fwd(x.reshape(N, -1), w.reshape(CO, -1), b)
    assert np.array_equal(y.reshape(N, CO), Y) and np.array_equal(S.reshape(N, CO), SY)
    dy = RNG.uniform(-1, 1, (N, CO, 1, 1))
    dw, _ = oracle.conv2d_bwd_dw(dy, x, w.shape)
    dW, _ = oracle.linear_bwd_dw(dy.reshape(N, CO), x.reshape(N, -1))
    assert np.array_equal(dw.reshape(CO, -1), dW)


def test_delta_input_places_the_kernel():
    # x = e at (c', h0, w0): y[0, co, i, j] = w[co, c', h0 - i s + p, w0 - j s + p] where in range
    C, H, W, CO, K, s, p = 2, 7, 7, 3, 3, 2, 1
    w = RNG.uniform(-1, 1, (CO, C, K, K))
    x = np.zeros((1, C, H, W))
    x[0, 1, 3, 4] = 1.0
    y, _ = oracle.conv2d_fwd(x, w, None, (s, s), (p, p))
    HO, WO = y.shape[2:]
    for co in range(CO):
        for i in range(HO):
            for j in range(WO):
                u, v = 3 - i * s + p, 4 - j * s + p
                want = w[co, 1, u, v] if 0 <= u < K and 0 <= v < K else 0.0
                assert y[0, co, i, j] == want


def test_integer_inputs_exact_against_int64():
    case = (2, 3, 8, 7, 4, 3, 3, (2, 1), (1, 2))
    N, C, H, W, CO, KH, KW, stride, pad = case
    xi = RNG.integers(-3, 4, (N, C, H, W))
    wi = RNG.integers(-3, 4, (CO, C, KH, KW))
    y, _ = oracle.conv2d_fwd(xi.astype(float), wi.astype(float), None, stride, pad)
    xp = np.pad(xi, ((0, 0), (0, 0), (pad[0], pad[0]), (pad[1], pad[1])))
    win = np.lib.stride_tricks.sliding_window_view(xp, (KH, KW), axis=(2, 3))
    win = win[:, :, ::stride[0], ::stride[1]][:, :, : y.shape[2], : y.shape[3]]
    want = np.einsum("nchwuv,ocuv->nohw", win, wi)   # int64 arithmetic: exact
    assert np.array_equal(y, want.astype(float))


def test_adjoint_identity():
    case = CASES[1]
    x, w, b, dy = _inputs(*case)
    y, _ = oracle.conv2d_fwd(x, w, None, case[7], case[8])
    dx, _ = oracle.conv2d_bwd_dx(dy, w, x.shape, case[7], case[8])
    dw, _ = oracle.conv2d_bwd_dw(dy, x, w.shape, case[7], case[8])
    a, bb, c = np.sum(dy * y), np.sum(dx * x), np.sum(dw * w)
    assert abs(a - bb) < 1e-12 * np.sum(np.abs(dy * y)) + 1e-12
    assert abs(a - c) < 1e-12 * np.sum(np.abs(dy * y)) + 1e-12


def test_sampled_equals_full_bit_exact():
    case = CASES[3]
    x, w, b, dy = _inputs(*case)
    st, pd = case[7], case[8]
    y, S = oracle.conv2d_fwd(x, w, b, st, pd)
    f = RNG.integers(0, y.size, 50)
    o, So = oracle.conv2d_fwd_at(x, w, b, f, st, pd)
    assert np.array_equal(o, y.flat[f]) and np.array_equal(So, S.flat[f])
    dx, Sx = oracle.conv2d_bwd_dx(dy, w, x.shape, st, pd)
    f = RNG.integers(0, dx.size, 50)
    assert np.array_equal(oracle.conv2d_bwd_dx_at(dy, w, x.shape, f, st, pd)[0], dx.flat[f])
    dw, Sw = oracle.conv2d_bwd_dw(dy, x, w.shape, st, pd)
    f = RNG.integers(0, dw.size, 50)
    assert np.array_equal(oracle.conv2d_bwd_dw_at(dy, x, w.shape, f, st, pd)[0], dw.flat[f])
