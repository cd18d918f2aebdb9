"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these compare the oracle with itself: each check is a closed form,
an invariant, an exact-arithmetic regime, a library routine (numpy, torch on
the CPU in float64) or central finite differences (Sec. 5, Eq. (11)).
"""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle

RNG = np.random.default_rng(1234)


def _rand(*shape):
    return RNG.uniform(-1, 1, size=shape)


# ---------------------------------------------------------------- golden --

def _read_golden(name):
    vals = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            key, rhs = line.split("=")
            rows = [[float(v) for v in r.split()] for r in rhs.split(";")]
            vals[key.strip()] = np.array(rows if len(rows) > 1 else rows[0])
    return vals


def test_golden_dense_by_hand():
    g = _read_golden("dense_bias_broadcast.txt")
    Y, _ = oracle.linear_fwd(g["X"], g["W"], g["b"])
    assert np.array_equal(Y, g["Y"])
    dX, _ = oracle.linear_bwd_dx(g["dY"], g["W"])
    assert np.array_equal(dX, g["dX"])
    dW, _ = oracle.linear_bwd_dw(g["dY"], g["X"])
    assert np.array_equal(dW, g["dW"])
    db, _ = oracle.linear_bwd_db(g["dY"])
    assert np.array_equal(db, g["db"])


# ---------------------------------------------------------------- shapes --

DIMS = (0, 1, 2, 3)


def _all_shapes(max_rank):
    for r in range(0, max_rank + 1):
        yield from itertools.product(DIMS, repeat=r)


def test_broadcast_shape_matches_numpy_exhaustive():
    shapes = list(_all_shapes(3))
    n = 0
    for a in shapes:
        for b in shapes:
            try:
                want = tuple(np.broadcast_shapes(a, b))
            except ValueError:
                want = None
            try:
                got = oracle.broadcast_shape(a, b)
            except ValueError:
                got = None
            assert got == want, (a, b, got, want)
            n += 1
    assert n == len(shapes) ** 2


def test_matmul_shape_matches_torch():
    shapes = [s for s in _all_shapes(4) if len(s) >= 1]
    rng = np.random.default_rng(7)
    pairs = [(shapes[i], shapes[j]) for i, j in rng.integers(0, len(shapes), size=(6000, 2))]
    # every (rank, rank) combination at least once with matching K
    for ra in range(1, 5):
        for rb in range(1, 5):
            pairs.append(((2,) * ra, (2,) * rb))
    for a, b in pairs:
        try:
            want = tuple(torch.matmul(torch.empty(a, dtype=torch.float64),
                                      torch.empty(b, dtype=torch.float64)).shape)
        except RuntimeError:
            want = None
        try:
            got = oracle.matmul_shape(a, b)
        except ValueError:
            got = None
        assert got == want, (a, b, got, want)


# ------------------------------------------------------------ linear pins --

def test_linear_matches_numpy_and_S_is_abs_product():
    M, N, K = 7, 5, 11  # all distinct: a transposed operand cannot pass
    X, W, b, dY = _rand(M, K), _rand(N, K), _rand(N), _rand(M, N)
    Y, S = oracle.linear_fwd(X, W, b)
    assert np.abs(Y - (X @ W.T + b)).max() <= 1e-12 * S.min()
    assert np.allclose(S, np.abs(X) @ np.abs(W).T + np.abs(b), rtol=1e-13, atol=0)
    Y0, S0 = oracle.linear_fwd(X, W, None)
    assert np.abs(Y0 - X @ W.T).max() <= 1e-12 * S0.min()
    dX, SX = oracle.linear_bwd_dx(dY, W)
    assert np.abs(dX - dY @ W).max() <= 1e-12 * SX.min()
    assert np.allclose(SX, np.abs(dY) @ np.abs(W), rtol=1e-13, atol=0)
    dW, SW = oracle.linear_bwd_dw(dY, X)
    assert np.abs(dW - dY.T @ X).max() <= 1e-12 * SW.min()
    assert np.allclose(SW, np.abs(dY).T @ np.abs(X), rtol=1e-13, atol=0)
    db, Sb = oracle.linear_bwd_db(dY)
    assert np.abs(db - dY.sum(0)).max() <= 1e-12 * Sb.min()
    assert np.allclose(Sb, np.abs(dY).sum(0), rtol=1e-13, atol=0)


def test_identity_and_permutation_bit_exact():
    M, K = 6, 9
    X, dY = _rand(M, K), _rand(M, K)
    I = np.eye(K)
    Y, _ = oracle.linear_fwd(X, I, np.zeros(K))
    assert np.array_equal(Y, X)
    dX, _ = oracle.linear_bwd_dx(dY, I)
    assert np.array_equal(dX, dY)
    # X = I (M = K): dW = dY^T X = dY^T
    dYs = _rand(K, 4)
    dW, _ = oracle.linear_bwd_dw(dYs, np.eye(K))
    assert np.array_equal(dW, dYs.T)
    perm = RNG.permutation(K)
    P = np.eye(K)[perm]          # row n of W is e_{perm[n]}
    Yp, _ = oracle.linear_fwd(X, P, None)
    assert np.array_equal(Yp, X[:, perm])
    dXp, _ = oracle.linear_bwd_dx(dY, P)   # dX[m,k] = dY[m, perm^-1[k]]
    inv = np.argsort(perm)
    assert np.array_equal(dXp, dY[:, inv])


def test_rank_one_closed_form():
    M, N, K = 5, 4, 8
    u, v, p, q, b = _rand(M), _rand(K), _rand(N), _rand(K), _rand(N)
    X, W = np.outer(u, v), np.outer(p, q)
    Y, S = oracle.linear_fwd(X, W, b)
    want = float(v @ q) * np.outer(u, p) + b
    assert np.abs(Y - want).max() <= 1e-12 * S.max()
    # dX = dY W with dY = r s^T: (s.p) r q^T ; dW = dY^T X = (r.u) s v^T
    r, s = _rand(M), _rand(N)
    dY = np.outer(r, s)
    dX, SX = oracle.linear_bwd_dx(dY, W)
    assert np.abs(dX - float(s @ p) * np.outer(r, q)).max() <= 1e-12 * SX.max()
    dW, SW = oracle.linear_bwd_dw(dY, X)
    assert np.abs(dW - float(r @ u) * np.outer(s, v)).max() <= 1e-12 * SW.max()


def test_ones_upstream():
    M, N, K = 13, 6, 4
    W = _rand(N, K)
    dY = np.ones((M, N))
    db, _ = oracle.linear_bwd_db(dY)
    assert np.array_equal(db, np.full(N, float(M)))
    dX, S = oracle.linear_bwd_dx(dY, W)
    assert np.abs(dX - W.sum(0)[None, :]).max() <= 1e-13 * S.max()


def test_integer_inputs_exact_against_int64():
    M, N, K = 37, 29, 53
    X = RNG.integers(-2, 3, size=(M, K))
    W = RNG.integers(-2, 3, size=(N, K))
    b = RNG.integers(-2, 3, size=N)
    dY = RNG.integers(-2, 3, size=(M, N))
    Y, _ = oracle.linear_fwd(X, W, b)
    assert np.array_equal(Y, (X @ W.T + b).astype(np.float64))
    dX, _ = oracle.linear_bwd_dx(dY, W)
    assert np.array_equal(dX, (dY @ W).astype(np.float64))
    dW, _ = oracle.linear_bwd_dw(dY, X)
    assert np.array_equal(dW, (dY.T @ X).astype(np.float64))
    db, _ = oracle.linear_bwd_db(dY)
    assert np.array_equal(db, dY.sum(0).astype(np.float64))


EPS = 2.0 ** -10


def _central_diff(loss, theta):
    g = np.empty_like(theta)
    for i in np.ndindex(theta.shape):
        tp, tm = theta.copy(), theta.copy()
        tp[i] += EPS
        tm[i] -= EPS
        g[i] = (loss(tp) - loss(tm)) / (2 * EPS)
    return g


def test_linear_gradients_match_central_differences():
    """Sec. 5 Eq. (11): L = <G, Dense(X; W, b)> is bilinear, so central
    differences equal the gradient up to rounding."""
    M, N, K = 3, 4, 5
    X, W, b, G = _rand(M, K), _rand(N, K), _rand(N), _rand(M, N)

    def L(X_, W_, b_):
        return float((G * oracle.linear_fwd(X_, W_, b_)[0]).sum())

    scale = np.abs(G).sum() * (np.abs(X).max() * np.abs(W).max() * K + 1)
    gx = _central_diff(lambda t: L(t, W, b), X)
    gw = _central_diff(lambda t: L(X, t, b), W)
    gb = _central_diff(lambda t: L(X, W, t), b)
    assert np.abs(oracle.linear_bwd_dx(G, W)[0] - gx).max() <= 1e-8 * scale
    assert np.abs(oracle.linear_bwd_dw(G, X)[0] - gw).max() <= 1e-8 * scale
    assert np.abs(oracle.linear_bwd_db(G)[0] - gb).max() <= 1e-8 * scale


def test_adjoint_identity():
    M, N, K = 17, 9, 12
    X, W, b, dY = _rand(M, K), _rand(N, K), _rand(N), _rand(M, N)
    Y, _ = oracle.linear_fwd(X, W, b)
    dX, _ = oracle.linear_bwd_dx(dY, W)
    dW, _ = oracle.linear_bwd_dw(dY, X)
    lhs = float((dY * (Y - b)).sum())
    assert abs(lhs - float((dX * X).sum())) <= 1e-12 * M * N * K
    assert abs(lhs - float((dW * W).sum())) <= 1e-12 * M * N * K


def test_sampled_equals_full_bit_exact():
    M, N, K = 23, 19, 31
    X, W, b, dY = _rand(M, K), _rand(N, K), _rand(N), _rand(M, N)
    Y, SY = oracle.linear_fwd(X, W, b)
    dX, SX = oracle.linear_bwd_dx(dY, W)
    dW, SW = oracle.linear_bwd_dw(dY, X)
    r, c = RNG.integers(0, M, 50), RNG.integers(0, N, 50)
    v, s = oracle.linear_fwd_at(X, W, b, r, c)
    assert np.array_equal(v, Y[r, c]) and np.array_equal(s, SY[r, c])
    r, c = RNG.integers(0, M, 50), RNG.integers(0, K, 50)
    v, s = oracle.linear_bwd_dx_at(dY, W, r, c)
    assert np.array_equal(v, dX[r, c]) and np.array_equal(s, SX[r, c])
    r, c = RNG.integers(0, N, 50), RNG.integers(0, K, 50)
    v, s = oracle.linear_bwd_dw_at(dY, X, r, c)
    assert np.array_equal(v, dW[r, c]) and np.array_equal(s, SW[r, c])


def test_zero_sizes():
    # K = 0: Y = b broadcast; M = 0: dW = 0 and db = 0; N = 0: empty
    b = _rand(3)
    Y, S = oracle.linear_fwd(np.zeros((4, 0)), np.zeros((3, 0)), b)
    assert np.array_equal(Y, np.tile(b, (4, 1)))
    assert np.array_equal(S, np.tile(np.abs(b), (4, 1)))
    dW, _ = oracle.linear_bwd_dw(np.zeros((0, 3)), np.zeros((0, 5)))
    assert dW.shape == (3, 5) and not dW.any()
    db, _ = oracle.linear_bwd_db(np.zeros((0, 3)))
    assert db.shape == (3,) and not db.any()
    Yn, _ = oracle.linear_fwd(np.zeros((4, 2)), np.zeros((0, 2)), np.zeros(0))
    assert Yn.shape == (4, 0)


# ---------------------------------------------------- broadcasting matmul --

MATMUL_SHAPES = [
    ((16, 1, 5, 7), (1, 8, 7, 3)),
    ((3, 1, 5, 4), (1, 2, 4, 3)),
    ((2, 3, 4), (4, 5)),
    ((4, 5), (2, 5, 3)),
    ((5,), (5,)),
    ((5,), (2, 5, 3)),
    ((2, 3, 4), (4,)),
    ((1, 1, 3, 2), (2, 2, 2)),
    ((2, 1, 3, 4), (3, 4, 2)),
    ((3, 0, 4), (4, 2)),
    ((3, 2, 0), (0, 2)),
]


@pytest.mark.parametrize("ashape,bshape", MATMUL_SHAPES)
def test_matmul_matches_numpy(ashape, bshape):
    A, B = _rand(*ashape), _rand(*bshape)
    C, S = oracle.matmul(A, B)
    want = np.matmul(A, B)
    assert C.shape == want.shape
    if C.size:
        assert np.abs(C - want).max() <= 1e-12 * max(S.max(), 1e-300)
        assert np.allclose(S, np.matmul(np.abs(A), np.abs(B)), rtol=1e-13, atol=0)


@pytest.mark.parametrize("ashape,bshape", MATMUL_SHAPES)
def test_matmul_bwd_matches_torch_autograd(ashape, bshape):
    A, B = _rand(*ashape), _rand(*bshape)
    cshape = oracle.matmul_shape(ashape, bshape)
    G = _rand(*cshape)
    ta = torch.tensor(A, requires_grad=True)
    tb = torch.tensor(B, requires_grad=True)
    torch.matmul(ta, tb).backward(torch.tensor(G))
    dA, SA, dB, SB = oracle.matmul_bwd(A, B, G)
    assert dA.shape == A.shape and dB.shape == B.shape
    if dA.size:
        assert np.abs(dA - ta.grad.numpy()).max() <= 1e-12 * max(SA.max(), 1.0)
    if dB.size:
        assert np.abs(dB - tb.grad.numpy()).max() <= 1e-12 * max(SB.max(), 1.0)


def test_matmul_gradients_match_central_differences_broadcast():
    """Eq. (11) on a tiny broadcast batch: pins the sum over broadcast axes."""
    ashape, bshape = (3, 1, 5, 4), (1, 2, 4, 3)
    A, B = _rand(*ashape), _rand(*bshape)
    G = _rand(*oracle.matmul_shape(ashape, bshape))

    def L(A_, B_):
        return float((G * oracle.matmul(A_, B_)[0]).sum())

    dA, _, dB, _ = oracle.matmul_bwd(A, B, G)
    scale = np.abs(G).sum() * 4 * 2
    assert np.abs(dA - _central_diff(lambda t: L(t, B), A)).max() <= 1e-8 * scale
    assert np.abs(dB - _central_diff(lambda t: L(A, t), B)).max() <= 1e-8 * scale


def test_matmul_integer_exact():
    A = RNG.integers(-2, 3, size=(4, 1, 9, 7))
    B = RNG.integers(-2, 3, size=(1, 3, 7, 5))
    G = RNG.integers(-2, 3, size=(4, 3, 9, 5))
    C, _ = oracle.matmul(A, B)
    assert np.array_equal(C, np.matmul(A, B).astype(np.float64))
    dA, _, dB, _ = oracle.matmul_bwd(A, B, G)
    wantA = np.matmul(G, np.swapaxes(B, -1, -2)).sum(axis=1, keepdims=True)
    wantB = np.matmul(np.swapaxes(A, -1, -2), G).sum(axis=0, keepdims=True)
    assert np.array_equal(dA, wantA.astype(np.float64))
    assert np.array_equal(dB, wantB.astype(np.float64))


@pytest.mark.parametrize("oshape,ishape", [
    ((16, 8, 5, 3), (16, 1, 5, 3)),
    ((16, 8, 5, 3), (1, 8, 5, 3)),
    ((16, 8, 5, 3), (8, 5, 3)),
    ((4, 6, 7), (6, 1)),
    ((4, 6, 7), (1, 1, 7)),
    ((4, 6, 7), ()),
    ((2, 3), (2, 3)),
    ((0, 3), (1, 3)),
])
def test_reduce_broadcast_matches_sum_to_size(oshape, ishape):
    g = _rand(*oshape)
    gin, S = oracle.reduce_broadcast(g, ishape)
    want = torch.tensor(g).sum_to_size(ishape).numpy() if len(oshape) else g
    assert gin.shape == tuple(ishape)
    assert np.abs(gin - want).max(initial=0.0) <= 1e-13 * max(S.max(initial=0.0), 1.0)
    wantS = torch.tensor(np.abs(g)).sum_to_size(ishape).numpy()
    assert np.allclose(S, wantS, rtol=1e-13, atol=0)


def test_reduce_broadcast_rejects_bad_target():
    with pytest.raises(ValueError):
        oracle.reduce_broadcast(np.zeros((4, 6)), (3, 6))
    with pytest.raises(ValueError):
        oracle.reduce_broadcast(np.zeros((4, 6)), (1, 4, 6))


def test_bf16_widening_all_bit_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.bf16_bits_to_f64(bits)
    want = torch.from_numpy(bits.astype(np.int32).astype(np.int16)).view(torch.bfloat16).to(
        torch.float64).numpy()
    assert np.array_equal(got, want, equal_nan=True)
