"""Plain fp64 CPU oracle for the dense layer and the broadcasting matmul.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, the smoke check and the
bench's CPU-baseline leg, never by the product path. It shares no code with
the HIP library (``paper_2602_00125_amd``) and does not import it.

The arithmetic lives in ``oracle.cpp`` (C++17, fp64 accumulation in ascending
order of the summed index, OpenMP over output rows only). This module only
builds/loads it and marshals numpy arrays. Every function returns the fp64
result and, per output element, ``S = sum |a_i b_i|`` over the products that
element sums (plus ``|b[n]|`` for the biased forward), which is what the
parity tolerances are scaled by.

Paper passages (MiniTensor): Sec. 3.1 Eq. (1) matmul and the broadcasting
rule; Sec. 3.2 Eq. (4) matmul pullbacks and the add pullback; Sec. 3.3
Eq. (5) dense layer; Sec. 3.3 Eq. (6) 2-D convolution and its pullbacks. bf16 inputs are widened bit-exactly (bits << 16 is the
fp32 value), see :func:`bf16_bits_to_f64`.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.cpp")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.POINTER(ctypes.c_int64)


def build() -> str:
    """Compile oracle.cpp into oracle/liboracle.so (g++, -O2, no fast-math)."""
    tmp = _LIB_PATH + ".tmp"
    cmd = ["g++", "-std=c++17", "-O2", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
           "-Wall", "-o", tmp, _SRC]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # a planted-mistake copy may be loaded instead by the oracle's own
    # mutation test (tests/test_oracle_mutants.py)
    path = os.environ.get("MT_ORACLE_LIB_OVERRIDE") or _LIB_PATH
    if path == _LIB_PATH and not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(path)
    i, i64, d = ctypes.c_int, ctypes.c_int64, _D
    lib.or_broadcast_shape.argtypes = [i, _I64, i, _I64, ctypes.POINTER(i), _I64]
    lib.or_matmul_shape.argtypes = [i, _I64, i, _I64, ctypes.POINTER(i), _I64]
    lib.or_linear_fwd.argtypes = [i64, i64, i64, d, d, d, d, d]
    lib.or_linear_bwd_dx.argtypes = [i64, i64, i64, d, d, d, d]
    lib.or_linear_bwd_dw.argtypes = [i64, i64, i64, d, d, d, d]
    lib.or_linear_bwd_db.argtypes = [i64, i64, d, d, d]
    for f in (lib.or_linear_fwd_at,):
        f.argtypes = [i64, i64, i64, d, d, d, i64, _I64, _I64, d, d]
    for f in (lib.or_linear_bwd_dx_at, lib.or_linear_bwd_dw_at):
        f.argtypes = [i64, i64, i64, d, d, i64, _I64, _I64, d, d]
    lib.or_matmul.argtypes = [i, _I64, d, i, _I64, d, d, d]
    lib.or_matmul_bwd.argtypes = [i, _I64, d, i, _I64, d, d, d, d, d, d]
    lib.or_reduce_broadcast.argtypes = [i, _I64, d, i, _I64, d, d]
    for f in (lib.or_broadcast_shape, lib.or_matmul_shape, lib.or_matmul, lib.or_matmul_bwd,
              lib.or_reduce_broadcast, lib.or_num_threads):
        f.restype = ctypes.c_int
    lib.or_conv2d_fwd.argtypes = [_I64, d, d, d, d, d]
    lib.or_conv2d_bwd_dx.argtypes = [_I64, d, d, d, d]
    lib.or_conv2d_bwd_dw.argtypes = [_I64, d, d, d, d]
    lib.or_conv2d_bwd_db.argtypes = [_I64, d, d, d]
    lib.or_conv2d_fwd_at.argtypes = [_I64, d, d, d, i64, _I64, d, d]
    lib.or_conv2d_bwd_dx_at.argtypes = [_I64, d, d, i64, _I64, d, d]
    lib.or_conv2d_bwd_dw_at.argtypes = [_I64, d, d, i64, _I64, d, d]
    _lib = lib
    return lib


def num_threads() -> int:
    """OpenMP threads the oracle uses (OMP_NUM_THREADS, else all cores)."""
    return int(_load().or_num_threads())


def _f64(x) -> np.ndarray:
    a = np.asarray(x, dtype=np.float64)   # keeps 0-d arrays 0-d
    return a if a.flags.c_contiguous else a.copy()


def _p(a: np.ndarray | None):
    if a is None:
        return None
    return a.ctypes.data_as(_D)


def _shape_arr(shape) -> np.ndarray:
    return np.ascontiguousarray(np.array(list(shape) + [0], dtype=np.int64))


def bf16_bits_to_f64(bits) -> np.ndarray:
    """bf16 bit patterns (uint16/int16) -> their exact values as fp64.

    A bf16 number is the upper half of an fp32 number: shifting its 16 bits
    left by 16 gives the fp32 bit pattern, which widens exactly to fp64.
    """
    b = np.asarray(bits).astype(np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


_SHAPE_ERRORS = {1: "bad rank", 2: "incompatible shapes"}


def broadcast_shape(a, b) -> tuple:
    """Broadcast of two shapes (Sec. 3.1); raises ValueError when invalid."""
    lib = _load()
    out = np.zeros(9, dtype=np.int64)
    n = ctypes.c_int(0)
    r = lib.or_broadcast_shape(len(a), _shape_arr(a).ctypes.data_as(_I64), len(b),
                               _shape_arr(b).ctypes.data_as(_I64), ctypes.byref(n),
                               out.ctypes.data_as(_I64))
    if r:
        raise ValueError(_SHAPE_ERRORS.get(r, str(r)))
    return tuple(int(v) for v in out[: n.value])


def matmul_shape(a, b) -> tuple:
    """Output shape of the broadcasting matmul; raises ValueError when invalid."""
    lib = _load()
    out = np.zeros(9, dtype=np.int64)
    n = ctypes.c_int(0)
    r = lib.or_matmul_shape(len(a), _shape_arr(a).ctypes.data_as(_I64), len(b),
                            _shape_arr(b).ctypes.data_as(_I64), ctypes.byref(n),
                            out.ctypes.data_as(_I64))
    if r:
        raise ValueError(_SHAPE_ERRORS.get(r, str(r)))
    return tuple(int(v) for v in out[: n.value])


# --------------------------------------------------------------- linear --

def linear_fwd(X, W, b=None):
    """Eq. (5): Y = X W^T + 1 b^T (b=None gives Eq. (1)). Returns (Y, S)."""
    X, W = _f64(X), _f64(W)
    M, K = X.shape
    N = W.shape[0]
    assert W.shape == (N, K)
    bb = None if b is None else _f64(b)
    if bb is not None:
        assert bb.shape == (N,)
    Y = np.empty((M, N))
    S = np.empty((M, N))
    _load().or_linear_fwd(M, N, K, _p(X), _p(W), _p(bb), _p(Y), _p(S))
    return Y, S


def linear_bwd_dx(dY, W):
    """Eq. (4): dX = dY W. Returns (dX, S)."""
    dY, W = _f64(dY), _f64(W)
    M, N = dY.shape
    K = W.shape[1]
    assert W.shape == (N, K)
    dX = np.empty((M, K))
    S = np.empty((M, K))
    _load().or_linear_bwd_dx(M, N, K, _p(dY), _p(W), _p(dX), _p(S))
    return dX, S


def linear_bwd_dw(dY, X):
    """Eq. (4): dW = dY^T X. Returns (dW, S)."""
    dY, X = _f64(dY), _f64(X)
    M, N = dY.shape
    K = X.shape[1]
    assert X.shape == (M, K)
    dW = np.empty((N, K))
    S = np.empty((N, K))
    _load().or_linear_bwd_dw(M, N, K, _p(dY), _p(X), _p(dW), _p(S))
    return dW, S


def linear_bwd_db(dY):
    """Add pullback through the broadcast bias: db = 1^T dY. Returns (db, S)."""
    dY = _f64(dY)
    M, N = dY.shape
    db = np.empty(N)
    S = np.empty(N)
    _load().or_linear_bwd_db(M, N, _p(dY), _p(db), _p(S))
    return db, S


def _idx(rows, cols):
    r = np.ascontiguousarray(rows, dtype=np.int64)
    c = np.ascontiguousarray(cols, dtype=np.int64)
    assert r.shape == c.shape and r.ndim == 1
    return r, c


def linear_fwd_at(X, W, b, rows, cols):
    """Y[rows[i], cols[i]] and its S, one sampled element at a time."""
    X, W = _f64(X), _f64(W)
    M, K = X.shape
    N = W.shape[0]
    r, c = _idx(rows, cols)
    assert (r >= 0).all() and (r < M).all() and (c >= 0).all() and (c < N).all()
    bb = None if b is None else _f64(b)
    out = np.empty(len(r))
    S = np.empty(len(r))
    _load().or_linear_fwd_at(M, N, K, _p(X), _p(W), _p(bb), len(r), r.ctypes.data_as(_I64),
                             c.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S


def linear_bwd_dx_at(dY, W, rows, cols):
    """dX[rows[i], cols[i]] (m, k) and its S."""
    dY, W = _f64(dY), _f64(W)
    M, N = dY.shape
    K = W.shape[1]
    r, c = _idx(rows, cols)
    assert (r >= 0).all() and (r < M).all() and (c >= 0).all() and (c < K).all()
    out = np.empty(len(r))
    S = np.empty(len(r))
    _load().or_linear_bwd_dx_at(M, N, K, _p(dY), _p(W), len(r), r.ctypes.data_as(_I64),
                                c.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S


def linear_bwd_dw_at(dY, X, rows, cols):
    """dW[rows[i], cols[i]] (n, k) and its S."""
    dY, X = _f64(dY), _f64(X)
    M, N = dY.shape
    K = X.shape[1]
    r, c = _idx(rows, cols)
    assert (r >= 0).all() and (r < N).all() and (c >= 0).all() and (c < K).all()
    out = np.empty(len(r))
    S = np.empty(len(r))
    _load().or_linear_bwd_dw_at(M, N, K, _p(dY), _p(X), len(r), r.ctypes.data_as(_I64),
                                c.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S


# ---------------------------------------------------- broadcasting matmul --

def matmul(A, B):
    """Broadcasting matmul (Eq. (1) per batch, Sec. 3.1 rules). Returns (C, S)."""
    A, B = _f64(A), _f64(B)
    shape = matmul_shape(A.shape, B.shape)
    C = np.empty(shape)
    S = np.empty(shape)
    r = _load().or_matmul(A.ndim, _shape_arr(A.shape).ctypes.data_as(_I64), _p(A), B.ndim,
                          _shape_arr(B.shape).ctypes.data_as(_I64), _p(B), _p(C), _p(S))
    if r:
        raise ValueError(_SHAPE_ERRORS.get(r, str(r)))
    return C, S


def matmul_bwd(A, B, dC, need_a=True, need_b=True):
    """Pullbacks of the broadcasting matmul, summed over broadcast batch axes.

    Returns (dA, SA, dB, SB); dA/SA (dB/SB) are None when not requested.
    """
    A, B, dC = _f64(A), _f64(B), _f64(dC)
    shape = matmul_shape(A.shape, B.shape)
    assert dC.shape == shape, (dC.shape, shape)
    dA = SA = dB = SB = None
    if need_a:
        dA, SA = np.empty(A.shape), np.empty(A.shape)
    if need_b:
        dB, SB = np.empty(B.shape), np.empty(B.shape)
    r = _load().or_matmul_bwd(A.ndim, _shape_arr(A.shape).ctypes.data_as(_I64), _p(A), B.ndim,
                              _shape_arr(B.shape).ctypes.data_as(_I64), _p(B), _p(dC), _p(dA),
                              _p(SA), _p(dB), _p(SB))
    if r:
        raise ValueError(_SHAPE_ERRORS.get(r, str(r)))
    return dA, SA, dB, SB


def reduce_broadcast(g_out, in_shape):
    """Sum a gradient over the axes along which ``in_shape`` was broadcast.

    Returns (g_in, S) with g_in of shape ``in_shape``.
    """
    g = _f64(g_out)
    in_shape = tuple(int(v) for v in in_shape)
    gin = np.empty(in_shape)
    S = np.empty(in_shape)
    r = _load().or_reduce_broadcast(g.ndim, _shape_arr(g.shape).ctypes.data_as(_I64), _p(g),
                                    len(in_shape), _shape_arr(in_shape).ctypes.data_as(_I64),
                                    _p(gin), _p(S))
    if r:
        raise ValueError(_SHAPE_ERRORS.get(r, str(r)))
    return gin, S


# ----------------------------------------------------------- convolution --
# Sec. 3.3 Eq. (6): 2-D convolution (cross-correlation as written there) with
# stride (sh, sw) and zero padding (ph, pw), batched; NCHW arrays, 0-based
# indices. Output size Ho = (H + 2 ph - KH) // sh + 1 (likewise Wo).

def conv2d_out_hw(H, W, KH, KW, stride, pad):
    sh, sw = stride
    ph, pw = pad
    return (H + 2 * ph - KH) // sh + 1, (W + 2 * pw - KW) // sw + 1


def _conv_dims(xshape, wshape, stride, pad):
    N, C, H, W = (int(v) for v in xshape)
    CO, C2, KH, KW = (int(v) for v in wshape)
    assert C2 == C, (xshape, wshape)
    sh, sw = (int(v) for v in stride)
    ph, pw = (int(v) for v in pad)
    assert sh >= 1 and sw >= 1 and ph >= 0 and pw >= 0
    HO, WO = conv2d_out_hw(H, W, KH, KW, stride, pad)
    assert HO >= 1 and WO >= 1
    dims = np.ascontiguousarray([N, C, H, W, CO, KH, KW, sh, sw, ph, pw], dtype=np.int64)
    return dims, (N, CO, HO, WO)


def conv2d_fwd(x, w, b, stride=(1, 1), pad=(0, 0)):
    """y = conv(x, w) + b per Eq. (6). Returns (y, S)."""
    x, w = _f64(x), _f64(w)
    bb = None if b is None else _f64(b)
    dims, yshape = _conv_dims(x.shape, w.shape, stride, pad)
    y, S = np.empty(yshape), np.empty(yshape)
    _load().or_conv2d_fwd(dims.ctypes.data_as(_I64), _p(x), _p(w), _p(bb), _p(y), _p(S))
    return y, S


def conv2d_bwd_dx(dy, w, xshape, stride=(1, 1), pad=(0, 0)):
    """Pullback to the input. Returns (dx, S)."""
    dy, w = _f64(dy), _f64(w)
    dims, yshape = _conv_dims(xshape, w.shape, stride, pad)
    assert dy.shape == yshape, (dy.shape, yshape)
    dx, S = np.empty(tuple(xshape)), np.empty(tuple(xshape))
    _load().or_conv2d_bwd_dx(dims.ctypes.data_as(_I64), _p(dy), _p(w), _p(dx), _p(S))
    return dx, S


def conv2d_bwd_dw(dy, x, wshape, stride=(1, 1), pad=(0, 0)):
    """Pullback to the weights. Returns (dw, S)."""
    dy, x = _f64(dy), _f64(x)
    dims, yshape = _conv_dims(x.shape, wshape, stride, pad)
    assert dy.shape == yshape, (dy.shape, yshape)
    dw, S = np.empty(tuple(wshape)), np.empty(tuple(wshape))
    _load().or_conv2d_bwd_dw(dims.ctypes.data_as(_I64), _p(dy), _p(x), _p(dw), _p(S))
    return dw, S


def conv2d_bwd_db(dy):
    """Pullback to the bias: sums over n, i, j. Returns (db, S)."""
    dy = _f64(dy)
    N, CO, HO, WO = dy.shape
    dims = np.ascontiguousarray([N, 1, 1, 1, CO, 1, 1, 1, 1, 0, 0], dtype=np.int64)
    # with H = W = 1, KH = KW = 1 the dims only serve N, CO; Ho, Wo come from dy
    dims[2], dims[3] = HO, WO
    db, S = np.empty(CO), np.empty(CO)
    _load().or_conv2d_bwd_db(dims.ctypes.data_as(_I64), _p(dy), _p(db), _p(S))
    return db, S


def _flat(idx):
    f = np.ascontiguousarray(idx, dtype=np.int64)
    assert f.ndim == 1
    return f


def conv2d_fwd_at(x, w, b, flat, stride=(1, 1), pad=(0, 0)):
    """y.flat[flat[t]] and its S, one sampled element at a time."""
    x, w = _f64(x), _f64(w)
    bb = None if b is None else _f64(b)
    dims, yshape = _conv_dims(x.shape, w.shape, stride, pad)
    f = _flat(flat)
    assert (f >= 0).all() and (f < np.prod(yshape)).all()
    out, S = np.empty(len(f)), np.empty(len(f))
    _load().or_conv2d_fwd_at(dims.ctypes.data_as(_I64), _p(x), _p(w), _p(bb), len(f),
                             f.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S


def conv2d_bwd_dx_at(dy, w, xshape, flat, stride=(1, 1), pad=(0, 0)):
    """dx.flat[flat[t]] and its S."""
    dy, w = _f64(dy), _f64(w)
    dims, yshape = _conv_dims(xshape, w.shape, stride, pad)
    assert dy.shape == yshape
    f = _flat(flat)
    assert (f >= 0).all() and (f < np.prod(xshape)).all()
    out, S = np.empty(len(f)), np.empty(len(f))
    _load().or_conv2d_bwd_dx_at(dims.ctypes.data_as(_I64), _p(dy), _p(w), len(f),
                                f.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S


def conv2d_bwd_dw_at(dy, x, wshape, flat, stride=(1, 1), pad=(0, 0)):
    """dw.flat[flat[t]] and its S."""
    dy, x = _f64(dy), _f64(x)
    dims, yshape = _conv_dims(x.shape, wshape, stride, pad)
    assert dy.shape == yshape
    f = _flat(flat)
    assert (f >= 0).all() and (f < np.prod(wshape)).all()
    out, S = np.empty(len(f)), np.empty(len(f))
    _load().or_conv2d_bwd_dw_at(dims.ctypes.data_as(_I64), _p(dy), _p(x), len(f),
                                f.ctypes.data_as(_I64), _p(out), _p(S))
    return out, S
