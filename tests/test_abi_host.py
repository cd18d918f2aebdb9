"""Host-side checks of libminitensor_hip: it loads, exports every declared
symbol, its shape bookkeeping is exact, and every validation error is
reported with the documented status before any HIP call (no GPU needed;
no case here passes validation, so nothing is ever launched)."""
import ctypes
import itertools
import os
import re

import numpy as np
import pytest

import oracle
from helpers import load_binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "minitensor_hip.h")

b = load_binding()


def test_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:mt_status|size_t|int|const char\*)\s+(mt_\w+)\s*\(", text, re.M))
    assert len(declared) >= 10
    for name in declared:
        assert hasattr(b.lib, name), name
    assert declared == set(b.EXPORTS)


DIMS = (0, 1, 2, 3)


def _shapes(max_rank):
    for r in range(0, max_rank + 1):
        yield from itertools.product(DIMS, repeat=r)


def test_broadcast_shape_bit_exact_vs_oracle_and_numpy():
    shapes = list(_shapes(3))
    for a in shapes:
        for c in shapes:
            try:
                want = tuple(np.broadcast_shapes(a, c))
            except ValueError:
                want = None
            try:
                o = oracle.broadcast_shape(a, c)
            except ValueError:
                o = None
            try:
                got = b.broadcast_shape(a, c)
            except b.MtError as e:
                assert e.status == 3
                got = None
            assert got == want == o, (a, c, got, want, o)


def test_matmul_shape_bit_exact_vs_oracle():
    shapes = [s for s in _shapes(4) if len(s) >= 1]
    rng = np.random.default_rng(3)
    pairs = [(shapes[i], shapes[j]) for i, j in rng.integers(0, len(shapes), size=(8000, 2))]
    pairs += [((16, 1, 509, 257), (1, 8, 257, 383)), ((5,), (5,)), ((7,), (3, 7, 2)), ((2, 3, 7), (7,))]
    for x, y in pairs:
        try:
            want = oracle.matmul_shape(x, y)
        except ValueError:
            want = None
        try:
            got = b.matmul_shape(x, y)
        except b.MtError as e:
            assert e.status in (2, 3)
            got = None
        assert got == want, (x, y, got, want)


FAKE = 0x10000  # never dereferenced: each case fails validation first
F32, BF16 = b.F32, b.BF16


def D(shape, dtype=F32, ptr=FAKE, stride=None):
    if stride is None:
        stride, acc = [], 1
        for s in reversed(shape):
            stride.insert(0, acc)
            acc *= s
    return b.raw_desc(ptr, dtype, shape, stride)


def R(d):
    return None if d is None else ctypes.byref(d)


def fwd(x, w, bias, y):
    return b.lib.mt_linear_fwd(R(x), R(w), R(bias), R(y), None)


def bwd(x, w, dy, dx, dw, db, flags=0):
    return b.lib.mt_linear_bwd(R(x), R(w), R(dy), R(dx), R(dw), R(db), flags, None, 0, None)


def test_linear_fwd_validation():
    X, W, B, Y = D([8, 4], ptr=0x10000), D([6, 4], ptr=0x20000), D([6], ptr=0x30000), D([8, 6], ptr=0x40000)
    assert fwd(None, W, B, Y) == 1
    assert fwd(D([8, 4], ptr=0), W, B, Y) == 1                 # null data
    assert fwd(D([8, 4, 1]), W, B, Y) == 2                      # rank
    assert fwd(X, D([6, 5], ptr=0x20000), B, Y) == 3            # K mismatch
    assert fwd(X, W, B, D([8, 7], ptr=0x40000)) == 3            # y shape
    assert fwd(X, W, D([5], ptr=0x30000), Y) == 3               # bias length
    assert fwd(X, D([6, 4], BF16, 0x20000), B, Y) == 4          # dtype mix
    assert fwd(X, W, B, D([8, 6], BF16, 0x40000)) == 4          # bf16 output
    assert fwd(D([8, 4], stride=[1, 8]), W, B, Y) == 5          # inner dim strided
    assert fwd(X, W, B, D([8, 6], ptr=0x10000 + 16)) == 6       # y overlaps x
    assert fwd(D([8, 4], stride=[-4, 1]), W, B, Y) == 5          # negative stride
    assert fwd(X, W, D([6], stride=[2], ptr=0x30000), Y) == 5   # strided bias
    assert b.lib.mt_last_error()


def test_linear_bwd_validation():
    X, W, dY = D([8, 4], ptr=0x10000), D([6, 4], ptr=0x20000), D([8, 6], ptr=0x30000)
    dX, dW, db = D([8, 4], ptr=0x40000), D([6, 4], ptr=0x50000), D([6], ptr=0x60000)
    assert bwd(X, W, None, dX, dW, db) == 1
    assert bwd(None, W, dY, dX, dW, db) == 1                    # dw needs x
    assert bwd(X, None, dY, dX, dW, db) == 1                    # dx needs w
    assert bwd(X, W, dY, D([8, 5], ptr=0x40000), dW, db) == 3
    assert bwd(X, W, dY, dX, D([4, 6], ptr=0x50000), db) == 3
    assert bwd(X, W, dY, dX, dW, D([8], ptr=0x60000)) == 3
    assert bwd(X, W, D([8, 6], BF16, 0x30000), dX, dW, db) == 4
    assert bwd(X, W, dY, dX, D([6, 4], ptr=0x40000 + 8), db) == 6   # outputs overlap
    assert bwd(X, W, dY, D([8, 4], ptr=0x30000), dW, db) == 6       # dx overlaps dy
    assert bwd(X, W, dY, dX, dW, db, flags=8) == 9                  # unknown flag


def test_matmul_validation():
    A, B_ = D([2, 3, 4], ptr=0x10000), D([4, 5], ptr=0x20000)
    mm = lambda a, c, out, fl=0: b.lib.mt_matmul(R(a), R(c), R(out), fl, None, 0, None)
    assert mm(A, B_, D([2, 3, 6], ptr=0x30000)) == 3                      # wrong N
    assert mm(A, D([5, 5], ptr=0x20000), D([2, 3, 5], ptr=0x30000)) == 3  # K mismatch
    assert mm(A, B_, D([3, 5], ptr=0x30000)) == 3                         # reduced without flag
    assert mm(A, B_, D([2, 3, 5], ptr=0x30000, stride=[15, 1, 3])) == 5   # c not row-major
    assert mm(D([2, 3, 4], stride=[24, 2, 6]), B_, D([2, 3, 5], ptr=0x30000)) == 5  # no unit stride
    assert mm(A, B_, D([2, 3, 5], ptr=0x20000 + 4)) == 6                  # c overlaps b
    assert mm(A, D([4, 5], BF16, 0x20000), D([2, 3, 5], ptr=0x30000)) == 4
    assert mm(A, B_, D([2, 3, 5], ptr=0x30000), 4) == 9
    assert mm(A, B_, None) == 1


def test_reduce_validation():
    G = D([4, 6, 5], ptr=0x10000)
    rd = lambda g, out, fl=0: b.lib.mt_reduce_broadcast_grad(R(g), R(out), fl, None, 0, None)
    assert rd(G, D([3, 1, 5], ptr=0x20000)) == 3
    assert rd(G, D([1, 4, 6, 5], ptr=0x20000)) == 2
    assert rd(G, D([6, 5], ptr=0x10000 + 8)) == 6
    assert rd(G, D([6, 5], BF16, 0x20000)) == 4
    assert rd(G, D([6, 5], ptr=0x20000), 2) == 9
    assert rd(G, D([6, 5], ptr=0x20000, stride=[1, 6])) == 5


def test_pitch_beyond_tile_offset_range_rejected():
    """Rows 2**25 floats apart: even the smallest tile (64 rows) would span
    2**33 bytes of offsets, beyond the kernels' 32-bit range, so every tile
    configuration rejects the call on the host with MT_ERR_LAYOUT."""
    G = 1 << 40  # fake, well-separated addresses; nothing is dereferenced
    x = b.raw_desc(G, F32, (300, 8), (1 << 25, 1))
    w = b.raw_desc(2 * G, F32, (300, 8), (8, 1))
    y = b.raw_desc(3 * G, F32, (300, 300), (300, 1))
    assert fwd(x, w, None, y) == 5
    assert "offset" in b.lib.mt_last_error().decode()


def test_empty_problems_need_no_gpu():
    # M == 0 or N == 0: valid, nothing to do, nothing launched
    assert fwd(D([0, 4], ptr=0), D([6, 4], ptr=0x20000), None, D([0, 6], ptr=0)) == 0
    # M == 0: dx is empty and db has no rows... but db would be zero-filled, so
    # only dx is requested here
    assert bwd(D([0, 4], ptr=0), D([6, 4]), D([0, 6], ptr=0), D([0, 4], ptr=0), None, None) == 0


def test_workspace_queries_are_host_only():
    n = ctypes.c_size_t(123)
    G = 1 << 32  # fake, well-separated addresses
    x, w, dy = D([4096, 1024], ptr=G), D([1024, 1024], ptr=2 * G), D([4096, 1024], ptr=3 * G)
    dx, dw, db = D([4096, 1024], ptr=4 * G), D([1024, 1024], ptr=5 * G), D([1024], ptr=6 * G)
    assert b.lib.mt_linear_bwd_workspace(R(x), R(w), R(dy), R(dx), R(dw), R(db), ctypes.byref(n)) == 0
    assert n.value % 4 == 0
    g, gi = D([16, 8, 509, 257], ptr=0x100000), D([16, 1, 509, 257], ptr=0x900000000)
    assert b.lib.mt_reduce_broadcast_grad_workspace(R(g), R(gi), ctypes.byref(n)) == 0


def test_debug_knobs_validate():
    assert b.lib.mt_debug_set(b"nope", 0) == -1
    for key, bad in (("cfg", -2), ("cfg", b.NUM_GEMM_CFG), ("vec1", 2), ("splits", -1), ("parts", 5000),
                     ("conv_gather", 2), ("stream_k", 3), ("sk_blocks", -1), ("phase_grid", 3),
                     ("persist", 2), ("persist", -1)):
        assert b.lib.mt_debug_set(key.encode(), bad) == -2, (key, bad)
    for key, ok in (("cfg", b.NUM_GEMM_CFG - 1), ("cfg", -1), ("vec1", 1), ("vec1", 0), ("splits", 7), ("splits", 0),
                    ("parts", 3), ("parts", 0), ("stream_k", 1), ("sk_blocks", 0), ("conv_gather", 1),
                    ("persist", 0), ("persist", 1)):
        assert b.lib.mt_debug_set(key.encode(), ok) == 0, (key, ok)


def test_status_strings():
    for code in range(10):
        assert b.status_str(code)


def test_generic_workspace_query_matches_the_per_op_ones():
    """mt_workspace_bytes gives the per-op *_workspace answer for each op it
    covers, and SIZE_MAX for an unknown op, a wrong count or bad tensors."""
    SIZE_MAX = ctypes.c_size_t(-1).value

    def ws(op, *ts):
        arr = (b._P * len(ts))(*[ctypes.pointer(t) if t is not None else b._P() for t in ts])
        return b.lib.mt_workspace_bytes(op, arr, len(ts))

    n = ctypes.c_size_t(0)
    X, W, dY = D([4096, 1024], ptr=0x100000), D([1024, 1024], ptr=0x20000000), D([4096, 1024], ptr=0x30000000)
    dX, dW, dB = D([4096, 1024], ptr=0x40000000), D([1024, 1024], ptr=0x50000000), D([1024], ptr=0x60000000)
    assert b.lib.mt_linear_bwd_workspace(R(X), R(W), R(dY), R(dX), R(dW), R(dB), ctypes.byref(n)) == 0
    assert n.value > 0 and ws(b.OP["linear_bwd"], X, W, dY, dX, dW, dB) == n.value
    assert ws(b.OP["linear_bwd"], X, W, dY, None, dW, None) >= 0
    assert ws(b.OP["linear_fwd"], X, W, dB, dY) == 0
    A = D([16, 1, 509, 257], ptr=0x100000)
    B = D([1, 8, 257, 383], ptr=0x10000000)
    C = D([16, 8, 509, 383], ptr=0x20000000)
    assert b.lib.mt_matmul_workspace(R(A), R(B), R(C), 0, ctypes.byref(n)) == 0
    assert ws(b.OP["matmul"], A, B, C) == n.value
    G, Gi = D([16, 8, 509, 257], ptr=0x100000), D([16, 1, 509, 257], ptr=0x900000000)
    assert b.lib.mt_reduce_broadcast_grad_workspace(R(G), R(Gi), ctypes.byref(n)) == 0
    assert ws(b.OP["reduce_broadcast_grad"], G, Gi) == n.value
    P, T = D([1024, 1024], ptr=0x100000), D([1024, 1024], ptr=0x10000000)
    assert b.lib.mt_mse_loss_workspace(R(P), R(T), ctypes.byref(n)) == 0
    assert ws(b.OP["mse_loss"], P, T) == n.value
    assert ws(99, P, T) == SIZE_MAX
    assert ws(b.OP["mse_loss"], P) == SIZE_MAX                      # wrong count
    assert ws(b.OP["matmul"], A, D([1, 8, 256, 383], ptr=0x10000000), C) == SIZE_MAX  # shape
    assert b.lib.mt_last_error()                                    # the reason is recorded


def test_planner_split_decisions():
    """The measured split-K rules, seen through the workspace queries (host
    only): the 4096 x 1024 x 1024 layer runs dX whole (one 128x128 tile per
    CU) and dW split four ways on the 64-deep 128x128 tile (4 x 1024 x 1024
    partial floats); 8192^3 needs no split; a 256-row layer splits dX four
    ways on the 8-wave 128x128 tile; db takes its row-slice partials."""
    n = ctypes.c_size_t(0)
    G = 1 << 32

    def need(M, N, K, which):
        x, w, dy = D([M, K], ptr=G), D([N, K], ptr=2 * G), D([M, N], ptr=3 * G)
        outs = {"dx": D([M, K], ptr=4 * G), "dw": D([N, K], ptr=5 * G), "db": D([N], ptr=6 * G)}
        args = [R(outs[k]) if k == which else None for k in ("dx", "dw", "db")]
        assert b.lib.mt_linear_bwd_workspace(R(x), R(w), R(dy), *args, ctypes.byref(n)) == 0
        return n.value

    assert need(4096, 1024, 1024, "dx") == 0
    assert need(4096, 1024, 1024, "dw") == 4 * 1024 * 1024 * 4
    assert need(4096, 1024, 1024, "db") == 16 * 1024 * 4
    # dw with db: db is summed inside the split dW product, one sum of the
    # 1024 columns per run after the (256-byte aligned) partial tiles
    x, w, dy = D([4096, 1024], ptr=G), D([1024, 1024], ptr=2 * G), D([4096, 1024], ptr=3 * G)
    assert b.lib.mt_linear_bwd_workspace(R(x), R(w), R(dy), None, R(D([1024, 1024], ptr=5 * G)),
                                         R(D([1024], ptr=6 * G)), ctypes.byref(n)) == 0
    assert n.value == 4 * 1024 * 1024 * 4 + 4 * 1024 * 4
    assert need(8192, 8192, 8192, "dx") == 0 and need(8192, 8192, 8192, "dw") == 0
    assert need(256, 1024, 4096, "dx") == 4 * 256 * 4096 * 4


def test_planner_broadcast_batch_tiles():
    """The odd-pitch tiles chosen for the 16x1x509x257 @ 1x8x257x383 products,
    seen through the workspace queries (host only): dA (509 x 257 outputs)
    covers its 257 columns with three 96-wide tiles, 2 x 3 x 16 = 96 tiles
    split five ways; dB (257 x 383 outputs) covers its 257 rows with five
    64-row tiles of 384 columns, 40 tiles split twelve ways; the forward
    (512 tiles of 256 x 192, two full rounds) needs no split."""
    G = 1 << 36
    n = ctypes.c_size_t(0)
    A, B, C = D([16, 1, 509, 257], ptr=G), D([1, 8, 257, 383], ptr=2 * G), D([16, 8, 509, 383], ptr=3 * G)
    dA, dB = D([16, 1, 509, 257], ptr=4 * G), D([1, 8, 257, 383], ptr=5 * G)
    Bt = D([1, 8, 383, 257], ptr=2 * G, stride=[8 * 257 * 383, 257 * 383, 1, 383])
    At = D([16, 1, 257, 509], ptr=G, stride=[509 * 257, 509 * 257, 1, 257])
    assert b.lib.mt_matmul_workspace(R(A), R(B), R(C), 0, ctypes.byref(n)) == 0 and n.value == 0
    assert b.lib.mt_matmul_workspace(R(C), R(Bt), R(dA), b.REDUCE_INTO, ctypes.byref(n)) == 0
    assert n.value == 5 * 16 * 509 * 257 * 4
    assert b.lib.mt_matmul_workspace(R(At), R(C), R(dB), b.REDUCE_INTO, ctypes.byref(n)) == 0
    assert n.value == 12 * 8 * 257 * 383 * 4
