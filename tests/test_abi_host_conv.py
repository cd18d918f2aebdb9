"""Host-side validation of the convolution entry points: bad arguments are
reported with the documented status before any HIP call, and the workspace
size is the unfolded input (plus split-K partials for dw). No case here
passes validation, so nothing is launched and no GPU is needed."""
import ctypes

import pytest

from helpers import load_binding

b = load_binding()

from test_abi_host import BF16, D, R  # noqa: E402


def cl(shape, ptr):
    N, C, H, W = shape
    return D(shape, ptr=ptr, stride=[H * W * C, 1, W * C, C])


def fwd(x, w, bias, y, st=(1, 1), pd=(1, 1), ws=None, nbytes=0):
    return b.lib.mt_conv2d_fwd(R(x), R(w), R(bias), R(y), st[0], st[1], pd[0], pd[1], ws, nbytes,
                               None)


def test_conv_fwd_validation():
    X = cl([2, 8, 9, 9], 0x100000)
    Wt = D([16, 8, 3, 3], ptr=0x200000)
    B = D([16], ptr=0x300000)
    Y = cl([2, 16, 9, 9], 0x400000)
    assert fwd(X, Wt, B, Y, st=(0, 1)) == 9                           # stride 0
    assert fwd(X, Wt, B, Y, pd=(-1, 0)) == 9                          # negative padding
    assert fwd(X, D([16, 7, 3, 3], ptr=0x200000), B, Y) == 3          # channel mismatch
    assert fwd(X, D([16, 8, 12, 3], ptr=0x200000), B, Y) == 3         # kernel > padded image
    assert fwd(X, Wt, B, cl([2, 16, 8, 9], 0x400000)) == 3            # wrong output size
    assert fwd(X, Wt, B, D([2, 16, 9, 9], ptr=0x400000)) == 5         # y not channels-last
    assert fwd(X, D([16, 8, 3, 3], ptr=0x200000, stride=[72, 1, 24, 16]), B, Y) == 5  # taps gapped
    assert fwd(X, D([16, 8, 3, 3], BF16, 0x200000), B, Y) == 4
    assert fwd(X, Wt, D([15], ptr=0x300000), Y) == 3
    assert fwd(X, Wt, B, cl([2, 16, 9, 9], 0x100000 + 64)) == 6       # y overlaps x
    assert fwd(X, Wt, B, Y) == 7                                      # no workspace
    n = ctypes.c_size_t(0)
    assert b.lib.mt_conv2d_fwd_workspace(R(X), R(Wt), R(B), R(Y), 1, 1, 1, 1, ctypes.byref(n)) == 0
    assert n.value == (2 * 9 * 9 * 72 * 4 + 255) // 256 * 256         # N Ho Wo x C KH KW floats
    # strided output, odd tap count: the unfolded rows are padded to 4 floats
    Wp = D([16, 3, 3, 3], ptr=0x200000)
    Xp = D([1, 3, 10, 10], ptr=0x100000)
    Yp = cl([1, 16, 5, 5], 0x400000)
    assert b.lib.mt_conv2d_fwd_workspace(R(Xp), R(Wp), None, R(Yp), 2, 2, 1, 1, ctypes.byref(n)) == 0
    assert n.value == (25 * 28 * 4 + 255) // 256 * 256


def bwd(x, w, dy, dx, dw, db, flags=0, ws=None, nbytes=0):
    return b.lib.mt_conv2d_bwd(R(x), R(w), R(dy), R(dx), R(dw), R(db), 1, 1, 1, 1, flags, ws,
                               nbytes, None)


def test_conv_bwd_validation():
    X = cl([2, 8, 9, 9], 0x100000)
    Wt = D([16, 8, 3, 3], ptr=0x200000)
    dY = cl([2, 16, 9, 9], 0x300000)
    dX = cl([2, 8, 9, 9], 0x400000)
    dW = D([16, 8, 3, 3], ptr=0x500000)
    dB = D([16], ptr=0x600000)
    assert bwd(X, Wt, dY, dX, dW, dB, flags=2) == 9
    assert bwd(X, Wt, D([2, 16, 9, 9], ptr=0x300000), dX, dW, dB) == 5          # dy not channels-last
    assert bwd(X, Wt, dY, D([2, 8, 9, 9], ptr=0x400000, stride=[1, 2, 3, 4]), dW, dB) == 5
    assert bwd(X, Wt, dY, dX, D([16, 8, 3, 3], ptr=0x500000, stride=[72, 1, 24, 8]), dB) == 5
    assert bwd(X, Wt, dY, cl([2, 8, 9, 8], 0x400000), dW, dB) == 3
    assert bwd(X, Wt, dY, dX, dW, D([17], ptr=0x600000)) == 3
    assert bwd(X, Wt, dY, cl([2, 8, 9, 9], 0x300000 + 16), dW, dB) == 6         # dx overlaps dy
    assert bwd(X, Wt, dY, dX, dW, dB) == 7                                      # no workspace
    n = ctypes.c_size_t(0)
    assert b.lib.mt_conv2d_bwd_workspace(R(X), R(Wt), R(dY), R(dX), R(dW), R(dB), 1, 1, 1, 1,
                                         ctypes.byref(n)) == 0
    assert n.value >= 2 * 9 * 9 * 72 * 4


def test_conv_gather_needs_no_unfolded_input():
    """Channels-last x and w with C a multiple of 32: the forward product and
    the weight gradient gather the image in their loads, so the forward needs
    no workspace and a backward without dx none for the unfolded input. Other
    layouts (or the gather switched off) keep the unfolded workspace (plus
    any split partials after it)."""
    X = cl([2, 32, 9, 9], 0x1000000)
    Wt = cl([16, 32, 3, 3], 0x2000000)
    B = D([16], ptr=0x3000000)
    Y = cl([2, 16, 9, 9], 0x4000000)
    col = (2 * 9 * 9 * 288 * 4 + 255) // 256 * 256
    n = ctypes.c_size_t(123)

    def fwd_ws(x, w):
        assert b.lib.mt_conv2d_fwd_workspace(R(x), R(w), R(B), R(Y), 1, 1, 1, 1, ctypes.byref(n)) == 0
        return n.value

    def bwd_ws(dx, dw, db):
        assert b.lib.mt_conv2d_bwd_workspace(R(X), R(Wt), R(Y), R(dx), R(dw), R(db), 1, 1, 1, 1,
                                             ctypes.byref(n)) == 0
        return n.value

    dX = cl([2, 32, 9, 9], 0x5000000)
    dW = cl([16, 32, 3, 3], 0x6000000)
    try:
        assert fwd_ws(X, Wt) == 0
        assert fwd(X, Wt, B, Y, st=(0, 1)) == 9        # still validated first
        assert fwd_ws(X, D([16, 32, 3, 3], ptr=0x2000000)) >= col   # [CO][C][KH][KW] weights
        assert fwd_ws(D([2, 32, 9, 9], ptr=0x1000000), Wt) >= col   # [N][C][H][W] input
        assert fwd_ws(cl([2, 32, 9, 9], 0x1000004), Wt) >= col      # x not 16-byte aligned
        assert bwd_ws(None, dW, None) < col                          # dW gathers: partials only
        assert bwd_ws(dX, dW, None) >= col                           # dU for dx (CO % 32 != 0)
        # CO a multiple of 32 and stride 1: dx gathers dy as well, no dU
        W32, dW32 = cl([32, 32, 3, 3], 0x2000000), cl([32, 32, 3, 3], 0x6000000)
        dY32 = cl([2, 32, 9, 9], 0x4000000)
        assert b.lib.mt_conv2d_bwd_workspace(R(X), R(W32), R(dY32), R(dX), R(dW32), None, 1, 1, 1, 1,
                                             ctypes.byref(n)) == 0
        assert n.value < col
        dY5 = cl([2, 32, 5, 5], 0x4000000)
        assert b.lib.mt_conv2d_bwd_workspace(R(X), R(W32), R(dY5), R(dX), R(dW32), None, 2, 2, 1, 1,
                                             ctypes.byref(n)) == 0
        assert n.value < (2 * 5 * 5 * 288 * 4 + 255) // 256 * 256   # stride 2: sub-pixel phases
        dY3 = cl([2, 32, 3, 3], 0x4000000)                           # stride 4 > 3x3 window
        assert b.lib.mt_conv2d_bwd_workspace(R(X), R(W32), R(dY3), R(dX), R(dW32), None, 4, 4, 1, 1,
                                             ctypes.byref(n)) == 0
        assert n.value >= (2 * 3 * 3 * 288 * 4 + 255) // 256 * 256  # a phase without taps: dU and the fold
        assert b.lib.mt_debug_set(b"conv_gather", 0) == 0
        assert fwd_ws(X, Wt) >= col
        assert bwd_ws(None, dW, None) >= col
    finally:
        b.lib.mt_debug_set(b"conv_gather", 1)
    assert b.lib.mt_debug_set(b"conv_gather", 2) == -2
