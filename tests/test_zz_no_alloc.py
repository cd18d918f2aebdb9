"""mt_linear_bwd_noalloc, the dense layer's backward without a caller
workspace (its split-K partials and db row-slice sums in the library's
scratch array), checked against mt_linear_bwd given a workspace of the
queried size: bit-identical on two calls in a row, the second smaller, both
also within the fp32 bar of the fp64 oracle. The host-only part checks that
sizes beyond the scratch maximum are refused before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from helpers import assert_close, load_binding, to_f64

b = load_binding()

DEV = "cuda:0"
FAKE = 1 << 32  # host-only cases: never dereferenced


def _inputs(M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(M, K, generator=g)
    w = (torch.rand(N, K, generator=g) * 2 - 1) / K ** 0.5
    dy = torch.randn(M, N, generator=g)
    return x, w, dy


def _outputs(M, N, K, prior=None):
    outs = [torch.full(s, float("nan"), device=DEV) for s in ((M, K), (N, K), (N,))]
    if prior is not None:
        for o, p in zip(outs, prior):
            o.copy_(p)
    return outs


@pytest.mark.gpu
def test_noalloc_bit_identical_to_workspace_entry_point_on_two_calls():
    cases = (((4096, 1024, 1024), 1), ((2048, 256, 520), 2))
    for (M, N, K), seed in cases:
        x, w, dy = (t.to(DEV) for t in _inputs(M, N, K, seed))
        ref = _outputs(M, N, K)
        need = b.linear_bwd_workspace(x, w, dy, *ref)
        assert 0 < need <= b.NOALLOC_SCRATCH_BYTES, need
        ws = torch.empty(need // 4 + 64, device=DEV)
        b.linear_bwd(x, w, dy, *ref, workspace=ws)
        got = _outputs(M, N, K)
        b.linear_bwd_noalloc(x, w, dy, *got)
        torch.cuda.synchronize()
        for name, g_, r_ in zip(("dX", "dW", "db"), got, ref):
            assert torch.equal(g_, r_), f"{M}x{N}x{K} {name}: noalloc differs from the workspace call"
        X, W, dY = (to_f64(t) for t in (x, w, dy))
        want = {"dX": oracle.linear_bwd_dx(dY, W), "dW": oracle.linear_bwd_dw(dY, X),
                "db": oracle.linear_bwd_db(dY)}
        for name, g_ in zip(("dX", "dW", "db"), got):
            assert_close(to_f64(g_), *want[name], what=f"{M}x{N}x{K} {name}")


@pytest.mark.gpu
def test_noalloc_accumulate_matches_workspace_entry_point():
    M, N, K = 2048, 256, 520
    x, w, dy = (t.to(DEV) for t in _inputs(M, N, K, 3))
    prior = [torch.randn(s, device=DEV) for s in ((M, K), (N, K), (N,))]
    ref = _outputs(M, N, K, prior)
    need = b.linear_bwd_workspace(x, w, dy, *ref)
    ws = torch.empty(need // 4 + 64, device=DEV)
    b.linear_bwd(x, w, dy, *ref, accumulate=True, workspace=ws)
    got = _outputs(M, N, K, prior)
    b.linear_bwd_noalloc(x, w, dy, *got, accumulate=True)
    torch.cuda.synchronize()
    for g_, r_ in zip(got, ref):
        assert torch.equal(g_, r_)


def _d(shape, ptr):
    stride, acc = [], 1
    for s in reversed(shape):
        stride.insert(0, acc)
        acc *= s
    return b.raw_desc(ptr, b.F32, shape, stride)


def _noalloc(x, w, dy, dx, dw, db, flags=0):
    R = lambda d: None if d is None else ctypes.byref(d)
    return b.lib.mt_linear_bwd_noalloc(R(x), R(w), R(dy), R(dx), R(dw), R(db), flags, None)


def test_noalloc_refuses_sizes_beyond_its_scratch_on_the_host():
    """A 65536 x 2048 x 2048 layer splits dW over four runs of 2048 x 2048
    partial floats (64 MiB): more than the scratch holds, so the call fails
    with MT_ERR_WORKSPACE before any HIP call (the pointers are fake)."""
    M, N, K = 65536, 2048, 2048
    x, w, dy = _d([M, K], FAKE), _d([N, K], 2 * FAKE), _d([M, N], 3 * FAKE)
    dx, dw, db = _d([M, K], 4 * FAKE), _d([N, K], 5 * FAKE), _d([N], 6 * FAKE)
    n = ctypes.c_size_t(0)
    R = ctypes.byref
    assert b.lib.mt_linear_bwd_workspace(R(x), R(w), R(dy), R(dx), R(dw), R(db), R(n)) == 0
    assert n.value > b.NOALLOC_SCRATCH_BYTES
    assert _noalloc(x, w, dy, dx, dw, db) == 7
    assert "scratch" in b.lib.mt_last_error().decode()
    # validation runs first, with mt_linear_bwd's statuses
    assert _noalloc(x, w, dy, dx, dw, db, flags=8) == 9
    assert _noalloc(x, w, None, dx, dw, db) == 1
    assert _noalloc(x, w, dy, _d([M, K + 1], 4 * FAKE), dw, db) == 3
