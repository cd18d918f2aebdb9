"""Shared test utilities: tolerance checks and host copies for the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle

# fp32 bar: |gpu - oracle| <= 1e-4 * S + 1e-6, S = sum |a_i b_i| of that output
F32_REL, F32_ABS = 1e-4, 1e-6


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact fp64 copy of a (device or host) fp32 / bf16 tensor."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return oracle.bf16_bits_to_f64(t.view(torch.int16).numpy())
    return t.numpy().astype(np.float64)


def assert_close(got, want, S, rel=F32_REL, abs_=F32_ABS, what=""):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    S = np.asarray(S, dtype=np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    if got.size == 0:
        return
    assert np.isfinite(got).all(), f"{what}: non-finite values in the GPU result"
    err = np.abs(got - want)
    bound = rel * S + abs_
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err - bound), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} elements out of tolerance; worst at "
                             f"{i}: got {got[i]!r} want {want[i]!r} err {err[i]:.3e} bound {bound[i]:.3e}")


def sample_positions(rows: int, cols: int, n_random: int, seed: int = 0, tile=256):
    """Tile-boundary rows/cols (+-1) crossed with each other, plus random pairs."""
    rng = np.random.default_rng(seed)

    def edges(n):
        e = {0, 1, n - 1, n - 2}
        for t in (32, 64, 128, tile):
            for k in range(t, n, t * max(1, n // (t * 8))):
                e.update((k - 1, k))
        return sorted(x for x in e if 0 <= x < n)

    er, ec = edges(rows), edges(cols)
    r = np.repeat(er, len(ec))
    c = np.tile(ec, len(er))
    r = np.concatenate([r, rng.integers(0, rows, n_random)])
    c = np.concatenate([c, rng.integers(0, cols, n_random)])
    return r.astype(np.int64), c.astype(np.int64)


def hip_runtime_loads() -> bool:
    """Whether the HIP runtime library can be loaded on this host (it can on
    any ROCm install, GPU or not; only then is the C-ABI library loadable)."""
    import ctypes

    try:
        ctypes.CDLL("libamdhip64.so")
        return True
    except OSError:
        return False


def load_binding():
    """The ctypes binding. Where the HIP runtime loads, a missing or broken
    library is an error (never a skip); without a HIP runtime the host-ABI
    checks are skipped."""
    import pytest

    if not hip_runtime_loads():
        pytest.skip("libamdhip64 does not load on this host", allow_module_level=True)
    from paper_2602_00125_amd import binding

    return binding
