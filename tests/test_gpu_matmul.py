"""GPU parity of the broadcasting matmul (Eq. (1) per batch element with the
Sec. 3.1 broadcasting rule), its gradients summed over broadcast axes, and
the broadcast-gradient reduction, against the fp64 oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_00125_amd import workloads as wl

from helpers import assert_close, to_f64

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"


def gpu_matmul(a, c_shape, bb, accumulate=False, reduce_into=False, prior=None, use_ws=True):
    out = torch.full(c_shape, float("nan"), device=DEV)
    if prior is not None:
        out.copy_(prior)
    ws = None
    if use_ws:
        n = b.matmul_workspace(a, bb, out, accumulate=accumulate, reduce_into=reduce_into)
        ws = torch.empty(n // 4 + 64, device=DEV) if n else None
    b.matmul(a, bb, out, accumulate=accumulate, reduce_into=reduce_into, workspace=ws)
    torch.cuda.synchronize()
    return out


def bmm_grads_folded(A, B, dC, use_ws=True):
    """dA, dB by folding the broadcast-axis sums into the products."""
    dA = gpu_matmul(dC, A.shape, B.transpose(-1, -2), reduce_into=True, use_ws=use_ws)
    dB = gpu_matmul(A.transpose(-1, -2), B.shape, dC, reduce_into=True, use_ws=use_ws)
    return dA, dB


def test_bmm_broadcast_16x1x509x257_by_1x8x257x383():
    inp = wl.BMM_BCAST_16x1x509x257_1x8x257x383_F32.make()
    A, B, dC = (inp[k].to(DEV) for k in ("A", "B", "dC"))
    C = gpu_matmul(A, (16, 8, 509, 383), B)
    dA, dB = bmm_grads_folded(A, B, dC)
    An, Bn, dCn = (to_f64(inp[k]) for k in ("A", "B", "dC"))
    Cr, SC = oracle.matmul(An, Bn)
    assert_close(to_f64(C), Cr, SC, what="C")
    dAr, SA, dBr, SB = oracle.matmul_bwd(An, Bn, dCn)
    assert_close(to_f64(dA), dAr, SA, what="dA (folded)")
    assert_close(to_f64(dB), dBr, SB, what="dB (folded)")
    # materialised per-batch gradients, then the broadcast-gradient reduction
    dA_full = gpu_matmul(dC, (16, 8, 509, 257), B.transpose(-1, -2))
    dB_full = gpu_matmul(A.transpose(-1, -2), (16, 8, 257, 383), dC)
    dA2 = torch.full((16, 1, 509, 257), float("nan"), device=DEV)
    dB2 = torch.full((1, 8, 257, 383), float("nan"), device=DEV)
    for g, gi in ((dA_full, dA2), (dB_full, dB2)):
        n = b.reduce_broadcast_grad_workspace(g, gi)
        ws = torch.empty(n // 4 + 64, device=DEV) if n else None
        b.reduce_broadcast_grad(g, gi, workspace=ws)
    torch.cuda.synchronize()
    # the two-stage sum rounds the per-batch products first: S still bounds it
    assert_close(to_f64(dA2), dAr, SA, what="dA (materialised + reduce)")
    assert_close(to_f64(dB2), dBr, SB, what="dB (materialised + reduce)")
    # deterministic reruns
    dA_again, dB_again = bmm_grads_folded(A, B, dC)
    assert torch.equal(dA, dA_again) and torch.equal(dB, dB_again)
    # without workspace (no split-K): the same bar
    dA3, dB3 = bmm_grads_folded(A, B, dC, use_ws=False)
    assert_close(to_f64(dA3), dAr, SA, what="dA (folded, unsplit)")
    assert_close(to_f64(dB3), dBr, SB, what="dB (folded, unsplit)")
    # forced split counts, including splits that cut a summed batch index
    for splits in (2, 3, 7):
        b.debug_set("splits", splits)
        try:
            dA4, dB4 = bmm_grads_folded(A, B, dC)
        finally:
            b.debug_set("splits", 0)
        assert_close(to_f64(dA4), dAr, SA, what=f"dA (splits={splits})")
        assert_close(to_f64(dB4), dBr, SB, what=f"dB (splits={splits})")


def _rand_case(rng):
    """A random broadcasting matmul: shapes, optional transposed / expanded views."""
    nb = int(rng.integers(0, 3))
    batch = [int(rng.choice([1, 2, 3, 4])) for _ in range(nb)]
    M, K, N = (int(rng.choice([1, 3, 8, 31, 64, 97, 130])) for _ in range(3))
    abatch = [d if rng.random() < 0.6 else 1 for d in batch]
    bbatch = [d if rng.random() < 0.6 else 1 for d in batch]
    if nb and rng.random() < 0.3:
        abatch = abatch[int(rng.integers(0, nb)):]
    ashape = abatch + [M, K]
    bshape = bbatch + [K, N]
    if rng.random() < 0.1:
        ashape = [K]
    if rng.random() < 0.1:
        bshape = [K]
    return ashape, bshape


def _view(t, rng):
    """Same values, different strides: transposed storage and/or stride-0 expansion."""
    if t.dim() >= 2 and rng.random() < 0.4:
        t = t.transpose(-1, -2).contiguous().transpose(-1, -2)
    return t


@pytest.mark.parametrize("seed", range(40))
def test_bmm_random_broadcast_shapes(seed):
    rng = np.random.default_rng(seed)
    ashape, bshape = _rand_case(rng)
    A = wl.tensor(ashape, ("uniform", 1.0), seed=seed)
    B = wl.tensor(bshape, ("uniform", 1.0), seed=seed + 1000)
    cshape = oracle.matmul_shape(ashape, bshape)
    dC = wl.tensor(cshape, ("normal",), seed=seed + 2000)
    Ad, Bd = _view(A.to(DEV), rng), _view(B.to(DEV), rng)
    C = gpu_matmul(Ad, cshape, Bd)
    Cr, SC = oracle.matmul(A.double().numpy(), B.double().numpy())
    assert_close(to_f64(C), Cr, SC, what=f"C {ashape}@{bshape}")
    if len(ashape) >= 2 and len(bshape) >= 2:
        dA, dB = bmm_grads_folded(Ad, Bd, dC.to(DEV), use_ws=bool(seed % 2))
        dAr, SA, dBr, SB = oracle.matmul_bwd(A.double().numpy(), B.double().numpy(), dC.double().numpy())
        assert_close(to_f64(dA), dAr, SA, what="dA")
        assert_close(to_f64(dB), dBr, SB, what="dB")


def test_bmm_stride_zero_expanded_operand():
    base = wl.tensor((1, 37, 29), ("uniform", 1.0), seed=1)
    A = base.to(DEV).expand(6, 37, 29)          # stride 0 on a size-6 dim
    B = wl.tensor((6, 29, 41), ("uniform", 1.0), seed=2)
    C = gpu_matmul(A, (6, 37, 41), B.to(DEV))
    Cr, SC = oracle.matmul(base.expand(6, 37, 29).double().numpy(), B.double().numpy())
    assert_close(to_f64(C), Cr, SC, what="C")


def test_bmm_aligned_vector_path_and_accumulate():
    A = wl.tensor((4, 1, 64, 32), ("uniform", 1.0), seed=3).to(DEV)
    B = wl.tensor((1, 3, 32, 48), ("uniform", 1.0), seed=4).to(DEV)
    prior = torch.randn(4, 3, 64, 48, device=DEV)
    C = gpu_matmul(A, (4, 3, 64, 48), B, accumulate=True, prior=prior)
    Cr, SC = oracle.matmul(to_f64(A), to_f64(B))
    assert_close(to_f64(C), Cr + to_f64(prior), SC + 1, what="C+=")


def test_bmm_aligned_rows_with_wide_edge_tiles():
    """Aligned rows (pitches 260 and 384) on sizes where 256x256 tiles would
    cover 384 columns as 512: the products take the smaller tiles; all three
    against the oracle, the gradients summed over the broadcast axes."""
    A = wl.tensor((4, 1, 509, 260), ("uniform", 1.0), seed=5)
    B = wl.tensor((1, 8, 260, 384), ("uniform", 1.0), seed=6)
    dC = wl.tensor((4, 8, 509, 384), ("normal",), seed=7)
    Ad, Bd, dCd = A.to(DEV), B.to(DEV), dC.to(DEV)
    C = gpu_matmul(Ad, (4, 8, 509, 384), Bd)
    dA, dB = bmm_grads_folded(Ad, Bd, dCd)
    An, Bn, dCn = A.double().numpy(), B.double().numpy(), dC.double().numpy()
    Cr, SC = oracle.matmul(An, Bn)
    assert_close(to_f64(C), Cr, SC, what="C")
    dAr, SA, dBr, SB = oracle.matmul_bwd(An, Bn, dCn)
    assert_close(to_f64(dA), dAr, SA, what="dA")
    assert_close(to_f64(dB), dBr, SB, what="dB")


def test_bmm_empty_and_zero_k():
    A = torch.randn(3, 4, 0, device=DEV)
    B = torch.randn(0, 5, device=DEV)
    C = gpu_matmul(A, (3, 4, 5), B)
    assert torch.equal(C, torch.zeros(3, 4, 5, device=DEV))
    C0 = gpu_matmul(torch.randn(0, 4, 2, device=DEV), (0, 4, 5), torch.randn(2, 5, device=DEV))
    assert C0.numel() == 0


REDUCE_CASES = [
    ((16, 8, 509, 257), (16, 1, 509, 257), None),
    ((16, 8, 257, 383), (1, 8, 257, 383), None),
    ((16, 8, 257, 383), (8, 257, 383), None),
    ((64, 1000), (1000,), None),          # column sums (outer axis)
    ((1000, 64), (1000, 1), None),        # row sums (inner axis, DPP)
    ((7, 300, 5), (1, 300, 1), None),     # inner + outer together
    ((33, 17), (), None),                 # everything
    ((5, 6, 7), (5, 6, 7), None),         # nothing to sum
    ((16, 8, 5), (16, 1, 5), "transposed"),
    ((0, 4), (1, 4), None),
]


@pytest.mark.parametrize("oshape,ishape,layout", REDUCE_CASES)
@pytest.mark.parametrize("parts", [0, 3])
def test_reduce_broadcast_grad(oshape, ishape, layout, parts):
    g = wl.tensor(oshape, ("normal",), seed=len(oshape) * 100 + sum(oshape))
    gd = g.to(DEV)
    if layout == "transposed":
        gd = gd.transpose(0, 1).contiguous().transpose(0, 1)
    gi = torch.full(ishape, float("nan"), device=DEV)
    b.debug_set("parts", parts)
    try:
        n = b.reduce_broadcast_grad_workspace(gd, gi)
        ws = torch.empty(n // 4 + 64, device=DEV) if n else None
        b.reduce_broadcast_grad(gd, gi, workspace=ws)
        torch.cuda.synchronize()
    finally:
        b.debug_set("parts", 0)
    want, S = oracle.reduce_broadcast(g.double().numpy(), ishape)
    assert_close(to_f64(gi), want, S, what=f"{oshape}->{ishape}")


# the 256x96 tile (cfg 14) takes a K-contiguous B only, so only the nt layout
_STAGED_CASES = [(cfg, layout) for cfg in (6, 8, 9, 10, 13, 14, 15) for layout in ("nn", "tn", "nt")
                 if cfg != 14 or layout == "nt"]


@pytest.mark.parametrize("cfg,layout", _STAGED_CASES)
@pytest.mark.parametrize("acc", [False, True])
def test_bmm_odd_pitch_staged_epilogue(cfg, acc, layout):
    """Odd pitches run on the DMA tiles with 4-byte lanes and stage their
    output rows through LDS. Whole 32-row slabs take the straight-line store
    path (columns past N dropped by the buffer stores); slabs cut by the last
    row, and every accumulating product, take the per-row loop. C (+)= A B
    against the oracle, in each operand layout (tn: A an M-contiguous view;
    nt: B a K-contiguous view), on every DMA tile that serves odd pitches."""
    M, K, N = 301, 67, 389
    if layout == "tn":
        A = wl.tensor((2, 1, K, M), ("uniform", 1.0), seed=11).transpose(-1, -2)
    else:
        A = wl.tensor((2, 1, M, K), ("uniform", 1.0), seed=11)
    if layout == "nt":
        B = wl.tensor((1, 3, N, K), ("uniform", 1.0), seed=12).transpose(-1, -2)
    else:
        B = wl.tensor((1, 3, K, N), ("uniform", 1.0), seed=12)
    prior = torch.randn(2, 3, M, N) if acc else None
    b.debug_set("cfg", cfg)
    try:
        C = gpu_matmul(A.to(DEV), (2, 3, M, N), B.to(DEV), accumulate=acc,
                       prior=prior.to(DEV) if acc else None)
    finally:
        b.debug_set("cfg", -1)
    Cr, SC = oracle.matmul(A.double().numpy(), B.double().numpy())
    if acc:
        Cr, SC = Cr + prior.double().numpy(), SC + 1
    assert_close(to_f64(C), Cr, SC, what=f"C{'+' if acc else ''}= cfg {cfg} {layout}")
