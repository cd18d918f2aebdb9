"""The library's launches captured in a HIP graph (torch.cuda.CUDAGraph on
ROCm) and replayed: no allocation, copy or synchronisation happens inside a
call, so a captured step replays the same kernels. Every replay, with eager
work of the program in between, must equal the eager result bit for bit."""
import pytest
import torch

from paper_2602_00125_amd import workloads as wl

pytestmark = pytest.mark.gpu

from paper_2602_00125_amd import binding as b  # noqa: E402  (a missing library fails the module)
DEV = "cuda:0"


@pytest.mark.parametrize("M,N,K", [(64, 32, 128), (520, 392, 264), (256, 1024, 4096)])
def test_linear_step_replays_from_a_graph(M, N, K):
    w = wl.linear(M, N, K, dist={"X": ("normal",), "dY": ("normal",)})
    inp = w.make()
    x, wt, bias, dy = (inp[k].to(DEV) for k in ("X", "W", "b", "dY"))
    y, dx = torch.empty(M, N, device=DEV), torch.empty(M, K, device=DEV)
    dw, db = torch.empty(N, K, device=DEV), torch.empty(N, device=DEV)
    n = b.linear_bwd_workspace(x, wt, dy, dx, dw, db)
    ws = torch.empty(n // 4 + 64, device=DEV)

    def step():
        b.linear_fwd(x, wt, bias, y)
        b.linear_bwd(x, wt, dy, dx, dw, db, workspace=ws)

    step()
    torch.cuda.synchronize()
    eager = [t.clone() for t in (y, dx, dw, db)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(3):
        for t in (y, dx, dw, db):
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for got, want, name in zip((y, dx, dw, db), eager, ("y", "dx", "dw", "db")):
            assert torch.equal(got, want), f"replay {r}: {name}"
        # eager work of the program between replays, on the same buffers
        step()
        torch.cuda.synchronize()
        for got, want in zip((y, dx, dw, db), eager):
            assert torch.equal(got, want)


def test_convolution_step_replays_from_a_graph():
    """The gathered convolution products (forward and dx in stream-K order
    with their finish passes, dW split with its finish) captured and replayed."""
    from test_gpu_conv import make, to_dev
    case = (4, 64, 20, 20, 64, 3, 3, (1, 1), (1, 1), "cl", "cl")
    x, w, bias, dy = make(case, seed=61)
    N, C, H, W, CO, KH, KW, st, pd, wlay, xlay = case
    CL = torch.channels_last
    xd, wd, bd, dyd = to_dev(x, xlay), to_dev(w, wlay), bias.to(DEV), to_dev(dy, "cl")
    y = torch.empty(N, CO, H, W, device=DEV).contiguous(memory_format=CL)
    dx = torch.empty(N, C, H, W, device=DEV).contiguous(memory_format=CL)
    dw, db = torch.empty_like(wd), torch.empty(CO, device=DEV)
    try:
        b.debug_set("stream_k", 2)
        b.debug_set("sk_blocks", 13)
        need = max(b.conv2d_fwd_workspace(xd, wd, bd, y, st, pd),
                   b.conv2d_bwd_workspace(xd, wd, dyd, dx, dw, db, st, pd))
        ws = torch.empty(need // 4 + 64, device=DEV)

        def step():
            b.conv2d_fwd(xd, wd, bd, y, st, pd, workspace=ws)
            b.conv2d_bwd(xd, wd, dyd, dx, dw, db, st, pd, workspace=ws)

        step()
        torch.cuda.synchronize()
        eager = [t.clone() for t in (y, dx, dw, db)]
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
        for r in range(3):
            for t in (y, dx, dw, db):
                t.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            for got, want, name in zip((y, dx, dw, db), eager, ("y", "dx", "dw", "db")):
                assert torch.equal(got, want), f"replay {r}: {name}"
            step()
            torch.cuda.synchronize()
    finally:
        b.debug_set("sk_blocks", 0)
        b.debug_set("stream_k", 1)
