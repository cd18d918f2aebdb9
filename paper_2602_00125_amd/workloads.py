"""Seeded synthetic inputs for the dense-layer and broadcasting-matmul workloads.

Shared by the tests, the bench and the smoke check; it holds no arithmetic of
the method (no products, sums or reductions), only the random draws. Every
draw uses a CPU ``torch.Generator`` seeded once per workload and takes the
tensors in the order they are listed. ``uniform(a)`` draws ``a * (2 U - 1)``
with U ~ U[0, 1) in fp32, ``normal`` draws N(0, 1) in fp32; bf16 tensors are
the fp32 draws rounded to nearest even. ``integers(lo, hi)`` draws integers in
[lo, hi] stored as floats (an exact-arithmetic regime: small integer products
summed below 2**24 are exact in any order).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch


def _draw(g: torch.Generator, shape, dist) -> torch.Tensor:
    kind = dist[0]
    if kind == "uniform":
        a = float(dist[1])
        return a * (2.0 * torch.rand(shape, generator=g, dtype=torch.float32) - 1.0)
    if kind == "normal":
        return torch.randn(shape, generator=g, dtype=torch.float32)
    if kind == "integers":
        lo, hi = int(dist[1]), int(dist[2])
        return torch.randint(lo, hi + 1, shape, generator=g).to(torch.float32)
    if kind == "zeros":
        return torch.zeros(shape, dtype=torch.float32)
    raise ValueError(f"unknown distribution {dist!r}")


@dataclass
class LinearWorkload:
    """Y = X W^T + b and its backward: X[M,K], W[N,K], b[N], dY[M,N].

    ``dtype`` is the storage type of X, W and dY ("f32" or "bf16"); b and every
    output are fp32.
    """
    name: str
    M: int
    N: int
    K: int
    dtype: str = "f32"
    dist: dict = field(default_factory=dict)
    seed: int = 0

    def flops(self) -> float:
        """Multiply-adds of the three products, counted as 2 flops each."""
        return 6.0 * self.M * self.N * self.K

    def make(self, seed: int | None = None) -> dict:
        g = torch.Generator("cpu")
        g.manual_seed(self.seed if seed is None else seed)
        shapes = {"X": (self.M, self.K), "W": (self.N, self.K), "b": (self.N,),
                  "dY": (self.M, self.N)}
        out = {}
        for name in ("X", "W", "b", "dY"):
            out[name] = _draw(g, shapes[name], self.dist.get(name, ("uniform", 1.0)))
        if self.dtype == "bf16":
            for name in ("X", "W", "dY"):
                out[name] = out[name].to(torch.bfloat16)
        elif self.dtype != "f32":
            raise ValueError(self.dtype)
        return out


@dataclass
class BmmWorkload:
    """C = A @ B with broadcast batch dims, and its backward from dC."""
    name: str
    ashape: tuple
    bshape: tuple
    cshape: tuple
    dist: dict = field(default_factory=dict)
    seed: int = 0

    def flops(self) -> float:
        """2*M*N*K per output batch element, for the forward and both grads."""
        M, K = self.ashape[-2], self.ashape[-1]
        N = self.bshape[-1]
        nb = math.prod(self.cshape[:-2])
        return 3 * 2.0 * nb * M * N * K

    def make(self, seed: int | None = None) -> dict:
        g = torch.Generator("cpu")
        g.manual_seed(self.seed if seed is None else seed)
        shapes = {"A": self.ashape, "B": self.bshape, "dC": self.cshape}
        return {n: _draw(g, shapes[n], self.dist.get(n, ("uniform", 1.0))) for n in ("A", "B", "dC")}


@dataclass
class MlpWorkload:
    """A two-layer perceptron training step: P = Dense2(act(Dense1(X))), the
    mean squared error against T, the backward pass and an Adam update of
    W1, b1, W2, b2. X[M,D0], W1[D1,D0], b1[D1], W2[D2,D1], b2[D2], T[M,D2],
    all fp32."""
    name: str
    M: int
    D0: int
    D1: int
    D2: int
    act: str = "gelu"
    dist: dict = field(default_factory=dict)
    seed: int = 0

    def flops(self) -> float:
        """Multiply-adds of the five products of a step (both forwards, dH1,
        dW2, dW1; the input layer's dX is not needed), 2 flops each."""
        return 2.0 * self.M * (2 * self.D0 * self.D1 + 3 * self.D1 * self.D2)

    def make(self, seed: int | None = None) -> dict:
        g = torch.Generator("cpu")
        g.manual_seed(self.seed if seed is None else seed)
        shapes = {"X": (self.M, self.D0), "W1": (self.D1, self.D0), "b1": (self.D1,),
                  "W2": (self.D2, self.D1), "b2": (self.D2,), "T": (self.M, self.D2)}
        return {n: _draw(g, shapes[n], self.dist.get(n, ("uniform", 1.0)))
                for n in ("X", "W1", "b1", "W2", "b2", "T")}


@dataclass
class ConvWorkload:
    """2-D convolution forward and backward: x[N,C,H,W], w[CO,C,KH,KW], b[CO],
    dy[N,CO,Ho,Wo], fp32, stride and zero padding; drawn in that order."""
    name: str
    N: int
    C: int
    H: int
    W: int
    CO: int
    KH: int
    KW: int
    stride: tuple = (1, 1)
    pad: tuple = (0, 0)
    dist: dict = field(default_factory=dict)
    seed: int = 0

    def out_hw(self):
        return ((self.H + 2 * self.pad[0] - self.KH) // self.stride[0] + 1,
                (self.W + 2 * self.pad[1] - self.KW) // self.stride[1] + 1)

    def flops(self) -> float:
        """Multiply-adds of the three products (forward, dW, dX), 2 flops each."""
        HO, WO = self.out_hw()
        return 3 * 2.0 * self.N * HO * WO * self.CO * self.C * self.KH * self.KW

    def make(self, seed: int | None = None) -> dict:
        g = torch.Generator("cpu")
        g.manual_seed(self.seed if seed is None else seed)
        HO, WO = self.out_hw()
        shapes = {"x": (self.N, self.C, self.H, self.W), "w": (self.CO, self.C, self.KH, self.KW),
                  "b": (self.CO,), "dy": (self.N, self.CO, HO, WO)}
        return {n: _draw(g, shapes[n], self.dist.get(n, ("uniform", 1.0)))
                for n in ("x", "w", "b", "dy")}


def _u(a):
    return ("uniform", a)


N01 = ("normal",)

# The five workloads the hot path is measured and checked on.
LINEAR_64x32x128_F32 = LinearWorkload(
    "linear_64x32x128_f32", M=64, N=32, K=128, dtype="f32",
    dist={"X": _u(1), "W": _u(1), "b": _u(1), "dY": _u(1)})
LINEAR_4096x1024x1024_F32 = LinearWorkload(
    "linear_4096x1024x1024_f32", M=4096, N=1024, K=1024, dtype="f32",
    dist={"X": N01, "W": _u(1 / math.sqrt(1024)), "b": _u(1 / math.sqrt(1024)), "dY": N01})
LINEAR_8192x8192x8192_F32 = LinearWorkload(
    "linear_8192x8192x8192_f32", M=8192, N=8192, K=8192, dtype="f32",
    dist={"X": N01, "W": _u(1 / math.sqrt(8192)), "b": _u(1 / math.sqrt(8192)), "dY": N01})
BMM_BCAST_16x1x509x257_1x8x257x383_F32 = BmmWorkload(
    "bmm_bcast_16x1x509x257_1x8x257x383_f32", ashape=(16, 1, 509, 257), bshape=(1, 8, 257, 383),
    cshape=(16, 8, 509, 383), dist={"A": _u(1), "B": _u(1), "dC": N01})
LINEAR_16384x8192x8192_BF16 = LinearWorkload(
    "linear_16384x8192x8192_bf16", M=16384, N=8192, K=8192, dtype="bf16",
    dist={"X": N01, "W": _u(1 / math.sqrt(8192)), "b": _u(1 / math.sqrt(8192)), "dY": N01})

# The training step around the dense layer: 8192 rows through 8192 -> 8192
# (GELU) -> 8192 under MSE with Adam; weights scaled like the dense layers above.
MLP2_8192x8192x8192x8192_F32_GELU = MlpWorkload(
    "mlp2_8192x8192x8192x8192_f32_gelu", M=8192, D0=8192, D1=8192, D2=8192, act="gelu",
    dist={"X": N01, "W1": _u(1 / math.sqrt(8192)), "b1": _u(1 / math.sqrt(8192)),
          "W2": _u(1 / math.sqrt(8192)), "b2": _u(1 / math.sqrt(8192)), "T": N01})

# A 3x3 convolution layer of the size found mid-way through image classifiers:
# 32 images of 256 channels at 56 x 56, 256 filters, stride 1, padding 1.
CONV2D_32x256x56x56_256x3x3_F32 = ConvWorkload(
    "conv2d_32x256x56x56_256x3x3_s1p1_f32", N=32, C=256, H=56, W=56, CO=256, KH=3, KW=3,
    stride=(1, 1), pad=(1, 1),
    dist={"x": N01, "w": _u(1 / math.sqrt(256 * 9)), "b": _u(1 / math.sqrt(256 * 9)), "dy": N01})

# the same layer downsampling (stride 2): its input gradient runs by sub-pixel phases
CONV2D_32x256x56x56_256x3x3_S2_F32 = ConvWorkload(
    "conv2d_32x256x56x56_256x3x3_s2p1_f32", N=32, C=256, H=56, W=56, CO=256, KH=3, KW=3,
    stride=(2, 2), pad=(1, 1),
    dist={"x": N01, "w": _u(1 / math.sqrt(256 * 9)), "b": _u(1 / math.sqrt(256 * 9)), "dy": N01})

WORKLOADS = {w.name: w for w in (LINEAR_64x32x128_F32, LINEAR_4096x1024x1024_F32,
                                 LINEAR_8192x8192x8192_F32, BMM_BCAST_16x1x509x257_1x8x257x383_F32,
                                 LINEAR_16384x8192x8192_BF16, MLP2_8192x8192x8192x8192_F32_GELU,
                                 CONV2D_32x256x56x56_256x3x3_F32, CONV2D_32x256x56x56_256x3x3_S2_F32)}


def linear(M, N, K, dtype="f32", dist=None, seed=0, name=None) -> LinearWorkload:
    """A linear workload of any size; default draws uniform[-1, 1]."""
    return LinearWorkload(name or f"linear_{M}x{N}x{K}_{dtype}", M=M, N=N, K=K, dtype=dtype,
                          dist=dist or {}, seed=seed)


def integers(lo, hi):
    return ("integers", lo, hi)


def tensor(shape, dist, seed=0) -> torch.Tensor:
    """One seeded fp32 tensor of the given distribution."""
    g = torch.Generator("cpu")
    g.manual_seed(seed)
    return _draw(g, tuple(shape), dist)
