"""Seeded synthetic GEMM workloads.

This module holds the workload list (shapes, dtypes, seeds, search-space
shape, budgets) and the seeded input generator. It is shared by the tests,
the benchmark and the oracle checks; it contains none of the method's
arithmetic (no products, no configuration logic).

The paper measures perceptron GEMMs on synthetic square shapes (§5); the
workloads below stand in for them with fixed seeds and distributions.
Inputs are drawn on the CPU with ``torch.Generator().manual_seed(seed)``,
A first and then B, in fp32; bf16 workloads round the fp32 draw to bf16
(round-to-nearest-even, torch's ``.to(torch.bfloat16)``).
"""
from __future__ import annotations

import dataclasses
import math

import torch

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    dtype: str          # "f32" or "bf16"
    seed: int
    dist: str           # "uniform" (U[-1,1)), "normal", "normal_sqrtk", "normal002"
    d: tuple            # levels per dimension, order (m, k, n)
    mfma_coord: bool    # MFMA shape {16,32} is a search coordinate
    budget: int         # configurations timed by the search

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K


WORKLOADS = {
    w.name: w
    for w in [
        Workload("gemm256_f32", 256, 256, 256, F32, 0, "uniform", (3, 3, 3), False, 64),
        Workload("gemm1024_f32", 1024, 1024, 1024, F32, 1, "uniform", (4, 4, 4), False, 200),
        Workload("gemm2048_f32", 2048, 2048, 2048, F32, 2, "normal", (4, 4, 4), False, 500),
        Workload("gemm4096_bf16", 4096, 4096, 4096, BF16, 3, "normal_sqrtk", (4, 4, 4), True, 1000),
        Workload("mlp4096x11008x4096_bf16", 4096, 11008, 4096, BF16, 4, "normal002", (4, 4, 4), True, 1000),
        Workload("skinny64x4096x4096_bf16", 64, 4096, 4096, BF16, 4, "normal002", (4, 4, 4), True, 1000),
        # one GPU's share of the 4096³ product split eight ways along M (its
        # level-0 grid factor): the slab each GPU would tune and run alone
        Workload("slab512x4096x4096_bf16", 512, 4096, 4096, BF16, 3, "normal_sqrtk", (4, 4, 4), True,
                 1000),
        # the same eighth of the product split two ways along M and four along N
        Workload("slab1024x2048x4096_bf16", 1024, 2048, 4096, BF16, 3, "normal_sqrtk", (4, 4, 4), True,
                 1000),
    ]
}


def _draw(gen: torch.Generator, shape, dist: str, K: int) -> torch.Tensor:
    if dist == "uniform":
        return torch.rand(shape, generator=gen, dtype=torch.float32) * 2.0 - 1.0
    if dist == "normal":
        return torch.randn(shape, generator=gen, dtype=torch.float32)
    if dist == "normal_sqrtk":
        return torch.randn(shape, generator=gen, dtype=torch.float32) / math.sqrt(K)
    if dist == "normal002":
        return torch.randn(shape, generator=gen, dtype=torch.float32) * 0.02
    if dist == "smallint":
        return torch.randint(-4, 5, shape, generator=gen).to(torch.float32)
    raise ValueError(f"unknown distribution {dist!r}")


def make_inputs(M: int, N: int, K: int, dtype: str, seed: int, dist: str):
    """Return host tensors (A: M×K, B: K×N), row-major, in the input dtype."""
    gen = torch.Generator().manual_seed(seed)
    A = _draw(gen, (M, K), dist, K)
    B = _draw(gen, (K, N), dist, K)
    if dtype == BF16:
        A = A.to(torch.bfloat16)
        B = B.to(torch.bfloat16)
    elif dtype != F32:
        raise ValueError(f"unknown dtype {dtype!r}")
    return A.contiguous(), B.contiguous()


def make_large_smallint_inputs(M: int, N: int, K: int, dtype: str, seed: int, bound: int = 4):
    """Small-integer A (M×K) and B (K×N), integers in [-bound, bound] (the
    "smallint" values of make_inputs for bound 4), drawn directly as int8 so
    that operands of several GiB need no wider intermediate (a different
    random stream from make_inputs)."""
    gen = torch.Generator().manual_seed(seed)
    t = torch.bfloat16 if dtype == BF16 else torch.float32
    A = torch.randint(-bound, bound + 1, (M, K), generator=gen, dtype=torch.int8).to(t)
    B = torch.randint(-bound, bound + 1, (K, N), generator=gen, dtype=torch.int8).to(t)
    return A.contiguous(), B.contiguous()


# The paper's own protocol (§5): perceptron layers Y = WᵀX of sizes
# (m, k, n) = 512³, 1024³, 2048³ in fp32, d = (4, 2, 4), neighbours between
# any two levels (Eq.6), s0 = [[m,1,1,1],[k,1],[n,1,1,1]], ρ = 5, and a budget
# of 0.1 % of the space: ⌈0.001·|ξ|⌉ of 484,000, 899,756 and 1,589,952.
PAPER_PROTOCOL = [
    Workload("perceptron512_f32", 512, 512, 512, F32, 0, "uniform", (4, 2, 4), False, 484),
    Workload("perceptron1024_f32", 1024, 1024, 1024, F32, 0, "uniform", (4, 2, 4), False, 900),
    Workload("perceptron2048_f32", 2048, 2048, 2048, F32, 0, "uniform", (4, 2, 4), False, 1590),
]


def make_perceptron_inputs(M: int, N: int, K: int, dtype: str, seed: int, dist: str):
    """Host tensors of the perceptron layer Y = WᵀX of §5: W (K×M) drawn
    first, then X (K×N), row-major, in the input dtype."""
    gen = torch.Generator().manual_seed(seed)
    W = _draw(gen, (K, M), dist, K)
    X = _draw(gen, (K, N), dist, K)
    if dtype == BF16:
        W, X = W.to(torch.bfloat16), X.to(torch.bfloat16)
    elif dtype != F32:
        raise ValueError(f"unknown dtype {dtype!r}")
    return W.contiguous(), X.contiguous()


def workload_inputs(w: Workload):
    return make_inputs(w.M, w.N, w.K, w.dtype, w.seed, w.dist)


def raw_bytes(t: torch.Tensor):
    """The exact bytes of a host tensor as a numpy uint8 array (bf16 has no numpy dtype)."""
    t = t.contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint8")
    return t.numpy().view("uint8")
