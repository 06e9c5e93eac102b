"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This module holds no arithmetic of the method: it only names the workloads
(shapes, dtypes, value distributions, tile sizes) and draws their inputs
from a seed.  Inputs are drawn in fp32 with a CPU ``torch.Generator`` and
rounded once (round-to-nearest-even, by torch) to the input dtype; both sides
then consume the same 16-bit patterns.

Seeding: A of a GEMM workload comes from ``seed_stream(seed, 0)``; the
column shard B_r of rank r comes from ``seed_stream(seed, 1 + r)``, so the
gathered right operand is ``[B_0 | ... | B_{w-1}]`` and any one shard can be
drawn without drawing the others.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class GemmWorkload:
    name: str
    M: int
    K: int
    N_local: int
    world: int
    dtype: str            # "f16" or "bf16": input and output element type
    dist: str             # "uniform", "normal_sqrtk" or "uniform_sqrtk"
    tile_m: int
    tile_n: int
    rank: int = 0

    @property
    def N_gathered(self) -> int:
        return self.world * self.N_local

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N_local * self.K


@dataclass(frozen=True)
class CopyWorkload:
    name: str
    world: int
    rows: int
    cols: int
    tiles: tuple = field(default=(64, 128, 256))
    shift: int = 1

    @property
    def bytes_moved(self) -> int:
        # every rank's send block is read once and written once
        return 2 * self.world * self.rows * self.cols * 4


# The five synthetic workloads of the evaluation: the tiny two-rank case, the
# 256 MiB heap tile copy, and three eight-rank GEMM + All-Scatter shapes.
TINY = GemmWorkload("gas_f16_w2_m128_k256_n64", 128, 256, 64, 2, "f16", "uniform", 64, 64)
HEAP_COPY = CopyWorkload("heap_copy_f32_w8_2048x2048", 8, 2048, 2048)
SMALL_BF16 = GemmWorkload("gas_bf16_w8_m1024_k4096_n1024", 1024, 4096, 1024, 8, "bf16",
                          "normal_sqrtk", 256, 256)
LARGE_BF16 = GemmWorkload("gas_bf16_w8_m4096_k8192_n3584", 4096, 8192, 3584, 8, "bf16",
                          "normal_sqrtk", 256, 256)
WIDE_F16 = GemmWorkload("gas_f16_w8_m8192_k8192_n1024", 8192, 8192, 1024, 8, "f16",
                        "uniform_sqrtk", 256, 256)

GEMM_WORKLOADS = {w.name: w for w in (TINY, SMALL_BF16, LARGE_BF16, WIDE_F16)}


def seed_stream(seed: int, stream: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed) * 1_000_003 + int(stream))
    return g


def torch_dtype(dtype: str) -> torch.dtype:
    return {"f16": torch.float16, "bf16": torch.bfloat16}[dtype]


def _draw(shape, dist: str, K: int, gen: torch.Generator) -> torch.Tensor:
    if dist == "uniform":
        return torch.rand(shape, generator=gen, dtype=torch.float32) * 2.0 - 1.0
    if dist == "uniform_sqrtk":
        return (torch.rand(shape, generator=gen, dtype=torch.float32) * 2.0 - 1.0) / math.sqrt(K)
    if dist == "normal_sqrtk":
        return torch.randn(shape, generator=gen, dtype=torch.float32) / math.sqrt(K)
    raise ValueError(f"unknown distribution {dist!r}")


def gemm_A(M: int, K: int, dtype: str, dist: str, seed: int = 0) -> torch.Tensor:
    """A [M, K] in the input dtype (CPU tensor)."""
    return _draw((M, K), dist, K, seed_stream(seed, 0)).to(torch_dtype(dtype))


def gemm_B_shard(K: int, N_local: int, rank: int, dtype: str, dist: str,
                 seed: int = 0) -> torch.Tensor:
    """Rank ``rank``'s column shard B_r [K, N_local] in the input dtype."""
    return _draw((K, N_local), dist, K, seed_stream(seed, 1 + rank)).to(torch_dtype(dtype))


def workload_inputs(w: GemmWorkload, seed: int = 0, rank: int | None = None):
    """(A, B_rank) CPU tensors for workload ``w``."""
    r = w.rank if rank is None else rank
    return (gemm_A(w.M, w.K, w.dtype, w.dist, seed),
            gemm_B_shard(w.K, w.N_local, r, w.dtype, w.dist, seed))


def copy_send(w: CopyWorkload, seed: int = 0) -> torch.Tensor:
    """send blocks [world, rows, cols] fp32, uniform [0, 1)."""
    return torch.rand((w.world, w.rows, w.cols), generator=seed_stream(seed, 0),
                      dtype=torch.float32)


def bits(t: torch.Tensor) -> np.ndarray:
    """The 16-bit patterns of a float16/bfloat16 CPU tensor as numpy uint16."""
    if t.dtype not in (torch.float16, torch.bfloat16):
        raise TypeError("bits() expects a 16-bit float tensor")
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def random_ints(shape, lo: int, hi: int, seed: int) -> torch.Tensor:
    """Small integers in [lo, hi] as fp32 (exact in every 16-bit format)."""
    return torch.randint(lo, hi + 1, shape, generator=seed_stream(seed, 7),
                         dtype=torch.int64).to(torch.float32)
