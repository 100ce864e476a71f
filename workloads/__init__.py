"""Seeded synthetic inputs for the signaled + reordered GEMM path.

This module only draws random numbers and stores them as fp16/bf16 bit
patterns. It holds none of the method's arithmetic (no GEMM, no reorder, no
consumer sum, no normalisation), so both the CPU oracle's tests and the GPU
path can take their inputs from here without sharing any computation.

The paper evaluates on randomly generated inputs only and names no dataset
(artifact appendix, "Benchmarks"). The shapes below are tensor-parallel /
expert-parallel shard GEMMs inside the operator sizes the paper evaluates
(Section 6.1, Table 3: M*N of 4..400 x 1024^2, K of 2..16 x 1024).

Draw order per workload, from ``numpy.random.default_rng(seed)``:
A, then B (logical [K, N]), then the peer partial, then the workload's extra
arrays (destination permutation sigma, or the row-to-bucket map), then bias,
then gamma.  Values are drawn in float64 and rounded to nearest-even into the
storage dtype; bf16 rounding goes through float32 first (both steps RNE).
The GEMM's second operand is handed over transposed, as W = B^T with shape
[N, K] (the weight layout of a linear layer, K contiguous).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

FP16 = "fp16"
BF16 = "bf16"

# Patterns of the pre-communication reorder (Section 3.3, Approach):
TILE = "tile"            # AllReduce: whole tiles, column of tiles
SUBTILE = "subtile"      # ReduceScatter: tiles split into R row slices
SUBTOKEN = "subtoken"    # All-to-All: tile rows sent to per-destination pools
ROWMAJOR = "rowmajor"    # plain GEMM output, no reorder


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    dtype: str
    tile_m: int
    tile_n: int
    order: str               # "rowmajor" or "xcd" dispatch order of tiles
    pattern: str
    seed: int
    dist: str                # "uniform" or "normal"
    num_dest: int = 0        # R (subtile) or B (subtoken)
    group_unit: str = "waves"
    groups: Optional[tuple] = None   # None: chosen by the planner's search
    sweep: Optional[tuple] = None    # group sizes (in waves) to sweep
    bias: bool = False
    rmsnorm: bool = False
    gamma: bool = False
    eps: float = 1e-6
    description: str = ""

    @property
    def flops(self) -> float:
        return 2.0 * self.M * self.N * self.K

    def with_shape(self, M: int, N: int, K: int, name: Optional[str] = None) -> "Workload":
        return dataclasses.replace(self, M=M, N=N, K=K, name=name or f"{self.name}@{M}x{N}x{K}")


WORKLOADS = {
    "tiny": Workload(
        name="tiny", M=256, N=256, K=256, dtype=FP16, tile_m=64, tile_n=64,
        order="rowmajor", pattern=TILE, seed=0, dist="uniform",
        group_unit="tiles", groups=(4, 4, 4, 4),
        description="fp16 256^3, 64x64 tiles, 4 groups of 4 tiles in row-major "
                    "tile order, peer-partial sum, row-major restore"),
    "ar_2048x4096x4096": Workload(
        name="ar_2048x4096x4096", M=2048, N=4096, K=4096, dtype=FP16,
        tile_m=256, tile_n=128, order="xcd", pattern=TILE, seed=1,
        dist="uniform", num_dest=2,
        description="row-parallel linear shard, AllReduce stand-in (R=2: one "
                    "simulated peer partial), groups from the planner"),
    "rs_8192x8192x3584": Workload(
        name="rs_8192x8192x3584", M=8192, N=8192, K=3584, dtype=FP16,
        tile_m=256, tile_n=256, order="xcd", pattern=SUBTILE, seed=2,
        dist="uniform", num_dest=4, sweep=(1, 2, 4, 8),
        description="MLP down-projection shard (hidden 8192, FFN 28672/8), "
                    "ReduceScatter stand-in: subtile k plus peer into one of 4 "
                    "seeded destination slot buffers"),
    "ar_rmsnorm_16384x4096x3584_bf16": Workload(
        name="ar_rmsnorm_16384x4096x3584_bf16", M=16384, N=4096, K=3584,
        dtype=BF16, tile_m=256, tile_n=256, order="xcd", pattern=TILE, seed=3,
        dist="normal", num_dest=2, bias=True, rmsnorm=True, gamma=True,
        description="long-prefill shard, AllReduce stand-in, restore fused "
                    "with bias add and RMSNorm over N=4096"),
    "a2a_4096x7168x2048": Workload(
        name="a2a_4096x7168x2048", M=4096, N=7168, K=2048, dtype=FP16,
        tile_m=256, tile_n=256, order="xcd", pattern=SUBTOKEN, seed=4,
        dist="uniform", num_dest=8, rmsnorm=True,
        description="MoE-style output projection, All-to-All stand-in: rows "
                    "go to 8 seeded buckets, restore fused with RMSNorm over "
                    "N=7168"),
}


def _to_fp16_bits(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x.astype(np.float16)).view(np.uint16)


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    f = np.ascontiguousarray(x.astype(np.float32)).view(np.uint32)
    # round-to-nearest-even on the 16 dropped bits (inputs are finite)
    bias = np.uint32(0x7FFF) + ((f >> np.uint32(16)) & np.uint32(1))
    return ((f + bias) >> np.uint32(16)).astype(np.uint16)


def to_bits(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the storage dtype and return the raw bits."""
    if dtype == FP16:
        return _to_fp16_bits(x)
    if dtype == BF16:
        return _to_bf16_bits(x)
    raise ValueError(dtype)


def bits_to_float32(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening of stored fp16/bf16 bits (for display and statistics)."""
    if dtype == FP16:
        return bits.view(np.float16).astype(np.float32)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Inputs:
    A: np.ndarray                 # uint16 [M, K]
    W: np.ndarray                 # uint16 [N, K]  (= B^T)
    peer: np.ndarray              # uint16 [M*N], peer partial in reordered layout
    sigma: Optional[np.ndarray]   # int32 [R]  destination buffer of subtile k
    bucket: Optional[np.ndarray]  # int32 [M]  destination bucket of each row
    bias: Optional[np.ndarray]    # uint16 [N]
    gamma: Optional[np.ndarray]   # uint16 [N]


def make_inputs(w: Workload) -> Inputs:
    rng = np.random.default_rng(w.seed)
    M, N, K = w.M, w.N, w.K
    if w.dist == "uniform":
        A = rng.uniform(-1.0, 1.0, size=(M, K))
        B = rng.uniform(-1.0, 1.0, size=(K, N)) / math.sqrt(K)
        peer = rng.uniform(-1.0, 1.0, size=M * N)
    elif w.dist == "normal":
        A = rng.standard_normal(size=(M, K))
        B = rng.standard_normal(size=(K, N)) / math.sqrt(K)
        peer = rng.standard_normal(size=M * N)
    else:
        raise ValueError(w.dist)
    A_bits = to_bits(A, w.dtype)
    del A
    W_bits = np.ascontiguousarray(to_bits(B, w.dtype).T)
    del B
    peer_bits = to_bits(peer, w.dtype)
    del peer
    sigma = bucket = None
    if w.pattern == SUBTILE:
        sigma = rng.permutation(w.num_dest).astype(np.int32)
    elif w.pattern == SUBTOKEN:
        bucket = rng.integers(0, w.num_dest, size=M).astype(np.int32)
    bias = gamma = None
    if w.bias:
        bias = to_bits(rng.uniform(-0.1, 0.1, size=N), w.dtype)
    if w.gamma:
        gamma = to_bits(rng.uniform(0.5, 1.5, size=N), w.dtype)
    return Inputs(A=A_bits, W=W_bits, peer=peer_bits, sigma=sigma,
                  bucket=bucket, bias=bias, gamma=gamma)


def uniform_bits(shape, seed: int, dtype: str = FP16, lo=-1.0, hi=1.0) -> np.ndarray:
    """Seeded U[lo, hi] values stored as fp16/bf16 bits (small test buffers)."""
    rng = np.random.default_rng(seed)
    return to_bits(rng.uniform(lo, hi, size=shape), dtype)
