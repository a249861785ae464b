"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and places them; it holds none of the
Pici method's arithmetic.  Both the CPU oracle's tests and the GPU path take
their inputs from here, so the two sides always see the same arrays.

Recipe (the paper's microbenchmarks use unstructured, uniformly random
nonzero positions with a distinct seed per process, Sec. VI-A; its training
study prunes gradient buckets to 99% sparsity, Sec. VI-B):

* exact nonzero count ``nnz = round((1 - sigma) * n)`` at distinct positions
  drawn uniformly without replacement (``numpy.random.Generator.choice``);
* values drawn as float64, cast to float32 with round-to-nearest-even, and
  for bfloat16 rounded again from float32 to bfloat16 (nearest-even on the
  bit pattern);
* a value whose cast bit pattern is all zero would silently lower nnz, so it
  is drawn again until every placed value is nonzero;
* seeds are ``numpy.random.default_rng([config, rank, segment, permille])``
  so that any (rank, segment) of a large configuration can be regenerated on
  its own.

Arrays are returned as numpy ``float32`` for fp32 and ``uint16`` (the raw
bfloat16 bit patterns) for bf16.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

F32 = "f32"
BF16 = "bf16"

TILE = 4096


def nnz_for(n: int, permille: int) -> int:
    """round((1 - permille/1000) * n), computed exactly in integers (ties up)."""
    return (n * (1000 - permille) * 2 + 1000) // 2000


def _bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); raw bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def _draw_values(rng: np.random.Generator, k: int, dist: str, scale: float, dtype: str) -> np.ndarray:
    """k values whose bit patterns (in dtype) are all nonzero."""
    def draw(m):
        if dist == "normal":
            v = rng.normal(0.0, scale, m)
        elif dist == "laplace":
            v = rng.laplace(0.0, scale, m)
        else:
            raise ValueError(dist)
        v = v.astype(np.float32)
        return _bf16_bits_from_f32(v) if dtype == BF16 else v

    out = draw(k)
    while True:
        zero = (out.view(np.uint16) == 0) if dtype == BF16 else (out.view(np.uint32) == 0)
        bad = np.flatnonzero(zero)
        if bad.size == 0:
            return out
        out[bad] = draw(bad.size)


def empty(n: int, dtype: str) -> np.ndarray:
    return np.zeros(n, dtype=np.uint16 if dtype == BF16 else np.float32)


def sparse_array(n: int, nnz: int, seed, dtype: str = F32, dist: str = "normal",
                 scale: float = 1.0) -> np.ndarray:
    """n elements, exactly nnz of them nonzero at uniform random distinct positions."""
    if not 0 <= nnz <= n:
        raise ValueError("nnz out of range")
    rng = np.random.default_rng(seed)
    pos = rng.choice(n, size=nnz, replace=False) if nnz < n else np.arange(n)
    out = empty(n, dtype)
    out[pos] = _draw_values(rng, nnz, dist, scale, dtype)
    return out


# ---- the five workloads ----------------------------------------------------

CFG1_N = 1 << 20
CFG1_NNZ = 10486          # sigma = 99%


def cfg1():
    """1,048,576 fp32, 10,486 nonzeros, N(0,1): operand a (seed 0), b (seed 1)."""
    a = sparse_array(CFG1_N, CFG1_NNZ, 0, F32)
    b = sparse_array(CFG1_N, CFG1_NNZ, 1, F32)
    return a, b


CFG2_N = 1 << 26          # 256 MiB of fp32
CFG2_PERMILLE = (500, 900, 990, 999)


def cfg2(permille: int, operand: int = 0, n: int = CFG2_N):
    """The codec sweep array at sparsity permille/1000 (operand 1 = second reduce input)."""
    return sparse_array(n, nnz_for(n, permille), [2, operand, 0, permille], F32)


CFG3_P = 8
CFG3_N = 1 << 25          # 33,554,432 fp32 per rank
CFG3_PERMILLE = 990


def cfg3_rank(rank: int, n: int = CFG3_N, permille: int = CFG3_PERMILLE):
    """Reduce-scatter input of one virtual rank: sigma = 99%, independent positions."""
    return sparse_array(n, nnz_for(n, permille), [3, rank, 0, permille], F32)


CFG4_P = 8
CFG4_N = 1 << 24          # 16,777,216 bf16 per rank
CFG4_PERMILLE = 999


def cfg4_rank(rank: int, n: int = CFG4_N, permille: int = CFG4_PERMILLE):
    """All-gather contribution of one virtual rank: bf16, sigma = 99.9%, N(0, 0.02)."""
    return sparse_array(n, nnz_for(n, permille), [4, rank, 0, permille], BF16, "normal", 0.02)


CFG5_P = 8
CFG5_SEGMENTS = 64
CFG5_SEG = 1 << 22        # 4,194,304 elements per segment
CFG5_SHARED = 0.7


@dataclass
class Cfg5Plan:
    """Per-segment sparsity and shared positions, common to all ranks."""
    seg_len: int
    sigmas: np.ndarray
    nnz: np.ndarray
    shared: list

    @property
    def n(self) -> int:
        return self.seg_len * len(self.sigmas)


def cfg5_plan(segments: int = CFG5_SEGMENTS, seg_len: int = CFG5_SEG) -> Cfg5Plan:
    """Segment sparsities ~ U[0.5, 0.99] and the 70% shared positions of each segment."""
    srng = np.random.default_rng([5, 1000, segments, seg_len])
    sigmas = srng.uniform(0.5, 0.99, segments)
    nnz = np.rint((1.0 - sigmas) * seg_len).astype(np.int64)
    shared = []
    for s in range(segments):
        k_sh = int(np.rint(CFG5_SHARED * nnz[s]))
        rng = np.random.default_rng([5, 2000, s, seg_len])
        shared.append(np.sort(rng.choice(seg_len, size=k_sh, replace=False)))
    return Cfg5Plan(seg_len, sigmas, nnz, shared)


def cfg5_segment(plan: Cfg5Plan, rank: int, seg: int) -> np.ndarray:
    """One 'layer' segment of one rank: shared positions plus private ones, Laplace(0, 1e-3)."""
    L = plan.seg_len
    shared = plan.shared[seg]
    n_priv = int(plan.nnz[seg]) - shared.size
    rng = np.random.default_rng([5, rank, seg, L])
    mask = np.zeros(L, dtype=bool)
    mask[shared] = True
    comp = np.flatnonzero(~mask)
    priv = comp[rng.choice(comp.size, size=n_priv, replace=False)]
    out = np.zeros(L, dtype=np.float32)
    pos = np.concatenate([shared, priv])
    out[pos] = _draw_values(rng, pos.size, "laplace", 1e-3, F32)
    return out


def cfg5_rank(plan: Cfg5Plan, rank: int, out: np.ndarray | None = None) -> np.ndarray:
    """The whole pruned-gradient-like buffer of one rank (segments concatenated)."""
    if out is None:
        out = np.empty(plan.n, dtype=np.float32)
    for s in range(len(plan.sigmas)):
        out[s * plan.seg_len:(s + 1) * plan.seg_len] = cfg5_segment(plan, rank, s)
    return out
