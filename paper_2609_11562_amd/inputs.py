"""Seeded synthetic inputs for the GEMM + tile-reduce path.

This module only draws random numbers and rounds them to bfloat16.  It holds
none of the method's arithmetic, so both the HIP path (through the binding)
and the CPU oracle can consume the same arrays without sharing any code.

Every array is returned as raw bfloat16 bit patterns (``numpy.uint16``):

* ``A``      M x K, row-major (K contiguous)
* ``B``      K x N, row-major (N contiguous)
* ``peers``  P-1 arrays of M x N, row-major; peer ``q`` stands for the q-th
             rank other than the local one, in ascending rank order.
* layer epilogue (``make_layer_inputs``): the residual stream, rows x N
  row-major, and the RMSNorm weight gamma, length N.

Draws come from numpy's PCG64 generator: A from ``seed``, B from ``seed + 1``
and peer ``q`` from ``seed + 2 + q``.  Values are drawn in float32 and rounded
to bfloat16 with round-to-nearest-even (torch's CPU conversion).
"""
from __future__ import annotations

import dataclasses

import numpy as np
import torch

BASE_SEED = 2609_11562


@dataclasses.dataclass(frozen=True)
class Dist:
    """A value distribution: ``kind`` is "uniform" (on [-a, a]), "normal"
    (mean 0, standard deviation a), "int" (integers uniform on [-a, a]) or
    "const" (every value equals a)."""

    kind: str
    a: float


def _draw_f32(rng: np.random.Generator, shape, dist: Dist) -> np.ndarray:
    if dist.kind == "uniform":
        return rng.uniform(-dist.a, dist.a, size=shape).astype(np.float32)
    if dist.kind == "normal":
        x = rng.standard_normal(size=shape, dtype=np.float32)
        x *= np.float32(dist.a)
        return x
    if dist.kind == "int":
        lo = -int(dist.a)
        return rng.integers(lo, -lo + 1, size=shape).astype(np.float32)
    if dist.kind == "const":
        return np.full(shape, dist.a, dtype=np.float32)
    raise ValueError(f"unknown distribution {dist.kind!r}")


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest-even) and return the bits."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def draw_bf16(seed: int, shape, dist: Dist) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64(seed))
    return to_bf16_bits(_draw_f32(rng, shape, dist))


@dataclasses.dataclass
class Problem:
    M: int
    N: int
    K: int
    P: int
    A: np.ndarray
    B: np.ndarray
    peers: list


def make_problem(M: int, N: int, K: int, P: int, ab: Dist, peer: Dist,
                 seed: int = BASE_SEED) -> Problem:
    A = draw_bf16(seed, (M, K), ab)
    B = draw_bf16(seed + 1, (K, N), ab)
    peers = [draw_bf16(seed + 2 + q, (M, N), peer) for q in range(P - 1)]
    return Problem(M, N, K, P, A, B, peers)


def make_layer_inputs(rows: int, N: int, seed: int = BASE_SEED, residual: Dist = Dist("normal", 1.0)):
    """(R, gamma) for the residual addition + RMSNorm after the reduce-scatter:
    R ~ ``residual`` (hidden states of order one by default) from
    ``seed + 100``, gamma ~ U[0.5, 1.5] from ``seed + 101``."""
    R = draw_bf16(seed + 100, (rows, N), residual)
    rng = np.random.Generator(np.random.PCG64(seed + 101))
    gamma = to_bf16_bits(rng.uniform(0.5, 1.5, size=N).astype(np.float32))
    return R, gamma


def bits_to_torch(bits: np.ndarray) -> torch.Tensor:
    """View a uint16 bit array as a torch bfloat16 tensor (CPU, no copy)."""
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
