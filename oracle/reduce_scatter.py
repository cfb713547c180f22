"""Plain CPU statement of what one rank's GEMM-ReduceScatter computes.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this module;
only the tests, the smoke check and the benchmark's CPU-baseline leg do.

Definition followed (paper, Section 2.1 "GEMM-ReduceScatter Execution" and
Section 3.1 "Coordinating Tiled Computation and Communication"): with W ranks
(here P chunks), every rank r holds a K-slice of the reduction and computes an
M x N partial V[r] = A_r B_r.  Output row partition d (rows d*M/P ... ) is the
sum over all ranks of their partials restricted to those rows.  On one GPU the
local rank's partial is A B, and the P-1 other ranks' partials are supplied
as "peer" matrices Pi_q (q = 0 .. P-2, ascending rank order), so

    O_d = (A B)[R_d, :] + sum_q Pi_q[R_d, :],    R_d = rows [d M/P, (d+1) M/P).

Tile order, ready flags and the reducer's CU budget change *when* this is
computed, never *what* (the consumer reads a tile only after every
contribution to it has been published; Section 4.2).  The oracle therefore
evaluates the definition directly, in float64: every bf16 x bf16 product is
exact in float64, and a K-term float64 sum carries at most ~K * 2^-53 relative
error, far below bf16 resolution.  No blocking, reordering or fusion.

Inputs are raw bfloat16 bit patterns (uint16 arrays); decoding them is part of
this module so that it depends on nothing but numpy.
"""
from __future__ import annotations

import numpy as np

# Unit roundoff of the two formats the GPU path rounds through (round to
# nearest even): bfloat16 keeps 8 significant bits, float32 keeps 24.
U_BF16 = 2.0 ** -8
U_F32 = 2.0 ** -24

# Correctness gate of the paper's evaluation protocol (Section 5.1,
# "Protocol"): |got - ref| <= ATOL + RTOL * |ref| elementwise.
PAPER_ATOL = 0.1
PAPER_RTOL = 0.05


def bf16_to_f64(bits) -> np.ndarray:
    """Decode bfloat16 bit patterns: a bfloat16 is the upper half of a
    float32 word, so shift the 16 bits up and reinterpret."""
    b = np.asarray(bits, dtype=np.uint16)
    with np.errstate(invalid="ignore"):      # signalling-NaN patterns stay NaN
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def chunk_rows(M: int, P: int, d: int) -> slice:
    """Row partition R_d of destination d: equal, contiguous row blocks."""
    if M % P:
        raise ValueError("M must split into P equal row chunks")
    h = M // P
    return slice(d * h, (d + 1) * h)


def local_partial(A_bits, B_bits) -> np.ndarray:
    """The local rank's contribution C = A B in float64 (M x N)."""
    return bf16_to_f64(A_bits) @ bf16_to_f64(B_bits)


def reduce_chunk(C: np.ndarray, peer_bits, P: int, d: int) -> np.ndarray:
    """O_d: the local contribution to chunk d plus every peer's contribution
    to the same rows, peers added in rank order (Section 4.2)."""
    rows = chunk_rows(C.shape[0], P, d)
    out = np.array(C[rows], dtype=np.float64, copy=True)
    for q in range(P - 1):
        out += bf16_to_f64(peer_bits[q][rows])
    return out


def gemm_reduce_scatter(A_bits, B_bits, peer_bits, P: int, dest: int) -> np.ndarray:
    """Reference output.  ``dest`` in [0, P) returns O_dest ((M/P) x N);
    ``dest == -1`` returns every chunk stacked in row order (M x N)."""
    if len(peer_bits) != P - 1:
        raise ValueError("need exactly P-1 peer partials")
    C = local_partial(A_bits, B_bits)
    if dest == -1:
        return np.concatenate([reduce_chunk(C, peer_bits, P, d) for d in range(P)], axis=0)
    if not 0 <= dest < P:
        raise ValueError("dest out of range")
    return reduce_chunk(C, peer_bits, P, dest)


def output_rows(A_bits, B_bits, peer_bits, rows) -> np.ndarray:
    """The reduced output at the given *global* row indices (len(rows) x N),
    evaluated row by row; used to check full-size runs on sampled rows."""
    rows = np.asarray(rows, dtype=np.int64)
    C = bf16_to_f64(np.asarray(A_bits)[rows]) @ bf16_to_f64(B_bits)
    for pb in peer_bits:
        C += bf16_to_f64(np.asarray(pb)[rows])
    return C


def error_bound_rows(A_bits, B_bits, peer_bits, rows, final_rounding: bool = True) -> np.ndarray:
    """Elementwise rounding-error bound for a path that (1) accumulates the
    GEMM in float32, (2) stores the local partial as bfloat16, (3) sums the
    partial and the peers in float32 and (4) rounds the result to bfloat16.

    First-order bound (standard summation analysis, e.g. Higham, "Accuracy and
    Stability of Numerical Algorithms", 2nd ed., Section 3.1):
        (1) K u32 (|A||B|)          (2) u16 |C|
        (3) (P-1) u32 (|C| + sum|Pi|)   (4) u16 |O|
    It is returned doubled to absorb second-order terms:
        2 u16 (|O| + |C|) + 2 u32 (K |A||B| + P (|C| + sum|Pi|)).
    With ``final_rounding`` False, term (4) is left out: the bound on the
    float32 sum itself, for paths that keep computing with it.
    """
    rows = np.asarray(rows, dtype=np.int64)
    a = bf16_to_f64(np.asarray(A_bits)[rows])
    b = bf16_to_f64(B_bits)
    K = a.shape[1]
    P = len(peer_bits) + 1
    C = a @ b
    absAB = np.abs(a) @ np.abs(b)
    O = C.copy()
    abs_peers = np.zeros_like(C)
    for pb in peer_bits:
        v = bf16_to_f64(np.asarray(pb)[rows])
        O += v
        abs_peers += np.abs(v)
    return 2 * U_BF16 * ((np.abs(O) if final_rounding else 0.0) + np.abs(C)) + 2 * U_F32 * (
        K * absAB + P * (np.abs(C) + abs_peers))


def paper_gate(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Elementwise pass mask of the paper's correctness gate."""
    return np.abs(got - ref) <= PAPER_ATOL + PAPER_RTOL * np.abs(ref)


def f32_to_bf16_rne_bits(x) -> np.ndarray:
    """Round float32 values to bfloat16, nearest-even, returning the bits:
    keep the upper 16 bits after adding 0x7FFF plus the lowest kept bit
    (ties go to the even neighbour); NaN stays a quiet NaN."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounded = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    return np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), rounded)


def reduce_tile_f32(partial_bits, peer_bits) -> np.ndarray:
    """The reducer's own arithmetic on bf16 contributions (Section 4.2,
    ReduceTile): start from the local contribution, add the peers one at a
    time in rank order, each addition rounded to float32, then round the sum
    to bfloat16.  Returns bf16 bits; bit-exact by definition."""
    acc = bf16_to_f64(partial_bits).astype(np.float32)
    for pb in peer_bits:
        acc = (acc + bf16_to_f64(pb).astype(np.float32)).astype(np.float32)
    return f32_to_bf16_rne_bits(acc)
