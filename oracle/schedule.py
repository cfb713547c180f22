"""Plain statement of the producer traversal and consumer task assignment.

TEST INFRASTRUCTURE ONLY (imported by tests, never by the product path).

Terms (paper, Section 3.1):
* A producer block at logical position p computes a BM x BN region of the
  M x N partial.  The output is split into P equal row partitions
  (destinations); partition d holds rows [d M/P, (d+1) M/P).
* Interleaved production, Equation 1:  d = p mod P,  l = floor(p / P).
  l is the block's index inside partition d, counted in the consumer's order,
  which walks the partition's blocks N-major (column index fastest; the
  paper's evaluation, Section 5.3.1, states the interleaved map follows the
  consumer's N-major order within each partition).
* Two comparison orders: partition-contiguous traversal with N fastest over
  the whole output (Figure 1, top panel: every tile of partition 0 first,
  then partition 1, ...), and M-major traversal (M fastest), the producer
  default used as the ablation baseline in Section 5.3.1.
* The reduction unit is a T x T tile, T = 128 (Section 4.2).  A block covers
  c = (BM/T)(BN/T) tiles; each stays a separate reduction task.  Inside its
  partition, tile numbers follow producer order: the c tiles of block l get
  numbers l*c .. l*c + c - 1, in N-major order inside the block (the paper's
  1 x 2 example: block p=1 yields t0 and t1).
* Consumer block j of x processes tiles j, j+x, j+2x, ... below Q, where Q is
  the partition's tile count ("Matching task order").
"""
from __future__ import annotations

INTERLEAVED = 0
ROW_MAJOR = 1
M_MAJOR = 2
TILE = 128


def producer_block(order: int, p: int, M: int, N: int, P: int, BM: int, BN: int):
    """Map logical position p to (d, l, mb, nb): destination partition,
    index inside the partition (N-major), and the block's row / column index
    in the M/BM x N/BN block grid."""
    MB, NB = M // BM, N // BN
    rows_per_part = (M // P) // BM          # block rows in one partition
    if not 0 <= p < MB * NB:
        raise ValueError("position out of range")
    if order == INTERLEAVED:
        d = p % P                            # Equation 1
        l = p // P
        mb = d * rows_per_part + l // NB
        nb = l % NB
    elif order == ROW_MAJOR:
        mb, nb = p // NB, p % NB
        d = mb // rows_per_part
        l = (mb % rows_per_part) * NB + nb
    elif order == M_MAJOR:
        mb, nb = p % MB, p // MB
        d = mb // rows_per_part
        l = (mb % rows_per_part) * NB + nb
    else:
        raise ValueError("unknown order")
    return d, l, mb, nb


def block_tiles(mb: int, nb: int, BM: int, BN: int):
    """Global (tile_row, tile_col) of the tiles a block covers, in the
    block's N-major order."""
    out = []
    for ti in range(BM // TILE):
        for tj in range(BN // TILE):
            out.append((mb * (BM // TILE) + ti, nb * (BN // TILE) + tj))
    return out


def partition_tile_number(l: int, i: int, BM: int, BN: int) -> int:
    """Number of the i-th tile of partition block l: t = l*c + i."""
    c = (BM // TILE) * (BN // TILE)
    return l * c + i


def full_schedule(order: int, M: int, N: int, P: int, BM: int, BN: int):
    """Per logical position: (d, l, mb, nb, [(t, tile_row, tile_col), ...])."""
    nblocks = (M // BM) * (N // BN)
    sched = []
    for p in range(nblocks):
        d, l, mb, nb = producer_block(order, p, M, N, P, BM, BN)
        tiles = [(partition_tile_number(l, i, BM, BN), tr, tc)
                 for i, (tr, tc) in enumerate(block_tiles(mb, nb, BM, BN))]
        sched.append((d, l, mb, nb, tiles))
    return sched


def tiles_per_partition(M: int, N: int, P: int) -> int:
    return ((M // P) // TILE) * (N // TILE)


def consumer_tasks(j: int, x: int, Q: int):
    """Tiles processed, in order, by consumer block j of x."""
    return list(range(j, Q, x))


def all_chunk_consumer_tasks(j: int, x: int, P: int, Q: int):
    """One-GPU emulation of every destination: the x consumer blocks are
    split evenly over the P partitions (x a multiple of P); block j serves
    partition j mod P as its (j div P)-th block with stride x / P."""
    if x % P:
        raise ValueError("x must be a multiple of P")
    d = j % P
    return d, consumer_tasks(j // P, x // P, Q)
