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

The paper fixes the walk inside a partition to N-major.  The build also has
an L2-friendly walk (group_m > 1) that is not from the paper: with workgroup
b running on XCD b mod 8, partition d is served by G = 8 / P XCDs (P | 8) and
index l goes to stripe l mod G (column stripes when they divide the block
columns, else row stripes, else one stripe); each stripe is walked in groups
of group_m block rows (the largest divisor of the stripe's rows not above
group_m), M fastest inside a group, then the stripes are interleaved.  It is
restated here from that description, independently of the library.
"""
from __future__ import annotations

INTERLEAVED = 0
ROW_MAJOR = 1
M_MAJOR = 2
TILE = 128


def partition_walk(RB: int, NB: int, P: int, group_m: int = 1, xcds: int = 8):
    """Block coordinates (row, col) inside one partition (RB x NB blocks), in
    the order the partition's blocks are produced and consumed."""
    if group_m <= 1:
        return [(l // NB, l % NB) for l in range(RB * NB)]      # N-major (paper)
    G = xcds // P if (P <= xcds and xcds % P == 0) else 1
    if NB % G == 0:
        stripes = [(0, RB, s * (NB // G), NB // G) for s in range(G)]
    elif RB % G == 0:
        stripes = [(s * (RB // G), RB // G, 0, NB) for s in range(G)]
    else:
        G, stripes = 1, [(0, RB, 0, NB)]
    walks = []
    for r0, nr, c0, nc in stripes:
        gm = max(k for k in range(1, min(group_m, nr) + 1) if nr % k == 0)
        walk = []
        for grp in range(nr // gm):
            for c in range(nc):
                for r in range(gm):
                    walk.append((r0 + grp * gm + r, c0 + c))
        walks.append(walk)
    return [walks[l % G][l // G] for l in range(RB * NB)]


def producer_block(order: int, p: int, M: int, N: int, P: int, BM: int, BN: int, group_m: int = 1):
    """Map logical position p to (d, l, mb, nb): destination partition,
    index inside the partition (its walk), and the block's row / column
    index in the M/BM x N/BN block grid."""
    MB, NB = M // BM, N // BN
    rows_per_part = (M // P) // BM          # block rows in one partition
    if not 0 <= p < MB * NB:
        raise ValueError("position out of range")
    walk = partition_walk(rows_per_part, NB, P, group_m)
    if order == INTERLEAVED:
        d = p % P                            # Equation 1
        l = p // P
        r, c = walk[l]
        mb, nb = d * rows_per_part + r, c
    elif order in (ROW_MAJOR, M_MAJOR):
        if order == ROW_MAJOR:
            mb, nb = p // NB, p % NB
        else:
            mb, nb = p % MB, p // MB
        d = mb // rows_per_part
        l = walk.index((mb % rows_per_part, nb))
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


def full_schedule(order: int, M: int, N: int, P: int, BM: int, BN: int, group_m: int = 1):
    """Per logical position: (d, l, mb, nb, [(t, tile_row, tile_col), ...])."""
    nblocks = (M // BM) * (N // BN)
    sched = []
    for p in range(nblocks):
        d, l, mb, nb = producer_block(order, p, M, N, P, BM, BN, group_m)
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
