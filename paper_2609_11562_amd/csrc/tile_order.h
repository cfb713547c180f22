// tile_order.h - producer traversal and consumer task maps, usable on host
// and device.
//
// Paper Section 3.1: output partition d (P equal row chunks) collects the
// tiles reduced by destination d.  Interleaved production (Equation 1) maps a
// producer block's logical position p to destination d = p mod P and index
// l = p div P inside that partition; l walks the partition's blocks N-major,
// the consumer's order.  The comparison orders are the partition-contiguous
// traversal (N fastest over the whole output, Figure 1 top) and the M-major
// default traversal of the ablation (Section 5.3.1).
//
// A BM x BN producer block covers c = (BM/128)(BN/128) reduction tiles.  In
// partition d the tiles are numbered in producer order, t = l*c + i, with i
// N-major inside the block.  Consumer workgroup j of x processes t = j, j+x,
// ... below Q, the partition's tile count ("Matching task order").
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define ENTWINE_HD __host__ __device__ __forceinline__
#else
#define ENTWINE_HD inline
#endif

namespace entwine {

constexpr int kTile = 128;

struct BlockGrid {
  int MB, NB;          // block rows / cols of the M x N output
  int rows_per_part;   // block rows in one partition (M/P/BM)
  int P;
  int TBM, TBN;        // tiles per block along M / N (BM/128, BN/128)
};

ENTWINE_HD BlockGrid make_grid(int M, int N, int P, int BM, int BN) {
  BlockGrid g;
  g.MB = M / BM;
  g.NB = N / BN;
  g.rows_per_part = (M / P) / BM;
  g.P = P;
  g.TBM = BM / kTile;
  g.TBN = BN / kTile;
  return g;
}

struct BlockPos {
  int d, l, mb, nb;
};

// Logical position p -> (partition, index in partition, block row, block col).
ENTWINE_HD BlockPos block_of_position(int order, int p, const BlockGrid& g) {
  BlockPos b;
  if (order == 0) {            // interleaved, Equation 1
    b.d = p % g.P;
    b.l = p / g.P;
    b.mb = b.d * g.rows_per_part + b.l / g.NB;
    b.nb = b.l % g.NB;
  } else {
    if (order == 1) {          // partition-contiguous, N fastest
      b.mb = p / g.NB;
      b.nb = p % g.NB;
    } else {                   // M fastest
      b.mb = p % g.MB;
      b.nb = p / g.MB;
    }
    b.d = b.mb / g.rows_per_part;
    b.l = (b.mb % g.rows_per_part) * g.NB + b.nb;
  }
  return b;
}

// Tile number t inside partition d -> global tile coordinates.
ENTWINE_HD void tile_of_number(int d, int t, const BlockGrid& g, int* tile_row, int* tile_col) {
  const int c = g.TBM * g.TBN;
  const int l = t / c, i = t % c;
  const int mb = d * g.rows_per_part + l / g.NB;
  const int nb = l % g.NB;
  *tile_row = mb * g.TBM + i / g.TBN;
  *tile_col = nb * g.TBN + i % g.TBN;
}

ENTWINE_HD int tiles_per_partition(int M, int N, int P) { return (M / P / kTile) * (N / kTile); }

// Consumer assignment.  dest >= 0: workgroup j of x takes partition dest,
// tiles j, j+x, ...  dest < 0 (every partition): x is a multiple of P and
// workgroup j takes partition j mod P, tiles (j div P), + x/P, ...
struct ConsumerSeq {
  int part, first, stride;
};

ENTWINE_HD ConsumerSeq consumer_seq(int dest, int P, int x, int j) {
  ConsumerSeq s;
  if (dest >= 0) {
    s.part = dest;
    s.first = j;
    s.stride = x;
  } else {
    s.part = j % P;
    s.first = j / P;
    s.stride = x / P;
  }
  return s;
}

}  // namespace entwine
