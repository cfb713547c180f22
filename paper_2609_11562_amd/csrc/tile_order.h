// tile_order.h - producer traversal and consumer task maps, usable on host
// and device.
//
// Paper Section 3.1: output partition d (P equal row chunks) collects the
// tiles reduced by destination d.  Interleaved production (Equation 1) maps a
// producer block's logical position p to destination d = p mod P and index
// l = p div P inside that partition.  The comparison orders are the
// partition-contiguous traversal (N fastest over the whole output, Figure 1
// top) and the M-major default traversal of the ablation (Section 5.3.1).
//
// Order of the blocks inside a partition (what l means).  With group_m <= 1
// it is the paper's N-major walk (column index fastest), the consumer's
// order.  With group_m > 1 it is an L2-friendly walk for a GPU whose
// workgroups are dispatched round-robin over 8 XCDs (workgroup b runs on XCD
// b mod 8, each XCD with its own L2): position p = P l + d lands on XCD
// (P l + d) mod 8, so when P divides 8 the partition is served by G = 8 / P
// XCDs and l mod G says which.  The partition is cut into G stripes (column
// stripes, else row stripes), stripe s = l mod G, and inside a stripe the
// blocks are walked in groups of group_m block rows, M fastest within a group
// (so the ~32 blocks an XCD runs at once form a compact patch that shares A
// and B panels in its L2).  Equation 1 across partitions is unchanged, and
// the consumer still follows production order.
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
constexpr int kXcds = 8;

struct BlockGrid {
  int MB, NB;          // block rows / cols of the M x N output
  int RB;              // block rows in one partition (M/P/BM)
  int P;
  int TBM, TBN;        // tiles per block along M / N (BM/128, BN/128)
  // within-partition walk (group_m > 1)
  int grouped;         // 0: N-major
  int G;               // stripes per partition
  int col_stripes;     // 1: stripes split columns, 0: rows
  int SR, SC;          // stripe size in blocks (rows, cols)
  int gm;              // rows per group inside a stripe (divides SR)
};

ENTWINE_HD BlockGrid make_grid(int M, int N, int P, int BM, int BN, int group_m = 1) {
  BlockGrid g;
  g.MB = M / BM;
  g.NB = N / BN;
  g.RB = (M / P) / BM;
  g.P = P;
  g.TBM = BM / kTile;
  g.TBN = BN / kTile;
  g.grouped = group_m > 1;
  g.G = (P <= kXcds && kXcds % P == 0) ? kXcds / P : 1;
  if (g.NB % g.G == 0) {
    g.col_stripes = 1;
    g.SR = g.RB;
    g.SC = g.NB / g.G;
  } else if (g.RB % g.G == 0) {
    g.col_stripes = 0;
    g.SR = g.RB / g.G;
    g.SC = g.NB;
  } else {
    g.G = 1;
    g.col_stripes = 1;
    g.SR = g.RB;
    g.SC = g.NB;
  }
  g.gm = 1;
  for (int k = (group_m < g.SR ? group_m : g.SR); k >= 1; --k)
    if (g.SR % k == 0) {
      g.gm = k;
      break;
    }
  return g;
}

// Index l inside a partition -> (row, col) of the block inside the partition.
ENTWINE_HD void partition_block(int l, const BlockGrid& g, int* r, int* c) {
  if (!g.grouped) {
    *r = l / g.NB;
    *c = l % g.NB;
    return;
  }
  const int s = l % g.G, u = l / g.G;
  const int per_group = g.gm * g.SC;
  const int grp = u / per_group, w = u % per_group;
  const int rr = grp * g.gm + w % g.gm;      // M fastest inside a group
  const int cc = w / g.gm;
  if (g.col_stripes) {
    *r = rr;
    *c = s * g.SC + cc;
  } else {
    *r = s * g.SR + rr;
    *c = cc;
  }
}

ENTWINE_HD int partition_index(int r, int c, const BlockGrid& g) {
  if (!g.grouped) return r * g.NB + c;
  int s, rr, cc;
  if (g.col_stripes) {
    s = c / g.SC;
    cc = c % g.SC;
    rr = r;
  } else {
    s = r / g.SR;
    rr = r % g.SR;
    cc = c;
  }
  const int u = (rr / g.gm) * (g.gm * g.SC) + cc * g.gm + rr % g.gm;
  return u * g.G + s;
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
    int r, c;
    partition_block(b.l, g, &r, &c);
    b.mb = b.d * g.RB + r;
    b.nb = c;
  } else {
    if (order == 1) {          // partition-contiguous, N fastest
      b.mb = p / g.NB;
      b.nb = p % g.NB;
    } else {                   // M fastest
      b.mb = p % g.MB;
      b.nb = p / g.MB;
    }
    b.d = b.mb / g.RB;
    b.l = partition_index(b.mb % g.RB, b.nb, g);
  }
  return b;
}

// Tile number t inside partition d -> global tile coordinates.
ENTWINE_HD void tile_of_number(int d, int t, const BlockGrid& g, int* tile_row, int* tile_col) {
  const int c = g.TBM * g.TBN;
  const int l = t / c, i = t % c;
  int r, cc;
  partition_block(l, g, &r, &cc);
  *tile_row = (d * g.RB + r) * g.TBM + i / g.TBN;
  *tile_col = cc * g.TBN + i % g.TBN;
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
