// tile_reducer.h - the consumer: a persistent grid of x workgroups that
// reduces 128 x 128 tiles as soon as all their contributions are published
// (paper Section 3.1 "Matching task order", Section 4.2 ReduceTile).
//
// Workgroup j walks tiles j, j+x, j+2x, ... of its partition in producer
// order.  For each tile, lanes 0 .. P-1 of the first wave poll the local flag
// and the P-1 peer flags together (one memory round trip per poll instead of
// P), then one lane issues an acquire fence and the workgroup synchronises.
// The workgroup then reduces the tile: every element is initialised from the
// local bf16 contribution, the peer values are added in rank order in fp32,
// and the result is rounded to bf16 (nearest even) and stored once - each
// output element has a single writer.
//
// Data movement: a tile row is 256 bytes = 16 lanes x 16 bytes, so each wave
// moves 4 full rows per instruction (coalesced).  Contributions are read once
// and the output written once, so both use non-temporal accesses to keep the
// producer's A/B panels in cache.  A reducer CU is bound by how many bytes it
// keeps in flight, so each lane issues up to 32 independent 16-byte loads
// (G vectors of every contribution) before consuming any, and the first poll
// of the next tile's flags is issued right behind the current tile's loads,
// so its round trip overlaps theirs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/entwine.h"
#include "flags.h"
#include "tile_order.h"

namespace entwine {

struct ReduceArgs {
  const uint16_t* partial;
  const uint16_t* peers[ENTWINE_MAX_P - 1];
  uint16_t* out;
  int64_t ldc, ldp, ldo;
  int M, N, dest, x, BM, BN, group_m;
  const int* flags;        // local flags, one per global tile
  const int* peer_flags;   // (P-1) x ntiles synthetic peer flags
  uint32_t epoch;
  int* status;             // {code, tile, src}
  uint64_t timeout_ticks;  // bound on one tile's waits, wall-clock ticks
  int publish_peers;       // 1: publish the synthetic peers' flags of this
                           // workgroup's tiles before consuming them
  int withhold_peer;       // with publish_peers: peer left unpublished, or -1
  unsigned int* task_ctr;  // dynamic tasks: {next task, finished workgroups}
  int ntasks;              // dynamic tasks of this call
  int call_tiles;          // tiles the call reduces (their peer flags are published)
  // Layer epilogue (residual addition + RMSNorm after the reduce-scatter):
  // tasks are output rows; `out` receives the residual stream h = sum +
  // residual and `y` the normalised rows.
  int layer;
  const uint16_t* residual;  // rows like `out`, leading dimension ldr
  int64_t ldr, ldy;
  const uint16_t* gamma;     // N weights
  uint16_t* y;
  float eps;
};

typedef uint32_t r_u32x4_t __attribute__((ext_vector_type(4)));
typedef float r_f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 r_bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t rnd_pack_bf16x2(float lo, float hi) {
  r_f32x2_t f = {lo, hi};
  r_bf16x2_t b = __builtin_convertvector(f, r_bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ r_u32x4_t ld_stream(const uint16_t* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const r_u32x4_t*>(p));
}

__device__ __forceinline__ r_u32x4_t ld_stream_at(const uint16_t* base, uint32_t byte_off) {
  return __builtin_nontemporal_load(reinterpret_cast<const r_u32x4_t*>(reinterpret_cast<const char*>(base) + byte_off));
}

constexpr int pow2_floor(int v) {
  int p = 1;
  while (p * 2 <= v) p *= 2;
  return p;
}

// Dynamic reduction tasks are 1 / kTaskSplit of a tile (kTile / kTaskSplit
// rows): small enough that the end of a call, when every workgroup reduces,
// splits evenly, large enough to keep each lane's loads in flight.
constexpr int kTaskSplit = 2;

// Flag polled by lane `lane` of a waiting wave for global tile gt: lane 0
// the local flag, lane q+1 peer q's.
__device__ __forceinline__ const int* flag_of_lane(const ReduceArgs& a, int lane, int ntiles, int gt) {
  return lane == 0 ? a.flags + gt : a.peer_flags + static_cast<int64_t>(lane - 1) * ntiles + gt;
}

// One wave (lanes 0 .. np-1 poll): wait until every flag of tile gt equals
// the epoch (`seen` holds a first poll already made by this lane), sleeping
// `nap` units between polls.  Returns false, after recording the timeout in
// the status word, if the deadline passes first.
__device__ __forceinline__ bool wave_await_tile(const ReduceArgs& a, int gt, int ntiles, int np, int seen, int nap) {
  const int lane = threadIdx.x & 63;
  const bool poller = lane < np;
  const int epoch = static_cast<int>(a.epoch);
  bool ready = !poller || seen == epoch;
  const uint64_t deadline = wall_clock64() + a.timeout_ticks;
  while (__ballot(!ready) != 0) {
    if (wall_clock64() > deadline) {
      const int first = __builtin_ctzll(__ballot(!ready));
      if (lane == 0 && atomicCAS(a.status, 0, ENTWINE_ETIMEOUT) == 0) {
        atomicExch(a.status + 1, gt);
        atomicExch(a.status + 2, first == 0 ? -1 : first - 1);   // -1 local, q peer q
      }
      return false;
    }
    if (nap > 1) __builtin_amdgcn_s_sleep(8);
    else __builtin_amdgcn_s_sleep(1);
    if (!ready) ready = poll_relaxed(flag_of_lane(a, lane, ntiles, gt)) == epoch;
  }
  return true;
}

// Reduces ROWS rows of global tile gt, starting at row `row0` of the tile,
// with THREADS threads: every element starts from the local contribution,
// the peers are added in rank order in fp32, the result is rounded to bf16
// and stored once.  G vectors of every contribution are loaded per lane
// before any is consumed (at most MAXLOADS loads in flight per lane);
// `after_first_loads` runs right after the first batch of loads is issued
// (used to overlap a flag poll).
template <int THREADS, int NP, int ROWS = kTile, int MAXLOADS = 32, typename Hook>
__device__ __forceinline__ void reduce_tile(const ReduceArgs& a, int gt, int tiles_n, int row0, Hook after_first_loads) {
  constexpr int VPT = (ROWS * kTile * 2 / 16) / THREADS;   // 16-byte vectors per thread
  constexpr int GMAX = MAXLOADS / NP;                       // loads in flight per lane <= MAXLOADS
  constexpr int G = pow2_floor(VPT < GMAX ? VPT : GMAX);    // vectors per batch
  static_assert(VPT >= 1 && VPT % G == 0, "batch must divide the per-thread vectors");
  const int64_t grow0 = static_cast<int64_t>(gt / tiles_n) * kTile + row0;
  const int64_t gcol0 = static_cast<int64_t>(gt % tiles_n) * kTile;
  const int64_t orow0 = a.dest >= 0 ? grow0 - static_cast<int64_t>(a.dest) * (a.M / NP) : grow0;
#pragma unroll
  for (int v0 = 0; v0 < VPT; v0 += G) {
    r_u32x4_t lv[G];
    r_u32x4_t pv[NP > 1 ? NP - 1 : 1][G];
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      const int v = threadIdx.x + THREADS * (v0 + gi);
      const int64_t r = v >> 4, cc = (v & 15) * 8;
      lv[gi] = ld_stream(a.partial + (grow0 + r) * a.ldc + gcol0 + cc);
#pragma unroll
      for (int q = 0; q < NP - 1; ++q) pv[q][gi] = ld_stream(a.peers[q] + (grow0 + r) * a.ldp + gcol0 + cc);
    }
    if (v0 == 0) after_first_loads();
#pragma unroll
    for (int gi = 0; gi < G; ++gi) {
      float acc[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = __builtin_bit_cast(float, lv[gi][e] << 16);
        acc[2 * e + 1] = __builtin_bit_cast(float, lv[gi][e] & 0xffff0000u);
      }
#pragma unroll
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += __builtin_bit_cast(float, pv[q][gi][e] << 16);
          acc[2 * e + 1] += __builtin_bit_cast(float, pv[q][gi][e] & 0xffff0000u);
        }
      r_u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = rnd_pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
      const int v = threadIdx.x + THREADS * (v0 + gi);
      const int64_t r = v >> 4, cc = (v & 15) * 8;
      __builtin_nontemporal_store(o, reinterpret_cast<r_u32x4_t*>(a.out + (orow0 + r) * a.ldo + gcol0 + cc));
    }
  }
}

// The reducer role of workgroup j of x (blockDim.x == THREADS), with the
// paper's static task order (tiles j, j+x, ... of its partition); `s_abort`
// is one int of LDS.  Used by tile_reducer.
template <int THREADS, int NP>
__device__ __forceinline__ void reducer_body(const ReduceArgs& a, const int j, int& s_abort) {
  static_assert(NP <= 64, "one polling lane per contribution");
  const BlockGrid grid = make_grid(a.M, a.N, NP, a.BM, a.BN, a.group_m);
  const int Q = tiles_per_partition(a.M, a.N, NP);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const ConsumerSeq seq = consumer_seq(a.dest, NP, a.x, j);
  const int lane = threadIdx.x & 63;
  const bool poller = threadIdx.x < NP;       // lanes 0 .. NP-1 of wave 0
  const int epoch = static_cast<int>(a.epoch);

  auto global_tile = [&](int t) {
    int tr, tc;
    tile_of_number(seq.part, t, grid, &tr, &tc);
    return tr * tiles_n + tc;
  };

  // Synthetic peers: their producers have nothing left to compute on this
  // GPU, so the flags of this workgroup's tiles are published up front, by
  // the lanes that poll them.
  if (a.publish_peers && threadIdx.x >= 1 && threadIdx.x < NP && threadIdx.x - 1 != a.withhold_peer) {
    for (int tt = seq.first; tt < Q; tt += seq.stride)
      publish_relaxed(const_cast<int*>(a.peer_flags) + static_cast<int64_t>(threadIdx.x - 1) * ntiles + global_tile(tt),
                      a.epoch);
  }

  int t = seq.first;
  if (t >= Q) return;
  int gt = global_tile(t);
  int seen = poller ? poll_relaxed(flag_of_lane(a, lane, ntiles, gt)) : epoch;
  while (true) {
    if (threadIdx.x < 64) {
      const bool ok = wave_await_tile(a, gt, ntiles, NP, seen, 1);
      if (ok && lane == 0) acquire_fence();
      if (lane == 0) s_abort = !ok;
    }
    __syncthreads();
    if (s_abort) return;
    const int tn = t + seq.stride;
    const int gtn = tn < Q ? global_tile(tn) : 0;
    seen = epoch;
    // The first poll of the next tile's flags rides behind this tile's loads.
    reduce_tile<THREADS, NP>(a, gt, tiles_n, 0, [&] {
      if (poller && tn < Q) seen = poll_relaxed(flag_of_lane(a, lane, ntiles, gtn));
    });
    if (tn >= Q) break;
    t = tn;
    gt = gtn;
    __syncthreads();   // s_abort is rewritten next
  }
}

// Publishes, as part of one launch, the synthetic peers' flags of the
// a.call_tiles tiles the call reduces, split over all nb workgroups; peer
// `withhold_peer` stays unpublished.
__device__ __forceinline__ void publish_peer_slice(const ReduceArgs& a, int np, int b, int nb) {
  const BlockGrid grid = make_grid(a.M, a.N, np, a.BM, a.BN, a.group_m);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const int call_tiles = a.call_tiles;
  const int64_t n = static_cast<int64_t>(np - 1) * call_tiles;
  for (int64_t i = static_cast<int64_t>(b) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(nb) * blockDim.x) {
    const int q = static_cast<int>(i / call_tiles), u = static_cast<int>(i % call_tiles);
    if (q == a.withhold_peer) continue;
    const int part = a.dest >= 0 ? a.dest : u % np;
    const int idx = a.dest >= 0 ? u : u / np;
    int tr, tc;
    tile_of_number(part, idx, grid, &tr, &tc);
    publish_relaxed(const_cast<int*>(a.peer_flags) + static_cast<int64_t>(q) * ntiles + tr * tiles_n + tc, a.epoch);
  }
}

// The reducer role with dynamic tasks: workgroups take tile parts (SPLIT per
// tile, kTaskSplit in the fused launch) from a device counter in consumer
// order (task t is part t % SPLIT of tile u = t / SPLIT of the destination's
// partition; with every destination, tile u / P of partition u % P, which
// interleaves the partitions as Equation 1 does), so the dedicated reducers
// and every producer that has finished its blocks share the remaining work;
// parts keep every workgroup busy when a chunk has fewer tiles than the
// device has CUs.  `taken`, if not ~0u, is the first task, already taken.
// Each workgroup ends with one failed take; the last workgroup of the grid to
// finish returns both counters to zero, ready for the next call.  After a
// timeout waits are skipped (the call's output is then undefined) but the
// task accounting stays exact.  s: two ints of LDS.
template <int THREADS, int NP, int SPLIT>
__device__ __forceinline__ void reducer_dynamic(const ReduceArgs& a, int* s, unsigned long long* first_ready,
                                                unsigned int taken) {
  static_assert(kTile % SPLIT == 0 && SPLIT >= 1, "a task is kTile / SPLIT rows of a tile");
  const BlockGrid grid = make_grid(a.M, a.N, NP, a.BM, a.BN, a.group_m);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const int lane = threadIdx.x & 63;
  auto task_tile = [&](int task) {
    const int u = task / SPLIT;
    const int part = a.dest >= 0 ? a.dest : u % NP;
    const int idx = a.dest >= 0 ? u : u / NP;
    int tr, tc;
    tile_of_number(part, idx, grid, &tr, &tc);
    return tr * tiles_n + tc;
  };
  __syncthreads();   // producer waves are done with the LDS
  if (threadIdx.x == 0) s[0] = static_cast<int>(taken != ~0u ? taken : atomicAdd(a.task_ctr, 1u));
  __syncthreads();
  int task = s[0];
  bool timed_out = false;   // wave 0
  if (first_ready && threadIdx.x == 0) *first_ready = 0;
  while (task < a.ntasks) {
    const int gt = task_tile(task);
    const int row0 = (task % SPLIT) * (kTile / SPLIT);
    if (threadIdx.x < 64) {
      // The next task is taken now and stored once this one's flags are in,
      // so the two round trips overlap.
      const unsigned int nxt = threadIdx.x == 0 ? atomicAdd(a.task_ctr, 1u) : 0u;
      if (!timed_out) {
        const int seen = lane < NP ? poll_relaxed(flag_of_lane(a, lane, ntiles, gt)) : static_cast<int>(a.epoch);
        timed_out = !wave_await_tile(a, gt, ntiles, NP, seen, 8);
      }
      if (lane == 0) {
        acquire_fence();
        s[1] = static_cast<int>(nxt);
      }
    }
    __syncthreads();
    if (first_ready && threadIdx.x == 0) {
      *first_ready = wall_clock64();
      first_ready = nullptr;
    }
    const int next = s[1];
    reduce_tile<THREADS, NP, kTile / SPLIT>(a, gt, tiles_n, row0, [] {});
    __syncthreads();   // s[1] is rewritten next
    task = next;
  }
  if (threadIdx.x == 0 && atomicAdd(a.task_ctr + 1, 1u) == gridDim.x - 1) {
    atomicExch(a.task_ctr, 0u);
    atomicExch(a.task_ctr + 1, 0u);
  }
}

// ------------------------------------------------------------ layer epilogue
// Residual addition and RMSNorm after the reduce-scatter (paper Section 5.2,
// layer-level evaluation), as tasks of the same launch.  A task is one output
// row over all N columns: each of its 256 threads owns 8 columns in every
// step of 2048, reduces them exactly as ReduceTile does (local contribution,
// then the peers in rank order, in fp32), adds the residual in fp32, stores
// the bf16 residual stream h and keeps it in registers.  The row's sum of
// squares of the stored h is folded across the workgroup through the LDS, and
// y = bf16(h * (sum / N + eps)^(-1/2) * gamma) is stored next.  A row needs
// every tile of its tile row, so wave 0 waits for all of their flags; the
// first poll for the next task's tile row is issued behind the current row's
// first loads.  A task writes only its own row, which nothing else in the call
// reads, so it publishes nothing.
constexpr int kLayerThreads = 256;
constexpr int kLayerCols = kLayerThreads * 8;   // columns per step
constexpr int kLayerMaxSteps = 8;
constexpr int kLayerMaxN = kLayerCols * kLayerMaxSteps;

// Lane `lane` of wave 0: are the NP flags of every tile it checks in tile row
// tr (columns lane, lane + 64, ...) at the epoch?
template <int NP>
__device__ __forceinline__ bool row_flags_ready(const ReduceArgs& a, int tr, int tiles_n, int ntiles) {
  const int epoch = static_cast<int>(a.epoch);
  bool ok = true;
  for (int tc = threadIdx.x & 63; tc < tiles_n; tc += 64) {
#pragma unroll
    for (int q = 0; q < NP; ++q) ok &= poll_relaxed(flag_of_lane(a, q, ntiles, tr * tiles_n + tc)) == epoch;
  }
  return ok;
}

// Wave 0: wait until every flag of tile row tr is at the epoch (`ok` is this
// lane's first poll).  On timeout records the first missing flag's tile and
// source (-1 local, q peer q) and returns false.
template <int NP>
__device__ __forceinline__ bool wave_await_row(const ReduceArgs& a, int tr, int tiles_n, int ntiles, bool ok) {
  const int epoch = static_cast<int>(a.epoch);
  const uint64_t deadline = wall_clock64() + a.timeout_ticks;
  while (__ballot(!ok) != 0) {
    if (wall_clock64() > deadline) {
      if ((threadIdx.x & 63) == __builtin_ctzll(__ballot(!ok))) {
        int tile = tr * tiles_n, src = -1;   // this lane's first missing flag
        for (int tc = threadIdx.x & 63, found = 0; tc < tiles_n && !found; tc += 64)
          for (int q = 0; q < NP && !found; ++q)
            if (poll_relaxed(flag_of_lane(a, q, ntiles, tr * tiles_n + tc)) != epoch) {
              tile = tr * tiles_n + tc;
              src = q - 1;
              found = 1;
            }
        if (atomicCAS(a.status, 0, ENTWINE_ETIMEOUT) == 0) {
          atomicExch(a.status + 1, tile);
          atomicExch(a.status + 2, src);
        }
      }
      return false;
    }
    __builtin_amdgcn_s_sleep(8);
    if (!ok) ok = row_flags_ready<NP>(a, tr, tiles_n, ntiles);
  }
  return true;
}

// Loads of one batch of output row `orow` (kLayerBatch steps of 2048
// columns from step s0): this thread's 16 bytes of the local contribution, of
// every peer and of the residual, per step.
constexpr int kLayerBatch = 4;
static_assert(kLayerMaxSteps % kLayerBatch == 0, "batches tile the steps");

template <int NP>
struct LayerLoads {
  r_u32x4_t lv[kLayerBatch], rv[kLayerBatch];
  r_u32x4_t pv[NP > 1 ? NP - 1 : 1][kLayerBatch];
};

template <int NP>
__device__ __forceinline__ void layer_issue(const ReduceArgs& a, int64_t orow, int s0, LayerLoads<NP>& L) {
  const int64_t grow = orow + (a.dest >= 0 ? static_cast<int64_t>(a.dest) * (a.M / NP) : 0);
  const int c0 = threadIdx.x * 8;
#pragma unroll
  for (int b = 0; b < kLayerBatch; ++b) {
    const int c = (s0 + b) * kLayerCols + c0;
    if (c < a.N) {
      L.lv[b] = ld_stream(a.partial + grow * a.ldc + c);
#pragma unroll
      for (int q = 0; q < NP - 1; ++q) L.pv[q][b] = ld_stream(a.peers[q] + grow * a.ldp + c);
      L.rv[b] = ld_stream(a.residual + orow * a.ldr + c);
    }
  }
}

// Consumes a batch: h = bf16(local + peers in rank order + residual) in fp32,
// stored to `out` and kept in h[]; returns this thread's sum of squares of
// the stored h.
template <int NP>
__device__ __forceinline__ float layer_consume(const ReduceArgs& a, int64_t orow, int s0, const LayerLoads<NP>& L,
                                               r_u32x4_t* h) {
  const int c0 = threadIdx.x * 8;
  float ss = 0.0f;
#pragma unroll
  for (int b = 0; b < kLayerBatch; ++b) {
    const int c = (s0 + b) * kLayerCols + c0;
    h[s0 + b] = r_u32x4_t{0u, 0u, 0u, 0u};
    if (c >= a.N) continue;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] = __builtin_bit_cast(float, L.lv[b][e] << 16);
      acc[2 * e + 1] = __builtin_bit_cast(float, L.lv[b][e] & 0xffff0000u);
    }
#pragma unroll
    for (int q = 0; q < NP - 1; ++q)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += __builtin_bit_cast(float, L.pv[q][b][e] << 16);
        acc[2 * e + 1] += __builtin_bit_cast(float, L.pv[q][b][e] & 0xffff0000u);
      }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += __builtin_bit_cast(float, L.rv[b][e] << 16);
      acc[2 * e + 1] += __builtin_bit_cast(float, L.rv[b][e] & 0xffff0000u);
    }
    r_u32x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = rnd_pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
      const float lo = __builtin_bit_cast(float, o[e] << 16);
      const float hi = __builtin_bit_cast(float, o[e] & 0xffff0000u);
      ss += lo * lo + hi * hi;
    }
    h[s0 + b] = o;
    __builtin_nontemporal_store(o, reinterpret_cast<r_u32x4_t*>(a.out + orow * a.ldo + c));
  }
  return ss;
}

// The layer epilogue's task loop (blockDim.x == kLayerThreads): output rows
// taken from the device counter in order, each once all tiles of its tile
// row are published; counters returned to zero as in reducer_dynamic.
// Rows are pipelined: once a row's h is stored, wave 0 takes the next row
// and checks its tile row's flags; if they are all in, the next row's loads
// are issued right after the workgroup barrier that folds the current row's
// sum of squares, before the current row's y is computed and stored, so the
// workgroup keeps loads in flight between rows.  Otherwise the next row
// waits at the top of the loop as the first one does.
// s: sixteen ints of LDS (task ids, early-issue flags, two sets of row sums).
template <int NP>
__device__ __forceinline__ void reducer_layer(const ReduceArgs& a, int* s, unsigned int taken) {
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const int steps = (a.N + kLayerCols - 1) / kLayerCols;
  const int64_t first_row = a.dest >= 0 ? static_cast<int64_t>(a.dest) * (a.M / NP) : 0;
  auto tile_row = [&](int task) { return static_cast<int>((first_row + task) / kTile); };
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float* red = reinterpret_cast<float*>(s + 8);   // [2][4]: row sums, alternating by row
  // gamma is the same for every row: loaded once, kept in registers (an
  // input of the call, so no acquire orders it).
  r_u32x4_t g[kLayerMaxSteps];
#pragma unroll
  for (int st = 0; st < kLayerMaxSteps; ++st) {
    const int c = st * kLayerCols + threadIdx.x * 8;
    g[st] = c < a.N ? *reinterpret_cast<const r_u32x4_t*>(a.gamma + c) : r_u32x4_t{0u, 0u, 0u, 0u};
  }
  __syncthreads();   // producer waves are done with the LDS
  if (threadIdx.x == 0) s[0] = static_cast<int>(taken != ~0u ? taken : atomicAdd(a.task_ctr, 1u));
  __syncthreads();
  int task = s[0];
  bool timed_out = false;   // wave 0
  bool issued = false;      // this task's first batch of loads is in flight
  int parity = 0;
  LayerLoads<NP> L;
  while (task < a.ntasks) {
    if (!issued) {
      if (threadIdx.x < 64) {
        const int tr = tile_row(task);
        if (!timed_out) timed_out = !wave_await_row<NP>(a, tr, tiles_n, ntiles, row_flags_ready<NP>(a, tr, tiles_n, ntiles));
        if (lane == 0) acquire_fence();
      }
      __syncthreads();
      layer_issue<NP>(a, task, 0, L);
    }
    // The next task, taken while this row's loads are in flight.
    int next_w0 = 0;
    if (threadIdx.x < 64) {
      const unsigned int nx = lane == 0 ? atomicAdd(a.task_ctr, 1u) : 0u;
      next_w0 = static_cast<int>(__shfl(nx, 0));
    }
    r_u32x4_t h[kLayerMaxSteps];
    float ss = layer_consume<NP>(a, task, 0, L, h);
#pragma unroll
    for (int s0 = kLayerBatch; s0 < kLayerMaxSteps; s0 += kLayerBatch) {
      if (s0 < steps) {
        layer_issue<NP>(a, task, s0, L);
        ss += layer_consume<NP>(a, task, s0, L, h);
      } else {
#pragma unroll
        for (int b = 0; b < kLayerBatch; ++b) h[s0 + b] = r_u32x4_t{0u, 0u, 0u, 0u};
      }
    }
    // Wave 0: are the next row's flags all in?  Then acquire now.
    if (threadIdx.x < 64) {
      bool ready = false;
      if (next_w0 < a.ntasks && !timed_out) {
        ready = __ballot(!row_flags_ready<NP>(a, tile_row(next_w0), tiles_n, ntiles)) == 0;
        if (ready && lane == 0) acquire_fence();
      }
      if (lane == 0) {
        s[1 + parity] = next_w0;
        s[3 + parity] = ready;
      }
    }
    ss += __shfl_xor(ss, 32);
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 8);
    ss += __shfl_xor(ss, 4);
    ss += __shfl_xor(ss, 2);
    ss += __shfl_xor(ss, 1);
    if (lane == 0) red[4 * parity + wave] = ss;
    __syncthreads();   // row sums, the next task and its readiness are visible; loads after the acquire
    static_assert(kLayerThreads == 256, "four wave sums");
    const float* rs = red + 4 * parity;
    const float rstd = rsqrtf(((rs[0] + rs[1]) + (rs[2] + rs[3])) * (1.0f / static_cast<float>(a.N)) + a.eps);
    const int next = s[1 + parity];
    const bool early = s[3 + parity] != 0;
    if (early) layer_issue<NP>(a, next, 0, L);
#pragma unroll
    for (int st = 0; st < kLayerMaxSteps; ++st) {
      const int c = st * kLayerCols + threadIdx.x * 8;
      if (st >= steps || c >= a.N) continue;
      r_u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = __builtin_bit_cast(float, h[st][e] << 16) * rstd * __builtin_bit_cast(float, g[st][e] << 16);
        const float hi = __builtin_bit_cast(float, h[st][e] & 0xffff0000u) * rstd *
                         __builtin_bit_cast(float, g[st][e] & 0xffff0000u);
        o[e] = rnd_pack_bf16x2(lo, hi);
      }
      __builtin_nontemporal_store(o, reinterpret_cast<r_u32x4_t*>(a.y + task * a.ldy + c));
    }
    task = next;
    issued = early;
    parity ^= 1;
  }
  if (threadIdx.x == 0 && atomicAdd(a.task_ctr + 1, 1u) == gridDim.x - 1) {
    atomicExch(a.task_ctr, 0u);
    atomicExch(a.task_ctr + 1, 0u);
  }
}

template <int THREADS, int NP>
__global__ __launch_bounds__(THREADS) void tile_reducer(ReduceArgs a) {
  __shared__ int s_abort;
  reducer_body<THREADS, NP>(a, blockIdx.x, s_abort);
}

// The shared-pool form (paper Section 5.3.2, shared versus partitioned
// resources): reducer workgroups small enough to sit beside a producer
// workgroup on the same CU, so the reduction is spread over every CU instead
// of taking CUs away from the GEMM.  A producer wave holds at most 448 of the
// 512 registers per lane of its SIMD and the producer fills the LDS, so a
// reducer wave here uses at most 64 registers and no LDS.
//   * Only wave 0 polls a tile's flags (lanes 0 .. P-1), backing off between
//     polls, so idle reducers take few issue slots and memory requests from
//     the producer beside them; the other waves wait at the workgroup
//     barrier, which needs no LDS.
//   * After the barrier every wave reads the flags once itself and acquires,
//     then reduces its own quarter of the tile (32 rows, 16-byte lanes, one
//     vector of every contribution in flight per lane).
//   * No wave leaves early, so every wave reaches every barrier.  After a
//     timeout (recorded in the status word) wave 0 stops waiting; the output
//     of such a call is undefined.
template <int NP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(8, 8))) void tile_reducer_shared(ReduceArgs a) {
  const BlockGrid grid = make_grid(a.M, a.N, NP, a.BM, a.BN, a.group_m);
  const int Q = tiles_per_partition(a.M, a.N, NP);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const ConsumerSeq seq = consumer_seq(a.dest, NP, a.x, blockIdx.x);
  const int chunk_rows = a.M / NP;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool poller = lane < NP;
  const int epoch = static_cast<int>(a.epoch);

  auto global_tile = [&](int t) {
    int tr, tc;
    tile_of_number(seq.part, t, grid, &tr, &tc);
    return tr * tiles_n + tc;
  };
  auto flag_of = [&](int gt) {
    return lane == 0 ? a.flags + gt : a.peer_flags + static_cast<int64_t>(lane - 1) * ntiles + gt;
  };
  if (a.publish_peers && wave == 0 && lane >= 1 && lane < NP && lane - 1 != a.withhold_peer) {
    for (int tt = seq.first; tt < Q; tt += seq.stride)
      publish_relaxed(const_cast<int*>(a.peer_flags) + static_cast<int64_t>(lane - 1) * ntiles + global_tile(tt),
                      a.epoch);
  }

  bool timed_out = false;   // wave 0 only
  for (int t = seq.first; t < Q; t += seq.stride) {
    const int gt = global_tile(t);
    if (wave == 0 && !timed_out) {
      bool ready = !poller || poll_relaxed(flag_of(gt)) == epoch;
      const uint64_t deadline = wall_clock64() + a.timeout_ticks;
      while (__ballot(!ready) != 0) {
        if (wall_clock64() > deadline) {
          const int first = __builtin_ctzll(__ballot(!ready));
          if (lane == 0 && atomicCAS(a.status, 0, ENTWINE_ETIMEOUT) == 0) {
            atomicExch(a.status + 1, gt);
            atomicExch(a.status + 2, first == 0 ? -1 : first - 1);
          }
          timed_out = true;
          break;
        }
        __builtin_amdgcn_s_sleep(8);
        if (!ready) ready = poll_relaxed(flag_of(gt)) == epoch;
      }
    }
    __builtin_amdgcn_s_barrier();
    // This wave's own observation of the (monotonic) flags, then acquire.
    if (poller) (void)poll_relaxed(flag_of(gt));
    acquire_fence();

    const int64_t grow0 = static_cast<int64_t>(gt / tiles_n) * kTile + wave * 32;
    const int64_t gcol0 = static_cast<int64_t>(gt % tiles_n) * kTile;
    const int64_t orow0 = a.dest >= 0 ? grow0 - static_cast<int64_t>(a.dest) * chunk_rows : grow0;
    // Byte offsets fit 32 bits (checked on the host), so each load is a
    // wave-uniform base plus one per-lane offset register.
#pragma unroll 1
    for (int i = 0; i < 8; ++i) {
      const int v = lane + 64 * i;
      const int64_t r = v >> 4, cc = (v & 15) * 8;
      const uint32_t offc = static_cast<uint32_t>(((grow0 + r) * a.ldc + gcol0 + cc) * 2);
      const uint32_t offp = static_cast<uint32_t>(((grow0 + r) * a.ldp + gcol0 + cc) * 2);
      const r_u32x4_t lv = ld_stream_at(a.partial, offc);
      r_u32x4_t pv[NP > 1 ? NP - 1 : 1];
#pragma unroll
      for (int q = 0; q < NP - 1; ++q) pv[q] = ld_stream_at(a.peers[q], offp);
      float acc[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] = __builtin_bit_cast(float, lv[e] << 16);
        acc[2 * e + 1] = __builtin_bit_cast(float, lv[e] & 0xffff0000u);
      }
#pragma unroll
      for (int q = 0; q < NP - 1; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += __builtin_bit_cast(float, pv[q][e] << 16);
          acc[2 * e + 1] += __builtin_bit_cast(float, pv[q][e] & 0xffff0000u);
        }
      r_u32x4_t o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = rnd_pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
      const uint32_t offo = static_cast<uint32_t>(((orow0 + r) * a.ldo + gcol0 + cc) * 2);
      __builtin_nontemporal_store(o, reinterpret_cast<r_u32x4_t*>(reinterpret_cast<char*>(a.out) + offo));
    }
  }
}

// Publishes the synthetic peers' flags for this call (they stand in for the
// other ranks' producers, which on one GPU have nothing left to compute).
// `skip_peer` >= 0 withholds that peer's flags (test hook for the timeout).
__global__ void publish_fill(int* flags, int64_t n, int64_t per_peer, int skip_peer, uint32_t epoch) {
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    if (skip_peer >= 0 && i / per_peer == skip_peer) continue;
    flags[i] = static_cast<int>(epoch);
  }
}

}  // namespace entwine
