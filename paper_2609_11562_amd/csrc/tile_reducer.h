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

constexpr int pow2_floor(int v) {
  int p = 1;
  while (p * 2 <= v) p *= 2;
  return p;
}

// The reducer role of workgroup j of x (blockDim.x == THREADS); `s_abort`
// is one int of LDS.  Used by tile_reducer and by the single-launch fused
// kernel, whose last x workgroups are reducers.
template <int THREADS, int NP>
__device__ __forceinline__ void reducer_body(const ReduceArgs& a, const int j, int& s_abort) {
  constexpr int VPT = (kTile * kTile * 2 / 16) / THREADS;  // 16-byte vectors per thread
  constexpr int GMAX = 32 / NP;                             // loads in flight per lane <= 32
  constexpr int G = pow2_floor(VPT < GMAX ? VPT : GMAX);    // vectors per batch
  static_assert(VPT % G == 0, "batch must divide the per-thread vectors");
  static_assert(NP <= 64, "one polling lane per contribution");

  const BlockGrid grid = make_grid(a.M, a.N, NP, a.BM, a.BN, a.group_m);
  const int Q = tiles_per_partition(a.M, a.N, NP);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const ConsumerSeq seq = consumer_seq(a.dest, NP, a.x, j);
  const int chunk_rows = a.M / NP;
  const int lane = threadIdx.x & 63;
  const bool poller = threadIdx.x < NP;       // lanes 0 .. NP-1 of wave 0
  const int epoch = static_cast<int>(a.epoch);

  auto global_tile = [&](int t) {
    int tr, tc;
    tile_of_number(seq.part, t, grid, &tr, &tc);
    return tr * tiles_n + tc;
  };
  // Flag polled by this lane: lane 0 the local flag, lane q+1 peer q's.
  auto flag_of = [&](int gt) {
    return lane == 0 ? a.flags + gt : a.peer_flags + static_cast<int64_t>(lane - 1) * ntiles + gt;
  };
  // Wave 0: wait until every flag of tile gt is ready (`seen` holds a first
  // poll already made), then acquire; returns false, after recording the
  // timeout, if the deadline passes first.  Called by wave 0 only.
  auto await_tile = [&](int gt, int seen) {
    bool ready = !poller || seen == epoch;
    const uint64_t deadline = wall_clock64() + a.timeout_ticks;
    while (__ballot(!ready) != 0) {
      if (wall_clock64() > deadline) {
        const uint64_t missing = __ballot(!ready);
        const int first = __builtin_ctzll(missing);
        if (lane == 0 && atomicCAS(a.status, 0, ENTWINE_ETIMEOUT) == 0) {
          atomicExch(a.status + 1, gt);
          atomicExch(a.status + 2, first == 0 ? -1 : first - 1);   // -1 local, q peer q
        }
        return false;
      }
      __builtin_amdgcn_s_sleep(1);
      if (!ready) ready = poll_relaxed(flag_of(gt)) == epoch;
    }
    if (lane == 0) acquire_fence();
    return true;
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
  if (threadIdx.x < 64) {
    const int seen = poller ? poll_relaxed(flag_of(gt)) : epoch;
    const bool ok = await_tile(gt, seen);
    if (lane == 0) s_abort = !ok;
  }
  __syncthreads();
  if (s_abort) return;

  while (true) {
    const int64_t grow0 = static_cast<int64_t>(gt / tiles_n) * kTile;
    const int64_t gcol0 = static_cast<int64_t>(gt % tiles_n) * kTile;
    const int64_t orow0 = a.dest >= 0 ? grow0 - static_cast<int64_t>(a.dest) * chunk_rows : grow0;
    const int tn = t + seq.stride;
    const int gtn = tn < Q ? global_tile(tn) : 0;
    int seen = epoch;

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
      // First poll of the next tile's flags, behind the first batch's loads.
      if (v0 == 0 && poller && tn < Q) seen = poll_relaxed(flag_of(gtn));
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
    if (tn >= Q) break;
    t = tn;
    gt = gtn;
    __syncthreads();   // s_abort is rewritten below
    if (threadIdx.x < 64) {
      const bool ok = await_tile(gt, seen);
      if (lane == 0) s_abort = !ok;
    }
    __syncthreads();
    if (s_abort) return;
  }
}

template <int THREADS, int NP>
__global__ __launch_bounds__(THREADS) void tile_reducer(ReduceArgs a) {
  __shared__ int s_abort;
  reducer_body<THREADS, NP>(a, blockIdx.x, s_abort);
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
