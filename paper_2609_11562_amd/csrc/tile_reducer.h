// tile_reducer.h - the consumer: a persistent grid of x workgroups that
// reduces 128 x 128 tiles as soon as all their contributions are published
// (paper Section 3.1 "Matching task order", Section 4.2 ReduceTile).
//
// Workgroup j walks tiles j, j+x, j+2x, ... of its partition in producer
// order.  For each tile one thread waits for the local flag and then for the
// P-1 peer flags, issues an acquire fence, and the workgroup synchronises.
// The workgroup then reduces the tile: every element is initialised from the
// local bf16 contribution, the peer values are added in rank order in fp32,
// and the result is rounded to bf16 (nearest even) and stored once - each
// output element has a single writer.
//
// Data movement: a tile row is 256 bytes = 16 lanes x 16 bytes, so each wave
// moves 4 full rows per instruction (coalesced).  Contributions are read once
// and the output written once, so both use non-temporal accesses to keep the
// producer's A/B panels in cache.  G vectors per contribution are loaded
// before any is consumed, giving G * P independent 16-byte loads in flight
// per lane.
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

template <int THREADS, int NP>
__global__ __launch_bounds__(THREADS) void tile_reducer(ReduceArgs a) {
  constexpr int VPT = (kTile * kTile * 2 / 16) / THREADS;  // 16-byte vectors per thread
  constexpr int G = (NP >= 6) ? 2 : 4;                      // vectors per batch
  static_assert(VPT % G == 0, "batch must divide the per-thread vectors");
  __shared__ int s_abort;

  const BlockGrid grid = make_grid(a.M, a.N, NP, a.BM, a.BN, a.group_m);
  const int Q = tiles_per_partition(a.M, a.N, NP);
  const int tiles_n = a.N / kTile;
  const int ntiles = (a.M / kTile) * tiles_n;
  const ConsumerSeq seq = consumer_seq(a.dest, NP, a.x, blockIdx.x);
  const int chunk_rows = a.M / NP;

  for (int t = seq.first; t < Q; t += seq.stride) {
    int tr, tc;
    tile_of_number(seq.part, t, grid, &tr, &tc);
    const int gt = tr * tiles_n + tc;

    if (threadIdx.x == 0) {
      const uint64_t deadline = wall_clock64() + a.timeout_ticks;
      int src = -2;   // -2: all ready, -1: local flag missing, q: peer q missing
      if (!await_flag(a.flags + gt, a.epoch, deadline)) src = -1;
      for (int q = 0; q < NP - 1 && src == -2; ++q)
        if (!await_flag(a.peer_flags + static_cast<int64_t>(q) * ntiles + gt, a.epoch, deadline)) src = q;
      if (src != -2) {
        if (atomicCAS(a.status, 0, ENTWINE_ETIMEOUT) == 0) {
          atomicExch(a.status + 1, gt);
          atomicExch(a.status + 2, src);
        }
      }
      acquire_fence();
      s_abort = (src != -2);
    }
    __syncthreads();
    if (s_abort) return;

    const int64_t grow0 = static_cast<int64_t>(tr) * kTile;
    const int64_t gcol0 = static_cast<int64_t>(tc) * kTile;
    const int64_t orow0 = a.dest >= 0 ? grow0 - static_cast<int64_t>(a.dest) * chunk_rows : grow0;

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
    __syncthreads();   // s_abort is rewritten for the next tile
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
