// gemm_reduce_fused.h - the fused path as one kernel launch: workgroups
// [0, G) are producers and [G, G + x) reducers (paper Section 4.3 runs the
// two as separate kernels on two streams).
//
// Both roles are persistent and one workgroup fits a CU (the producer's LDS
// stages fill it), so with G + x no larger than the CU count every workgroup
// is resident at once and the reducers run on their own x CUs, the paper's
// partition of the device between computation and communication.  Tiles are
// handed out in consumer order from a device counter, and a producer that has
// finished its blocks becomes a reducer too: at the end of the GEMM the
// remaining tiles are reduced by the whole device instead of by x CUs, and a
// block count that is not a multiple of G leaves no CU idle.  Only reducers
// ever wait, and only for producers, so progress never depends on residency
// order.  One launch replaces the two kernels, the synthetic peer-flag kernel
// and the two cross-stream event waits of the two-stream form, each of which
// costs microseconds of queue synchronisation per call.
#pragma once

#include "gemm_producer.h"
#include "tile_reducer.h"

namespace entwine {

constexpr int kStampsPerWg = 6;

// stamps: null, or kStampsPerWg per workgroup: {start, producer end (= start
// without producer work), first reduction task ready (0 if none), end} in
// wall-clock ticks, then the engine clock's cycle counter at the start and at
// the producer end, which over the wall-clock span give the clock the
// producer ran at (it falls under load, and depends on the data).
template <int BM, int BN, bool TAIL>
__global__ __launch_bounds__(256) void gemm_reduce_fused(GemmArgs g, ReduceArgs r, int G, int np,
                                                          unsigned long long* stamps) {
  __shared__ __attribute__((aligned(1024))) char smem[GemmShape<BM, BN>::LDS_BYTES];
  const int b = blockIdx.x;
  // Stamps are stored as they are taken, so none stays live in registers
  // across the producer; their address is recomputed from the (scalar)
  // kernel arguments at each use.
  const bool stamp = stamps != nullptr && threadIdx.x == 0;
  if (stamp) {
    unsigned long long* const st = stamps + kStampsPerWg * b;
    st[0] = wall_clock64();
    st[4] = __builtin_amdgcn_s_memtime();
    if (b >= G) {
      st[1] = st[0];
      st[5] = st[4];
    }
  }
  publish_peer_slice(r, np, b, gridDim.x);
  const unsigned int taken = b < G ? producer_body<BM, BN, TAIL>(g, b, G, smem) : ~0u;
  if (stamp && b < G) {
    unsigned long long* const st = stamps + kStampsPerWg * b;
    st[1] = wall_clock64();
    st[5] = __builtin_amdgcn_s_memtime();
  }
  int* s = reinterpret_cast<int*>(smem);
  static_assert(kLayerThreads == 256, "the layer tasks run on the fused launch's workgroups");
  if (r.layer) {
    switch (np) {
      case 1: reducer_layer<1>(r, s, taken); break;
      case 2: reducer_layer<2>(r, s, taken); break;
      case 3: reducer_layer<3>(r, s, taken); break;
      case 4: reducer_layer<4>(r, s, taken); break;
      case 5: reducer_layer<5>(r, s, taken); break;
      case 6: reducer_layer<6>(r, s, taken); break;
      case 7: reducer_layer<7>(r, s, taken); break;
      default: reducer_layer<8>(r, s, taken); break;
    }
  } else {
    unsigned long long* ready = stamps ? stamps + kStampsPerWg * b + 2 : nullptr;
    switch (np) {
      case 1: reducer_dynamic<256, 1, kTaskSplit>(r, s, ready, taken); break;
      case 2: reducer_dynamic<256, 2, kTaskSplit>(r, s, ready, taken); break;
      case 3: reducer_dynamic<256, 3, kTaskSplit>(r, s, ready, taken); break;
      case 4: reducer_dynamic<256, 4, kTaskSplit>(r, s, ready, taken); break;
      case 5: reducer_dynamic<256, 5, kTaskSplit>(r, s, ready, taken); break;
      case 6: reducer_dynamic<256, 6, kTaskSplit>(r, s, ready, taken); break;
      case 7: reducer_dynamic<256, 7, kTaskSplit>(r, s, ready, taken); break;
      default: reducer_dynamic<256, 8, kTaskSplit>(r, s, ready, taken); break;
    }
  }
  if (stamps) {
    __syncthreads();
    if (stamp) {
      unsigned long long* const st = stamps + kStampsPerWg * b;
      if (r.layer) st[2] = 0;
      st[3] = wall_clock64();
    }
  }
}

}  // namespace entwine
