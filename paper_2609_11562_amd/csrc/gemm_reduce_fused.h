// gemm_reduce_fused.h - the fused path as one kernel launch: workgroups
// [0, G) are producers and [G, G + x) reducers (paper Section 4.3 runs the
// two as separate kernels on two streams).
//
// Both roles are persistent and one workgroup fits a CU (the producer's LDS
// stages fill it), so with G + x no larger than the CU count every workgroup
// is resident at once and the reducers run on their own x CUs, the paper's
// partition of the device between computation and communication.  Only
// reducers ever wait, and only for producers, so progress never depends on
// residency order.  One launch replaces the two kernels, the synthetic
// peer-flag kernel and the two cross-stream event waits of the two-stream
// form, each of which costs microseconds of queue synchronisation per call.
#pragma once

#include "gemm_producer.h"
#include "tile_reducer.h"

namespace entwine {

// stamps: null, or 2 per workgroup {start, end} in wall-clock ticks.
template <int BM, int BN, bool TAIL>
__global__ __launch_bounds__(256) void gemm_reduce_fused(GemmArgs g, ReduceArgs r, int G, int np,
                                                          unsigned long long* stamps) {
  __shared__ __attribute__((aligned(1024))) char smem[GemmShape<BM, BN>::LDS_BYTES];
  const unsigned long long t0 = stamps ? wall_clock64() : 0;
  const int b = blockIdx.x;
  if (b < G) {
    producer_body<BM, BN, TAIL>(g, b, G, smem);
  } else {
    int& s_abort = *reinterpret_cast<int*>(smem);
    const int j = b - G;
    switch (np) {
      case 1: reducer_body<256, 1>(r, j, s_abort); break;
      case 2: reducer_body<256, 2>(r, j, s_abort); break;
      case 3: reducer_body<256, 3>(r, j, s_abort); break;
      case 4: reducer_body<256, 4>(r, j, s_abort); break;
      case 5: reducer_body<256, 5>(r, j, s_abort); break;
      case 6: reducer_body<256, 6>(r, j, s_abort); break;
      case 7: reducer_body<256, 7>(r, j, s_abort); break;
      default: reducer_body<256, 8>(r, j, s_abort); break;
    }
  }
  if (stamps) {
    __syncthreads();
    if (threadIdx.x == 0) {
      stamps[2 * b] = t0;
      stamps[2 * b + 1] = wall_clock64();
    }
  }
}

}  // namespace entwine
