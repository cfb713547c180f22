// flags.h - per-tile publication protocol between the producer GEMM and the
// tile reducer (paper Section 3.1 "Independent tile communication" and
// Section 4.2).
//
// Producer: every thread stores its part of the tile, the workgroup
// synchronises, then one thread issues a release fence and writes the tile's
// flag, so the flag is ordered after the stores of the whole workgroup.
// Consumer: one thread polls the local flag, then each peer flag, then issues
// an acquire fence and the workgroup synchronises, which orders every
// thread's reads of the tile after the producers' stores.
//
// Both kernels run on one device whose eight XCDs have separate L2 caches, so
// the scope is the agent (device): the release writes dirty L2 lines back and
// the acquire invalidates stale ones.  (The paper uses system scope because
// its peers are other GPUs.)
//
// Flags are reused across calls without clearing: a call with epoch e treats
// a flag as ready when it equals e.  Each wait is bounded by a deadline on the
// device's constant-rate wall clock; on expiry the consumer reports a timeout
// instead of hanging.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace entwine {

// Release fence once, then relaxed stores: one L2 write-back covers every
// flag a producer block publishes.  The wait for this wave's outstanding
// memory operations that the fence implies is also issued explicitly: the
// producer's tile stores and operand loads are inline asm, which the
// compiler's wait tracking does not see, so it would drop the fence's own
// wait as redundant and let a flag overtake the data it publishes.
__device__ __forceinline__ void release_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __builtin_amdgcn_s_waitcnt(0);   // vmcnt, expcnt and lgkmcnt all zero
}

__device__ __forceinline__ void publish_relaxed(int* flag, uint32_t epoch) {
  __hip_atomic_store(flag, static_cast<int>(epoch), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int poll_relaxed(const int* flag) {
  return __hip_atomic_load(const_cast<int*>(flag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Spin until *flag == epoch or the wall clock passes `deadline`.
__device__ __forceinline__ bool await_flag(const int* flag, uint32_t epoch, uint64_t deadline) {
  while (poll_relaxed(flag) != static_cast<int>(epoch)) {
    if (wall_clock64() > deadline) return false;
    __builtin_amdgcn_s_sleep(2);
  }
  return true;
}

__device__ __forceinline__ void acquire_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

}  // namespace entwine
