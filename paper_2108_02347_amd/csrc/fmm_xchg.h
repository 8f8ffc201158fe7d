// Exchange of partial results between the workgroups of one launch through
// memory (the one-launch apply kernel and the state kernel that also sums its
// segments).  A workgroup writes its partial result with ordinary stores,
// waits for them to reach L2 (s_waitcnt vmcnt(0)) and then writes a stamp
// with a device-scope atomic store; its peers poll the stamps with
// device-scope atomic loads (which skip the vector L1) and read the partial
// results only after all stamps are there.  The partial results are coherent
// only between workgroups that share an L2 (one XCD): a stamp carries the XCC
// id of its writer, and a stamp from another XCC, a peer that gave up, or a
// wait beyond its poll limit sends the caller down a path that does not need
// the peers.  Every stamp also carries the launch's epoch, which differs from
// launch to launch, also between replays of a captured graph, so stamps left
// in memory by an earlier launch never count as this launch's.
#pragma once

#include <hip/hip_runtime.h>

namespace fmm {

// stamps: (epoch << 8) | XCC id of the writer; this XCC id marks a workgroup
// that gave up on the exchange
constexpr unsigned kGaveUp = 0xffu;

// The dispatch's packet index on its queue (the hardware's 64-bit dispatch
// id, the same for every workgroup of one launch and new for every launch,
// also for each replay of a captured graph, whose kernel arguments are frozen).
extern "C" __device__ unsigned long long fmm_dispatch_id() __asm("llvm.amdgcn.dispatch.id");

// A launch's epoch (56 bits): the host's call number in bits 32-55 and, in
// bits 0-31, the host's per-process offset plus the dispatch id.
__device__ __forceinline__ unsigned long long launch_epoch(unsigned long long host) {
  return (host & 0x00ffffff00000000ull) |
         (unsigned)((unsigned)host + (unsigned)fmm_dispatch_id());
}

__device__ __forceinline__ unsigned xcc_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 0xfu;
}

// Wave 0 polls stamp[stride i + level] of the G peers (G <= 64) until all
// carry this launch's epoch; true when every one is `mine` (same epoch, same
// XCC), false as soon as a stamp of this epoch is anything else or after
// spin_limit polls.  Uniform over the workgroup; s_flag is one int of LDS.
__device__ __forceinline__ bool wait_stamps(const unsigned long long* stamp, int stride,
                                            int level, int G, unsigned long long epoch,
                                            unsigned long long mine, int spin_limit,
                                            int* s_flag) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    int res = 2;
    for (int it = 0; it <= spin_limit; ++it) {
      const unsigned long long x =
          lane < G ? __hip_atomic_load(stamp + stride * lane + level, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT)
                   : mine;
      const bool fresh = (x >> 8) == epoch;
      if (__any(fresh && x != mine)) break;
      if (__all(fresh)) {
        res = 1;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (lane == 0) *s_flag = res;
  }
  __syncthreads();
  const bool ok = *s_flag == 1;
  __syncthreads();  // the flag is reused by the next wait
  return ok;
}

__device__ __forceinline__ void put_stamp(unsigned long long* p, unsigned long long x) {
  __hip_atomic_store(p, x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace fmm
