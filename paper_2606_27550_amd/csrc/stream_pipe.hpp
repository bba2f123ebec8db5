// Device helpers of the LM-head kernels that stream W through LDS rings:
// vocabulary slicing, explicit load-count waits, direct global->LDS copies
// and a fence-free workgroup barrier.
#pragma once

#include "common.hpp"

namespace entmtp {

// First vocabulary row of slice b of G (multiples of 4; V past the last).
__device__ __forceinline__ int slice_begin(int b, int G, int V) {
  if (b >= G) return V;
  return static_cast<int>((static_cast<long long>(V) * b / G) & ~3ll);
}

// s_waitcnt vmcnt(N) lgkmcnt(0) (gfx9 encoding; expcnt not waited on): this
// wave's direct-to-LDS loads older than the last N have landed and its own
// LDS reads are complete.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
}

// One direct global->LDS copy of 16 bytes per lane: lane l's bytes land at
// lds + 16 * l (lds is wave-uniform).  Kept in a device-only function: in a
// kernel's (host+device) lambda this gfx950 builtin would keep the compiler
// from emitting the kernel's host launch stub.
__device__ __forceinline__ void lds_dma16(const void* src, void* lds) {
  __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
}

// Workgroup barrier without a memory-model fence.  __syncthreads() would add
// a release fence, which waits for every outstanding load (the LDS-DMA
// stages count as LDS writes) and so drains the pipeline; here the waits are
// explicit (wait_vmcnt) and the empty asm statements only stop the compiler
// from moving LDS accesses across the barrier.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace entmtp
