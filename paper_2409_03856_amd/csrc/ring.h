// Internal: helpers of the LDS-ring kernels, whose K blocks are moved into LDS by direct
// global-to-LDS loads and waited for by count.
#pragma once

#include <hip/hip_runtime.h>

namespace sirius {

// vmcnt(n) with the other counters left alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without the release fence of __syncthreads(), which would wait for every
// direct-to-LDS load still in flight. The ring's own wait counts make this wave's loads of the
// block complete before it; LDS needs no cache maintenance. The lgkmcnt(0) wait makes every
// ds_read this wave issued (of the slot about to be refilled) return its data to registers
// before the barrier, whatever the compiler did with the instructions that consume them: an
// MFMA is not a memory operation, so it (and the wait the compiler places for its operands)
// may be scheduled below the asm. vmcnt is left alone, so the ring's loads stay in flight. The
// memory clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace sirius
