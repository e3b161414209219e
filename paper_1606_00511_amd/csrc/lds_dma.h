// Direct global-to-LDS loads on gfx950 and the waits and barriers of the
// multi-stage K pipelines built on them (shared by the fp32 and bf16 GEMMs).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace hfk {

// 16 bytes per lane from global memory straight into LDS: lane i's bytes
// land at dst + 16 i (dst is the wave's LDS base, the same in every lane).
// Written as inline assembly: with the compiler builtin, any direct load in
// flight makes the compiler wait for every outstanding LDS read before each
// MFMA, which serialises the fragment loads with the MFMAs.  The kernels
// track these loads themselves (wait_vm before a stage is read).  M0 holds
// the wave's LDS base and needs one wait state before the load.
__device__ __forceinline__ void dma16(const void* src, void* dst) {
  const uint32_t lds_addr = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)dst);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(lds_addr) : "memory");
}

// Wait until at most N vector-memory operations of this wave are pending
// and every LDS operation has completed.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (0 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier that neither the compiler nor the scheduler may move
// memory operations across; unlike __syncthreads it does not drain the
// wave's outstanding direct loads.
__device__ __forceinline__ void stage_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

}  // namespace hfk
