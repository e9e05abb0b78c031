// gfx950 global->LDS DMA and vector-memory wait helpers shared by the MFMA kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace ssconv {

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from global address g into LDS at byte lds + 16 * lane
// (global_load_lds_dwordx4; M0 holds the wave-uniform LDS base, and one wait state
// separates the M0 write from the DMA that reads it).  Issued through inline
// assembly so that the compiler does not drain every outstanding load before the
// next LDS read; completion is tracked with wait_vm below.
__device__ __forceinline__ void dma16(const void* g, uint32_t lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(l), "v"(g) : "memory", "m0");
}

// Same, from the wave-uniform base address base plus this lane's 32-bit byte offset off.
__device__ __forceinline__ void dma16_off(const void* base, uint32_t off, uint32_t lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(l), "v"(off), "s"(base)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt vmcnt(N): at most N of this wavefront's vector-memory operations still in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

}  // namespace ssconv
