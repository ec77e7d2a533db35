// Direct global-to-LDS copies and the waits around them (gfx950).
#pragma once

#include "common.h"

namespace dpsgd {

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier that also orders the compiler's memory accesses (LDS
// reads cannot move across it) without making the hardware wait for
// outstanding loads, which the explicit vmcnt waits already account for.
__device__ __forceinline__ void barrier_no_wait() { asm volatile("s_barrier" ::: "memory"); }

// One 16-byte-per-lane copy from global memory into LDS at lds_addr + 16 * lane:
// lane i reads base + voff_i (base uniform, in SGPRs; voff a 32-bit byte offset).
// Issued as inline assembly so the compiler does not treat later LDS reads as
// aliasing an in-flight copy (it would otherwise wait for every outstanding
// copy before each read); completion is tracked with explicit vmcnt waits.
__device__ __forceinline__ void copy16_to_lds(const void* base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds_addr)
               : "m0", "memory");
}

// 32-bit LDS address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

}  // namespace dpsgd
