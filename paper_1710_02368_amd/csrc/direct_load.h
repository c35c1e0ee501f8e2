// Direct global->LDS loads (global_load_lds_dwordx4 on gfx950) and the
// waits and barrier that go with them, shared by the direct-load kernels.
#pragma once

#include "device_common.h"

namespace agn {
namespace {

// The direct loads, the barrier and the waits on their counter are written
// as inline assembly with a memory clobber: the compiler neither moves LDS
// reads across them nor adds waits of its own for the loads (it cannot tell
// which LDS stage a load writes, and would wait for all of them); the waits
// below count the load instructions exactly.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"

// LDS byte offset of a pointer into a __shared__ array
__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) char*)p);
}

// one 64-lane direct load: lane l's 16 bytes from src to LDS byte offset
// lds + 16*l (lds wave-uniform, in M0; one wait state between the M0 write
// and the load that reads it)
__device__ __forceinline__ void fire(const void* src, uint32_t lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m0), "v"(src)
               : "memory", "m0");
}

// at most N of this wave's vector memory loads still in flight
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

#pragma clang diagnostic pop

}  // namespace
}  // namespace agn
