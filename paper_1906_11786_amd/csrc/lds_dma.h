// Copies from global memory straight into LDS (global_load_lds_dwordx4),
// issued from inline assembly so that the compiler does not wait for them
// before unrelated LDS reads or barriers; the caller waits for exactly the
// copies it needs (s_waitcnt vmcnt counts them in issue order).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ggnn {
namespace dev {

// One wave-wide 1 KB copy: lane l's 16 bytes at gsrc go to LDS byte address
// lds + 16 l (lds wave-uniform).  M0 holds the LDS base; one wait state
// between writing M0 and the load that uses it.  M0 is listed as clobbered;
// the compiler keeps nothing else in M0 in the kernels that use this (none
// of their other instructions reads it, checked in the generated assembly).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* gsrc, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(gsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop
// Wait until at most N of this wave's vector-memory loads are outstanding
// (vmcnt only).
template <int N>
__device__ __forceinline__ void wait_copies() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0xF70 | N);
}

}  // namespace dev
}  // namespace ggnn
