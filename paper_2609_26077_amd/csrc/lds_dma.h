// HBM -> LDS transfers that bypass the register file (gfx950 global_load_lds).
//
// A transfer is issued from inline assembly so that the compiler neither waits
// for it (the builtin form makes it drain vmcnt before every later LDS read)
// nor reorders LDS reads across it; completion is tracked by the caller with
// an explicit s_waitcnt vmcnt(N), which counts these transfers in issue order.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace fmm {
namespace dma {

typedef __attribute__((address_space(3))) uint8_t lds_u8;

// LDS byte address of a __shared__ object, as M0 expects it
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T *p) {
  return (uint32_t)(uintptr_t)(lds_u8 *)p;
}

// one wave-wide transfer: lane l moves 16 bytes from base + off to LDS byte m0 + 16 l
__device__ __forceinline__ void copy16(uint32_t off, const uint8_t *base, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(m0)
               : "memory", "m0");
}
// one wave-wide transfer: lane l moves 4 bytes from base + off to LDS byte m0 + 4 l
__device__ __forceinline__ void copy4(uint32_t off, const uint8_t *base, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(base), "s"(m0)
               : "memory", "m0");
}
// wait until at most N of this wave's vector-memory operations are outstanding
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

}  // namespace dma
}  // namespace fmm
