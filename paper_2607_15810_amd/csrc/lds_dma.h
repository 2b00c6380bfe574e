// Direct global->LDS loads and hand-counted waits, shared by the GEMM
// kernels.
#pragma once
#include "common.h"

namespace qdl {

// Direct global->LDS loads: lane l's bytes land at M0 + l * size.  They are
// issued from inline assembly and their completion is counted by hand; the
// memory clobbers keep every LDS access on its side of the issue and of the
// waits.
__device__ __forceinline__ void dma16(const void *g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(g), "s"(lds_addr) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void *g, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :: "v"(g), "s"(lds_addr) : "memory", "m0");
}
// the same with a uniform 64-bit base in SGPRs and a 32-bit per-lane offset
__device__ __forceinline__ void dma16s(const void *base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_addr) : "memory", "m0");
}
__device__ __forceinline__ void dma4s(const void *base, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %0, %1"
               :: "v"(voff), "s"(base), "s"(lds_addr) : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
__device__ __forceinline__ void wait_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}
__device__ __forceinline__ uint32_t uni(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }
template <typename T>
__device__ __forceinline__ const T *uni_ptr(const T *p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint64_t r = ((uint64_t)uni((uint32_t)(v >> 32)) << 32) | uni((uint32_t)v);
  return reinterpret_cast<const T *>((uintptr_t)r);
}

}  // namespace qdl
