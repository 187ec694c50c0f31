// Direct global-to-LDS loads for gfx950 kernels (the attention ring and the
// MLP scorer's operand ring).
//
// 16 (or 4) bytes per lane go from global memory into LDS at l + 16 (4) x
// lane, l wave-uniform.  They are written as inline assembly so that the
// compiler does not track them: it would otherwise wait for every one in
// flight before any LDS read.  Completion is waited for explicitly with
// s_waitcnt vmcnt (loads retire in issue order); waits the compiler derives
// for other loads stay correct (untracked loads only make them wait longer).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gambit {

__device__ inline uint32_t lds_addr(const void* l) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)l;
}

// M0 carries the LDS address; it is saved and restored around the load, so
// the compiler's view of M0 never changes.
__device__ inline void dma16(const void* g, void* l) {
  uint32_t save;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off\n\ts_nop 0\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(save)
      : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds_addr(l)))
      : "memory");
}

__device__ inline void dma4(const void* g, void* l) {
  uint32_t save;
  asm volatile(
      "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dword %1, off\n\ts_nop 0\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(save)
      : "v"(g), "s"(__builtin_amdgcn_readfirstlane(lds_addr(l)))
      : "memory");
}

// s_waitcnt until at most N vector-memory loads of this wave are in flight
// (N < 64: vmcnt is bits 3:0 and 15:14 of the immediate; expcnt and lgkmcnt
// at their maxima, so they are not waited for).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Workgroup barrier that keeps the compiler from moving memory accesses
// across it but adds no wait for outstanding loads (a fenced barrier would
// wait for every in-flight direct load, emptying the ring).
__device__ inline void barrier_no_fence() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace gambit
