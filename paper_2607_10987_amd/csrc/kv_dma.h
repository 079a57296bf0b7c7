// Asynchronous global -> LDS copies for multi-stage pipelines (gfx950).
//
// lds_dma16 issues global_load_lds_dwordx4: lane i of the wavefront copies 16
// bytes from its global address to LDS bytes [16 i, 16 i + 16) after the
// wave-uniform LDS base `lds`.  It is written as inline assembly so that the
// compiler does not track the copy; the pipelines order it explicitly:
//   * wait_vmcnt<N>() (s_waitcnt vmcnt(N)) before reading a stage: the wave's
//     copies complete in issue order, so all but its N most recent are done;
//   * lds_barrier() (s_waitcnt lgkmcnt(0); s_barrier), a workgroup barrier
//     without the memory fence of __syncthreads(), whose vmcnt(0) would drain
//     every stage in flight.  After it, every wave's copies of the stage are
//     visible and every wave has finished reading the buffer about to be
//     refilled.  The "memory" clobbers keep the compiler from moving memory
//     accesses across either statement.
// Values loaded with ordinary global loads before a pipeline must be made
// ready with settle() so that the compiler's own wait for them is not placed
// inside the pipelined loop (where it would wait for every copy as well).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvs {

__device__ inline void lds_dma16(const void* gptr, void* lds) {
  const uint32_t la = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds);
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(la)
               : "memory", "m0");
}

// LDS byte address of a __shared__ pointer, wave-uniform.
__device__ inline uint32_t lds_addr(const void* lds) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds);
}

// The same copy with the global address split into a wave-uniform base
// (scalar registers) and a per-lane 32-bit byte offset; `lds` is an LDS byte
// address from lds_addr().
__device__ inline void lds_dma16_sv(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// lds_dma16_sv with the non-temporal cache policy (data read exactly once).
__device__ inline void lds_dma16_sv_nt(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1 nt"
               :
               : "v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

template <int N>
__device__ inline void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ inline void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Workgroup barrier alone, for a point where the wave's own LDS reads of
// the buffer other waves are about to refill have already been consumed.
__device__ inline void barrier_only() { asm volatile("s_barrier" ::: "memory"); }

template <typename T>
__device__ inline void settle(T& v) {
  asm volatile("" : "+v"(v));
}

}  // namespace kvs
