// Helpers for kernels that stream operands from global memory straight into
// LDS with global_load_lds_dwordx4 (16 bytes per lane, placed at a wave-uniform
// LDS base + 16 * lane).
//
// LDS that such a load fills is read only through inline assembly with explicit
// waits: vmcnt for the loads (then a barrier), lgkmcnt before the values are
// used.  Compiler-generated LDS accesses would each be preceded by a wait for
// every DMA load in flight.  A value read this way must reach its uses only
// through asm statements placed after its lgkmcnt wait (see the callers), and
// the kernels using it must not spill registers: a spill could copy a register
// before the LDS data has arrived (the build checks that they do not spill).
#pragma once

#include "gemm.h"

namespace mtgnn {

typedef __attribute__((address_space(3))) void* lds_void_ptr;

namespace dma {

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void barrier() { asm volatile("s_barrier" ::: "memory"); }

__device__ __forceinline__ f32x4 ds_read4(uint32_t addr) {
  f32x4 v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return v;
}

__device__ __forceinline__ void ds_zero4(uint32_t addr) {
  const f32x4 z = {0.f, 0.f, 0.f, 0.f};
  asm volatile("ds_write_b128 %0, %1" ::"v"(addr), "v"(z) : "memory");
}

__device__ __forceinline__ void ds_write4(uint32_t addr, const f32x4& v) {
  asm volatile("ds_write_b128 %0, %1" ::"v"(addr), "v"(v) : "memory");
}

__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Passes a value through an (empty) volatile asm statement: uses of the result are
// ordered after every asm statement before it, e.g. an lgkmcnt wait.
__device__ __forceinline__ void tie(f32x4& v) { asm volatile("" : "+v"(v)); }

// 16 bytes per lane from global memory to LDS at lds_base + 16 * lane (lds_base wave-uniform).
__device__ __forceinline__ void load16(const float* g, uint32_t lds_base) {
  __builtin_amdgcn_global_load_lds((void*)g, (lds_void_ptr)(uintptr_t)lds_base, 16, 0, 0);
}

}  // namespace dma

}  // namespace mtgnn
