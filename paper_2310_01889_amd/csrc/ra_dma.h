// Direct-to-LDS loads the compiler does not track, and an LDS-only workgroup barrier, for
// kernels that pipeline tile loads several stages deep (the GEMM).
#pragma once
#include "ra_common.h"

namespace ra {

// Direct-to-LDS loads issued from inline assembly, 16 or 4 bytes per lane (lane i lands at
// byte 16 i, or 4 i, of the wave-uniform LDS address lds_addr).  The compiler does not
// track these loads: a kernel that uses them waits for them itself with counted vmcnt
// waits, which lets the loads of later ring stages stay in flight while a stage is read
// (the compiler's own tracking of direct-to-LDS loads is too coarse for that and waits for
// all of them before reading any buffer).  M0 carries the LDS address; a kernel that uses
// these must have no compiler-generated code that relies on M0.
__device__ __forceinline__ void dma_lds16(const __amdgpu_buffer_rsrc_t& rsrc, unsigned lds_addr, int voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds_addr), "v"(voff), "s"(rsrc)
               : "memory");
}
// As dma_lds16, the read address plus a wave-uniform byte offset soff (scalar register).
__device__ __forceinline__ void dma_lds16_so(const __amdgpu_buffer_rsrc_t& rsrc, unsigned lds_addr, int voff, int soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(lds_addr), "v"(voff), "s"(rsrc),
               "s"(soff)
               : "memory");
}
__device__ __forceinline__ void dma_lds4(const __amdgpu_buffer_rsrc_t& rsrc, unsigned lds_addr, int voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds" ::"s"(lds_addr), "v"(voff), "s"(rsrc)
               : "memory");
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, num_bytes, 0x00020000);
}
__device__ __forceinline__ unsigned lds_addr(const void* p) { return (unsigned)(unsigned long long)(lds_void*)p; }

// Workgroup barrier that orders the waves' LDS instructions only: every LDS instruction
// of the wave issued before it has completed, and (memory clobber) the compiler moves no
// memory access across it.  Unlike __syncthreads() it does not wait for vector-memory
// operations (a fence would, since direct-to-LDS loads count as pending LDS writes), so
// tile loads issued earlier stay in flight; callers first wait, with an explicit vmcnt,
// for the loads whose data the other waves will read after the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace ra
