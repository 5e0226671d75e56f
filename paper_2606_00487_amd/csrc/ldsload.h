// Direct global-to-LDS loads and the explicit waits that order them, shared by the kernels
// that stream their operands through rings of LDS slots (tree attention, layer GEMM).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace taps {

typedef int i32x4 __attribute__((ext_vector_type(4)));

// s_waitcnt that waits until at most `n` vector-memory operations are outstanding
// (expcnt and lgkmcnt left at their maxima, i.e. not waited on)
#define TAPS_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))

// workgroup barrier for the stage buffers: the explicit vmcnt waits before it cover the
// direct loads; the memory clobber keeps the compiler from moving LDS accesses across it
#define TAPS_STAGE_BARRIER() asm volatile("s_barrier" ::: "memory")

// workgroup barrier after LDS writes: waits for this wave's LDS operations only, so the
// direct loads in flight stay in flight (__syncthreads would also wait for them)
#define TAPS_LDS_BARRIER()                                                   \
  do {                                                                       \
    __builtin_amdgcn_s_waitcnt(0xF | (7 << 4) | (0 << 8) | (3 << 14));       \
    asm volatile("s_barrier" ::: "memory");                                  \
  } while (0)

// Buffer resource over `bytes` bytes from p (raw buffer, no stride): accesses at offsets
// >= bytes read as zeros without touching memory.
__device__ inline i32x4 buffer_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)p;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// 16 bytes per lane from buffer offset `off` straight into LDS at dst + 16 * lane, issued
// as inline assembly so that the compiler does not track it.  Its own bookkeeping of
// direct-to-LDS loads cannot tell the slots of a ring apart and would make every LDS read
// wait for all but the newest loads in flight, which cuts the look-ahead of the ring to
// one step.  Callers order every global read of the kernel with explicit vmcnt waits.
// m0 carries the LDS address; nothing else in the kernels that call this uses m0.  A
// direct-to-LDS load must not follow the scalar write of m0 immediately (one wait state).
__device__ inline void load_lds16(const i32x4& rs, unsigned char* dst, uint32_t off) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)dst);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :: "s"(m0v), "v"(off), "s"(rs) : "memory");
}

// 4 bytes per lane into LDS at dst + 4 * lane (same conventions as load_lds16)
__device__ inline void load_lds4(const i32x4& rs, unsigned char* dst, uint32_t off) {
  const uint32_t m0v = __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)dst);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
               :: "s"(m0v), "v"(off), "s"(rs) : "memory");
}

}  // namespace taps
