// Device helpers of the kernels that stream history tiles into LDS with
// direct global-to-LDS loads (fast.hip, reordered.hip).
#pragma once

#include "common.h"

namespace stca {

// s_waitcnt on vector memory: at most n (rounded down to even, <= 6) of this
// wave's vector memory operations still outstanding; LDS operations drained.
__device__ __forceinline__ void wait_vm(int n) {
  // gfx9 immediate: vmcnt[3:0], expcnt[6:4] = 7 (no wait), lgkmcnt[11:8] = 0
  if (n >= 6)
    __builtin_amdgcn_s_waitcnt(0x0076);
  else if (n >= 4)
    __builtin_amdgcn_s_waitcnt(0x0074);
  else if (n >= 2)
    __builtin_amdgcn_s_waitcnt(0x0072);
  else
    __builtin_amdgcn_s_waitcnt(0x0070);
}

// Direct global-to-LDS load of 16 bytes per lane: lane i's bytes land at
// lds + 16 i (lds wave-uniform).  Issued as inline assembly so that the
// compiler does not treat every later LDS read as possibly aliasing it (it
// would wait for all loads in flight before each read); the kernel waits for
// these loads itself (wait_vm).  The compiler's own vector-memory waits only
// become more conservative, as the counter retires operations in order.
__device__ __forceinline__ void dma16(const void* src, const unsigned char* lds) {
  const uint32_t m0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const __attribute__((address_space(3))) unsigned char*)lds));
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(__builtin_amdgcn_readfirstlane(m0)));
}

// Workgroup barrier without the fences of __syncthreads (whose release would
// wait for every load in flight, including the ring's prefetches); the memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void ring_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Transposing LDS read of 16-bit data (gfx950): within each group of 16
// lanes, lane s reads the 4 consecutive elements at its own address (a
// 4-element vector V_s), and lane j of the group receives element k of
// V_(4 k + j / 4) at position j % 4, for k = 0..3.  With lane s addressing
// row s / 4 and columns 4 (s % 4) .. + 3 of a row-major 4 x 16 block, lane j
// receives column j of the block: four rows of one column.
typedef short tr16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ tr16x4 lds_read_tr16(const unsigned char* lds) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) tr16x4*)((__attribute__((address_space(3))) unsigned char*)lds));
}

}  // namespace stca
