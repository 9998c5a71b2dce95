// Direct global->LDS loads (LDS DMA) with manual completion tracking.
//
// global_load_lds_dwordx4 copies 16 bytes per lane from a global address to
// LDS at M0 + 16*lane.  It is issued through inline asm so that the compiler
// does not track it: the compiler cannot tell which LDS bytes such a load
// writes and would otherwise wait for every one of them to land before the
// next LDS read, which serialises a multi-stage ring.  Completion is
// therefore the kernel's job: wait_vmcnt<N>() (per wave, in issue order)
// followed by barrier() (all waves) before the LDS data is read.
//
// These kernels use M0 for nothing else; the asm sets it before each load.
#pragma once
#include "common.h"

namespace lmop {

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// lds_base must be the same for all lanes of the wave
LMOP_DEVICE void g2l16(const void* gaddr, void* lds_base) {
  const uint32_t m0 =
      __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_ptr_t)lds_base);
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gaddr), "s"(m0)
               : "memory");
}

// the same with the address split into a wave-uniform base (scalar
// registers) plus a per-lane 32-bit byte offset, and the LDS destination
// given as a wave-uniform LDS address
LMOP_DEVICE void g2l16_m0(const void* sbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_addr)
               : "memory");
}

// s_waitcnt vmcnt(N), other counters untouched (gfx9 encoding)
template <int N>
LMOP_DEVICE void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// workgroup barrier without the memory fence of __syncthreads (which would
// wait for every outstanding load, including the prefetches in flight);
// the empty asm statements keep the compiler from moving memory accesses
// across it
LMOP_DEVICE void barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

}  // namespace lmop
