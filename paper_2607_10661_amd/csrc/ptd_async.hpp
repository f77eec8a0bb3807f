// Asynchronous HBM -> LDS copies and the waits that go with them (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ptd {

// Asynchronous HBM -> LDS copy (gfx950 global_load_lds_dwordx4): every lane
// copies 16 bytes from its own global address and the wave's 64 x 16 bytes
// land contiguously at the wave-uniform LDS byte address `lds`.  The copy is
// issued from inline asm so that the compiler's wait-count insertion does not
// make later LDS reads wait for every copy in flight; completion is tracked
// with explicit vmcnt waits (vector-memory operations retire in issue order,
// so a wait also covers every older load).  M0 is saved and restored inside
// the asm, and one wait state separates the M0 write from the copy.
__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(gptr)
      : "memory");
}

// Same copy from a wave-uniform base address (SGPR pair) plus a per-lane
// 32-bit byte offset: moving to the next tile changes only the scalar base.
// The base must be uniform over the wave; it is moved to SGPRs explicitly.
__device__ __forceinline__ void dma16_s(const void* base, uint32_t voff, uint32_t lds) {
  // (readfirstlane returns int: widen through uint32_t, never sign-extend)
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b)));
  const uint64_t sbase = (static_cast<uint64_t>(hi) << 32) | lo;
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(voff), "s"(sbase)
      : "memory");
}

// Same, 4 bytes per lane (lane l lands at lds + 4*l).
__device__ __forceinline__ void dma4(const void* gptr, uint32_t lds) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dword %2, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds), "v"(gptr)
      : "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most n of this wave's vector-memory operations are pending
// (n above 24 waits for 24: stricter, never wrong).
__device__ __forceinline__ void wait_vmcnt_le(int n) {
  switch (n) {
#define PTD_W(k) case k: wait_vmcnt<k>(); break;
    PTD_W(1) PTD_W(2) PTD_W(3) PTD_W(4) PTD_W(5) PTD_W(6) PTD_W(7) PTD_W(8)
    PTD_W(9) PTD_W(10) PTD_W(11) PTD_W(12) PTD_W(13) PTD_W(14) PTD_W(15) PTD_W(16)
    PTD_W(17) PTD_W(18) PTD_W(19) PTD_W(20) PTD_W(21) PTD_W(22) PTD_W(23)
#undef PTD_W
    case 0: wait_vmcnt<0>(); break;
    default: wait_vmcnt<24>(); break;
  }
}

// Workgroup barrier that also completes this wave's LDS reads; the asm memory
// clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

#define PTD_LDS __attribute__((address_space(3)))

// LDS byte address of a __shared__ object (address-space casts need C casts)
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const PTD_LDS char*)p));
}

}  // namespace ptd
