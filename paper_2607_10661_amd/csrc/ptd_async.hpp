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
__device__ __forceinline__ uint32_t uniform_u32(uint32_t x) {
  return static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(x)));
}

__device__ __forceinline__ void dma16(const void* gptr, uint32_t lds) {
  lds = uniform_u32(lds);
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
  lds = uniform_u32(lds);
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

// Two such copies (K and V parts of one sub-tile) with one save/restore of M0.
__device__ __forceinline__ void dma16_s2(const void* base0, uint32_t voff0, uint32_t lds0,
                                         const void* base1, uint32_t voff1, uint32_t lds1) {
  const uint64_t b0 = reinterpret_cast<uint64_t>(base0);
  const uint64_t b1 = reinterpret_cast<uint64_t>(base1);
  const uint64_t s0 = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b0 >> 32)))) << 32) |
                      static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b0)));
  const uint64_t s1 = (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b1 >> 32)))) << 32) |
                      static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b1)));
  lds0 = uniform_u32(lds0);
  lds1 = uniform_u32(lds1);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %4\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %5, %6\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds0), "v"(voff0), "s"(s0), "s"(lds1), "v"(voff1), "s"(s1)
      : "memory");
}

// Same, 4 bytes per lane (lane l lands at lds + 4*l).
__device__ __forceinline__ void dma4(const void* gptr, uint32_t lds) {
  lds = uniform_u32(lds);
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

// 4-byte global load into a VGPR from inline asm (not tracked by the
// compiler's wait counts; see wait_vmcnt_le and a register fence).
__device__ __forceinline__ uint32_t gload4(const void* p) {
  uint32_t v;
  asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
  return v;
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Wait until at most n of this wave's vector-memory operations are pending
// (n is clamped to [0, 63], the counter's range).
__device__ __forceinline__ void wait_vmcnt_le(int n) {
  switch (n) {
#define PTD_W(k) case k: wait_vmcnt<k>(); break;
    PTD_W(1) PTD_W(2) PTD_W(3) PTD_W(4) PTD_W(5) PTD_W(6) PTD_W(7) PTD_W(8)
    PTD_W(9) PTD_W(10) PTD_W(11) PTD_W(12) PTD_W(13) PTD_W(14) PTD_W(15) PTD_W(16)
    PTD_W(17) PTD_W(18) PTD_W(19) PTD_W(20) PTD_W(21) PTD_W(22) PTD_W(23) PTD_W(24)
    PTD_W(25) PTD_W(26) PTD_W(27) PTD_W(28) PTD_W(29) PTD_W(30) PTD_W(31) PTD_W(32)
    PTD_W(33) PTD_W(34) PTD_W(35) PTD_W(36) PTD_W(37) PTD_W(38) PTD_W(39) PTD_W(40)
    PTD_W(41) PTD_W(42) PTD_W(43) PTD_W(44) PTD_W(45) PTD_W(46) PTD_W(47) PTD_W(48)
    PTD_W(49) PTD_W(50) PTD_W(51) PTD_W(52) PTD_W(53) PTD_W(54) PTD_W(55) PTD_W(56)
    PTD_W(57) PTD_W(58) PTD_W(59) PTD_W(60) PTD_W(61) PTD_W(62)
#undef PTD_W
    case 0: wait_vmcnt<0>(); break;
    default:
      if (n < 0) wait_vmcnt<0>();
      else wait_vmcnt<63>();
      break;
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
