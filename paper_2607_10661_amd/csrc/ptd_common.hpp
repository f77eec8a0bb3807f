// Device and host helpers shared by the gfx950 kernels of the PTD hot path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ptd.h"

#define PTD_WAVE 64

namespace ptd {

// ---------------------------------------------------------------------------
// bf16 <-> fp32 (bf16 is the upper half of an IEEE binary32)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}
// round-to-nearest-even, finite inputs
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}
// Same rounding by the gfx950 packed converter (v_cvt_pk_bf16_f32, RNE).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  using bf16x2 = __bf16 __attribute__((ext_vector_type(2)));
  using f32x2 = float __attribute__((ext_vector_type(2)));
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// ---------------------------------------------------------------------------
// device-reported errors: first error wins
// ---------------------------------------------------------------------------
__device__ __forceinline__ void report(int32_t* dev_status, int32_t code) {
  if (dev_status) atomicCAS(dev_status, 0, code);
}

// ---------------------------------------------------------------------------
// wave (64-lane) reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, PTD_WAVE));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, PTD_WAVE);
  return v;
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int o) {
  uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), o, PTD_WAVE);
  uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), o, PTD_WAVE);
  return (static_cast<uint64_t>(hi) << 32) | lo;
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = shfl_xor_u64(v, o);
    v = w > v ? w : v;
  }
  return v;
}

}  // namespace ptd

// ---------------------------------------------------------------------------
// host helpers
// ---------------------------------------------------------------------------
#define PTD_RETURN_IF(cond, code) \
  do {                            \
    if (cond) return (code);      \
  } while (0)

static inline int ptd_launch_status() {
  return hipGetLastError() == hipSuccess ? PTD_OK : PTD_ERR_HIP;
}

static inline bool ptd_aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

// Ceil division for non-negative ints.
static inline __host__ __device__ int ptd_cdiv(int a, int b) { return (a + b - 1) / b; }
