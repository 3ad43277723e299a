// Device-side helpers shared by the HIP kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "divmagic.h"

namespace sc {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest even (the gfx950 conversion instruction rounds RNE).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

// n / d for n < 2^31 with a host-computed magic pair (divmagic.h).
__device__ __forceinline__ uint32_t fast_div(uint32_t n, DivMagic m) {
  return (__umulhi(n, m.mul) + n) >> m.shift;
}

// Work-group index remap for the 8 XCDs of MI355X: consecutive hardware
// work-group ids are dealt round-robin to the XCDs, so hand each XCD a
// contiguous range of logical work items (which then share its L2).
__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t n) {
  const uint32_t x = b & 7u, local = b >> 3, per = n >> 3, extra = n & 7u;
  return x * per + (x < extra ? x : extra) + local;
}

}  // namespace sc
