// Device helpers shared by the kernels of libkvb (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvb {

// float -> bfloat16 bit pattern, round to nearest even (finite inputs; NaN
// stays a quiet NaN).  Written with integer operations so the rounding rule
// is explicit.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (u >> 16) | 0x40u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// code of channel j from a row of stored codes (BITS 8: one byte per channel;
// BITS 4: two per byte, even channel in the low nibble)
template <int BITS>
__device__ __forceinline__ uint32_t code_at(const uint32_t* words, int j) {
  if constexpr (BITS == 8) {
    return (words[j >> 2] >> ((j & 3) * 8)) & 0xFFu;
  } else {
    return (words[j >> 3] >> ((j & 7) * 4)) & 0xFu;
  }
}

}  // namespace kvb
