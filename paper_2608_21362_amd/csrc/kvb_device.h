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

// two floats -> packed bfloat16 pair (lo in the low half), round to nearest
// even: one v_cvt_pk_bf16_f32, which rounds like f32_to_bf16_rne for every
// non-NaN input
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) float f2;
  typedef __attribute__((ext_vector_type(2))) __bf16 b2;
  const f2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2));
}

// packed bfloat16 pair -> packed fp16 pair (exact while |x| <= 65504 and x is
// not below the fp16 normal range)
__device__ __forceinline__ uint32_t bf16x2_to_f16x2(uint32_t w) {
  typedef __attribute__((ext_vector_type(2))) float f2;
  typedef __attribute__((ext_vector_type(2))) _Float16 h2;
  const f2 v = {__uint_as_float(w << 16), __uint_as_float(w & 0xFFFF0000u)};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, h2));
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
