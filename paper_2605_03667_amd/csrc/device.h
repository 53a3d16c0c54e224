// Device-side helpers shared by the kernel translation units: vector types,
// bf16 bit manipulation and the 2:4 top-2 selection (Algorithm 1 of ELAS on
// one group of 4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elas {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// float -> bf16 bits, round to nearest, ties to even.  Integer formulation:
// adding 0x7FFF plus the lowest kept bit carries into the kept half exactly
// when the dropped half is above one half ulp, or equal to it with an odd kept
// half.  Infinity stays infinity; finite values past the largest bf16 become
// infinity; NaN inputs are not expected here (keys are never NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float x) {
  uint32_t u = __builtin_bit_cast(uint32_t, x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t b) {
  return __builtin_bit_cast(float, b << 16);
}

// relu(h) as bf16 bits for a bf16 input: the bits themselves when h is a
// positive non-NaN number, else 0.  For non-negative bf16 the bit pattern
// orders exactly like the value, and (as h*h is exact in fp32 over the
// contract range) exactly like s = relu(h)^2, so the bits serve as the
// ranking key of Algorithm 1 on s.
__device__ __forceinline__ uint32_t relu_bits(uint32_t b) {
  return ((int32_t)(int16_t)b > 0 && b <= 0x7F80u) ? b : 0u;
}

// Stable top-2 of four keys (ties go to the lower index).  Returns the 4-bit
// code i0 | (i1 << 2) of the two kept positions, i0 < i1.  Element i beats
// element j (i < j) when key_i >= key_j; an element is kept when it beats at
// least two of the other three.
__device__ __forceinline__ uint32_t top2_code(uint32_t k0, uint32_t k1, uint32_t k2, uint32_t k3) {
  const uint32_t b01 = k0 >= k1, b02 = k0 >= k2, b03 = k0 >= k3;
  const uint32_t b12 = k1 >= k2, b13 = k1 >= k3, b23 = k2 >= k3;
  const uint32_t w0 = b01 + b02 + b03;
  const uint32_t w1 = 1u - b01 + b12 + b13;
  const uint32_t w2 = 2u - b02 - b12 + b23;
  const uint32_t w3 = 3u - b03 - b13 - b23;
  const uint32_t m = (w0 >= 2u) | ((w1 >= 2u) << 1) | ((w2 >= 2u) << 2) | ((w3 >= 2u) << 3);
  // keep-mask -> code: 0b0011->(0,1)=4, 0b0101->(0,2)=8, 0b0110->(1,2)=9,
  // 0b1001->(0,3)=12, 0b1010->(1,3)=13, 0b1100->(2,3)=14
  constexpr uint64_t kLut = (4ull << 12) | (8ull << 20) | (9ull << 24) | (12ull << 36) |
                            (13ull << 40) | (14ull << 48);
  return (uint32_t)(kLut >> (4u * m)) & 0xFu;
}

// The two kept entries of a group (v0..v3) for a code from top2_code.
__device__ __forceinline__ uint32_t pick_pair(uint32_t code, uint32_t v0, uint32_t v1, uint32_t v2,
                                              uint32_t v3) {
  const uint32_t i0 = code & 3u, i1 = code >> 2;
  const uint32_t a = i0 == 0u ? v0 : (i0 == 1u ? v1 : v2);
  const uint32_t b = i1 == 1u ? v1 : (i1 == 2u ? v2 : v3);
  return a | (b << 16);
}

}  // namespace elas
