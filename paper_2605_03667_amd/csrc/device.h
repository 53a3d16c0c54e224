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
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (the hardware conversion, round to nearest even)
// packed as lo | hi << 16: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
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

// relu on two packed bf16 (lo | hi << 16), with the same result as relu_bits
// on each half: negative values, -0 and NaN become 0.  After the signed
// max with 0, adding 0x7F moves exactly the NaN patterns (0x7F81..0x7FFF)
// past 0x7FFF; the second max sends them to 0x7F, and subtracting 0x7F
// restores every other value.  Four packed 16-bit operations.
__device__ __forceinline__ uint32_t relu_bits2(uint32_t p) {
  typedef short s16x2 __attribute__((ext_vector_type(2)));
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  const s16x2 zero = {0, 0}, c7f = {0x7F, 0x7F};
  const u16x2 u7f = {0x7F, 0x7F};
  s16x2 v = __builtin_elementwise_max(__builtin_bit_cast(s16x2, p), zero);
  v = __builtin_bit_cast(s16x2, __builtin_bit_cast(u16x2, v) + u7f);
  v = __builtin_elementwise_max(v, c7f);
  return __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, v) - u7f);
}

// Top-2 of a group of four from two packed relu'd pairs (p01 = r0 | r1 << 16,
// p23 = r2 | r3 << 16), as Algorithm 1 ranks them: by value, ties to the lower
// index.  Each element becomes the unique key r << 2 | (3 - i), so that a
// plain maximum implements the tie rule.  With a, b the larger and smaller
// key of elements 0, 1 and c, d those of 2, 3, the largest key is max(a, c)
// and the second largest max(min(a, c), max(b, d)).  Rotating the index bits
// to the top orders the two kept elements
// by index.
struct Top2 {
  uint32_t first, second;   // r | (3 - i) << 30 of the kept elements, i0 < i1
};
__device__ __forceinline__ Top2 top2_keys(uint32_t p01, uint32_t p23) {
  const uint32_t k0 = ((p01 & 0xFFFFu) << 2) | 3u;
  const uint32_t k1 = ((p01 >> 14) & 0x3FFFCu) | 2u;
  const uint32_t k2 = ((p23 & 0xFFFFu) << 2) | 1u;
  const uint32_t k3 = (p23 >> 14) & 0x3FFFCu;
  const uint32_t a = k0 > k1 ? k0 : k1, b = k0 > k1 ? k1 : k0;
  const uint32_t c = k2 > k3 ? k2 : k3, d = k2 > k3 ? k3 : k2;
  const uint32_t t1 = a > c ? a : c;
  const uint32_t e = b > d ? b : d, f = a > c ? c : a;
  const uint32_t t2 = e > f ? e : f;
  const uint32_t r1 = __builtin_amdgcn_alignbit(t1, t1, 2), r2 = __builtin_amdgcn_alignbit(t2, t2, 2);
  Top2 t;
  t.first = r1 > r2 ? r1 : r2;
  t.second = r1 > r2 ? r2 : r1;
  return t;
}
// Code i0 | i1 << 2 of a Top2 result.
__device__ __forceinline__ uint32_t top2_code_of(const Top2& t) {
  return 15u - ((t.first >> 30) | ((t.second >> 30) << 2));
}

// relu of an fp32 value with NaN sent to 0: v_max_f32 returns the non-NaN
// operand.  Written as one instruction because the compiler's fmaxf first
// quiets its input (a second instruction).
__device__ __forceinline__ float relu_f32(float x) {
  float r;
  asm("v_max_f32 %0, 0, %1" : "=v"(r) : "v"(x));
  return r;
}

// The same top-2 as top2_keys, for the fused epilogues, with fewer
// instructions.  The inputs hold non-negative bf16 pairs (p01 = r0 | r1 << 16,
// p23 = r2 | r3 << 16).  Key of element i: r << 16 | (3 - i), built with one
// instruction each.  With m and e the largest and middle key of elements
// 0..2, the largest of all four is max(m, k3) and the second largest
// max(e, min(m, k3)).  Rotating right by 2 moves the index bits to the top
// (r sits at bits 14..29, bits 0..13 are zero), which orders the kept pair by
// index; `first << 2` and `second << 2` are the kept values as fp32.
__device__ __forceinline__ Top2 top2_keys_hi(uint32_t p01, uint32_t p23) {
  const uint32_t k0 = (p01 << 16) | 3u;
  const uint32_t k1 = (p01 & 0xFFFF0000u) | 2u;
  const uint32_t k2 = (p23 << 16) | 1u;
  const uint32_t k3 = p23 & 0xFFFF0000u;
  uint32_t m, e;   // v_max3_u32 / v_med3_u32 (not formed from min/max by the compiler)
  asm("v_max3_u32 %0, %1, %2, %3" : "=v"(m) : "v"(k0), "v"(k1), "v"(k2));
  asm("v_med3_u32 %0, %1, %2, %3" : "=v"(e) : "v"(k0), "v"(k1), "v"(k2));
  const uint32_t t1 = __builtin_elementwise_max(m, k3);
  const uint32_t t2 = __builtin_elementwise_max(e, __builtin_elementwise_min(m, k3));
  const uint32_t r1 = __builtin_amdgcn_alignbit(t1, t1, 2), r2 = __builtin_amdgcn_alignbit(t2, t2, 2);
  Top2 t;
  t.first = __builtin_elementwise_max(r1, r2);
  t.second = __builtin_elementwise_min(r1, r2);
  return t;
}
// (3 - i0) | (3 - i1) << 2 of a top2_keys_hi result: the code XOR 15.
__device__ __forceinline__ uint32_t top2_code_xor15(const Top2& t) {
  return (t.first >> 30) | ((t.second >> 28) & 0xCu);
}

// Square root rounded to bf16 for a non-negative bf16 value s given as fp32.
// The raw v_sqrt_f32 result rounds to the same bf16 as the correctly rounded
// square root for every such s with a normal exponent (checked over all bf16
// inputs on gfx950); subnormal inputs, which v_sqrt_f32 flushes, are scaled
// by 2^64 first and the root by 2^-32 after (both exact).  The caller rounds.
__device__ __forceinline__ float sqrt_for_bf16(float s) {
  const bool tiny = s < 0x1p-126f;
  const float r = __builtin_amdgcn_sqrtf(tiny ? s * 0x1p64f : s);
  return tiny ? r * 0x1p-32f : r;
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
