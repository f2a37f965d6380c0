// Device-side types and helpers shared by the solfp4 kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace solfp4 {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Per-tensor scale divisor: largest E2M1 magnitude times largest E4M3 value.
constexpr float kAlphaDivisor = 6.0f * 448.0f;

__device__ __forceinline__ ushort2_t as_us2(uint32_t v) { return __builtin_bit_cast(ushort2_t, v); }
__device__ __forceinline__ uint32_t as_u32(ushort2_t v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }
__device__ __forceinline__ uint32_t h2_as_u32(half2_t v) { return __builtin_bit_cast(uint32_t, v); }

// Largest BF16 magnitude (as its 15-bit pattern) among the two halves of
// each word, combined into a packed pair: |x| of non-negative floats orders
// like the integers of their bit patterns, so this max is exact.
__device__ __forceinline__ ushort2_t absmax_pair(ushort2_t acc, uint32_t w) {
  return __builtin_elementwise_max(acc, as_us2(w & 0x7FFF7FFFu));
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, kWave));
  return v;
}

// E4M3 (OCP E4M3FN) code of a non-negative binary32 value: nearest, ties to
// the even code, saturating at 448.  Normal range: round the binary32
// significand to 3 bits with the carry allowed into the exponent; subnormal
// range (< 2^-6): the E4M3 grid is k * 2^-9, so round s * 512 (exact) to an
// integer.  Branch free: both candidates are formed and one is selected.
__device__ __forceinline__ uint32_t e4m3_rne_sat(float s) {
  const uint32_t u = __float_as_uint(s);
  const uint32_t normal = ((u + 0x7FFFFu + ((u >> 20) & 1u)) >> 20) - (120u << 3);
  const uint32_t sub = (uint32_t)__builtin_rintf(s * 512.0f);
  const uint32_t code = s < 0x1p-6f ? sub : normal;
  return s < 448.0f ? code : 0x7Eu;
}

// Exact value of an E4M3 byte (finite codes 0x00..0x7E).
__device__ __forceinline__ float e4m3_value(uint32_t c) {
  return c < 8u ? (float)c * 0x1p-9f : __uint_as_float((c + (120u << 3)) << 20);
}

// Round binary32 to BF16 bits (nearest, ties to even).  Finite inputs.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

}  // namespace solfp4
