// Pieces shared by the NVFP4 GEMM kernels that dequantize per lane (the
// lane kernel and the small-tile kernel): stage geometry, the exact FP16
// dequantization of 8 E2M1 codes under one E4M3 block scale, the scale
// bytes as FP16 bit patterns, and the BF16 output packing.
#pragma once

#include "device_common.h"

namespace solfp4 {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));

// Two FP32 values to a BF16 pair (round to nearest even), first in the low half.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_t{lo, hi}), bf16x2_t));
}

constexpr int kLBK = 128;                       // K elements per stage
constexpr int kLRowBytes = kLBK / 2;            // code bytes per row per stage
constexpr int kLThreads = 256;
constexpr int kLBufs = 4;                       // LDS stage buffers (loads run 3 stages ahead)
constexpr int kLScaleStride = 5;                // words per row in LDS (4 + 1 pad)

// The 8 elements of one K-step (codes of word w, element j in nibble j)
// times the scale pattern s (s * 2^-8 in both halves): 256 q from the
// converter, then one exact packed multiply per pair.
__device__ __forceinline__ half8_t dequant_step(uint32_t w, half2_t s) {
  const half2_t d0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 0) * s;
  const half2_t d1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 1) * s;
  const half2_t d2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 2) * s;
  const half2_t d3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 3) * s;
  typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
  const half4_t lo = __builtin_shufflevector(d0, d1, 0, 1, 2, 3);
  const half4_t hi = __builtin_shufflevector(d2, d3, 0, 1, 2, 3);
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Scale bytes b0 (low) and b1 of a word's byte pair, as the FP16 patterns
// b << 7 (s * 2^-8) in the low and high half.
__device__ __forceinline__ uint32_t scale_patterns(uint32_t w, bool high_pair) {
  return __builtin_amdgcn_perm(0u, w, high_pair ? 0x0C030C02u : 0x0C010C00u) << 7;
}

}  // namespace solfp4
