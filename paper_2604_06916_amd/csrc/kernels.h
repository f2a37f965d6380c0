// Internal launch interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace solfp4 {

// First quantize pass: at most this many partial maxima (workspace words).
constexpr int kMaxPartials = 1024;
// Encode pass: grid-stride loop over at most this many workgroups (eight
// per compute unit: more only adds per-workgroup set-up and an uneven tail).
constexpr int64_t kEncodeMaxGrid = 2048;
// MXFP4 quantize: grid-stride loop over at most this many workgroups.
constexpr int64_t kMxQuantMaxGrid = 8192;

int amax_partial_count(int64_t n_elems);

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                           uint8_t* scales, float* global_scale, uint32_t* partial,
                           hipStream_t stream);

// Whether a GEMM should run on 128 x 128 output tiles rather than 256 x 256
// ones, given the tile counts of both (host only).
bool small_tiles_pay(int64_t tiles256, int64_t tiles128);

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                       const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                       const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                       hipStream_t stream);

// MXFP4 (32-element blocks, E8M0 scales): one quantize pass, and the GEMM
// on the scaled FP4 matrix instructions.
hipError_t launch_mx_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                              uint8_t* scales, hipStream_t stream);

hipError_t launch_mx_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
                          const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M,
                          int64_t N, int64_t K, hipStream_t stream);

}  // namespace solfp4
