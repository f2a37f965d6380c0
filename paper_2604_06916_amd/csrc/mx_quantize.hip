// MXFP4 quantization (Preliminaries of arXiv 2604.06916: the OCP MX format
// with E2M1 elements and one power-of-two E8M0 scale per 32 elements).
//
// Per 32-element block, following the OCP MX conversion rule:
//   E = floor(log2(amax_b)) - 2   (2 = exponent of the largest E2M1 value, 6)
//   scale byte = clamp(E + 127, 0, 254), 0 for an all-zero block
//   q = E2M1_RNE_SAT(x / 2^E), sign kept on zeros.
// For a BF16 amax with exponent field f, floor(log2(amax_b)) + 127 = f, so the
// scale byte is max(f - 2, 0) (a subnormal or zero amax gives 0).  x / 2^E is
// a multiplication by the exact power of two 2^(127 - byte), so y is exact
// and the hardware converter (round to nearest even, saturating) gives the
// code.  One pass: 2 B/element read, 0.53125 B/element written.
#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kMxQuantThreads = 256;
constexpr int kMxQuantUnroll = 2;   // blocks per lane per iteration

__device__ __forceinline__ u32x4_t mx_stream_load(const u32x4_t* p) {
  return __builtin_nontemporal_load(p);
}

// Encode one 32-element block held in w[0..15] (element 2j in the low half
// of word j).  Writes 16 code bytes to c and returns the E8M0 byte.
__device__ __forceinline__ uint32_t mx_encode_block(const uint32_t (&w)[16], uint32_t (&c)[4]) {
  ushort2_t m = as_us2(w[0] & 0x7FFF7FFFu);
#pragma unroll
  for (int j = 1; j < 16; ++j) m = absmax_pair(m, w[j]);
  const uint32_t ab = max((uint32_t)m.x, (uint32_t)m.y);
  const uint32_t f = ab >> 7;                   // BF16 exponent field of amax_b
  const uint32_t sc = f > 2u ? f - 2u : 0u;
  const float inv = __uint_as_float((254u - sc) << 23);   // 2^(127 - sc)
  float e[32];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    e[2 * j] = __uint_as_float(w[j] << 16) * inv;
    e[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u) * inv;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t v = 0;
    v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, e[8 * i + 0], e[8 * i + 1], 1.0f, 0);
    v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, e[8 * i + 2], e[8 * i + 3], 1.0f, 1);
    v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, e[8 * i + 4], e[8 * i + 5], 1.0f, 2);
    v = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(v, e[8 * i + 6], e[8 * i + 7], 1.0f, 3);
    c[i] = v;
  }
  return sc;
}

template <bool kGuard>
__device__ __forceinline__ void mx_encode_iter(const u32x4_t* __restrict__ x, int64_t nblocks,
                                               int64_t base, u32x4_t* __restrict__ codes,
                                               uint8_t* __restrict__ scales) {
  const int lane = threadIdx.x & (kWave - 1);
  u32x4_t v[kMxQuantUnroll][4];
#pragma unroll
  for (int u = 0; u < kMxQuantUnroll; ++u) {
    const int64_t blk = base + u * kMxQuantThreads + threadIdx.x;
#pragma unroll
    for (int p = 0; p < 4; ++p)
      v[u][p] = (!kGuard || blk < nblocks) ? mx_stream_load(&x[4 * blk + p]) : u32x4_t{0, 0, 0, 0};
  }
#pragma unroll
  for (int u = 0; u < kMxQuantUnroll; ++u) {
    const int64_t blk = base + u * kMxQuantThreads + threadIdx.x;
    uint32_t w[16];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      w[4 * p + 0] = v[u][p].x;
      w[4 * p + 1] = v[u][p].y;
      w[4 * p + 2] = v[u][p].z;
      w[4 * p + 3] = v[u][p].w;
    }
    uint32_t c[4];
    const uint32_t sc = mx_encode_block(w, c);
    if (!kGuard || blk < nblocks) codes[blk] = u32x4_t{c[0], c[1], c[2], c[3]};
    // gather the scale bytes of each aligned lane quad into its first lane
    const uint32_t s1 = (uint32_t)__builtin_amdgcn_mov_dpp((int)sc, 0x55, 0xF, 0xF, false);
    const uint32_t s2 = (uint32_t)__builtin_amdgcn_mov_dpp((int)sc, 0xAA, 0xF, 0xF, false);
    const uint32_t s3 = (uint32_t)__builtin_amdgcn_mov_dpp((int)sc, 0xFF, 0xF, 0xF, false);
    if ((lane & 3) == 0) {
      if (!kGuard || blk + 3 < nblocks) {
        *reinterpret_cast<uint32_t*>(scales + blk) = sc | (s1 << 8) | (s2 << 16) | (s3 << 24);
      } else {
        if (blk < nblocks) scales[blk] = (uint8_t)sc;
        if (blk + 1 < nblocks) scales[blk + 1] = (uint8_t)s1;
        if (blk + 2 < nblocks) scales[blk + 2] = (uint8_t)s2;
      }
    }
  }
}

__global__ __launch_bounds__(kMxQuantThreads) void mxfp4_quantize_kernel(
    const u32x4_t* __restrict__ x, int64_t nblocks, u32x4_t* __restrict__ codes,
    uint8_t* __restrict__ scales) {
  const int64_t per_iter = (int64_t)kMxQuantThreads * kMxQuantUnroll;
  for (int64_t base = (int64_t)blockIdx.x * per_iter; base < nblocks;
       base += (int64_t)gridDim.x * per_iter) {
    if (base + per_iter <= nblocks)
      mx_encode_iter<false>(x, nblocks, base, codes, scales);
    else
      mx_encode_iter<true>(x, nblocks, base, codes, scales);
  }
}

hipError_t launch_mx_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                              uint8_t* scales, hipStream_t stream) {
  const int64_t nblocks = rows * K / 32;
  if (nblocks == 0) return hipSuccess;
  const int64_t per_wg = (int64_t)kMxQuantThreads * kMxQuantUnroll;
  int64_t grid = (nblocks + per_wg - 1) / per_wg;
  if (grid > kEncodeMaxGrid) grid = kEncodeMaxGrid;
  hipLaunchKernelGGL(mxfp4_quantize_kernel, dim3((unsigned)grid), dim3(kMxQuantThreads), 0, stream,
                     reinterpret_cast<const u32x4_t*>(x), nblocks,
                     reinterpret_cast<u32x4_t*>(codes), scales);
  return hipGetLastError();
}

}  // namespace solfp4
