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
//
// Layout of the work: a lane quad owns one block, each lane 8 elements (16
// bytes), so consecutive lanes read consecutive 16-byte pieces (every load
// instruction covers whole cache lines) and write consecutive 4-byte code
// words; the block maximum is combined across the quad with DPP.
#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kMxQuantThreads = 256;
constexpr int kMxQuantUnroll = 4;   // 16-byte pieces per lane per iteration

__device__ __forceinline__ u32x4_t mx_stream_load(const u32x4_t* p) {
  return __builtin_nontemporal_load(p);
}

// max over the aligned lane quad (quad_perm DPP: lanes 1,0,3,2 then 2,3,0,1)
__device__ __forceinline__ uint32_t quad_max(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false));
  return v;
}

template <bool kGuard>
__device__ __forceinline__ void mx_encode_iter(const u32x4_t* __restrict__ x, int64_t npieces,
                                               int64_t base, uint32_t* __restrict__ codes,
                                               uint8_t* __restrict__ scales) {
  const int lane = threadIdx.x & (kWave - 1);
  u32x4_t v[kMxQuantUnroll];
#pragma unroll
  for (int u = 0; u < kMxQuantUnroll; ++u) {
    const int64_t p = base + u * kMxQuantThreads + threadIdx.x;
    v[u] = (!kGuard || p < npieces) ? mx_stream_load(&x[p]) : u32x4_t{0, 0, 0, 0};
  }
#pragma unroll
  for (int u = 0; u < kMxQuantUnroll; ++u) {
    const int64_t p = base + u * kMxQuantThreads + threadIdx.x;
    const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    ushort2_t m = as_us2(w[0] & 0x7FFF7FFFu);
#pragma unroll
    for (int j = 1; j < 4; ++j) m = absmax_pair(m, w[j]);
    const uint32_t ab = quad_max(max((uint32_t)m.x, (uint32_t)m.y));
    const uint32_t f = ab >> 7;                   // BF16 exponent field of amax_b
    const uint32_t sc = f > 2u ? f - 2u : 0u;
    const float inv = __uint_as_float((254u - sc) << 23);   // 2^(127 - sc)
    uint32_t c = 0;
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[0] << 16) * inv,
                                                 __uint_as_float(w[0] & 0xFFFF0000u) * inv, 1.0f, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[1] << 16) * inv,
                                                 __uint_as_float(w[1] & 0xFFFF0000u) * inv, 1.0f, 1);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[2] << 16) * inv,
                                                 __uint_as_float(w[2] & 0xFFFF0000u) * inv, 1.0f, 2);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[3] << 16) * inv,
                                                 __uint_as_float(w[3] & 0xFFFF0000u) * inv, 1.0f, 3);
    if (!kGuard || p < npieces) {
      codes[p] = c;
      if ((lane & 3) == 0) scales[p >> 2] = (uint8_t)sc;
    }
  }
}

__global__ __launch_bounds__(kMxQuantThreads) void mxfp4_quantize_kernel(
    const u32x4_t* __restrict__ x, int64_t npieces, uint32_t* __restrict__ codes,
    uint8_t* __restrict__ scales) {
  const int64_t per_iter = (int64_t)kMxQuantThreads * kMxQuantUnroll;
  for (int64_t base = (int64_t)blockIdx.x * per_iter; base < npieces;
       base += (int64_t)gridDim.x * per_iter) {
    if (base + per_iter <= npieces)
      mx_encode_iter<false>(x, npieces, base, codes, scales);
    else
      mx_encode_iter<true>(x, npieces, base, codes, scales);
  }
}

hipError_t launch_mx_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                              uint8_t* scales, hipStream_t stream) {
  const int64_t npieces = rows * K / 8;      // 8 elements per lane, 4 lanes per block
  if (npieces == 0) return hipSuccess;
  const int64_t per_wg = (int64_t)kMxQuantThreads * kMxQuantUnroll;
  int64_t grid = (npieces + per_wg - 1) / per_wg;
  if (grid > kMxQuantMaxGrid) grid = kMxQuantMaxGrid;
  return launch_kernel(mxfp4_quantize_kernel, dim3((unsigned)grid), dim3(kMxQuantThreads), stream,
                       reinterpret_cast<const u32x4_t*>(x), npieces,
                       reinterpret_cast<uint32_t*>(codes), scales);
}

}  // namespace solfp4
