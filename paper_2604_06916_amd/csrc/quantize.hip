// NVFP4 quantization kernels (Preliminaries of arXiv 2604.06916: E2M1
// elements, one E4M3 scale per 16 elements, Q(x) = S * Pi_FP4(x / S); plus a
// per-tensor FP32 scale alpha = amax / (6 * 448)).
//
// The tensor is a flat run of 16-element blocks (K % 16 == 0, row-major), so
// both kernels treat it as one-dimensional:
//   1. amax_partial_kernel  streams x once (nontemporal loads, grid-stride
//      loop) and writes one partial |x| maximum (as a 15-bit BF16
//      magnitude) per workgroup;
//   2. nvfp4_encode_kernel  folds the partials into alpha, tabulates
//      r(s) = 1 / (s * alpha) for the 126 nonzero finite E4M3 scales in LDS,
//      then streams x again, one block per lane pair (8 elements per lane,
//      so every load instruction covers whole cache lines): block amax
//      across the pair, E4M3 scale, table lookup of r, then E2M1 encoding by
//      the hardware converter.
// Both passes are HBM-bound streaming reads (2 B/element each) plus the
// 0.5625 B/element of codes and scales written by the second.
//
// The FP32 operation order is fixed (it decides the codes bit for bit):
//   alpha = amax_g / 2688; t = alpha * 6; s_f = amax_b / t; s = E4M3(s_f);
//   d = s * alpha; r = 1 / d; y = x * r; q = E2M1(y)
// with correctly rounded division (hipcc's default) and no contraction.
#include <mutex>

#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kQuantThreads = 256;

constexpr int kEncodeUnroll = 8;   // pieces per lane per iteration (large tensors)
constexpr int kEncodeUnrollSmall = 2;   // for small tensors: four times the workgroups
// Tensors past the 256 MB memory-side cache: 4 pieces per lane on up to
// 4096 workgroups (measured 2.6-3.8% faster there, 1-3% slower on 113 MB).
constexpr int kEncodeUnrollHuge = 4;
constexpr int64_t kEncodeHugePieces = (int64_t)1 << 24;   // 16 Mi pieces, 256 MB of BF16
constexpr int64_t kEncodeMaxGridHuge = 4096;
constexpr int kAmaxUnroll = 4;     // amax pass, pieces per lane per iteration (large tensors)
constexpr int kAmaxUnrollSmall = 2;

// Whether the amax pass takes the large unroll: every one of its kMaxPartials
// workgroups then runs at least one whole iteration.
static bool amax_large(int64_t n_vec) {
  return n_vec >= (int64_t)kMaxPartials * kQuantThreads * kAmaxUnroll;
}

__device__ __forceinline__ ushort2_t absmax_piece(ushort2_t m, u32x4_t v) {
  m = absmax_pair(m, v.x);
  m = absmax_pair(m, v.y);
  m = absmax_pair(m, v.z);
  return absmax_pair(m, v.w);
}

template <int kU>
__global__ __launch_bounds__(kQuantThreads) void amax_partial_kernel(
    const u32x4_t* __restrict__ x, int64_t n_vec, uint32_t* __restrict__ partial) {
  // grid-stride loop: an iteration covers kU * 256 consecutive 16-byte
  // pieces of the workgroup, kU loads in flight per lane
  ushort2_t m = {0, 0};
  const int64_t per_iter = (int64_t)kU * kQuantThreads;
  int64_t base = (int64_t)blockIdx.x * per_iter;
  const int64_t stride = (int64_t)gridDim.x * per_iter;
  for (; base + per_iter <= n_vec; base += stride) {
    u32x4_t v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) v[u] = __builtin_nontemporal_load(&x[base + u * kQuantThreads + threadIdx.x]);
#pragma unroll
    for (int u = 0; u < kU; ++u) m = absmax_piece(m, v[u]);
  }
  // the one iteration that reaches past the end (at most one workgroup)
  if (base < n_vec) {
    for (int64_t i = base + threadIdx.x; i < n_vec; i += kQuantThreads) m = absmax_piece(m, x[i]);
  }
  uint32_t r = wave_max_u32(max((uint32_t)m.x, (uint32_t)m.y));
  __shared__ uint32_t red[kQuantThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = r;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = red[0];
#pragma unroll
    for (int w = 1; w < kQuantThreads / kWave; ++w) t = max(t, red[w]);
    partial[blockIdx.x] = t;
  }
}

// max over the aligned lane pair (quad_perm DPP: lanes 1, 0, 3, 2)
__device__ __forceinline__ uint32_t pair_max(uint32_t v) {
  return max(v, (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false));
}

// One grid-stride iteration: kEncodeUnroll 16-byte pieces (8 elements) per
// lane starting at piece `base`; a lane pair owns one 16-element block, so
// consecutive lanes read consecutive pieces and write consecutive 4-byte
// code words.  rtab[c] = 1 / (value(c) * alpha) (0 for c == 0, so a
// zero-scale block becomes signed zeros: x * 0 keeps the sign).  kGuard: the
// iteration reaches past the last piece (uniform choice per iteration).
template <bool kGuard, int kU>
__device__ __forceinline__ void encode_iter(const u32x4_t* __restrict__ x, int64_t npieces,
                                            int64_t base, float t, bool zero_tensor,
                                            const float* rtab, uint32_t* __restrict__ codes,
                                            uint8_t* __restrict__ scales) {
  const int lane = threadIdx.x & (kWave - 1);
  u32x4_t v[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t p = base + u * kQuantThreads + threadIdx.x;
    v[u] = (!kGuard || p < npieces) ? __builtin_nontemporal_load(&x[p]) : u32x4_t{0, 0, 0, 0};
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t p = base + u * kQuantThreads + threadIdx.x;
    const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
    ushort2_t m = as_us2(w[0] & 0x7FFF7FFFu);
#pragma unroll
    for (int j = 1; j < 4; ++j) m = absmax_pair(m, w[j]);
    const uint32_t ab = pair_max(max((uint32_t)m.x, (uint32_t)m.y));
    const float amax_b = __uint_as_float(ab << 16);
    const float q = amax_b / t;
    const uint32_t sc = e4m3_rne_sat(zero_tensor ? 0.0f : q);
    const float r = rtab[sc];
    // hardware E2M1 encode, two elements per byte (the first in the low nibble)
    uint32_t c = 0;
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[0] << 16) * r,
                                                 __uint_as_float(w[0] & 0xFFFF0000u) * r, 1.0f, 0);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[1] << 16) * r,
                                                 __uint_as_float(w[1] & 0xFFFF0000u) * r, 1.0f, 1);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[2] << 16) * r,
                                                 __uint_as_float(w[2] & 0xFFFF0000u) * r, 1.0f, 2);
    c = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(c, __uint_as_float(w[3] << 16) * r,
                                                 __uint_as_float(w[3] & 0xFFFF0000u) * r, 1.0f, 3);
    if (!kGuard || p < npieces) {
      codes[p] = c;
      if ((lane & 1) == 0) scales[p >> 1] = (uint8_t)sc;
    }
  }
}

template <int kU>
__global__ __launch_bounds__(kQuantThreads) void nvfp4_encode_kernel(
    const u32x4_t* __restrict__ x, int64_t npieces, const uint32_t* __restrict__ partial,
    int npartial, uint32_t* __restrict__ codes, uint8_t* __restrict__ scales,
    float* __restrict__ global_scale) {
  // fold the first pass's partial maxima (every workgroup does it; a few KB
  // from L2)
  __shared__ uint32_t red[kQuantThreads / kWave];
  __shared__ float rtab[128];
  uint32_t m = 0;
  for (int i = threadIdx.x; i < npartial; i += kQuantThreads) m = max(m, partial[i]);
  m = wave_max_u32(m);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = m;
  __syncthreads();
  uint32_t amax_bits = red[0];
#pragma unroll
  for (int w = 1; w < kQuantThreads / kWave; ++w) amax_bits = max(amax_bits, red[w]);

  const float amax_g = __uint_as_float(amax_bits << 16);
  const float alpha = amax_g / kAlphaDivisor;
  const float t = alpha * 6.0f;
  const bool zero_tensor = amax_bits == 0u;
  if (blockIdx.x == 0 && threadIdx.x == 0) *global_scale = alpha;
  // r(s) = 1 / (s * alpha), both operations rounded exactly as the encoding
  // prescribes; code 0 (and the unused NaN code) map to 0
  if (threadIdx.x < 128) {
    const uint32_t c = threadIdx.x;
    const float d = e4m3_value(c) * alpha;
    rtab[c] = (c == 0u || c == 0x7Fu) ? 0.0f : 1.0f / d;
  }
  __syncthreads();

  const int64_t per_iter = (int64_t)kQuantThreads * kU;
  for (int64_t base = (int64_t)blockIdx.x * per_iter; base < npieces;
       base += (int64_t)gridDim.x * per_iter) {
    if (base + per_iter <= npieces)
      encode_iter<false, kU>(x, npieces, base, t, zero_tensor, rtab, codes, scales);
    else
      encode_iter<true, kU>(x, npieces, base, t, zero_tensor, rtab, codes, scales);
  }
}

// Scratch of the allocation-free quantize: the amax pass's partial maxima,
// one word per workgroup of that pass, at most kMaxPartials (4 KiB).  Each
// device the library runs on holds its own copy until the process ends.
// Host code never passes `scratch` itself to a kernel (on the host the name
// stands for a host-side shadow, not a device address): the address comes
// from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint32_t scratch[kScratchWords];

hipError_t scratch_address(uint32_t** out) {
  constexpr int kMaxDevices = 64;
  static uint32_t* cached[kMaxDevices];
  static std::mutex mu;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!cached[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    cached[dev] = static_cast<uint32_t*>(p);
  }
  *out = cached[dev];
  return hipSuccess;
}

int amax_partial_count(int64_t n_elems) {
  // the grid of the amax pass, one partial maximum per workgroup: all
  // kMaxPartials once each runs a whole iteration of the large unroll;
  // below that one workgroup per iteration of the small unroll (4 Ki
  // elements), so that small tensors still spread over many CUs
  const int64_t n_vec = n_elems / 8;
  if (amax_large(n_vec)) return kMaxPartials;
  int64_t p = (n_vec + kQuantThreads * kAmaxUnrollSmall - 1) / (kQuantThreads * kAmaxUnrollSmall);
  if (p < 1) p = 1;
  if (p > kMaxPartials) p = kMaxPartials;
  return (int)p;
}

hipError_t launch_amax(const uint16_t* x, int64_t n, uint32_t* partial, hipStream_t stream) {
  const int64_t n_vec = n / 8;
  return launch_kernel(amax_large(n_vec) ? amax_partial_kernel<kAmaxUnroll> : amax_partial_kernel<kAmaxUnrollSmall>,
                       dim3(amax_partial_count(n)), dim3(kQuantThreads), stream,
                       reinterpret_cast<const u32x4_t*>(x), n_vec, partial);
}

hipError_t launch_encode(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                         uint8_t* scales, float* global_scale, const uint32_t* partial,
                         hipStream_t stream) {
  const int64_t n = rows * K;
  const int64_t npieces = n / 8;           // 8 elements per lane, 2 lanes per block
  const int npartial = amax_partial_count(n);
  // small tensors (under 64 workgroups of the large unroll) take the small
  // unroll, so that they spread over four times as many CUs; the arithmetic
  // per piece is the same
  const bool small = npieces < 64 * (int64_t)kQuantThreads * kEncodeUnroll;
  const bool huge = npieces >= kEncodeHugePieces;
  const int unroll = small ? kEncodeUnrollSmall : huge ? kEncodeUnrollHuge : kEncodeUnroll;
  const int64_t per_wg = (int64_t)kQuantThreads * unroll;
  int64_t grid = (npieces + per_wg - 1) / per_wg;
  const int64_t cap = huge ? kEncodeMaxGridHuge : kEncodeMaxGrid;
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  return launch_kernel(small  ? nvfp4_encode_kernel<kEncodeUnrollSmall>
                       : huge ? nvfp4_encode_kernel<kEncodeUnrollHuge>
                              : nvfp4_encode_kernel<kEncodeUnroll>,
                       dim3((unsigned)grid), dim3(kQuantThreads), stream,
                       reinterpret_cast<const u32x4_t*>(x), npieces, partial, npartial,
                       reinterpret_cast<uint32_t*>(codes), scales, global_scale);
}

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                           uint8_t* scales, float* global_scale, uint32_t* partial,
                           hipStream_t stream) {
  const hipError_t e = launch_amax(x, rows * K, partial, stream);
  if (e != hipSuccess) return e;
  return launch_encode(x, rows, K, codes, scales, global_scale, partial, stream);
}

}  // namespace solfp4
