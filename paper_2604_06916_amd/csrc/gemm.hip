// Block-scaled NVFP4 GEMM with BF16 output for gfx950.
//
//   out[m][n] = bf16( aA * aB * sum_k (sA qA)[m][k] (sB qB)[n][k] + bias[n] )
//
// How the E4M3-per-16 scales are applied.  CDNA4's scaled matrix
// instructions take one power-of-two (E8M0) scale per 32 K-elements, while an
// NVFP4 element decodes to q * s with an E4M3 s: up to 2 + 4 = 6 significant
// bits per operand, more than any FP4/FP6/FP8 matrix input format carries.
// The kernel therefore keeps the operands packed (0.5 B/element codes plus
// 1/16 B/element scales) in HBM and LDS and dequantizes each element exactly
// to FP16 in registers (hardware FP4->FP16 convert, then one packed FP16
// multiply by the block scale: products of <= 6 significant bits in
// [2^-10, 2688], exact), feeding the FP16 matrix cores
// (v_mfma_f32_32x32x16_f16) with FP32 accumulation.  Every product
// (sA qA)(sB qB) is exact; only the FP32 sums and the final BF16 rounding
// round.  The per-tensor scales and the bias are applied once, in the
// epilogue.
//
// Tiling: 256 x 256 output tile per workgroup of 4 waves (2 x 2), each wave
// owning 128 x 128 (4 x 4 MFMA tiles of 32 x 32, accumulators in AGPRs); K
// advances 128 elements (8 NVFP4 blocks) per LDS stage, double buffered.
// Inside a stage the wave walks 32-element chunks; lane (i, g) of a fragment
// takes row i and the whole 16-element block 2c+g of chunk c, whose first 8
// elements feed the chunk's first MFMA and last 8 its second (the same
// K permutation is used for both operands, so the sum is unchanged).
// The MFMA's first operand is the weight tile, so each lane's accumulators
// hold 4 consecutive output columns of one row (8-byte BF16 stores).
#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kBM = 256;
constexpr int kBN = 256;
constexpr int kBKB = 8;                    // NVFP4 blocks per K stage (128 elements)
constexpr int kCodeRow = kBKB * 8;         // code bytes per row per stage
constexpr int kCodeStride = kCodeRow + 8;  // padded LDS row, bytes
constexpr int kScaleStride = kBKB + 1;     // padded LDS row of f16x2 scales, words
constexpr int kGemmThreads = 256;
constexpr int kWaveTile = 128;
constexpr int kFrags = kWaveTile / 32;     // 32x32 MFMA tiles per wave dimension

struct Stage {
  uint8_t a_codes[kBM * kCodeStride];
  uint8_t b_codes[kBN * kCodeStride];
  uint32_t a_scales[kBM * kScaleStride];
  uint32_t b_scales[kBN * kScaleStride];
};

// f16x2 (s, s) bit pattern of an E4M3 scale byte (exact: every finite E4M3
// value is a normal FP16 number).
__device__ __forceinline__ uint32_t scale_f16x2(uint32_t c) {
  const _Float16 sub = (_Float16)(float)c * (_Float16)0x1p-9f;
  const uint32_t h = c >= 8u ? (c << 7) + 0x2000u : (uint32_t)__builtin_bit_cast(uint16_t, sub);
  return h | (h << 16);
}

// 8 E2M1 codes (one 32-bit word, element 2j in the low nibble of byte j)
// times the block scale, as 8 exact FP16 values.
__device__ __forceinline__ half8_t dequant8(uint32_t codes, uint32_t scale2) {
  const half2_t s = as_h2(scale2);
  const half2_t p0 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 0) * s;
  const half2_t p1 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 1) * s;
  const half2_t p2 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 2) * s;
  const half2_t p3 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, 3) * s;
  return half8_t{p0.x, p0.y, p1.x, p1.y, p2.x, p2.y, p3.x, p3.y};
}

// Register-staged copy of one operand's stage: 4 x 16 code bytes and 8
// scale bytes per thread.
struct OperandRegs {
  uint4 codes[4];
  uint32_t sc_lo, sc_hi;
};

// Thread t loads code units u = t + 256 p (p < 4), unit u = row u/4, bytes
// 16 (u%4) .. +16 of the stage; and the 8 scale bytes of row t.
// kFast: K % 128 == 0 (no partial stage; 16-byte code rows, 8-byte scale
// rows are aligned).  Otherwise loads go by 8-byte block and scale byte,
// each guarded against K.
template <bool kFast>
__device__ __forceinline__ void load_operand(OperandRegs& r, const uint8_t* __restrict__ codes,
                                             const uint8_t* __restrict__ scales, int64_t row0,
                                             int64_t rows, int64_t K, int stage) {
  const int t = threadIdx.x;
  const int64_t kb_total = K / 16;
  const int64_t kb0 = (int64_t)stage * kBKB;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int u = t + kGemmThreads * p;
    const int64_t row = row0 + (u >> 2);
    const int col = u & 3;
    const int64_t kb = kb0 + 2 * col;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row < rows) {
      const uint8_t* src = codes + row * (K / 2) + kb * 8;
      if (kFast) {
        v = *reinterpret_cast<const uint4*>(src);
      } else {
        if (kb < kb_total) {
          const uint2 lo = *reinterpret_cast<const uint2*>(src);
          v.x = lo.x;
          v.y = lo.y;
        }
        if (kb + 1 < kb_total) {
          const uint2 hi = *reinterpret_cast<const uint2*>(src + 8);
          v.z = hi.x;
          v.w = hi.y;
        }
      }
    }
    r.codes[p] = v;
  }
  const int64_t srow = row0 + t;
  r.sc_lo = 0;
  r.sc_hi = 0;
  if (srow < rows) {
    const uint8_t* src = scales + srow * kb_total + kb0;
    if (kFast) {
      const uint2 s = *reinterpret_cast<const uint2*>(src);
      r.sc_lo = s.x;
      r.sc_hi = s.y;
    } else {
      uint32_t lo = 0, hi = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (kb0 + j < kb_total) lo |= (uint32_t)src[j] << (8 * j);
        if (kb0 + 4 + j < kb_total) hi |= (uint32_t)src[4 + j] << (8 * j);
      }
      r.sc_lo = lo;
      r.sc_hi = hi;
    }
  }
}

__device__ __forceinline__ void store_operand(const OperandRegs& r, uint8_t* lds_codes,
                                              uint32_t* lds_scales) {
  const int t = threadIdx.x;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int u = t + kGemmThreads * p;
    uint8_t* dst = lds_codes + (u >> 2) * kCodeStride + (u & 3) * 16;
    *reinterpret_cast<uint2*>(dst) = make_uint2(r.codes[p].x, r.codes[p].y);
    *reinterpret_cast<uint2*>(dst + 8) = make_uint2(r.codes[p].z, r.codes[p].w);
  }
  uint32_t* srow = lds_scales + t * kScaleStride;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    srow[j] = scale_f16x2((r.sc_lo >> (8 * j)) & 0xFFu);
    srow[4 + j] = scale_f16x2((r.sc_hi >> (8 * j)) & 0xFFu);
  }
}

// Tile order: consecutive workgroups are dispatched round-robin over the 8
// XCDs, each with its own L2.  Remap so each XCD gets a contiguous range of
// tile ids, then walk tiles in groups of kGroupM row-tiles so the tiles an
// XCD runs together share A rows and B columns.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
  const int b = blockIdx.x;
  const int per_xcd = total / kXcds;
  const int t = b < per_xcd * kXcds ? (b % kXcds) * per_xcd + b / kXcds : b;
  const int group_size = kGroupM * tiles_n;
  const int group = t / group_size;
  const int first_m = group * kGroupM;
  const int gm = min(tiles_m - first_m, kGroupM);
  const int in_group = t % group_size;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

template <bool kFast, bool kVecOut>
__global__ __launch_bounds__(kGemmThreads, 1) void nvfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_gs, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_gs,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K) {
  __shared__ Stage smem[2];

  const int tiles_m = (int)((M + kBM - 1) / kBM);
  const int tiles_n = (int)((N + kBN - 1) / kBN);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kBM;
  const int64_t n0 = (int64_t)tn * kBN;

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int wm = wave >> 1;
  const int wn = wave & 1;
  const int li = lane & 31;
  const int lg = lane >> 5;

  floatx16_t acc[kFrags][kFrags];
#pragma unroll
  for (int i = 0; i < kFrags; ++i)
#pragma unroll
    for (int j = 0; j < kFrags; ++j) acc[i][j] = floatx16_t{};

  const int nstages = (int)((K + kBKB * 16 - 1) / (kBKB * 16));
  OperandRegs ra, rb;
  if (nstages > 0) {
    load_operand<kFast>(ra, a_codes, a_scales, m0, M, K, 0);
    load_operand<kFast>(rb, b_codes, b_scales, n0, N, K, 0);
    store_operand(ra, smem[0].a_codes, smem[0].a_scales);
    store_operand(rb, smem[0].b_codes, smem[0].b_scales);
  }
  __syncthreads();

  for (int s = 0; s < nstages; ++s) {
    const bool more = s + 1 < nstages;
    if (more) {
      load_operand<kFast>(ra, a_codes, a_scales, m0, M, K, s + 1);
      load_operand<kFast>(rb, b_codes, b_scales, n0, N, K, s + 1);
    }
    const Stage& st = smem[s & 1];
#pragma unroll
    for (int c = 0; c < kBKB / 2; ++c) {
      const int blk = 2 * c + lg;
      half8_t af[kFrags][2], bf[kFrags][2];
#pragma unroll
      for (int f = 0; f < kFrags; ++f) {
        const int ra_row = wm * kWaveTile + f * 32 + li;
        const uint2 ac = *reinterpret_cast<const uint2*>(st.a_codes + ra_row * kCodeStride + blk * 8);
        const uint32_t as = st.a_scales[ra_row * kScaleStride + blk];
        af[f][0] = dequant8(ac.x, as);
        af[f][1] = dequant8(ac.y, as);
        const int rb_row = wn * kWaveTile + f * 32 + li;
        const uint2 bc = *reinterpret_cast<const uint2*>(st.b_codes + rb_row * kCodeStride + blk * 8);
        const uint32_t bs = st.b_scales[rb_row * kScaleStride + blk];
        bf[f][0] = dequant8(bc.x, bs);
        bf[f][1] = dequant8(bc.y, bs);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int fn = 0; fn < kFrags; ++fn)
#pragma unroll
          for (int fm = 0; fm < kFrags; ++fm)
            acc[fn][fm] = __builtin_amdgcn_mfma_f32_32x32x16_f16(bf[fn][h], af[fm][h], acc[fn][fm], 0, 0, 0);
    }
    if (more) {
      Stage& nx = smem[(s + 1) & 1];
      store_operand(ra, nx.a_codes, nx.a_scales);
      store_operand(rb, nx.b_codes, nx.b_scales);
    }
    __syncthreads();
  }

  // epilogue: out = bf16(alpha * acc + bias), alpha = aA * aB in FP32
  const float alpha = a_gs[0] * b_gs[0];
#pragma unroll
  for (int fm = 0; fm < kFrags; ++fm) {
    const int64_t m = m0 + wm * kWaveTile + fm * 32 + li;
    if (m >= M) continue;
    uint16_t* orow = out + m * N;
#pragma unroll
    for (int fn = 0; fn < kFrags; ++fn) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t n = n0 + wn * kWaveTile + fn * 32 + 8 * k + 4 * lg;
        float v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = acc[fn][fm][4 * k + q];
        if (kVecOut && n + 3 < N) {
          float bv[4] = {0.f, 0.f, 0.f, 0.f};
          if (bias) {
            const uint2 b2 = *reinterpret_cast<const uint2*>(bias + n);
            bv[0] = __uint_as_float(b2.x << 16);
            bv[1] = __uint_as_float(b2.x & 0xFFFF0000u);
            bv[2] = __uint_as_float(b2.y << 16);
            bv[3] = __uint_as_float(b2.y & 0xFFFF0000u);
          }
          uint32_t o[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = f32_to_bf16_rne(__builtin_fmaf(alpha, v[q], bv[q]));
          *reinterpret_cast<uint2*>(orow + n) = make_uint2(o[0] | (o[1] << 16), o[2] | (o[3] << 16));
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (n + q < N) {
              const float bq = bias ? __uint_as_float((uint32_t)bias[n + q] << 16) : 0.f;
              orow[n + q] = (uint16_t)f32_to_bf16_rne(__builtin_fmaf(alpha, v[q], bq));
            }
          }
        }
      }
    }
  }
}

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                       const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                       const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                       hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  const dim3 grid((unsigned)tiles), block(kGemmThreads);
  const bool fast = K % 128 == 0;
  const bool vec = N % 4 == 0;
  if (fast && vec)
    hipLaunchKernelGGL((nvfp4_gemm_kernel<true, true>), grid, block, 0, stream, a_codes, a_scales,
                       a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K);
  else if (fast)
    hipLaunchKernelGGL((nvfp4_gemm_kernel<true, false>), grid, block, 0, stream, a_codes, a_scales,
                       a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K);
  else if (vec)
    hipLaunchKernelGGL((nvfp4_gemm_kernel<false, true>), grid, block, 0, stream, a_codes, a_scales,
                       a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K);
  else
    hipLaunchKernelGGL((nvfp4_gemm_kernel<false, false>), grid, block, 0, stream, a_codes, a_scales,
                       a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K);
  return hipGetLastError();
}

}  // namespace solfp4
