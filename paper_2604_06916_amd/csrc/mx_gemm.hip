// MXFP4 GEMM with BF16 output on the CDNA4 scaled FP4 matrix instructions.
//
//   out[m][n] = bf16( fp32( sum_k (X qA)[m][k] (X qB)[n][k] + bias[n] ) )
//
// A [M, K] and B [N, K] are MXFP4 (the OCP MX format named in the paper's
// Preliminaries): E2M1 codes, two per byte with the even element in the low
// nibble, and one E8M0 scale byte X = 2^(byte - 127) per 32 elements along
// K.  That is exactly what v_mfma_scale_f32_32x32x64_f8f6f4 consumes: each
// lane supplies 32 codes of one row (16 bytes) plus that row's scale byte for
// those 32 elements, so the packed codes travel from HBM to the matrix cores
// unconverted and the products run at the FP4 rate.
//
// Tiling: a 256 x 256 output tile per workgroup of 4 waves (one per SIMD),
// each wave owning 128 x 128 (4 x 4 MFMA tiles of 32 x 32, 256 FP32
// accumulators per lane in AGPRs).  K advances 128 elements (64 code bytes
// per row) per stage.  Codes move global -> registers -> LDS -> registers,
// through three LDS stage buffers whose rows are padded to 80 bytes (16-byte
// row reads and writes of 16 consecutive rows are bank-conflict free).  Scale
// bytes go straight from global memory to the lanes that use them: a lane
// needs the scales of its own 8 rows only.
//
// Pipeline of stage s: the MFMAs read LDS buffer s%3; the codes of stage s+2,
// fetched during stage s-1, are stored to buffer (s+2)%3; the codes of stage
// s+3 and the scales of stage s+1 are fetched; the operands of the first
// K-step of stage s+1 are read from LDS during the last K-step of stage s
// (that buffer was completed before the previous barrier), so the one barrier
// per stage does not expose LDS latency.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kMxTile = 256;                   // output tile edge (M and N)
constexpr int kMxBK = 128;                     // K elements per stage
constexpr int kMxRowBytes = kMxBK / 2;         // code bytes per row per stage
constexpr int kMxLdsRow = kMxRowBytes + 16;    // padded LDS row
constexpr int kMxThreads = 256;
constexpr int kMxWaveTile = 128;
constexpr int kMxFrags = kMxWaveTile / 32;     // 32 x 32 MFMA tiles per wave edge
constexpr int kMxSteps = kMxBK / 64;           // MFMA K-steps per stage
constexpr int kMxBufs = 3;
constexpr int kMxRounds = kMxTile * kMxRowBytes / 16 / kMxThreads;   // 16-byte loads per operand

struct MxSmem {
  uint8_t a[kMxBufs][kMxTile * kMxLdsRow];
  uint8_t b[kMxBufs][kMxTile * kMxLdsRow];
};

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v8i_t __attribute__((ext_vector_type(8)));

// An FP4 matrix operand occupies the low 4 registers of the 8-register
// operand; the rest are ignored for this format and left undefined.
__device__ __forceinline__ v8i_t fp4_operand(u32x4_t x) {
  const v4i_t y = __builtin_bit_cast(v4i_t, x);
  return __builtin_shufflevector(y, y, 0, 1, 2, 3, -1, -1, -1, -1);
}

// Scale bytes of kgroups 4*stage .. 4*stage+3 of one row, as one word.
// kFast: K % 128 == 0 (4-byte aligned, no stage reaches past K).  Otherwise
// byte loads, with kgroups past K zeroed (a stray 0xFF byte would be NaN).
template <bool kFast>
__device__ __forceinline__ uint32_t load_scale_word(__amdgpu_buffer_rsrc_t src, uint32_t off,
                                                    int64_t kgroups, int stage) {
  if (kFast) return __builtin_amdgcn_raw_buffer_load_b32(src, off, 0, 0);
  uint32_t w = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t b = __builtin_amdgcn_raw_buffer_load_b8(src, off + i, 0, 0);
    w |= ((int64_t)stage * 4 + i < kgroups ? b : 0u) << (8 * i);
  }
  return w;
}

template <bool kFast, bool kVecOut>
__global__ __launch_bounds__(kMxThreads, 1) void mxfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const uint8_t* __restrict__ b_codes, const uint8_t* __restrict__ b_scales,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K) {
  __shared__ MxSmem smem;

  const int tiles_m = (int)((M + kMxTile - 1) / kMxTile);
  const int tiles_n = (int)((N + kMxTile - 1) / kMxTile);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kMxTile;
  const int64_t n0 = (int64_t)tn * kMxTile;

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int wm = wave >> 1;
  const int wn = wave & 1;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t kgroups = K / 32;
  const int64_t valid_a = min<int64_t>(M - m0, kMxTile);
  const int64_t valid_b = min<int64_t>(N - n0, kMxTile);
  const __amdgpu_buffer_rsrc_t rca = uniform_rsrc(a_codes + m0 * row_bytes, valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rsa = uniform_rsrc(a_scales + m0 * kgroups, valid_a * kgroups);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * kgroups, valid_b * kgroups);

  // code staging: in round j this thread moves 16 bytes (piece `piece`) of
  // tile row 64 j + srow; a wave covers 16 whole rows per round
  const int srow = 16 * wave + (lane & 15);
  const int piece = lane >> 4;
  const uint32_t code_off = (uint32_t)(srow * row_bytes + 16 * piece);
  const uint32_t round_stride = (uint32_t)(64 * row_bytes);
  const int st_off = (srow * kMxLdsRow) + 16 * piece;
  // MFMA operand rows of this lane
  uint32_t sa_off[kMxFrags], sb_off[kMxFrags];
#pragma unroll
  for (int f = 0; f < kMxFrags; ++f) {
    sa_off[f] = (uint32_t)((wm * kMxWaveTile + f * 32 + li) * kgroups);
    sb_off[f] = (uint32_t)((wn * kMxWaveTile + f * 32 + li) * kgroups);
  }
  const int rd_a = (wm * kMxWaveTile + li) * kMxLdsRow + 16 * g;
  const int rd_b = (wn * kMxWaveTile + li) * kMxLdsRow + 16 * g;

  floatx16_t acc[kMxFrags][kMxFrags];
#pragma unroll
  for (int i = 0; i < kMxFrags; ++i)
#pragma unroll
    for (int j = 0; j < kMxFrags; ++j) acc[i][j] = floatx16_t{};

  u32x4_t stg[2][2][kMxRounds];          // [set][operand][round]
  uint32_t sca[2][kMxFrags], scb[2][kMxFrags];
  u32x4_t fa[2][kMxFrags], fb[2][kMxFrags];

  auto load_codes = [&](u32x4_t (&dst)[2][kMxRounds], int stage) {
    const bool ok = kFast || (int64_t)stage * kMxBK + 32 * piece < K;
#pragma unroll
    for (int j = 0; j < kMxRounds; ++j) {
      const uint32_t off = code_off + j * round_stride + (uint32_t)stage * kMxRowBytes;
      const u32x4_t va = __builtin_amdgcn_raw_buffer_load_b128(rca, off, 0, 0);
      const u32x4_t vb = __builtin_amdgcn_raw_buffer_load_b128(rcb, off, 0, 0);
      dst[0][j] = ok ? va : u32x4_t{0, 0, 0, 0};
      dst[1][j] = ok ? vb : u32x4_t{0, 0, 0, 0};
    }
  };
  auto store_codes = [&](const u32x4_t (&src)[2][kMxRounds], int buf) {
#pragma unroll
    for (int j = 0; j < kMxRounds; ++j) {
      *reinterpret_cast<u32x4_t*>(&smem.a[buf][st_off + 64 * j * kMxLdsRow]) = src[0][j];
      *reinterpret_cast<u32x4_t*>(&smem.b[buf][st_off + 64 * j * kMxLdsRow]) = src[1][j];
    }
  };
  auto load_scales = [&](uint32_t (&da)[kMxFrags], uint32_t (&db)[kMxFrags], int stage) {
#pragma unroll
    for (int f = 0; f < kMxFrags; ++f) {
      da[f] = load_scale_word<kFast>(rsa, sa_off[f] + 4 * stage, kgroups, stage);
      db[f] = load_scale_word<kFast>(rsb, sb_off[f] + 4 * stage, kgroups, stage);
    }
  };
  auto read_frags = [&](u32x4_t (&da)[kMxFrags], u32x4_t (&db)[kMxFrags], int buf, int st) {
#pragma unroll
    for (int f = 0; f < kMxFrags; ++f) {
      da[f] = *reinterpret_cast<const u32x4_t*>(&smem.a[buf][rd_a + f * 32 * kMxLdsRow + 32 * st]);
      db[f] = *reinterpret_cast<const u32x4_t*>(&smem.b[buf][rd_b + f * 32 * kMxLdsRow + 32 * st]);
    }
  };
  // one K-step: lane group g supplies kgroup 2 st + g of the stage, i.e.
  // byte 2 st + g of its scale words; after the shift by 8 g the byte
  // select is the constant 2 st for every lane
  auto mfma_step = [&](auto step, const u32x4_t (&xa)[kMxFrags], const u32x4_t (&xb)[kMxFrags],
                       const uint32_t (&ssa)[kMxFrags], const uint32_t (&ssb)[kMxFrags]) {
    constexpr int st = decltype(step)::value;
#pragma unroll
    for (int fn = 0; fn < kMxFrags; ++fn)
#pragma unroll
      for (int fm = 0; fm < kMxFrags; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            fp4_operand(xb[fn]), fp4_operand(xa[fm]), acc[fn][fm], 4, 4, 2 * st,
            (int)ssb[fn], 2 * st, (int)ssa[fm]);
  };

  const int nstages = (int)((K + kMxBK - 1) / kMxBK);
  // prologue: stages 0 and 1 into LDS buffers 0 and 1, stage 2 in flight,
  // scales of stage 0, operands of the first K-step
  load_codes(stg[0], 0);
  load_codes(stg[1], 1);
  load_scales(sca[0], scb[0], 0);
  store_codes(stg[0], 0);
  store_codes(stg[1], 1);
  load_codes(stg[0], 2);
  __syncthreads();
  read_frags(fa[0], fb[0], 0, 0);

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  auto run_stage = [&](auto phase, int s, int cur, int nxt, int wbuf) {
    constexpr int P = decltype(phase)::value;
    uint32_t ssa[kMxFrags], ssb[kMxFrags];
#pragma unroll
    for (int f = 0; f < kMxFrags; ++f) {
      ssa[f] = sca[P][f] >> (8 * g);
      ssb[f] = scb[P][f] >> (8 * g);
    }
    read_frags(fa[1], fb[1], cur, 1);
    load_codes(stg[P ^ 1], s + 3);
    load_scales(sca[P ^ 1], scb[P ^ 1], s + 1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(S0{}, fa[0], fb[0], ssa, ssb);
    store_codes(stg[P], wbuf);
    __builtin_amdgcn_sched_barrier(0);
    read_frags(fa[0], fb[0], nxt, 0);
    mfma_step(S1{}, fa[1], fb[1], ssa, ssb);
    __syncthreads();
  };

  int s = 0, cur = 0;
  for (; s + 2 <= nstages; s += 2) {
    const int c1 = cur == 2 ? 0 : cur + 1;
    const int c2 = c1 == 2 ? 0 : c1 + 1;
    run_stage(S0{}, s, cur, c1, c2);
    run_stage(S1{}, s + 1, c1, c2, cur);
    cur = c2;
  }
  if (s < nstages) {
    const int c1 = cur == 2 ? 0 : cur + 1;
    const int c2 = c1 == 2 ? 0 : c1 + 1;
    run_stage(S0{}, s, cur, c1, c2);
  }

  // epilogue: out = bf16(fp32(acc + bias))
#pragma unroll
  for (int fm = 0; fm < kMxFrags; ++fm) {
    const int64_t m = m0 + wm * kMxWaveTile + fm * 32 + li;
    if (m >= M) continue;
    uint16_t* orow = out + m * N;
#pragma unroll
    for (int fn = 0; fn < kMxFrags; ++fn) {
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int64_t n = n0 + wn * kMxWaveTile + fn * 32 + 8 * k + 4 * g;
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
          for (int q = 0; q < 4; ++q) o[q] = f32_to_bf16_rne(v[q] + bv[q]);
          *reinterpret_cast<uint2*>(orow + n) = make_uint2(o[0] | (o[1] << 16), o[2] | (o[3] << 16));
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            if (n + q < N) {
              const float bq = bias ? __uint_as_float((uint32_t)bias[n + q] << 16) : 0.f;
              orow[n + q] = (uint16_t)f32_to_bf16_rne(v[q] + bq);
            }
          }
        }
      }
    }
  }
}

hipError_t launch_mx_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
                          const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M,
                          int64_t N, int64_t K, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ((M + kMxTile - 1) / kMxTile) * ((N + kMxTile - 1) / kMxTile);
  const dim3 grid((unsigned)tiles), block(kMxThreads);
  const bool fast = K % kMxBK == 0;
  const bool vec = N % 4 == 0;
  if (fast && vec)
    hipLaunchKernelGGL((mxfp4_gemm_kernel<true, true>), grid, block, 0, stream, a_codes, a_scales,
                       b_codes, b_scales, bias, out, M, N, K);
  else if (fast)
    hipLaunchKernelGGL((mxfp4_gemm_kernel<true, false>), grid, block, 0, stream, a_codes, a_scales,
                       b_codes, b_scales, bias, out, M, N, K);
  else if (vec)
    hipLaunchKernelGGL((mxfp4_gemm_kernel<false, true>), grid, block, 0, stream, a_codes, a_scales,
                       b_codes, b_scales, bias, out, M, N, K);
  else
    hipLaunchKernelGGL((mxfp4_gemm_kernel<false, false>), grid, block, 0, stream, a_codes,
                       a_scales, b_codes, b_scales, bias, out, M, N, K);
  return hipGetLastError();
}

}  // namespace solfp4
