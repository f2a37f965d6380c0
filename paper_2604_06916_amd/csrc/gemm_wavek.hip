// NVFP4 GEMM for few tokens with the K loop dealt to the waves of a
// workgroup: one 32 x 32 output tile per workgroup of four waves, wave w
// taking stages w, w + 4, w + 8, ... of K (128 elements each).
//
// On few tokens the 64 x 64-tile kernel runs one K loop per wave, bound by
// the issue of its dequantization (two operand fragments converted per
// MFMA), on as many CUs as there are tiles.  Here each wave runs a quarter
// of that loop for a tile a quarter the size, so four times as many CUs
// work and each wave's loop is a quarter as long.  The arithmetic per
// K-step is the lane-dequantizing kernels': exact FP16 dequantization
// (q * s, at most 6 significant bits) and v_mfma_f32_32x32x16_f16 with FP32
// accumulation, in the same K order inside a stage.
//
// Each wave runs its own pipeline: its codes and scale bytes go by DMA into
// four LDS stage buffers of its own, three of its stages ahead, and it
// waits only for its own loads, so the main loop has no barrier.  The
// buffers take 72 KB, so two workgroups share a CU (1.16-1.39x faster than
// one per CU on launches of 280 to 1024 tiles; bit-identical).  At the
// end waves 1-3 park their partial sums in their own stage buffers and wave
// 0 adds them in the order 0 + 1, + 2, + 3 (so the result does not depend
// on timing) before the epilogue: one FP32 fused multiply-add of alpha and
// bias, then rounding to BF16.  The FP32 sums are formed in a different order than in
// the other kernels, so results agree with them to FP32 summation error,
// not bit for bit.  K must be a multiple of 128 (whole stages).
#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "nvfp4_gemm_common.h"
#include "solfp4.h"

namespace solfp4 {

constexpr int kWKTile = 32;                    // output tile edge
constexpr int kWKWaves = kLThreads / kWave;    // waves per workgroup, one K share each
// one stage buffer: A codes (two 16-row groups of 1 KB), B codes, then the
// scale bytes (A, then B: 64 words each, word l holding bytes 4 (l / 32) ..
// +3 of row l % 32's 8 for the stage)
constexpr int kWKCodes = kWKTile * kLRowBytes;       // 2 KB per operand
constexpr int kWKBuf = 2 * kWKCodes + 512;           // 4.5 KB: codes, then 512 B of scales
constexpr int kWKScales = 2 * kWKCodes;
// 72 KB of stage buffers per workgroup, so two workgroups fit one CU's LDS
static_assert(kWKWaves * kLBufs * kWKBuf <= 80 * 1024 - 64, "two workgroups per CU");
static_assert(4 * kWave * (int)sizeof(floatx4_t) <= kLBufs * kWKBuf, "partial sums fit a wave's buffers");

template <bool kVecOut>
__global__ __launch_bounds__(kLThreads, 2) void nvfp4_gemm_wavek_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_gs, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_gs,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K) {
  __shared__ __attribute__((aligned(1024))) uint8_t lbuf[kWKWaves][kLBufs][kWKBuf];
  __shared__ uint16_t lbias[kWKTile];

  const int tiles_m = (int)((M + kWKTile - 1) / kWKTile);
  const int tiles_n = (int)((N + kWKTile - 1) / kWKTile);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kWKTile;
  const int64_t n0 = (int64_t)tn * kWKTile;
  const int nstages = (int)(K / kLBK);

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t scale_row = K / 16;
  const int64_t valid_a = min<int64_t>(M - m0, kWKTile);
  const int64_t valid_b = min<int64_t>(N - n0, kWKTile);
  const __amdgpu_buffer_rsrc_t rca = uniform_rsrc(a_codes + m0 * row_bytes, valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rsa = uniform_rsrc(a_scales + m0 * scale_row, valid_a * scale_row);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * scale_row, valid_b * scale_row);

  // this wave's stages: wave + 4 i for i < count
  const int count = nstages > wave ? (nstages - wave + kWKWaves - 1) / kWKWaves : 0;

  // code DMA: lane quad l/4 reads the 64 bytes of row l/4 of a 16-row group
  // (rows past the operand read zero), lane l's 16 bytes land in slot l of
  // the group's 1 KB, the piece order of row r swizzled by (r >> 2) & 3 so
  // that 16 lanes reading one piece of 16 consecutive rows hit every bank
  // once
  const int dma_r = lane >> 2;
  const int piece = (lane & 3) ^ ((dma_r >> 2) & 3);
  const uint32_t dma_off = (uint32_t)(dma_r * row_bytes + 16 * piece);
  const uint32_t group_stride = (uint32_t)(16 * row_bytes);
  // operand slots of this lane (row li of A and of B): lane group g reads
  // piece g in K-steps 0-3 and piece 2 + g in K-steps 4-7
  const int swz = ((li & 15) >> 2) & 3;
  const int rd = (li >> 4) * 1024 + (li & 15) * 64;
  const int q_off[2] = {16 * (g ^ swz), 16 * ((2 + g) ^ swz)};
  // scale DMA: lane l fetches bytes 4 (l / 32) .. +3 of row l % 32's 8 for
  // the stage (one instruction per operand)
  const uint32_t sc_off = (uint32_t)((lane & 31) * scale_row + 4 * (lane >> 5));

  if (t < kWKTile) lbias[t] = bias && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc = floatx16_t{};

  // the loads of this wave's i-th stage into buffer B (6 instructions)
  auto issue = [&](auto buf, int i) {
    constexpr int B = decltype(buf)::value;
    const int stage = wave + kWKWaves * i;
    uint8_t* base = &lbuf[wave][B][0];
    const uint32_t off = dma_off + (uint32_t)stage * kLRowBytes;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(base), 16, off, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(base + 1024), 16, off + group_stride, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(base + kWKCodes), 16, off, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(base + kWKCodes + 1024), 16,
                                             off + group_stride, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_ptr_t)(base + kWKScales), 4, sc_off + 8 * stage, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)(base + kWKScales + 256), 4,
                                             sc_off + 8 * stage, 0, 0, 1);
  };
  constexpr int kPerStage = 6;   // vector-memory instructions per stage

  // one stage from buffer B: the lane's two code pieces of A and B, its
  // scale words (blocks 2g, 2g+1 for K-steps 0-3 and 4+2g, 5+2g after, as
  // FP16 patterns), then 8 K-steps of dequantization and MFMA
  auto compute = [&](auto buf) {
    constexpr int B = decltype(buf)::value;
    const uint8_t* base = &lbuf[wave][B][0];
    u32x4_t ca[2], cb[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      ca[h] = *reinterpret_cast<const u32x4_t*>(base + rd + q_off[h]);
      cb[h] = *reinterpret_cast<const u32x4_t*>(base + kWKCodes + rd + q_off[h]);
    }
    const uint32_t* sw = reinterpret_cast<const uint32_t*>(base + kWKScales);
    const uint32_t wa[2] = {scale_patterns(sw[li], g != 0), scale_patterns(sw[32 + li], g != 0)};
    const uint32_t wb[2] = {scale_patterns(sw[64 + li], g != 0), scale_patterns(sw[96 + li], g != 0)};
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int h = j >> 2, w = j & 3;
      const half2_t xa = as_h2(wa[h]), xb = as_h2(wb[h]);
      const half2_t s_a = (w & 2) ? __builtin_shufflevector(xa, xa, 1, 1) : __builtin_shufflevector(xa, xa, 0, 0);
      const half2_t s_b = (w & 2) ? __builtin_shufflevector(xb, xb, 1, 1) : __builtin_shufflevector(xb, xb, 0, 0);
      const half8_t oa = dequant_step(ca[h][w], s_a);
      const half8_t ob = dequant_step(cb[h][w], s_b);
      acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ob, oa, acc, 0, 0, 0);
    }
  };

  // stage i (buffer B = i % 4): the loads of stage i+3 go into the buffer
  // read in stage i-1, whose LDS reads the wait at the end of that stage
  // completed; then wait until stage i's loads have landed (only younger
  // stages' loads may stay in flight)
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using B2 = std::integral_constant<int, 2>;
  using B3 = std::integral_constant<int, 3>;
  auto run = [&](auto buf, int i) {
    constexpr int B = decltype(buf)::value;
    if (i + 3 < count) {
      issue(std::integral_constant<int, (B + 3) % kLBufs>{}, i + 3);
      wait_counts<3 * kPerStage, 0>();
    } else if (i + 2 < count) {
      wait_counts<2 * kPerStage, 0>();
    } else if (i + 1 < count) {
      wait_counts<kPerStage, 0>();
    } else {
      wait_counts<0, 0>();
    }
    compute(buf);
    wait_counts<63, 0>();   // this stage's LDS reads done before its buffer is refilled
  };

  // prologue: up to three stages in flight
  if (count > 0) issue(B0{}, 0);
  if (count > 1) issue(B1{}, 1);
  if (count > 2) issue(B2{}, 2);
  int i = 0;
  for (; i + 4 <= count; i += 4) {
    run(B0{}, i);
    run(B1{}, i + 1);
    run(B2{}, i + 2);
    run(B3{}, i + 3);
  }
  if (i < count) run(B0{}, i);
  if (i + 1 < count) run(B1{}, i + 1);
  if (i + 2 < count) run(B2{}, i + 2);
  wait_counts<0, 0>();

  // waves 1-3 park their sums in their own stage buffers (their loads and
  // reads are complete), wave 0 adds them in wave order
  if (wave > 0) {
    floatx4_t* red = reinterpret_cast<floatx4_t*>(&lbuf[wave][0][0]);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      red[q * kWave + lane] = floatx4_t{acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]};
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 1; w < kWKWaves; ++w)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const floatx4_t p = reinterpret_cast<const floatx4_t*>(&lbuf[w][0][0])[q * kWave + lane];
      acc[4 * q] += p[0];
      acc[4 * q + 1] += p[1];
      acc[4 * q + 2] += p[2];
      acc[4 * q + 3] += p[3];
    }

  // epilogue: out = bf16(fp32(fma(alpha, acc, bias))), alpha = aA * aB in
  // FP32.  Lane (li, g) holds row li and the column runs 8k + 4g .. +3
  // (k = 0..3); swapping halves with the lane 32 apart gives each lane two
  // runs of 8 consecutive columns (16-byte stores) through a buffer
  // resource over the tile's valid rows.
  const float alpha = a_gs[0] * b_gs[0];
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
  const uint32_t mrow = (uint32_t)(li * N);
  float v[16];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint2 b2 = *reinterpret_cast<const uint2*>(&lbias[8 * k + 4 * g]);
    const float bv[4] = {__uint_as_float(b2.x << 16), __uint_as_float(b2.x & 0xFFFF0000u),
                         __uint_as_float(b2.y << 16), __uint_as_float(b2.y & 0xFFFF0000u)};
#pragma unroll
    for (int q = 0; q < 4; ++q) v[4 * k + q] = __builtin_fmaf(alpha, acc[4 * k + q], bv[q]);
  }
  uint32_t p[4][2];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    p[k][0] = pack_bf16(v[4 * k], v[4 * k + 1]);
    p[k][1] = pack_bf16(v[4 * k + 2], v[4 * k + 3]);
  }
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    uint32_t r[4];   // 8 columns starting at 16 h + 8 g
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const auto x = __builtin_amdgcn_permlane32_swap(p[2 * h][d], p[2 * h + 1][d], false, false);
      r[d] = x[0];
      r[2 + d] = x[1];
    }
    const int64_t n = n0 + 16 * h + 8 * g;
    if (kVecOut) {
      const uint32_t off = n < N ? (mrow + (uint32_t)n) * 2 : kDrop;
      __builtin_amdgcn_raw_buffer_store_b128(u32x4_t{r[0], r[1], r[2], r[3]}, ro, off, 0, 0);
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const uint32_t off = n + q < N ? (mrow + (uint32_t)(n + q)) * 2 : kDrop;
        __builtin_amdgcn_raw_buffer_store_b16((uint16_t)(r[q / 2] >> (16 * (q & 1))), ro, off, 0, 0);
      }
    }
  }
}

hipError_t launch_gemm_wavek(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                             const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                             hipStream_t stream) {
  const int64_t tiles = ((M + kWKTile - 1) / kWKTile) * ((N + kWKTile - 1) / kWKTile);
  const dim3 grid((unsigned)tiles), block(kLThreads);
  return N % 8 == 0
             ? launch_kernel(nvfp4_gemm_wavek_kernel<true>, grid, block, stream, a_codes, a_scales,
                             a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K)
             : launch_kernel(nvfp4_gemm_wavek_kernel<false>, grid, block, stream, a_codes, a_scales,
                             a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K);
}

}  // namespace solfp4
