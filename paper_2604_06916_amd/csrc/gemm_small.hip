// NVFP4 GEMM for few tokens: 64 x 64 output tiles, and the linear layer with
// the activations quantized inside the GEMM (the "quantize fused into the
// GEMM prologue" step of the NVFP4 linear of Sec. 4.1).
//
// A GEMM with few rows (a 128-token layer, say) has too few 128 x 128 tiles
// to occupy the chip, and each of them runs its K loop on one compute unit:
// the launch is bound by the latency of that loop, not by arithmetic.  This
// kernel takes 64 x 64 tiles (four times as many workgroups, a quarter of
// the matrix work each), four waves of 32 x 32, with the arithmetic of the
// lane-dequantizing kernel: codes move into four LDS stage buffers by DMA
// three stages ahead, each wave dequantizes its own operands exactly to FP16
// (q * s has at most 6 significant bits) and multiplies them on the FP16
// matrix cores (v_mfma_f32_32x32x16_f16, FP32 accumulation), and the epilogue
// is one FP32 fused multiply-add of alpha and bias followed by rounding to
// BF16.  K must be a multiple of 128 (whole stages).
//
// kFuse: the activations arrive as BF16 X, not as codes, and the tiles are
// 32 x 128 (four waves side by side, so that a workgroup quantizes 32 rows;
// each wave computes a 32 x 32 block either way, so the results do not
// depend on the tile shape).  Every workgroup folds the amax pass's partial
// maxima into alpha = amax / 2688 and tabulates r(s) = 1 / (s * alpha), as
// the quantizer's encode pass does, and then quantizes its own rows of X
// stage by stage into the A stage
// buffers: the block amax, the E4M3 scale, r from the table, E2M1 codes
// from the hardware converter; the same operations in the
// same order as nvfp4_quantize, so codes, scales and alpha are bit-identical
// to it.  The tiles of column 0 also store their codes and scales (and
// workgroup 0 alpha) to memory, where nvfp4_linear documents them.  With
// the same tiles, K order and epilogue, the fused linear's output is
// bit-identical to nvfp4_quantize followed by the unfused kernel.  A row
// panel is quantized once per column tile it meets (N / 128 times), and the
// kernel is bound by VALU issue (the dequantization alone outweighs the
// matrix work on these tiles), so the quantization costs about as much as
// the encode pass it replaces: the fusion pays only where the saved launch
// dominates, for short K (the host fuses only up to K = 512).
//
// Per stage s (P = s % 4 selects the buffer, C = s % 2 the scale set), as
// in the lane kernel: the scale patterns of stage s+2 are parked in LDS set
// C, the scale bytes of stage s+3 fetched, the DMA of stage s+3 issued (one
// 16-row group per wave and operand), the codes of this stage read and
// converted K-step by K-step.  With kFuse the A side instead quantizes stage
// s+2 from registers (its BF16 loaded two stages earlier, into register set
// (s + 2) % 4), one 16-element block per thread between K-steps 0 and 1 and
// another between K-steps 2 and 3, into buffer (P + 2) % 4 and set C, and
// after the DMA loads the BF16 of stage s+4.  The wait that ends a stage
// leaves only the stage's own DMA and BF16 loads in flight.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"
#include "nvfp4_gemm_common.h"
#include "solfp4.h"

namespace solfp4 {

template <bool kFuse, bool kVecOut>
__global__ __launch_bounds__(kLThreads, 1) void nvfp4_gemm_small_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_gs, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_gs,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K, SmallFuse fuse) {
  // tile: 64 x 64 (2 x 2 waves), or with kFuse 32 x 128 (1 x 4 waves), so
  // that a workgroup quantizes 32 rows of X, not 64; each wave computes a
  // 32 x 32 block of the output either way
  constexpr int kTM = kFuse ? 32 : 64;
  constexpr int kTN = 4096 / kTM;
  constexpr int kWN = kTN / 32;                // waves along N
  constexpr int kGA = kFuse ? 0 : kTM / 64;    // A DMA groups (16 rows) per wave and stage
  constexpr int kGB = kTN / 64;                // B DMA groups per wave and stage
  constexpr int kDma = kGA + kGB;              // DMA instructions per wave and stage
  constexpr int kXLoads = kFuse ? 2 : 0;       // BF16 loads per thread and stage
  constexpr int kInFlight = kDma + kXLoads;    // may stay in flight past a stage's end
  __shared__ __attribute__((aligned(1024))) uint8_t la0[kTM * kLRowBytes], la1[kTM * kLRowBytes],
      la2[kTM * kLRowBytes], la3[kTM * kLRowBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t lb0[kTN * kLRowBytes], lb1[kTN * kLRowBytes],
      lb2[kTN * kLRowBytes], lb3[kTN * kLRowBytes];
  __shared__ uint32_t lsc[2][2][kTN * kLScaleStride];   // [stage parity][operand][row, word]
  __shared__ uint16_t lbias[kTN];
  __shared__ float rtab[128];
  __shared__ uint32_t red[kLThreads / kWave];
  uint8_t* const abuf[kLBufs] = {la0, la1, la2, la3};
  uint8_t* const bbuf[kLBufs] = {lb0, lb1, lb2, lb3};

  const int tiles_m = (int)((M + kTM - 1) / kTM);
  const int tiles_n = (int)((N + kTN - 1) / kTN);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kTM;
  const int64_t n0 = (int64_t)tn * kTN;
  const int nstages = (int)(K / kLBK);

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int wm = wave / kWN;
  const int wn = wave % kWN;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t scale_row = K / 16;
  const int64_t valid_a = min<int64_t>(M - m0, kTM);
  const int64_t valid_b = min<int64_t>(N - n0, kTN);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * scale_row, valid_b * scale_row);
  // A as codes and scales, or (kFuse) as BF16; the other pair is unused
  const __amdgpu_buffer_rsrc_t rca =
      uniform_rsrc(kFuse ? nullptr : a_codes + m0 * row_bytes, kFuse ? 0 : valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rsa =
      uniform_rsrc(kFuse ? nullptr : a_scales + m0 * scale_row, kFuse ? 0 : valid_a * scale_row);
  const __amdgpu_buffer_rsrc_t rx =
      uniform_rsrc(kFuse ? fuse.x + m0 * K : nullptr, kFuse ? valid_a * K * 2 : 0);

  float alpha_a = 0.0f, tq = 0.0f;   // fused: the activations' alpha and 6 alpha
  bool zero_tensor = false;

  // code DMA: wave w fills 16-row groups w, w + 4, ... of each operand;
  // lane quad l/4 reads the 64 bytes of row l/4 of the group, lane l's 16
  // bytes land in slot l of the group's 1 KB, the piece order of row r
  // swizzled by (r >> 2) & 3
  const int dma_r = lane >> 2;
  const int piece = (lane & 3) ^ ((dma_r >> 2) & 3);
  const uint32_t dma_off = (uint32_t)((16 * wave + dma_r) * row_bytes + 16 * piece);
  const uint32_t group4_stride = (uint32_t)(64 * row_bytes);   // four groups further on
  // scale staging: thread t moves the 8 scale bytes of tile row t (A: t <
  // kTM, B: t < kTN)
  const bool row_a = t < kTM;
  const bool row_b = t < kTN;
  const uint32_t sg_off = (uint32_t)(t * scale_row);
  // operand slots of this lane (row wm*32 + li of A, wn*32 + li of B): lane
  // group g reads piece g in K-steps 0-3 and piece 2 + g in K-steps 4-7
  const int swz = ((li & 15) >> 2) & 3;
  const int rd_a = ((wm * 32 + li) >> 4) * 1024 + (li & 15) * 64;
  const int rd_b = ((wn * 32 + li) >> 4) * 1024 + (li & 15) * 64;
  const int q_off[2] = {16 * (g ^ swz), 16 * ((2 + g) ^ swz)};
  const int rs_a = (wm * 32 + li) * kLScaleStride + g;
  const int rs_b = (wn * 32 + li) * kLScaleStride + g;

  // fused quantizer's share of a stage: 32 rows x 8 blocks of 16 elements,
  // thread t owns block qb = t % 8 of row t / 8 (8 lanes read a row's 256
  // bytes)
  const int qb = t & 7;
  const int qrow = t >> 3;
  const bool write_out = kFuse && tn == 0;

  const uint16_t bias_v = bias && row_b && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc = floatx16_t{};
  uint32_t sca[2][2], scb[2][2];   // [stage parity][half stage]
  u32x4_t ca[2], cb[2];            // code pieces, [half stage]
  half8_t oa[2], ob[2];            // FP16 operands, [K-step parity]
  u32x4_t xr[4][2];                // fused: BF16 of stage k in set k % 4

  auto dma = [&](int buf, int stage) {
    const uint32_t off = dma_off + (uint32_t)stage * kLRowBytes;
#pragma unroll
    for (int j = 0; j < kGA; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(abuf[buf] + (wave + 4 * j) * 1024),
                                               16, off + j * group4_stride, 0, 0, 1);
#pragma unroll
    for (int j = 0; j < kGB; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(bbuf[buf] + (wave + 4 * j) * 1024),
                                               16, off + j * group4_stride, 0, 0, 1);
  };
  struct ScaleFetch {
    u32x2_t a, b;
  };
  auto fetch_scales = [&](ScaleFetch& f, int stage) {
    const uint32_t off = sg_off + 8 * stage;
    if constexpr (!kFuse) f.a = __builtin_amdgcn_raw_buffer_load_b64(rsa, off, 0, 0);
    f.b = __builtin_amdgcn_raw_buffer_load_b64(rsb, off, 0, 0);
  };
  auto store_scales = [&](const ScaleFetch& f, int set) {
    if constexpr (!kFuse) {
      if (row_a) {
        uint32_t* da = &lsc[set][0][t * kLScaleStride];
        da[0] = scale_patterns(f.a.x, false);
        da[1] = scale_patterns(f.a.x, true);
        da[2] = scale_patterns(f.a.y, false);
        da[3] = scale_patterns(f.a.y, true);
      }
    }
    if (row_b) {
      uint32_t* db = &lsc[set][1][t * kLScaleStride];
      db[0] = scale_patterns(f.b.x, false);
      db[1] = scale_patterns(f.b.x, true);
      db[2] = scale_patterns(f.b.y, false);
      db[3] = scale_patterns(f.b.y, true);
    }
  };
  // fused: the BF16 of `stage` for this thread's block (two 16-byte loads)
  auto load_x = [&](u32x4_t (&v)[2], int stage) {
    const uint32_t off = (uint32_t)(((int64_t)qrow * K + (int64_t)stage * kLBK + 16 * qb) * 2);
    v[0] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0);
    v[1] = __builtin_amdgcn_raw_buffer_load_b128(rx, off + 16, 0, 0);
  };
  // fused: quantize this thread's block (its BF16 in v) into A buffer `buf`
  // and scale set `set`: the block amax, its E4M3 scale, r from the table,
  // then 16 codes from the hardware converter
  auto quantize_block = [&](const u32x4_t (&v)[2], int buf, int set) {
    const int row = qrow;
    const uint32_t w[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    ushort2_t m = as_us2(w[0] & 0x7FFF7FFFu);
#pragma unroll
    for (int j = 1; j < 8; ++j) m = absmax_pair(m, w[j]);
    const uint32_t ab = max((uint32_t)m.x, (uint32_t)m.y);
    const float amax_b = __uint_as_float(ab << 16);
    const float qv = amax_b / tq;
    const uint32_t sc = e4m3_rne_sat(zero_tensor ? 0.0f : qv);
    const float r = rtab[sc];
    uint32_t c[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      uint32_t x = 0;
      x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(x, __uint_as_float(w[4 * h] << 16) * r,
                                                   __uint_as_float(w[4 * h] & 0xFFFF0000u) * r, 1.0f, 0);
      x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(x, __uint_as_float(w[4 * h + 1] << 16) * r,
                                                   __uint_as_float(w[4 * h + 1] & 0xFFFF0000u) * r, 1.0f, 1);
      x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(x, __uint_as_float(w[4 * h + 2] << 16) * r,
                                                   __uint_as_float(w[4 * h + 2] & 0xFFFF0000u) * r, 1.0f, 2);
      x = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(x, __uint_as_float(w[4 * h + 3] << 16) * r,
                                                   __uint_as_float(w[4 * h + 3] & 0xFFFF0000u) * r, 1.0f, 3);
      c[h] = x;
    }
    // row `row` of the tile: the block is half qb % 2 of logical piece
    // qb / 2, stored at that piece's swizzled position
    const int r16 = row & 15;
    *reinterpret_cast<u32x2_t*>(abuf[buf] + (row >> 4) * 1024 + r16 * 64 +
                                16 * ((qb >> 1) ^ ((r16 >> 2) & 3)) + 8 * (qb & 1)) = u32x2_t{c[0], c[1]};
    reinterpret_cast<uint16_t*>(&lsc[set][0][row * kLScaleStride + (qb >> 1)])[qb & 1] =
        (uint16_t)(sc << 7);
  };
  // fused, tiles of column 0: `stage`'s codes (buffer `buf`, un-swizzled)
  // and scales (set `set`, patterns back to bytes) to memory, one 16-byte
  // piece per thread and the 8 scale bytes of a row per thread of the first
  // kTM; rows past M fall outside the buffer ranges and are dropped
  const __amdgpu_buffer_rsrc_t rco =
      uniform_rsrc(write_out ? fuse.codes_out + m0 * row_bytes : nullptr, write_out ? valid_a * row_bytes : 0);
  const __amdgpu_buffer_rsrc_t rso =
      uniform_rsrc(write_out ? fuse.scales_out + m0 * scale_row : nullptr, write_out ? valid_a * scale_row : 0);
  auto copy_out = [&](int buf, int set, int stage) {
    const int row = t >> 2, pc = t & 3, r16 = row & 15;
    if (row < kTM) {
      const u32x4_t c = *reinterpret_cast<const u32x4_t*>(abuf[buf] + (row >> 4) * 1024 + r16 * 64 +
                                                           16 * (pc ^ ((r16 >> 2) & 3)));
      __builtin_amdgcn_raw_buffer_store_b128(
          c, rco, (uint32_t)(row * row_bytes + (int64_t)stage * kLRowBytes + 16 * pc), 0, 0);
    }
    if (row_a) {
      const uint32_t* pw = &lsc[set][0][t * kLScaleStride];
      uint32_t b[2];
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const uint32_t w0 = pw[2 * k], w1 = pw[2 * k + 1];
        b[k] = ((w0 >> 7) & 0xFFu) | (((w0 >> 23) & 0xFFu) << 8) | (((w1 >> 7) & 0xFFu) << 16) |
               (((w1 >> 23) & 0xFFu) << 24);
      }
      __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{b[0], b[1]}, rso,
                                            (uint32_t)(t * scale_row + (int64_t)stage * 8), 0, 0);
    }
  };
  auto read_scales = [&](uint32_t (&da)[2], uint32_t (&db)[2], int stage) {
    const int set = stage & 1;
    da[0] = lsc[set][0][rs_a];
    da[1] = lsc[set][0][rs_a + 2];
    db[0] = lsc[set][1][rs_b];
    db[1] = lsc[set][1][rs_b + 2];
  };
  auto read_codes = [&](int half, int buf) {
    ca[half] = *reinterpret_cast<const u32x4_t*>(abuf[buf] + rd_a + q_off[half]);
    cb[half] = *reinterpret_cast<const u32x4_t*>(bbuf[buf] + rd_b + q_off[half]);
  };
  // operands of K-step j: lane group g takes elements 32 p + 8 (j % 4) ..
  // +7 of the stage, p = g for j < 4 and 2 + g after (both operands alike)
  auto convert = [&](auto step, const uint32_t (&ssa)[2], const uint32_t (&ssb)[2], int d) {
    constexpr int j = decltype(step)::value;
    constexpr int h = j >> 2, w = j & 3;
    const half2_t xa = as_h2(ssa[h]), xb = as_h2(ssb[h]);
    const half2_t sa = (w & 2) ? __builtin_shufflevector(xa, xa, 1, 1) : __builtin_shufflevector(xa, xa, 0, 0);
    const half2_t sb = (w & 2) ? __builtin_shufflevector(xb, xb, 1, 1) : __builtin_shufflevector(xb, xb, 0, 0);
    oa[d] = dequant_step(ca[h][w], sa);
    ob[d] = dequant_step(cb[h][w], sb);
  };
  auto mfma_step = [&](int d) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ob[d], oa[d], acc, 0, 0, 0);
  };

  using J0 = std::integral_constant<int, 0>;
  using J1 = std::integral_constant<int, 1>;
  using J2 = std::integral_constant<int, 2>;
  using J3 = std::integral_constant<int, 3>;
  using J4 = std::integral_constant<int, 4>;
  using J5 = std::integral_constant<int, 5>;
  using J6 = std::integral_constant<int, 6>;
  using J7 = std::integral_constant<int, 7>;

  // prologue: stages 0-2 of B (and A's codes, or A quantized from X for
  // stages 0 and 1 with stage 2's BF16 kept in registers); the scales of
  // stages 0 and 1 parked in LDS; then the first half stage's codes and
  // stage 0's scales read and K-step 0 converted
  // alpha of the activations: folded from the amax pass's partial maxima
  // (every workgroup does it; a few KB from L2) exactly as the quantizer's
  // encode pass does, while the prologue's loads are in flight; or read
  // from the quantizer's output in the epilogue
  // (the partial maxima, at most 1024 of them, are loaded first of all)
  uint32_t pm[kMaxPartials / kLThreads];
  auto load_partials = [&]() {
#pragma unroll
    for (int k = 0; k < kMaxPartials / kLThreads; ++k) {
      const int i = t + k * kLThreads;
      pm[k] = i < fuse.npartial ? fuse.partial[i] : 0u;
    }
  };
  auto fold_alpha = [&]() {
    uint32_t mx = pm[0];
#pragma unroll
    for (int k = 1; k < kMaxPartials / kLThreads; ++k) mx = max(mx, pm[k]);
    mx = wave_max_u32(mx);
    if (lane == 0) red[wave] = mx;
    // an LDS-only barrier: the DMA and BF16 loads stay in flight
    wait_counts<63, 0>();
    __builtin_amdgcn_s_barrier();
    uint32_t amax_bits = red[0];
#pragma unroll
    for (int w = 1; w < kLThreads / kWave; ++w) amax_bits = max(amax_bits, red[w]);
    const float amax_g = __uint_as_float(amax_bits << 16);
    alpha_a = amax_g / kAlphaDivisor;
    tq = alpha_a * 6.0f;
    zero_tensor = amax_bits == 0u;
    if (blockIdx.x == 0 && t == 0) *fuse.alpha_out = alpha_a;
    if (t < 128) {
      const uint32_t c = t;
      const float d = e4m3_value(c) * alpha_a;
      rtab[c] = (c == 0u || c == 0x7Fu) ? 0.0f : 1.0f / d;
    }
  };

  ScaleFetch sf, sf0, sf1;
  if constexpr (kFuse) load_partials();
  fetch_scales(sf0, 0);
  fetch_scales(sf1, 1);
  fetch_scales(sf, 2);
  if constexpr (kFuse) {
    load_x(xr[0], 0);
    load_x(xr[1], 1);
  }
  dma(0, 0);
  dma(1, 1);
  dma(2, 2);
  if (row_b) lbias[t] = bias_v;
  if constexpr (kFuse) {
    // the BF16 of stages 2 and 3 stays in flight into the main loop
    load_x(xr[2], 2);
    load_x(xr[3], 3);
    fold_alpha();
    // rtab complete (LDS-only barrier); the compiler waits for the BF16 of
    // stages 0 and 1
    wait_counts<63, 0>();
    __builtin_amdgcn_s_barrier();
    quantize_block(xr[0], 0, 0);
    quantize_block(xr[1], 1, 1);
  }
  store_scales(sf0, 0);
  store_scales(sf1, 1);
  wait_counts<kFuse ? 0 : kDma, 0>();
  __builtin_amdgcn_s_barrier();
  if (kFuse && write_out) copy_out(0, 0, 0);
  read_scales(sca[0], scb[0], 0);
  read_codes(0, 0);
  wait_counts<63, 0>();
  __builtin_amdgcn_s_barrier();
  convert(J0{}, sca[0], scb[0], 0);

  auto run_stage = [&](auto phase, int s) {
    constexpr int P = decltype(phase)::value;
    constexpr int C = P & 1;
    // fused: stage s+2 (its BF16 loaded during stage s-2, in register set
    // (s + 2) % 4) is quantized a block at a time between the K-steps, into
    // buffer (P + 2) % 4 (its last reader was stage s-2) and scale set C
    // (last read for stage s, during stage s-1)
    constexpr int XQ = (P + 2) % 4;
    __builtin_amdgcn_sched_barrier(0);
    store_scales(sf, C);
    // fused, tiles of column 0: stage s+1 (complete since the last barrier)
    // out to memory, before the DMA so that the stage-end wait covers it
    if constexpr (kFuse)
      if (write_out && s + 1 < nstages) copy_out((P + 1) % kLBufs, C ^ 1, s + 1);
    fetch_scales(sf, s + 3);
    dma((P + 3) % kLBufs, s + 3);
    // the BF16 of stage s+4 goes out after the DMA: with it, the youngest
    // kInFlight operations may stay in flight past the stage's end
    if constexpr (kFuse) load_x(xr[P], s + 4);
    read_codes(1, P);
    mfma_step(0);
    if constexpr (kFuse) quantize_block(xr[XQ], (P + 2) % kLBufs, C);
    convert(J1{}, sca[C], scb[C], 1);
    mfma_step(1);
    convert(J2{}, sca[C], scb[C], 0);
    mfma_step(0);
    convert(J3{}, sca[C], scb[C], 1);
    mfma_step(1);
    convert(J4{}, sca[C], scb[C], 0);
    read_codes(0, (P + 1) % kLBufs);
    read_scales(sca[C ^ 1], scb[C ^ 1], s + 1);
    mfma_step(0);
    convert(J5{}, sca[C], scb[C], 1);
    mfma_step(1);
    convert(J6{}, sca[C], scb[C], 0);
    mfma_step(0);
    convert(J7{}, sca[C], scb[C], 1);
    mfma_step(1);
    convert(J0{}, sca[C ^ 1], scb[C ^ 1], 0);
    __builtin_amdgcn_sched_barrier(0);
    // only operations of this stage may still be in flight: its DMA (and
    // the next BF16 loads); every stage issues at least kInFlight of them,
    // so everything older, the DMA of stage s+2 above all, has landed
    wait_counts<kInFlight, 0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };

  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  using P3 = std::integral_constant<int, 3>;
  int s = 0;
  for (; s + 4 <= nstages; s += 4) {
    run_stage(P0{}, s);
    run_stage(P1{}, s + 1);
    run_stage(P2{}, s + 2);
    run_stage(P3{}, s + 3);
  }
  {
    const int rest = nstages - s;
    if (rest > 0) run_stage(P0{}, s);
    if (rest > 1) run_stage(P1{}, s + 1);
    if (rest > 2) run_stage(P2{}, s + 2);
  }
  // no DMA may still be writing LDS when the workgroup ends
  wait_counts<0, 0>();

  // epilogue: out = bf16(fp32(fma(alpha, acc, bias))), alpha = aA * aB in
  // FP32.  Lane (li, g) holds row li and the column runs 8k + 4g .. +3
  // (k = 0..3) of its wave's 32 x 32 tile; swapping halves with the lane 32
  // apart gives each lane two runs of 8 consecutive columns (16-byte
  // stores) through a buffer resource over the tile's valid rows.
  const float alpha = (kFuse ? alpha_a : a_gs[0]) * b_gs[0];
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
  const uint32_t mrow = (uint32_t)((wm * 32 + li) * N);
  const int nb = wn * 32;   // this wave's first column in the tile
  float v[16];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint2 b2 = *reinterpret_cast<const uint2*>(&lbias[nb + 8 * k + 4 * g]);
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
    uint32_t r[4];   // 8 columns starting at nb + 16 h + 8 g
#pragma unroll
    for (int d = 0; d < 2; ++d) {
      const auto x = __builtin_amdgcn_permlane32_swap(p[2 * h][d], p[2 * h + 1][d], false, false);
      r[d] = x[0];
      r[2 + d] = x[1];
    }
    const int64_t n = n0 + nb + 16 * h + 8 * g;
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

hipError_t launch_gemm_small(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                             const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                             const SmallFuse* fuse, hipStream_t stream) {
  // 64 x 64 tiles, or 32 x 128 when fused
  const int64_t tiles = fuse ? ((M + 31) / 32) * ((N + 127) / 128) : ((M + 63) / 64) * ((N + 63) / 64);
  const dim3 grid((unsigned)tiles), block(kLThreads);
  const bool vec = N % 8 == 0;
  const SmallFuse f = fuse ? *fuse : SmallFuse{};
  if (fuse)
    return vec ? launch_kernel(nvfp4_gemm_small_kernel<true, true>, grid, block, stream, a_codes,
                               a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K, f)
               : launch_kernel(nvfp4_gemm_small_kernel<true, false>, grid, block, stream, a_codes,
                               a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K, f);
  return vec ? launch_kernel(nvfp4_gemm_small_kernel<false, true>, grid, block, stream, a_codes,
                             a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K, f)
             : launch_kernel(nvfp4_gemm_small_kernel<false, false>, grid, block, stream, a_codes,
                             a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K, f);
}

}  // namespace solfp4
