// Block-scaled NVFP4 GEMM with BF16 output for gfx950.
//
//   out[m][n] = bf16( fp32( aA * aB * sum_k (sA qA)[m][k] (sB qB)[n][k] + bias[n] ) )
//
// How the E4M3-per-16 scales are applied.  CDNA4's scaled matrix
// instructions take one power-of-two (E8M0) scale per 32 K-elements, while an
// NVFP4 element decodes to q * s with an E4M3 s: up to 2 + 4 = 6 significant
// bits per operand, more than any FP4/FP6/FP8 matrix input carries.  So the
// operands stay packed (0.5 B/element codes + 1/16 B/element scales) in HBM
// and L2, and each element is dequantized exactly to FP16 (q * s has at most
// 6 significant bits and lies in [2^-10, 2688]) before the FP16 matrix cores
// (v_mfma_f32_32x32x16_f16, FP32 accumulation) consume it.  Every product
// (sA qA)(sB qB) is exact; only the FP32 sums, the epilogue FMA and the BF16
// rounding round.  The per-tensor scales and the bias are applied once, in
// the epilogue.
//
// The dequantization is two instructions per pair of elements: the hardware
// FP4 converter (which applies only the exponent of its scale operand) with
// scale 2^8 gives 256 q exactly in FP16, and one packed FP16 multiply by the
// E4M3 byte shifted into an FP16 bit pattern (which reads as s * 2^-8, the
// two formats' mantissa fields being aligned and E4M3 subnormals landing on
// FP16 subnormals) gives q * s exactly.
//
// Two kernels:
//   nvfp4_gemm_lane_kernel (K % 128 == 0 or K % 64 == 32, and K % 128 == 64
//     where its 128 x 128 tiles or its split last round apply): codes travel
//     from HBM into LDS by DMA and each wave dequantizes its own MFMA operands
//     in registers, so LDS carries 0.5 B/element of codes instead of 2 B of
//     FP16 per operand read; with too few tiles for one 256 x 256 tile per
//     CU it runs on 128 x 128 tiles; a last round of at most a quarter of
//     the CUs' worth of 256 x 256 tiles runs in a second launch as their
//     128 x 128 quadrants (launch_gemm_quad), and otherwise a last round of
//     at most half the CUs' worth as two K halves per tile (SplitK);
//   nvfp4_gemm_kernel (the other K % 16 == 0): the workgroup converts each
//     stage once into FP16 tiles in LDS, which all waves read.
// Few tokens (K % 128 == 0, at most one 64 x 64 tile per CU) take one of
// two kernels of their own, chosen here by estimated time: 64 x 64 tiles
// (gemm_small.hip) or 32 x 32 tiles with the K stages dealt to the four
// waves of a workgroup (gemm_wavek.hip).
#include <type_traits>

#include "device_common.h"
#include "nvfp4_gemm_common.h"
#include "solfp4.h"
#include "kernels.h"

namespace solfp4 {

// ---------------------------------------------------------------------------
// nvfp4_gemm_kernel: workgroup-shared dequantization, any K % 16 == 0.
//
// Per K stage each pair of threads owns one row of the A tile and one row of
// the B tile, each thread converting 32 codes of each to FP16 and storing
// them to LDS, where all eight waves read their MFMA operands: each element
// is converted once per 256 x 256 output tile.  Tiling: 8 waves (2 x 4, two
// per SIMD so one wave's waits are covered by the other's MFMAs), each wave
// owning 128 x 64 (4 x 2 MFMA tiles of 32 x 32); K advances 64 elements
// (4 NVFP4 blocks) per stage.  LDS holds two stages of FP16 A and B tiles
// (rows padded to 144 bytes: conflict-free 16-byte row accesses).  Packed
// codes for stage s+2 are fetched into registers while stage s runs its
// MFMAs and stage s+1 is converted into the other LDS buffer, so each stage
// ends with a single barrier.  The two threads of a row load its 32 code
// bytes (and 4 scale bytes) with one coalesced request.  The MFMA's first
// operand is the weight tile, so each lane's accumulators hold runs of 4
// consecutive output columns of one row; one lane swap with the partner 32
// lanes away turns them into 16-byte runs for the stores.

constexpr int kBM = 256;
constexpr int kBN = 256;
constexpr int kBK = 64;                       // K elements per stage
constexpr int kBlocksPerStage = kBK / 16;     // NVFP4 blocks per row per stage
constexpr int kRowHalves = kBK + 8;           // padded LDS row (144 bytes)
constexpr int kGemmThreads = 512;
constexpr int kWaveTileM = 128;
constexpr int kWaveTileN = 64;
constexpr int kFragsM = kWaveTileM / 32;      // 32x32 MFMA tiles per wave, along M
constexpr int kFragsN = kWaveTileN / 32;      // and along N
constexpr int kSteps = kBK / 16;              // MFMA K-steps per stage

struct Smem {
  _Float16 a[2][kBM * kRowHalves];
  _Float16 b[2][kBN * kRowHalves];
  uint16_t bias[kBN];
};

// 8 E2M1 codes (element 2j in the low nibble of byte j) times the block
// scale, as 4 words of FP16 pairs (elements 2j, 2j+1); s2 holds s * 2^-8 in
// both halves.
__device__ __forceinline__ void dequant8(uint32_t w, uint32_t s2, uint32_t (&d)[4]) {
  const half2_t s = as_h2(s2);
  d[0] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 0) * s);
  d[1] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 1) * s);
  d[2] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 2) * s);
  d[3] = h2_as_u32(__builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 256.0f, 3) * s);
}

// One thread's share of a stage: half a row of one operand, 32 codes (16
// bytes, two NVFP4 blocks).  Scales arrive separately, four stages at a time.
struct HalfRow {
  uint4 c;
};

// Buffer resources for one operand's 256-row tile: rows past the end of the
// matrix fall outside num_records and read as zeros (code 0 with scale 0:
// the value 0), so no load needs a branch.
struct TileSrc {
  __amdgpu_buffer_rsrc_t codes, scales;
  uint32_t code_off, scale_off;   // this thread's half row / row, in bytes
};

__device__ __forceinline__ TileSrc make_tile_src(const uint8_t* codes, const uint8_t* scales,
                                                 int64_t row0, int64_t rows, int64_t K, int t) {
  const int64_t valid = min<int64_t>(rows - row0, 256);
  const int r = t >> 1, h = t & 1;
  TileSrc s;
  s.codes = uniform_rsrc(codes + row0 * (K / 2), valid * (K / 2));
  s.scales = uniform_rsrc(scales + row0 * (K / 16), valid * (K / 16));
  s.code_off = (uint32_t)(r * (K / 2) + 16 * h);
  s.scale_off = (uint32_t)(r * (K / 16));
  return s;
}

// Load this thread's 16 code bytes of `stage`.  kFast: K % 64 == 0 (every
// stage full, 16-byte offsets aligned).  Otherwise two 8-byte loads, and
// blocks past K are zeroed.
template <bool kFast>
__device__ __forceinline__ void load_codes(HalfRow& r, const TileSrc& src, int64_t K, int stage,
                                           int h) {
  const uint32_t co = src.code_off + (uint32_t)stage * (kBK / 2);
  if (kFast) {
    const u32x4_t a = __builtin_amdgcn_raw_buffer_load_b128(src.codes, co, 0, 0);
    r.c = make_uint4(a.x, a.y, a.z, a.w);
  } else {
    const int64_t kb_left = K / 16 - (int64_t)stage * kBlocksPerStage - 2 * h;
    u32x2_t blk[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      blk[j] = __builtin_amdgcn_raw_buffer_load_b64(src.codes, co + 8 * j, 0, 0);
      blk[j] = j < kb_left ? blk[j] : u32x2_t{0, 0};
    }
    r.c = make_uint4(blk[0].x, blk[0].y, blk[1].x, blk[1].y);
  }
}

// The row's 16 scale bytes for stages 4g .. 4g+3 (both threads of a row load
// the same bytes: one coalesced request).  Byte 4j + b is block b of stage
// 4g + j.  Blocks past K are zeroed.
template <bool kFast>
__device__ __forceinline__ u32x4_t load_scales(const TileSrc& src, int64_t K, int g) {
  const uint32_t so = src.scale_off + (uint32_t)g * 16;
  if (kFast && (K / 16) % 16 == 0) {
    return __builtin_amdgcn_raw_buffer_load_b128(src.scales, so, 0, 0);
  } else if (kFast) {
    // 4-byte aligned (K % 64 == 0); stages past K read other rows or zeros
    // and are never converted into a used buffer
    u32x4_t v;
    v.x = __builtin_amdgcn_raw_buffer_load_b32(src.scales, so, 0, 0);
    v.y = __builtin_amdgcn_raw_buffer_load_b32(src.scales, so + 4, 0, 0);
    v.z = __builtin_amdgcn_raw_buffer_load_b32(src.scales, so + 8, 0, 0);
    v.w = __builtin_amdgcn_raw_buffer_load_b32(src.scales, so + 12, 0, 0);
    return v;
  } else {
    const int64_t kb_left = K / 16 - (int64_t)g * 16;
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const uint32_t b = __builtin_amdgcn_raw_buffer_load_b8(src.scales, so + i, 0, 0);
      w[i / 4] |= (i < kb_left ? b : 0u) << (8 * (i % 4));
    }
    return u32x4_t{w[0], w[1], w[2], w[3]};
  }
}

// Convert block j (0 or 1) of a half row (scale bytes of its two blocks in
// sc2) and store its 16 FP16 values.  The
// E4M3 scale byte shifted into an FP16 bit pattern reads as s * 2^-8 (the
// two formats align their mantissa fields, and E4M3 subnormals become FP16
// subnormals); one exact multiply by 2^8 restores s.
__device__ __forceinline__ void convert_block(const HalfRow& r, uint32_t sc2, int j,
                                              _Float16* dst) {
  const uint32_t c = (sc2 >> (8 * j)) & 0xFFu;
  const uint32_t s2 = (c << 7) | (c << 23);   // s * 2^-8 in both FP16 halves
  const uint32_t w0 = j == 0 ? r.c.x : r.c.z;
  const uint32_t w1 = j == 0 ? r.c.y : r.c.w;
  uint32_t d[4], e[4];
  dequant8(w0, s2, d);
  dequant8(w1, s2, e);
  *reinterpret_cast<uint4*>(dst + 16 * j) = make_uint4(d[0], d[1], d[2], d[3]);
  *reinterpret_cast<uint4*>(dst + 16 * j + 8) = make_uint4(e[0], e[1], e[2], e[3]);
}

// Scheduling of one K-step segment (after its operand reads are fenced
// off): each of the 8 MFMAs is followed by up to 5 VALU instructions of the
// next stage's conversion, and the conversion's 2 LDS stores go last, so the
// conversion runs in the shadow of the matrix pipeline.
__device__ __forceinline__ void interleave_step() {
#pragma unroll
  for (int i = 0; i < kFragsM * kFragsN; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // MFMA
    __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);   // VALU
    if (i >= 6) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);    // DS write
  }
}

template <bool kFast, bool kVecOut>
__global__ __launch_bounds__(kGemmThreads, 1) void nvfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_gs, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_gs,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K) {
  __shared__ Smem smem;

  const int tiles_m = (int)((M + kBM - 1) / kBM);
  const int tiles_n = (int)((N + kBN - 1) / kBN);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kBM;
  const int64_t n0 = (int64_t)tn * kBN;

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int wm = wave >> 2;
  const int wn = wave & 3;
  const int li = lane & 31;
  const int lg = lane >> 5;
  const int h = t & 1;

  floatx16_t acc[kFragsN][kFragsM];
#pragma unroll
  for (int i = 0; i < kFragsN; ++i)
#pragma unroll
    for (int j = 0; j < kFragsM; ++j) acc[i][j] = floatx16_t{};

  const int nstages = (int)((K + kBK - 1) / kBK);
  const TileSrc src_a = make_tile_src(a_codes, a_scales, m0, M, K, t);
  const TileSrc src_b = make_tile_src(b_codes, b_scales, n0, N, K, t);
  // this thread's half row in an LDS stage buffer
  const int my = (t >> 1) * kRowHalves + 32 * h;
  // this thread's two scale bytes of stage s sit in word s%4 of its group's
  // scale registers, at byte offset 2h
  const int sshift = 16 * h;
  HalfRow ca[2], cb[2];
  u32x4_t sa4[2], sb4[2];
  // prologue: scales of stages 0-7, codes of stages 0-1; stage 0 converted
  // into buffer 0
  sa4[0] = load_scales<kFast>(src_a, K, 0);
  sb4[0] = load_scales<kFast>(src_b, K, 0);
  sa4[1] = load_scales<kFast>(src_a, K, 1);
  sb4[1] = load_scales<kFast>(src_b, K, 1);
  load_codes<kFast>(ca[0], src_a, K, 0, h);
  load_codes<kFast>(cb[0], src_b, K, 0, h);
  load_codes<kFast>(ca[1], src_a, K, 1, h);
  load_codes<kFast>(cb[1], src_b, K, 1, h);
  convert_block(ca[0], sa4[0].x >> sshift, 0, &smem.a[0][my]);
  convert_block(ca[0], sa4[0].x >> sshift, 1, &smem.a[0][my]);
  convert_block(cb[0], sb4[0].x >> sshift, 0, &smem.b[0][my]);
  convert_block(cb[0], sb4[0].x >> sshift, 1, &smem.b[0][my]);
  // the tile's bias (+0 without one: fma(alpha, acc, +0) == alpha * acc for
  // every accumulator, which never holds -0)
  if (t < kBN) smem.bias[t] = bias && n0 + t < N ? bias[n0 + t] : (uint16_t)0;
  __syncthreads();

  // One stage, branch free.  P = s % 8 selects the register sets: codes of
  // stage s+1 (converted now into buffer cur^1) are in set (P+1)%2 and the
  // loads of stage s+2 go to set P%2; scales of stage s+1 are in group set
  // ((P+1)/4)%2, and at P == 0 / P == 4 the scales of the group after next
  // are fetched into the set the previous group used.  Past the last stage
  // the loads read zeros or unused data and the conversion fills the buffer
  // nobody reads again.
  auto run_stage = [&](auto phase, int s) {
    constexpr int P = decltype(phase)::value;
    constexpr int kc = P & 1;              // code set loaded now (stage s+2)
    constexpr int kn = (P + 1) & 1;        // code set converted now (stage s+1)
    constexpr int gn = ((P + 1) >> 2) & 1; // scale set of stage s+1
    constexpr int wn_ = (P + 1) & 3;       // word of stage s+1 in its group
    const int cur = s & 1;
    if (P == 0 || P == 4) {
      constexpr int gl = P == 0 ? 1 : 0;   // set receiving group s/4 + 1
      sa4[gl] = load_scales<kFast>(src_a, K, s / 4 + 1);
      sb4[gl] = load_scales<kFast>(src_b, K, s / 4 + 1);
    }
    load_codes<kFast>(ca[kc], src_a, K, s + 2, h);
    load_codes<kFast>(cb[kc], src_b, K, s + 2, h);
    const uint32_t sca = sa4[gn][wn_] >> sshift;
    const uint32_t scb = sb4[gn][wn_] >> sshift;
    const _Float16* sa = smem.a[cur] + (wm * kWaveTileM + li) * kRowHalves + 8 * lg;
    const _Float16* sb = smem.b[cur] + (wn * kWaveTileN + li) * kRowHalves + 8 * lg;
    _Float16* na = &smem.a[cur ^ 1][my];
    _Float16* nb = &smem.b[cur ^ 1][my];
    half8_t af[2][kFragsM], bf[2][kFragsN];
#pragma unroll
    for (int f = 0; f < kFragsM; ++f) af[0][f] = *reinterpret_cast<const half8_t*>(sa + f * 32 * kRowHalves);
#pragma unroll
    for (int f = 0; f < kFragsN; ++f) bf[0][f] = *reinterpret_cast<const half8_t*>(sb + f * 32 * kRowHalves);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      const int c = st & 1;
      // operand reads for the next K-step go out first: they have this
      // step's MFMAs to complete
      if (st + 1 < kSteps) {
#pragma unroll
        for (int f = 0; f < kFragsM; ++f)
          af[c ^ 1][f] = *reinterpret_cast<const half8_t*>(sa + f * 32 * kRowHalves + 16 * (st + 1));
#pragma unroll
        for (int f = 0; f < kFragsN; ++f)
          bf[c ^ 1][f] = *reinterpret_cast<const half8_t*>(sb + f * 32 * kRowHalves + 16 * (st + 1));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int fn = 0; fn < kFragsN; ++fn)
#pragma unroll
        for (int fm = 0; fm < kFragsM; ++fm)
          acc[fn][fm] = __builtin_amdgcn_mfma_f32_32x32x16_f16(bf[c][fn], af[c][fm], acc[fn][fm], 0, 0, 0);
      // a quarter of the next stage's conversion per K-step
      if (st == 0) convert_block(ca[kn], sca, 0, na);
      if (st == 1) convert_block(ca[kn], sca, 1, na);
      if (st == 2) convert_block(cb[kn], scb, 0, nb);
      if (st == 3) convert_block(cb[kn], scb, 1, nb);
      interleave_step();
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
  };

  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  using P3 = std::integral_constant<int, 3>;
  using P4 = std::integral_constant<int, 4>;
  using P5 = std::integral_constant<int, 5>;
  using P6 = std::integral_constant<int, 6>;
  using P7 = std::integral_constant<int, 7>;
  int s = 0;
  for (; s + 8 <= nstages; s += 8) {
    run_stage(P0{}, s);
    run_stage(P1{}, s + 1);
    run_stage(P2{}, s + 2);
    run_stage(P3{}, s + 3);
    run_stage(P4{}, s + 4);
    run_stage(P5{}, s + 5);
    run_stage(P6{}, s + 6);
    run_stage(P7{}, s + 7);
  }
  const int rest = nstages - s;
  if (rest > 0) run_stage(P0{}, s);
  if (rest > 1) run_stage(P1{}, s + 1);
  if (rest > 2) run_stage(P2{}, s + 2);
  if (rest > 3) run_stage(P3{}, s + 3);
  if (rest > 4) run_stage(P4{}, s + 4);
  if (rest > 5) run_stage(P5{}, s + 5);
  if (rest > 6) run_stage(P6{}, s + 6);

  // epilogue: out = bf16(fp32(fma(alpha, acc, bias))), alpha = aA * aB in
  // FP32.  Lane (li, lg) holds, per MFMA tile, row m = li and the column runs
  // 8k + 4lg .. 8k + 4lg + 3 (k = 0..3); swapping halves with the lane 32
  // apart gives each lane two runs of 8 consecutive columns (16-byte
  // stores).  Stores go through a buffer resource covering the tile's valid
  // rows, so rows past M are dropped by the hardware range check; columns
  // past N get an offset beyond the range.
  const float alpha = a_gs[0] * b_gs[0];
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, min<int64_t>(M - m0, kBM) * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
#pragma unroll
  for (int fm = 0; fm < kFragsM; ++fm) {
    const uint32_t mrow = (uint32_t)((wm * kWaveTileM + fm * 32 + li) * N);
#pragma unroll
    for (int fn = 0; fn < kFragsN; ++fn) {
      const int nb = wn * kWaveTileN + fn * 32;
      float v[16];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint2 b2 = *reinterpret_cast<const uint2*>(&smem.bias[nb + 8 * k + 4 * lg]);
        const float bv[4] = {__uint_as_float(b2.x << 16), __uint_as_float(b2.x & 0xFFFF0000u),
                             __uint_as_float(b2.y << 16), __uint_as_float(b2.y & 0xFFFF0000u)};
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * k + q] = __builtin_fmaf(alpha, acc[fn][fm][4 * k + q], bv[q]);
      }
      uint32_t p[4][2];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        p[k][0] = pack_bf16(v[4 * k], v[4 * k + 1]);
        p[k][1] = pack_bf16(v[4 * k + 2], v[4 * k + 3]);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t r[4];   // 8 columns starting at nb + 16 h + 8 lg
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          const auto x = __builtin_amdgcn_permlane32_swap(p[2 * h][d], p[2 * h + 1][d], false, false);
          r[d] = x[0];
          r[2 + d] = x[1];
        }
        const int64_t n = n0 + nb + 16 * h + 8 * lg;
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
  }
}

// ---------------------------------------------------------------------------
// nvfp4_gemm_lane_kernel: lane-side dequantization, K % 32 == 0.
//
// Tiling and data movement follow the MXFP4 GEMM: a 2 kWT x 2 kWT output
// tile per workgroup of 4 waves (one per SIMD), each wave owning kWT x kWT
// (kWT = 128: 4 x 4 MFMA tiles of 32 x 32, 256 FP32 accumulators per lane;
// kWT = 64, for GEMMs with too few 256 x 256 tiles to fill the chip: 2 x 2
// tiles, a quarter of the work per workgroup); K advances 128
// elements (64 code bytes per row) per stage; codes go from global memory
// straight into four LDS stage buffers by DMA, three stages ahead, each lane
// quad reading the 64 contiguous bytes of one row, stored as [row][piece] x
// 16 bytes with the piece order of row r swizzled by (r >> 2) & 3 (no bank
// conflicts on the operand reads).
//
// Each wave turns its own operands into FP16 in registers.  The order of K
// inside a stage is free as long as both operands use the same one, so lane
// group g (lanes 32g .. 32g+31) of K-step j supplies the 8 elements
// 32 p + 8 (j % 4) .. +7 with p = g for j < 4 and p = 2 + g after: one
// 16-byte LDS read of a row's piece p feeds four K-steps, and the 8 elements
// of a K-step always sit in one NVFP4 block.  Scales are staged through LDS
// already as FP16 patterns (s * 2^-8, two blocks per word), so a lane reads
// the word of its row and piece and a packed multiply with the half selected
// by op_sel applies the block scale.  Per K-step a kWT = 128 wave converts 8
// fragments (64 VALU instructions) under 16 MFMAs.

// kFull: K % 128 == 0, every stage lies inside the rows and a stage's 8
// scale bytes per row are one aligned 8-byte load.  Otherwise (K % 32 == 0)
// the last stage is partial: its code pieces past K read bytes of the next
// row (or zeros past the tile), which stay harmless because the scales of
// those blocks are set to zero (E2M1 codes are all finite, and q * 0 = 0).
// A row's scales then start at an even offset only; the 8-byte load works
// at any byte alignment, but the buffer range check drops a whole 4-byte
// word that straddles the end of the range, so the one lane whose stage
// reaches past the operand's last scale byte (the last row, last stage)
// fetches its bytes as four 2-byte loads instead.
template <bool kVecOut, bool kFull, int kWT>
__global__ __launch_bounds__(kLThreads, 1) void nvfp4_gemm_lane_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const float* __restrict__ a_gs, const uint8_t* __restrict__ b_codes,
    const uint8_t* __restrict__ b_scales, const float* __restrict__ b_gs,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K, SplitK split) {
  static_assert(kWT == 128 || kWT == 64, "wave tile edge");
  constexpr int kT = 2 * kWT;                // output tile edge (M and N)
  constexpr int kFr = kWT / 32;              // 32 x 32 MFMA tiles per wave edge
  constexpr int kStage = kT * kLRowBytes;    // one operand, one stage
  constexpr int kGw = kT / 64;               // 16-row DMA groups per wave and operand
  constexpr int kDma = 2 * kGw;              // DMA instructions per wave and stage
  // one array per stage buffer and operand, so the compiler can tell the
  // buffer being filled by DMA from the one being read
  __shared__ __attribute__((aligned(1024))) uint8_t la0[kStage], la1[kStage],
      la2[kStage], la3[kStage];
  __shared__ __attribute__((aligned(1024))) uint8_t lb0[kStage], lb1[kStage],
      lb2[kStage], lb3[kStage];
  __shared__ uint32_t lsc[2][2][kT * kLScaleStride];   // [stage parity][operand][row, word]
  __shared__ uint16_t lbias[kT];
  uint8_t* const abuf[kLBufs] = {la0, la1, la2, la3};
  uint8_t* const bbuf[kLBufs] = {lb0, lb1, lb2, lb3};

  const int tiles_m = (int)((M + kT - 1) / kT);
  const int tiles_n = (int)((N + kT - 1) / kT);
  // workgroups past split.dp_tiles each take one K range of a remainder tile
  const int sub = (int)blockIdx.x - split.dp_tiles;
  const int rem = sub < 0 ? -1 : sub / split.splits;
  const int part_idx = sub < 0 ? 0 : sub - rem * split.splits;
  int tm, tn;
  const int tile_id = sub < 0 ? (int)blockIdx.x : split.dp_tiles + rem;
  if constexpr (kWT == 64) {
    if (split.quad_base >= 0) {
      // quadrant tile_id % 4 of 256 x 256 tile quad_base + tile_id / 4
      tile_coords_at(split.quad_base + tile_id / 4, (int)((M + 255) / 256), (int)((N + 255) / 256),
                     tm, tn);
      tm = 2 * tm + ((tile_id >> 1) & 1);
      tn = 2 * tn + (tile_id & 1);
      if ((int64_t)tm * kT >= M || (int64_t)tn * kT >= N) return;   // quadrant outside the output
    } else {
      tile_coords_at(tile_id, tiles_m, tiles_n, tm, tn);
    }
  } else {
    tile_coords_at(tile_id, tiles_m, tiles_n, tm, tn);
  }
  const int64_t m0 = (int64_t)tm * kT;
  const int64_t n0 = (int64_t)tn * kT;
  const int all_stages = (int)((K + kLBK - 1) / kLBK);
  const int s_first = sub < 0 ? 0 : part_idx * split.stages;
  const int nstages = sub < 0 ? all_stages : min(all_stages - s_first, split.stages);

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int wm = wave >> 1;
  const int wn = wave & 1;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t scale_row = K / 16;
  const int64_t valid_a = min<int64_t>(M - m0, kT);
  const int64_t valid_b = min<int64_t>(N - n0, kT);
  const __amdgpu_buffer_rsrc_t rca = uniform_rsrc(a_codes + m0 * row_bytes, valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rsa = uniform_rsrc(a_scales + m0 * scale_row, valid_a * scale_row);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * scale_row, valid_b * scale_row);

  // code DMA: wave w fills 16-row groups kGw w .. kGw w + kGw - 1 of each
  // operand; lane quad l/4 reads the 64 bytes of row l/4 of the group, lane
  // l's 16 bytes land in slot l of the group's 1 KB
  const int dma_r = lane >> 2;
  const int piece = (lane & 3) ^ ((dma_r >> 2) & 3);
  const uint32_t dma_off =
      (uint32_t)((16 * kGw * wave + dma_r) * row_bytes + 16 * piece + s_first * kLRowBytes);
  const uint32_t group_stride = (uint32_t)(16 * row_bytes);
  // scale staging: thread t moves the 8 scale bytes of tile row t of A and B
  // (threads past the tile's rows load zeros out of range and store nothing)
  const uint32_t sg_off = (uint32_t)(t * scale_row + 8 * s_first);
  // operand slots of this lane: row r of the tile lives in group r / 16 at
  // byte (r % 16) * 64 + 16 * (piece ^ ((r % 16) >> 2)); lane group g reads
  // piece g in K-steps 0-3 and piece 2 + g in K-steps 4-7
  const int swz = ((li & 15) >> 2) & 3;
  const int rd_a = ((wm * kWT + li) >> 4) * 1024 + (li & 15) * 64;
  const int rd_b = ((wn * kWT + li) >> 4) * 1024 + (li & 15) * 64;
  const int q_off[2] = {16 * (g ^ swz), 16 * ((2 + g) ^ swz)};
  // and its scale words: word p of a row holds the patterns of blocks 2p, 2p+1
  const int rs_a = (wm * kWT + li) * kLScaleStride + g;
  const int rs_b = (wn * kWT + li) * kLScaleStride + g;

  // the tile's bias (+0 without one: fma(alpha, acc, +0) == alpha * acc for
  // every accumulator, which never holds -0); parked in LDS once the
  // prologue's loads are out, so its latency overlaps theirs
  constexpr bool kAllRows = kT == kLThreads;   // every thread stages one tile row
  const bool row_thread = kAllRows || t < kT;
  const uint16_t bias_v = bias && row_thread && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc[kFr][kFr];
#pragma unroll
  for (int i = 0; i < kFr; ++i)
#pragma unroll
    for (int j = 0; j < kFr; ++j) acc[i][j] = floatx16_t{};

  uint32_t sca[2][kFr][2], scb[2][kFr][2];   // [stage parity][frag][half stage]
  u32x4_t ca[2][kFr], cb[2][kFr];            // code pieces, [half stage][frag]
  half8_t oa[2][kFr], ob[2][kFr];            // FP16 operands, [K-step parity][frag]

  // kDma DMA instructions per wave: stage `stage` into buffer `buf`.
  // Stages past K read bytes of later rows or zeros into buffers never
  // computed.
  auto dma_stage = [&](int buf, int stage) {
    const uint32_t base = dma_off + (uint32_t)stage * kLRowBytes;
#pragma unroll
    for (int j = 0; j < kGw; ++j) {
      const uint32_t off = base + j * group_stride;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rca, (lds_ptr_t)(abuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rcb, (lds_ptr_t)(bbuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
    }
  };
  // group j of the DMA of `stage` (2 of its kDma instructions)
  auto dma_part = [&](int buf, int stage, int j) {
    const uint32_t off = dma_off + (uint32_t)stage * kLRowBytes + j * group_stride;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rca, (lds_ptr_t)(abuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rcb, (lds_ptr_t)(bbuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
  };
  // one stage's scale bytes of this thread's A and B rows, in flight
  const uint32_t range_a = (uint32_t)(valid_a * scale_row);
  const uint32_t range_b = (uint32_t)(valid_b * scale_row);
  struct ScaleFetch {
    u32x2_t a, b;            // one 8-byte load each
    uint32_t ha[4], hb[4];   // !kFull, a stage straddling the end of the range: 2-byte loads
    bool whole_a, whole_b;   // the 8-byte load holds every in-range byte
  };
  auto fetch_scales = [&](ScaleFetch& f, int stage) {
    const uint32_t off = sg_off + 8 * stage;
    f.a = __builtin_amdgcn_raw_buffer_load_b64(rsa, off, 0, 0);
    f.b = __builtin_amdgcn_raw_buffer_load_b64(rsb, off, 0, 0);
    if (!kFull) {
      f.whole_a = off + 8 <= range_a || off >= range_a;
      f.whole_b = off + 8 <= range_b || off >= range_b;
      if (!(f.whole_a && f.whole_b)) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f.ha[j] = __builtin_amdgcn_raw_buffer_load_b16(rsa, off + 2 * j, 0, 0);
          f.hb[j] = __builtin_amdgcn_raw_buffer_load_b16(rsb, off + 2 * j, 0, 0);
        }
      }
    }
  };
  // scale bytes of `stage` (fetched earlier into f) into set `set`, as FP16
  // patterns; blocks at or past K/16 get scale 0
  auto store_scales = [&](ScaleFetch& f, int set, int stage) {
    u32x2_t ga = f.a, gb = f.b;
    if (!kFull) {
      if (!f.whole_a) ga = u32x2_t{f.ha[0] | (f.ha[1] << 16), f.ha[2] | (f.ha[3] << 16)};
      if (!f.whole_b) gb = u32x2_t{f.hb[0] | (f.hb[1] << 16), f.hb[2] | (f.hb[3] << 16)};
      const int64_t valid = scale_row - 8 * (int64_t)(s_first + stage);   // blocks inside K
      if (valid < 8) {
        const uint64_t keep = valid <= 0 ? 0ull : (~0ull >> (64 - 8 * valid));
        ga.x &= (uint32_t)keep;
        ga.y &= (uint32_t)(keep >> 32);
        gb.x &= (uint32_t)keep;
        gb.y &= (uint32_t)(keep >> 32);
      }
    }
    if (row_thread) {
      uint32_t* da = &lsc[set][0][t * kLScaleStride];
      uint32_t* db = &lsc[set][1][t * kLScaleStride];
      da[0] = scale_patterns(ga.x, false);
      da[1] = scale_patterns(ga.x, true);
      da[2] = scale_patterns(ga.y, false);
      da[3] = scale_patterns(ga.y, true);
      db[0] = scale_patterns(gb.x, false);
      db[1] = scale_patterns(gb.x, true);
      db[2] = scale_patterns(gb.y, false);
      db[3] = scale_patterns(gb.y, true);
    }
  };
  // this lane's scale words of `stage` (its 4 A rows and 4 B rows, both pieces)
  auto read_scales = [&](uint32_t (&da)[kFr][2], uint32_t (&db)[kFr][2], int stage) {
    const int set = stage & 1;
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      da[f][0] = lsc[set][0][rs_a + f * 32 * kLScaleStride];
      da[f][1] = lsc[set][0][rs_a + f * 32 * kLScaleStride + 2];
      db[f][0] = lsc[set][1][rs_b + f * 32 * kLScaleStride];
      db[f][1] = lsc[set][1][rs_b + f * 32 * kLScaleStride + 2];
    }
  };
  auto read_codes = [&](int half, int buf) {
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      ca[half][f] = *reinterpret_cast<const u32x4_t*>(abuf[buf] + rd_a + f * 2048 + q_off[half]);
      cb[half][f] = *reinterpret_cast<const u32x4_t*>(bbuf[buf] + rd_b + f * 2048 + q_off[half]);
    }
  };
  // K-step j of a stage (scale words ss) into operand set d
  auto convert = [&](auto step, const uint32_t (&ssa)[kFr][2],
                     const uint32_t (&ssb)[kFr][2], int d) {
    constexpr int j = decltype(step)::value;
    constexpr int h = j >> 2, w = j & 3;
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      const half2_t xa = as_h2(ssa[f][h]), xb = as_h2(ssb[f][h]);
      const half2_t sa = (w & 2) ? __builtin_shufflevector(xa, xa, 1, 1) : __builtin_shufflevector(xa, xa, 0, 0);
      const half2_t sb = (w & 2) ? __builtin_shufflevector(xb, xb, 1, 1) : __builtin_shufflevector(xb, xb, 0, 0);
      oa[d][f] = dequant_step(ca[h][f][w], sa);
      ob[d][f] = dequant_step(cb[h][f][w], sb);
    }
  };
  auto mfma_step = [&](int d) {
#pragma unroll
    for (int fn = 0; fn < kFr; ++fn)
#pragma unroll
      for (int fm = 0; fm < kFr; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ob[d][fn], oa[d][fm], acc[fn][fm], 0, 0, 0);
  };
  // kFr^2 MFMAs, each followed by up to 16 / kFr VALU instructions of the
  // next K-step's conversion and a share of the step's kR pairs of LDS
  // reads, kV memory loads and kW LDS writes (one of each per MFMA for the
  // 128 x 128 wave tile, four for the 64 x 64 one)
  auto interleave = [&](auto reads, auto vmem, auto writes) {
    constexpr int kR = decltype(reads)::value, kV = decltype(vmem)::value,
                  kW = decltype(writes)::value;
    constexpr int kPer = 16 / (kFr * kFr);
#pragma unroll
    for (int i = 0; i < kFr * kFr; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                          // MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 16 / kFr, 0);                   // VALU
      if (i * kPer < kR) __builtin_amdgcn_sched_group_barrier(0x100, 2 * kPer, 0);   // DS read
      if (i * kPer < kV) __builtin_amdgcn_sched_group_barrier(0x020, kPer, 0);       // VMEM read
      if (i * kPer < kW) __builtin_amdgcn_sched_group_barrier(0x200, kPer, 0);       // DS write
    }
  };

  using I0 = std::integral_constant<int, 0>;
  using I4 = std::integral_constant<int, 4>;
  using I8 = std::integral_constant<int, 8>;
  using I12 = std::integral_constant<int, 12>;
  using J0 = std::integral_constant<int, 0>;
  using J1 = std::integral_constant<int, 1>;
  using J2 = std::integral_constant<int, 2>;
  using J3 = std::integral_constant<int, 3>;
  using J4 = std::integral_constant<int, 4>;
  using J5 = std::integral_constant<int, 5>;
  using J6 = std::integral_constant<int, 6>;
  using J7 = std::integral_constant<int, 7>;

  constexpr int kSL = 2;   // vector-memory instructions of one scale fetch (but for one stage of one lane)
  // prologue: the scales of stages 0-2, then the codes of stages 0-2, all go
  // out first; the scales of stages 0 and 1 are parked in LDS as they land
  // (each store waits only for its own, older loads), stage 2's stay in
  // registers; once stages 0 and 1 have landed (only stage 2's DMA, the
  // youngest loads, may still be in flight), the first half stage's codes
  // and the scales of stage 0 are read and K-step 0 converted.  The second
  // barrier keeps stage 0 from parking stage 2's scales over set 0 before
  // every wave has read it.
  ScaleFetch sf, sf0, sf1;   // sf: the stage in flight during the main loop
  fetch_scales(sf0, 0);
  fetch_scales(sf1, 1);
  fetch_scales(sf, 2);
  dma_stage(0, 0);
  dma_stage(1, 1);
  dma_stage(2, 2);
  if (row_thread) lbias[t] = bias_v;
  store_scales(sf0, 0, 0);
  store_scales(sf1, 1, 1);
  wait_counts<kDma, 0>();
  __builtin_amdgcn_s_barrier();
  read_scales(sca[0], scb[0], 0);
  read_codes(0, 0);
  wait_counts<63, 0>();
  __builtin_amdgcn_s_barrier();
  convert(J0{}, sca[0], scb[0], 0);

  // Stage s with P = s % 4 (buffer P, scale parity C = P % 2).  K-steps 0
  // .. kGw-1 issue the DMA of stage s+3 into buffer (P + 3) % 4 (last read in
  // stage s-1); K-step 0 parks the scales of stage s+2 in set C (last read in stage s-1,
  // next read in stage s+1) and fetches those of stage s+3, and reads this
  // stage's second code half; K-step 4 reads the next stage's first code
  // half and scales; K-step 7 converts the next stage's K-step 0.  The
  // barrier that ends stage s waits for this wave's DMA of stage s+2, so in
  // stage s+1 both its own buffer and the next one are complete.
  auto run_stage = [&](auto phase, int s) {
    constexpr int P = decltype(phase)::value;
    constexpr int C = P & 1;
    __builtin_amdgcn_sched_barrier(0);
    // the scale loads go out before the DMA, so the wait that ends the stage
    // can count the DMA alone (the compiler may merge the scale loads into
    // fewer instructions than written)
    store_scales(sf, C, s + 2);
    fetch_scales(sf, s + 3);
    // the DMA of stage s+3 goes out a group (2 instructions) per K-step over
    // K-steps 0 .. kGw-1: issued at once, the 8 instructions of a 128 x 128
    // wave tile filled the texture addresser's queues and held up the MFMA
    // issue behind them (3% slower)
    using I2 = std::integral_constant<int, 2>;
    dma_part((P + 3) % kLBufs, s + 3, 0);
    read_codes(1, P);
    mfma_step(0);
    convert(J1{}, sca[C], scb[C], 1);
    interleave(I4{}, std::integral_constant<int, 2 + kSL>{}, I8{});
    __builtin_amdgcn_sched_barrier(0);
    dma_part((P + 3) % kLBufs, s + 3, 1);
    mfma_step(1);
    convert(J2{}, sca[C], scb[C], 0);
    interleave(I0{}, I2{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    if (kGw > 2) dma_part((P + 3) % kLBufs, s + 3, 2);
    mfma_step(0);
    convert(J3{}, sca[C], scb[C], 1);
    interleave(I0{}, std::integral_constant<int, (kGw > 2 ? 2 : 0)>{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    if (kGw > 3) dma_part((P + 3) % kLBufs, s + 3, 3);
    mfma_step(1);
    convert(J4{}, sca[C], scb[C], 0);
    interleave(I0{}, std::integral_constant<int, (kGw > 3 ? 2 : 0)>{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    read_codes(0, (P + 1) % kLBufs);
    read_scales(sca[C ^ 1], scb[C ^ 1], s + 1);
    mfma_step(0);
    convert(J5{}, sca[C], scb[C], 1);
    interleave(I12{}, I0{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(1);
    convert(J6{}, sca[C], scb[C], 0);
    interleave(I0{}, I0{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(0);
    convert(J7{}, sca[C], scb[C], 1);
    interleave(I0{}, I0{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    mfma_step(1);
    convert(J0{}, sca[C ^ 1], scb[C ^ 1], 0);
    interleave(I0{}, I0{}, I0{});
    __builtin_amdgcn_sched_barrier(0);
    // this stage's kDma DMA instructions, the last vector-memory operations
    // it issued, may stay in flight; everything older (the DMA of stage s+2
    // and this stage's scale loads) is complete
    wait_counts<kDma, 0>();
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

  if (sub >= 0) {
    // One of the two K halves of a remainder tile: park the FP32
    // accumulators in the workspace; the second of the tile's two
    // workgroups to finish adds the other half's sums to its own (FP32
    // addition is commutative, so the result does not depend on which one
    // that is) and runs the epilogue.  The partial sums are written and read
    // with the sc1 cache policy (written through to memory, read past this
    // XCD's L2), so they are coherent across XCDs without writing back or
    // invalidating whole L2 caches; a half's stores are complete before its
    // workgroup counts itself in.  Lane-major 16-byte slots: each store or
    // load instruction covers 1 KB.
    constexpr int kSlots = kFr * kFr * 4;           // 16-byte slots per lane
    constexpr uint32_t kSlotBytes = 16 * kWave;     // one slot of a wave
    constexpr uint32_t kHalfBytes = 4 * kSlots * kSlotBytes;   // one half's partial tile
    constexpr int kSc1 = 16;                        // cache policy bits: sc1
    const __amdgpu_buffer_rsrc_t rp = uniform_rsrc(
        reinterpret_cast<const uint8_t*>(split.part) + (size_t)rem * 2 * kHalfBytes,
        (int64_t)2 * kHalfBytes);
    const uint32_t lane_off = (uint32_t)wave * kSlots * kSlotBytes + 16u * lane;
#pragma unroll
    for (int fn = 0; fn < kFr; ++fn)
#pragma unroll
      for (int fm = 0; fm < kFr; ++fm)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const floatx16_t& a = acc[fn][fm];
          const u32x4_t v = {__float_as_uint(a[4 * q]), __float_as_uint(a[4 * q + 1]),
                             __float_as_uint(a[4 * q + 2]), __float_as_uint(a[4 * q + 3])};
          __builtin_amdgcn_raw_buffer_store_b128(
              v, rp, lane_off + part_idx * kHalfBytes + ((fn * kFr + fm) * 4 + q) * kSlotBytes, 0, kSc1);
        }
    __shared__ int last_flag;
    wait_counts<0, 0>();   // this thread's partial sums have reached memory
    __syncthreads();
    if (t == 0) {
      const uint64_t mine = kSplitToken ^ (uint64_t)(2 * rem + part_idx);
      const uint64_t before = __hip_atomic_exchange(&split.slots[rem], mine, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
      last_flag = before == (mine ^ 1u);   // the other half's token: it finished first
      if (last_flag)
        __hip_atomic_store(&split.slots[rem], (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last_flag) return;
    // The other half's sums come in through LDS, whose stage buffers are
    // free now: each wave moves its own slots by DMA (no registers held
    // while the loads are in flight), half of them at a time into two of
    // the stage buffers, then reads each slot back and adds it.
    constexpr int kPerBuf = kStage / 1024;   // 1 KB slots per stage buffer
    constexpr int kPass = kSlots / 2;
    static_assert(kSlots % 2 == 0 && kPass <= 2 * kPerBuf, "slots per pass");
    uint8_t* const lds_lo = wave == 0 ? la0 : wave == 1 ? la2 : wave == 2 ? lb0 : lb2;
    uint8_t* const lds_hi = wave == 0 ? la1 : wave == 1 ? la3 : wave == 2 ? lb1 : lb3;
    const uint32_t other = lane_off + (1 - part_idx) * kHalfBytes;
#pragma unroll
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
      for (int i = 0; i < kPass; ++i) {
        uint8_t* const dst = (i < kPerBuf ? lds_lo : lds_hi) + (i % kPerBuf) * 1024;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rp, (lds_ptr_t)dst, 16,
                                                 other + (pass * kPass + i) * kSlotBytes, 0, 0, kSc1);
      }
      wait_counts<0, 0>();
#pragma unroll
      for (int i = 0; i < kPass; ++i) {
        const int slot = pass * kPass + i;
        const int fn = slot / (4 * kFr), fm = (slot / 4) % kFr, q = slot % 4;
        const uint8_t* const src = (i < kPerBuf ? lds_lo : lds_hi) + (i % kPerBuf) * 1024 + 16 * lane;
        const u32x4_t v = *reinterpret_cast<const u32x4_t*>(src);
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[fn][fm][4 * q + e] += __uint_as_float(v[e]);
      }
    }
  }

  // epilogue: out = bf16(fp32(fma(alpha, acc, bias))), alpha = aA * aB in
  // FP32.  Lane (li, g) holds, per MFMA tile, row m = li and the column runs
  // 8k + 4g .. 8k + 4g + 3 (k = 0..3); swapping halves with the lane 32 apart
  // gives each lane two runs of 8 consecutive columns (16-byte stores).
  // Stores go through a buffer resource covering the tile's valid rows, so
  // rows past M are dropped by the hardware range check; columns past N get
  // an offset beyond the range.
  const float alpha = a_gs[0] * b_gs[0];
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
#pragma unroll
  for (int fm = 0; fm < kFr; ++fm) {
    const uint32_t mrow = (uint32_t)((wm * kWT + fm * 32 + li) * N);
#pragma unroll
    for (int fn = 0; fn < kFr; ++fn) {
      const int nb = wn * kWT + fn * 32;
      float v[16];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint2 b2 = *reinterpret_cast<const uint2*>(&lbias[nb + 8 * k + 4 * g]);
        const float bv[4] = {__uint_as_float(b2.x << 16), __uint_as_float(b2.x & 0xFFFF0000u),
                             __uint_as_float(b2.y << 16), __uint_as_float(b2.y & 0xFFFF0000u)};
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * k + q] = __builtin_fmaf(alpha, acc[fn][fm][4 * k + q], bv[q]);
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
  }
}

// Compute units of the current device (256 on MI355X), queried once per
// device.
int device_cu_count() {
  constexpr int kMaxDevices = 64;
  static int cached[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int v = __atomic_load_n(&cached[dev], __ATOMIC_RELAXED);
  if (v <= 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    __atomic_store_n(&cached[dev], v, __ATOMIC_RELAXED);
  }
  return v;
}

// Whether 128 x 128 tiles finish sooner than 256 x 256 ones: one workgroup
// per CU at a time, so a launch takes about ceil(tiles / CUs) rounds of one
// tile's time, and a small tile takes kSmallTileCost of a large one's
// (measured; ideal would be 1/4).
bool small_tiles_pay(int64_t tiles256, int64_t tiles128) {
#ifndef SOLFP4_SMALL_TILE_COST
#define SOLFP4_SMALL_TILE_COST 0.46
#endif
  const int64_t cus = device_cu_count();
  const double big = (double)((tiles256 + cus - 1) / cus);
  const double small = (double)((tiles128 + cus - 1) / cus) * SOLFP4_SMALL_TILE_COST;
  return small < big;
}

// Quadrants of the last round split in K halves from this many stages on
// (measured: 8 stages 0.92x of whole quadrants, 18 stages 1.01x, 24-96
// stages 1.05-1.10x).
constexpr int64_t kQuadHalvesMinStages = 16;

SplitPlan plan_split(int64_t tiles, int64_t nstages, double fixed_cost, double part_cost,
                     size_t part_tile_bytes, bool quad_ok) {
  SplitPlan plan;
  plan.dp_tiles = tiles;
  plan.stages = nstages;
  const int64_t cus = device_cu_count();
  const int64_t rem = tiles % cus;
  if (rem == 0) return plan;
  if (quad_ok && tiles > cus && 4 * rem <= cus) {
    plan.quad = true;
    plan.rem_tiles = rem;
    plan.dp_tiles = tiles - rem;
    if (8 * rem <= cus && nstages >= kQuadHalvesMinStages) {
      const int64_t quads = 4 * rem;
      plan.splits = 2;
      plan.stages = (nstages + 1) / 2;
      plan.bytes = ((size_t)quads * 8 + 255) / 256 * 256 + (size_t)quads * 2 * (part_tile_bytes / 4);
    }
    return plan;
  }
  if (nstages < 2) return plan;
  // two K halves per remainder tile (the kernels add exactly two), when
  // both halves of every remainder tile fit in one round
  if (2 * rem > cus) return plan;
  const double whole = (double)nstages + fixed_cost;
  const double halves = (double)((nstages + 1) / 2) + fixed_cost + 2.0 * part_cost;
  if (!(halves < whole)) return plan;
  plan.stages = (nstages + 1) / 2;
  plan.splits = 2;
  plan.rem_tiles = rem;
  plan.dp_tiles = tiles - rem;
  plan.bytes = ((size_t)rem * 8 + 255) / 256 * 256 + (size_t)(rem * plan.splits) * part_tile_bytes;
  return plan;
}

SplitK split_args(const SplitPlan& plan, void* workspace) {
  SplitK a{};
  a.dp_tiles = (int)plan.dp_tiles;
  a.splits = (int)plan.splits;
  a.stages = (int)plan.stages;
  if (plan.active()) {
    a.slots = static_cast<uint64_t*>(workspace);
    a.part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                      ((size_t)plan.rem_tiles * 8 + 255) / 256 * 256);
  }
  return a;
}

// Timing estimates in units of one K stage of the NVFP4 lane kernel
// (measured about 5.1k cycles on a busy chip): prologue plus epilogue of a
// tile about 3.3 stages; writing one 256 KB partial tile, or reading one
// back, with every remainder workgroup doing so at once, 2-3.5 stages.
#ifndef SOLFP4_SPLIT_FIXED
#define SOLFP4_SPLIT_FIXED 3.3
#endif
#ifndef SOLFP4_SPLIT_PART
#define SOLFP4_SPLIT_PART 2.5
#endif
// The same for 128 x 128 tiles, in units of their own (latency-bound) stage:
// fitted to the measured gain of the split on the 128-token 3072 -> 3072
// (1.32x), 128-token 1152 -> 1152 at K = 4608 (1.49x), 512-token 2240 ->
// 2240 (1.16x) and 128-token 1152 -> 1152 (none) layers.
#ifndef SOLFP4_SPLIT_FIXED_SMALL
#define SOLFP4_SPLIT_FIXED_SMALL 9.0
#endif
#ifndef SOLFP4_SPLIT_PART_SMALL
#define SOLFP4_SPLIT_PART_SMALL 2.0
#endif

// The lane kernel is the one that splits, on either tile size.
// The lane kernel takes K % 128 == 0 and K % 64 == 32 always.  At
// K % 128 == 64 (a half last stage) the workgroup-shared kernel is 1-2%
// faster on whole rounds of 256 x 256 tiles (the 8192-token 2240 -> 6720
// and 2240 -> 5600 layers), so the lane kernel takes those shapes only
// where its 128 x 128 tiles or its split last round apply (2240 -> 2240:
// 1.08x; 300 x 260: 2.6x).  K % 32 == 16 is the shared kernel's alone.
static SplitPlan gemm_plan(int64_t M, int64_t N, int64_t K, bool* small_out) {
  SplitPlan plan;
  const bool lane_ok = K % 32 == 0;
  const int64_t t256 = ((M + 255) / 256) * ((N + 255) / 256);
  const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
  const bool small = lane_ok && small_tiles_pay(t256, t128);
  if (small_out) *small_out = small;
  plan.dp_tiles = small ? t128 : t256;
  if (!lane_ok) return plan;
  const int64_t nstages = (K + kLBK - 1) / kLBK;
  if (small)
    return plan_split(t128, nstages, SOLFP4_SPLIT_FIXED_SMALL, SOLFP4_SPLIT_PART_SMALL, 128 * 128 * 4,
                      false);
  return plan_split(t256, nstages, SOLFP4_SPLIT_FIXED, SOLFP4_SPLIT_PART, 256 * 256 * 4, true);
}

size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0 || use_small_gemm(M, N, K)) return 0;
  return gemm_plan(M, N, K, nullptr).bytes;
}

void describe_gemm(int64_t M, int64_t N, int64_t K, bool with_workspace, int* kernel, int* tile,
                   int64_t* workgroups, int* splits) {
  if (use_wavek_gemm(M, N, K)) {
    *kernel = SOLFP4_KERNEL_NVFP4_WAVEK;
    *tile = 32;
    *splits = 1;
    *workgroups = ((M + 31) / 32) * ((N + 31) / 32);
    return;
  }
  if (use_small_gemm(M, N, K)) {
    *kernel = SOLFP4_KERNEL_NVFP4_SMALL;
    *tile = 64;
    *splits = 1;
    *workgroups = ((M + 63) / 64) * ((N + 63) / 64);
    return;
  }
  bool small = false;
  SplitPlan plan = gemm_plan(M, N, K, &small);
  const bool split = plan.active() && with_workspace;
  const bool lane = K % kLBK == 0 || K % 64 == 32 || (K % 32 == 0 && (small || split || plan.quad));
  *kernel = lane ? SOLFP4_KERNEL_NVFP4_LANE : SOLFP4_KERNEL_NVFP4_SHARED;
  *tile = small ? 128 : 256;
  *splits = split ? (int)plan.splits : 1;
  const int64_t tiles = small ? ((M + 127) / 128) * ((N + 127) / 128)
                              : ((M + 255) / 256) * ((N + 255) / 256);
  if (plan.quad)
    *workgroups = plan.dp_tiles + 4 * plan.rem_tiles * (split ? plan.splits : 1);
  else
    *workgroups = split ? plan.dp_tiles + plan.rem_tiles * plan.splits : tiles;
}

// The small-tile kernel takes the shapes whose 64 x 64 tiles fit in one
// round (one workgroup per CU).  Measured against the 128 x 128 / 256 x 256
// kernels, graph-replayed: 128 x 1152 x 1152 6.96 vs 11.46 us, 128 x 3072 x
// 3072 13.3 vs 17.8, 768 x 1152 x 1152 7.4 vs 11.6; past one round it loses
// (384 x 3072 x 3072 0.96x, 1024 x 3072 x 3072 0.85x, 128 x 9216 x 3072
// 0.95x) or gains little (1024 x 1152 x 1152 1.16x at 288 tiles).
bool use_small_gemm(int64_t M, int64_t N, int64_t K) {
  if (K % kLBK != 0 || M <= 0 || N <= 0 || K <= 0) return false;
  const int64_t t64 = ((M + 63) / 64) * ((N + 63) / 64);
  return t64 <= device_cu_count();
}

// Among the shapes the small-tile kernel takes, the wave-K kernel (32 x 32
// tiles, each workgroup's K stages dealt to its four waves) where its
// estimated time is lower.  Its LDS lets two workgroups share a CU, so a
// launch of t tiles puts ceil(t / CUs) of them on the busiest CU, and each
// one past the first adds 0.52 of a lone workgroup's time (two at once run
// 1.28-1.6x as long as one alone, longer K towards the top).  A lone
// workgroup costs a fixed part plus one per stage of its longest wave; the
// 64 x 64 kernel never takes more than one round here.  The costs, in
// microseconds, are fitted to measurements on one box (50 launches per
// timing): the 64 x 64 kernel 3.35 + 0.40 per stage, the wave-K kernel
// 2.83 + 0.52 per stage (128 x 1152 x 1152 6.9 -> 4.4 us, 128 x 3072 x 12288
// 42.4 -> 23.6 at 384 tiles, 256 x 3072 x 3072 13.7 -> 12.4 at 768; kept on
// 64 x 64 tiles: 512 x 2048 x 2048, 10.6 against 11.9 at 1024 tiles).  On
// 15 shapes of 7 to 512 tokens the estimate picks the faster kernel on all
// but one, 128 x 6144 x 1536, where wave-K would be 3% faster.
bool use_wavek_gemm(int64_t M, int64_t N, int64_t K) {
  if (!use_small_gemm(M, N, K)) return false;
  const int64_t cus = device_cu_count();
  const int64_t t32 = ((M + 31) / 32) * ((N + 31) / 32);
  const int64_t stages = K / kLBK;
  const double small = 3.35 + 0.40 * (double)stages;
  const double per_cu = (double)((t32 + cus - 1) / cus);
  const double wavek = (1.0 + 0.52 * (per_cu - 1.0)) * (2.83 + 0.52 * (double)((stages + 3) / 4));
  return wavek < small;
}

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                       const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                       const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  if (use_wavek_gemm(M, N, K))
    return launch_gemm_wavek(a_codes, a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K,
                             stream);
  if (use_small_gemm(M, N, K))
    return launch_gemm_small(a_codes, a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K,
                             nullptr, stream);
  return launch_gemm_regular(a_codes, a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K,
                             workspace, workspace_bytes, stream);
}

// The whole tiles in one launch of 256 x 256 tiles, then the last round's
// tiles as four 128 x 128 quadrants each (their K halves added through the
// workspace when the plan splits them).  The quadrants run the same MFMAs
// per output element in the same order as whole tiles (or, split, as two K
// halves of a whole tile), so the output is bit-identical to the one-launch
// plan that leaves those tiles whole (or splits them in two).  Measured on
// one box against the one-launch plans: shapes with one round plus 8 to 64
// tiles 1.04-1.20x (K = 256 to 12288), 18432 x 9216 x 3072 1.017x.
static hipError_t launch_gemm_quad(const uint8_t* a_codes, const uint8_t* a_scales,
                                   const float* a_gs, const uint8_t* b_codes,
                                   const uint8_t* b_scales, const float* b_gs,
                                   const uint16_t* bias, uint16_t* out, int64_t M, int64_t N,
                                   int64_t K, const SplitPlan& plan, void* workspace,
                                   hipStream_t stream) {
  const bool vec = N % 8 == 0, full = K % kLBK == 0;
  const int all_stages = (int)((K + kLBK - 1) / kLBK);
  SplitK whole{};
  whole.dp_tiles = (int)plan.dp_tiles;
  whole.splits = 1;
  whole.stages = all_stages;
  const int64_t quads = 4 * plan.rem_tiles;
  SplitK tail{};
  tail.quad_base = (int)plan.dp_tiles;
  if (plan.active()) {
    tail.dp_tiles = 0;
    tail.splits = (int)plan.splits;
    tail.stages = (int)plan.stages;
    tail.slots = static_cast<uint64_t*>(workspace);
    tail.part = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                         ((size_t)quads * 8 + 255) / 256 * 256);
  } else {
    tail.dp_tiles = (int)quads;
    tail.splits = 1;
    tail.stages = all_stages;
  }
  const dim3 block(kLThreads);
#define SOLFP4_QUAD_LAUNCH(V, F, W, G, S)                                                       \
  launch_kernel(nvfp4_gemm_lane_kernel<V, F, W>, G, block, stream, a_codes, a_scales, a_gs,     \
                b_codes, b_scales, b_gs, bias, out, M, N, K, S)
#define SOLFP4_QUAD_PICK(W, G, S)                                                               \
  (vec && full ? SOLFP4_QUAD_LAUNCH(true, true, W, G, S)                                       \
   : full      ? SOLFP4_QUAD_LAUNCH(false, true, W, G, S)                                      \
   : vec       ? SOLFP4_QUAD_LAUNCH(true, false, W, G, S)                                      \
               : SOLFP4_QUAD_LAUNCH(false, false, W, G, S))
  if (plan.dp_tiles > 0) {
    const hipError_t e = SOLFP4_QUAD_PICK(128, dim3((unsigned)plan.dp_tiles), whole);
    if (e != hipSuccess) return e;
  }
  const hipError_t e = SOLFP4_QUAD_PICK(64, dim3((unsigned)(quads * tail.splits)), tail);
#undef SOLFP4_QUAD_PICK
#undef SOLFP4_QUAD_LAUNCH
  return e;
}

hipError_t launch_gemm_regular(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                               const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  const dim3 grid((unsigned)tiles);
  const bool vec = N % 8 == 0;
  // Kernel choice as in gemm_plan (at K = 5600, where the shared kernel
  // must take its unaligned path, the lane kernel is 1.46x faster).
  bool small = false;
  SplitPlan plan = gemm_plan(M, N, K, &small);
  if (plan.active() && (workspace == nullptr || workspace_bytes < plan.bytes)) {
    // no room: every tile (or quadrant) whole
    const bool quad = plan.quad;
    const int64_t rem = plan.rem_tiles;
    plan = SplitPlan{};
    plan.dp_tiles = small ? ((M + 127) / 128) * ((N + 127) / 128) : ((M + 255) / 256) * ((N + 255) / 256);
    plan.stages = (K + kLBK - 1) / kLBK;
    if (quad) {
      plan.quad = true;
      plan.rem_tiles = rem;
      plan.dp_tiles -= rem;
    }
  }
  if (plan.quad)
    return launch_gemm_quad(a_codes, a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K,
                            plan, workspace, stream);
  if (K % kLBK == 0 || K % 64 == 32 || (K % 32 == 0 && (small || plan.active()))) {
    const SplitK split = split_args(plan, workspace);
    const dim3 lgrid((unsigned)(plan.dp_tiles + plan.rem_tiles * plan.splits));
#define SOLFP4_LANE_LAUNCH(V, F, W)                                                           \
  launch_kernel(nvfp4_gemm_lane_kernel<V, F, W>, lgrid, dim3(kLThreads), stream, a_codes,      \
                a_scales, a_gs, b_codes, b_scales, b_gs, bias, out, M, N, K, split)
    const bool full = K % kLBK == 0;
    hipError_t e;
    if (small) {
      if (vec && full) e = SOLFP4_LANE_LAUNCH(true, true, 64);
      else if (full) e = SOLFP4_LANE_LAUNCH(false, true, 64);
      else if (vec) e = SOLFP4_LANE_LAUNCH(true, false, 64);
      else e = SOLFP4_LANE_LAUNCH(false, false, 64);
    } else {
      if (vec && full) e = SOLFP4_LANE_LAUNCH(true, true, 128);
      else if (full) e = SOLFP4_LANE_LAUNCH(false, true, 128);
      else if (vec) e = SOLFP4_LANE_LAUNCH(true, false, 128);
      else e = SOLFP4_LANE_LAUNCH(false, false, 128);
    }
#undef SOLFP4_LANE_LAUNCH
    return e;
  }
  const dim3 block(kGemmThreads);
  const bool fast = K % kBK == 0;
#define SOLFP4_SHARED_LAUNCH(F, V)                                                             \
  launch_kernel(nvfp4_gemm_kernel<F, V>, grid, block, stream, a_codes, a_scales, a_gs, b_codes, \
                b_scales, b_gs, bias, out, M, N, K)
  if (fast && vec) return SOLFP4_SHARED_LAUNCH(true, true);
  if (fast) return SOLFP4_SHARED_LAUNCH(true, false);
  if (vec) return SOLFP4_SHARED_LAUNCH(false, true);
  return SOLFP4_SHARED_LAUNCH(false, false);
#undef SOLFP4_SHARED_LAUNCH
}

}  // namespace solfp4
