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
// Dequantization is shared by the whole workgroup: per K stage each pair of
// threads owns one row of the A tile and one row of the B tile, each thread
// converting 32 codes of each to FP16 and storing them to LDS, where all
// eight waves read their MFMA operands.  Each element is converted once per
// 256 x 256 output tile.
// The conversion avoids the (half-rate) FP4 convert instructions: E2M1 values
// have at most 2 significant bits, so the low byte of their FP16 encoding is
// zero and the high byte comes from an 8-entry byte table indexed with
// v_perm_b32 (sign bits are copied in by mask); one packed FP16 multiply then
// applies the E4M3 block scale.
//
// Tiling: 256 x 256 output tile per workgroup of 8 waves (2 x 4, two per
// SIMD so one wave's waits are covered by the other's MFMAs), each wave
// owning 128 x 64 (4 x 2 MFMA tiles of 32 x 32, accumulators in AGPRs); K
// advances 64 elements (4 NVFP4 blocks) per stage.  LDS holds two stages of
// FP16 A and B tiles (rows padded to 144 bytes: conflict-free 16-byte row
// accesses).  Packed codes for stage s+2 are fetched into registers while
// stage s runs its MFMAs and stage s+1 is converted into the other LDS
// buffer, so each stage ends with a single barrier.  The two threads of a
// row load its 32 code bytes (and 4 scale bytes) with one coalesced request.
// The MFMA's first operand is the weight tile, so each lane's accumulators
// hold runs of 4 consecutive output columns of one row; one lane swap with
// the partner 32 lanes away turns them into 16-byte runs for the stores.
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace solfp4 {

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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));

// Two FP32 values to a BF16 pair (round to nearest even), first in the low half.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_t{lo, hi}), bf16x2_t));
}

// High bytes of the FP16 encodings of the E2M1 magnitudes 0, .5, 1, 1.5, 2,
// 3, 4, 6 (their low bytes are 0), as the two source words of v_perm_b32.
constexpr uint32_t kLutLo = 0x3E3C3800u;
constexpr uint32_t kLutHi = 0x46444240u;

// 8 E2M1 codes (element 2j in the low nibble of byte j) times the block
// scale s2 = (s, s) in FP16, as 4 words of FP16 pairs (elements 2j, 2j+1).
__device__ __forceinline__ void dequant8(uint32_t w, uint32_t s2, uint32_t (&d)[4]) {
  // high bytes of the even elements (0, 2, 4, 6), signs in bit 7
  const uint32_t ev = __builtin_amdgcn_perm(kLutHi, kLutLo, w & 0x07070707u) |
                      ((w << 4) & 0x80808080u);
  // and of the odd elements (1, 3, 5, 7)
  const uint32_t od = __builtin_amdgcn_perm(kLutHi, kLutLo, (w >> 4) & 0x07070707u) |
                      (w & 0x80808080u);
  // interleave into FP16 pairs: [0, ev.byte j, 0, od.byte j]
  const half2_t s = as_h2(s2);
  d[0] = h2_as_u32(as_h2(__builtin_amdgcn_perm(od, ev, 0x040C000Cu)) * s);
  d[1] = h2_as_u32(as_h2(__builtin_amdgcn_perm(od, ev, 0x050C010Cu)) * s);
  d[2] = h2_as_u32(as_h2(__builtin_amdgcn_perm(od, ev, 0x060C020Cu)) * s);
  d[3] = h2_as_u32(as_h2(__builtin_amdgcn_perm(od, ev, 0x070C030Cu)) * s);
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
  const half2_t k256 = {(_Float16)256.0f, (_Float16)256.0f};
  const uint32_t c = (sc2 >> (8 * j)) & 0xFFu;
  const uint32_t s2 = h2_as_u32(as_h2((c << 7) | (c << 23)) * k256);
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

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                       const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                       const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                       hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
  const dim3 grid((unsigned)tiles), block(kGemmThreads);
  const bool fast = K % kBK == 0;
  const bool vec = N % 8 == 0;
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
