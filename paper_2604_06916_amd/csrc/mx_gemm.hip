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
// accumulators per lane in AGPRs); or, for GEMMs with too few such tiles to
// fill the chip, 128 x 128 tiles with 64 x 64 per wave, and for few tokens
// 64 x 64 tiles with one 32 x 32 MFMA tile per wave (mx_tile_edge chooses;
// every size runs the same sequence of MFMAs per output element, so the
// results are bit-identical across sizes; the wave-K kernel further down,
// for few tokens, sums in another order).  A last round of few 256 x 256
// tiles runs in a second launch as their 128 x 128 quadrants (quad_base;
// mx_quad_tiles).  K advances 128
// elements (64 code bytes per row) per stage.  Codes go from global memory straight into LDS by
// buffer loads with the LDS-destination bit (no register staging), into four
// stage buffers: the loads for stage s+3 are issued while stage s computes,
// so about two stages of time cover their latency.  A DMA instruction puts
// lane l's 16 bytes at slot l of a 1 KB block; each lane quad reads the 64
// contiguous bytes of one row, so the request coalesces (with the 16 rows in
// adjacent lanes instead, the memory pipeline spent most of its time on 64
// separate 16-byte accesses per instruction).  A block holds 16 rows as
// [row][piece] x 16 bytes, the piece order of row r swizzled by (r >> 2) & 3,
// so that the 16 lanes reading one piece of 16 consecutive rows for an MFMA
// operand hit every bank once (no bank conflicts, no padding).  The loads
// skip allocation in the per-CU vector cache (sc0): every line is used once
// from there.  Scale bytes are fetched 16 per row (four stages) by one
// thread per tile row with a single load, parked in LDS, and read by the
// lanes that use them: a lane needs the scale words of its own 8 rows,
// which would otherwise cost a 32-cache-line load per row and stage.
//
// Pipeline of stage s (buffer s % 4): the DMA of stage s+3 goes to the buffer
// read in stage s-1; the scales and operands of the first K-step of stage
// s+1 are read during the last K-step of stage s; the barrier that ends
// stage s first waits for this wave's DMA of stage s+2 (the barrier is a
// plain s_barrier with explicit counter waits: a release fence would wait
// for every DMA in flight).  Every wait counts only DMA instructions, which
// are always the youngest vector-memory operations when it is reached.

#include <type_traits>

#include "device_common.h"
#include "solfp4.h"
#include "kernels.h"

namespace solfp4 {

constexpr int kMxBK = 128;                     // K elements per stage
constexpr int kMxRowBytes = kMxBK / 2;         // code bytes per row per stage
constexpr int kMxThreads = 256;
constexpr int kMxBufs = 4;                     // LDS stage buffers (loads run 3 stages ahead)
constexpr int kMxGroup = 4;                    // stages per scale group (16 scale bytes per row)
constexpr int kMxScaleStride = 5;              // words per row in LDS (4 + 1 pad: no bank conflicts)

typedef int v4i_t __attribute__((ext_vector_type(4)));
typedef int v8i_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float floatx2_t __attribute__((ext_vector_type(2)));

// An FP4 matrix operand occupies the low 4 registers of the 8-register
// operand; the rest are ignored for this format and left undefined.
__device__ __forceinline__ v8i_t fp4_operand(u32x4_t x) {
  const v4i_t y = __builtin_bit_cast(v4i_t, x);
  return __builtin_shufflevector(y, y, 0, 1, 2, 3, -1, -1, -1, -1);
}

// Two FP32 values to a BF16 pair (round to nearest even), first in the low half.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2_t{lo, hi}), bf16x2_t));
}

// The 16 scale bytes of one row for stages 4 grp .. 4 grp + 3 (byte 4 j + i
// is kgroup i of stage 4 grp + j), one 16-byte load: buffer loads read
// correctly at any byte offset.  kFast: K % 128 == 0, so the bytes of every
// stage that is computed lie inside the row (a group reaching past K only
// covers stages that are never computed), and with rows of a multiple of 4
// bytes every 4-byte word of the load lies inside the operand's range or
// past it.  Otherwise kgroups past K are zeroed (a stray 0xFF byte would be
// NaN), and the range check, which drops a whole word straddling the end of
// the range, would drop in-range bytes of the one lane whose group reaches
// past the operand's last scale byte: that lane loads bytes instead.
template <bool kFast>
__device__ __forceinline__ u32x4_t load_scale_group(__amdgpu_buffer_rsrc_t src, uint32_t off,
                                                    int64_t kgroups, int grp, uint32_t range) {
  if (kFast) return __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
  u32x4_t v;
  if (off + 16 <= range || off >= range) {
    v = __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
  } else {
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 16; ++i)
      w[i / 4] |= __builtin_amdgcn_raw_buffer_load_b8(src, off + i, 0, 0) << (8 * (i % 4));
    v = u32x4_t{w[0], w[1], w[2], w[3]};
  }
  const int64_t valid = kgroups - (int64_t)grp * 16;   // bytes of this group inside K
  if (valid < 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int64_t n = valid - 4 * q;                  // valid bytes of word q
      v[q] &= n >= 4 ? 0xFFFFFFFFu : n <= 0 ? 0u : (1u << (8 * n)) - 1u;
    }
  }
  return v;
}


template <bool kFast, bool kVecOut, int kWT>
__global__ __launch_bounds__(kMxThreads, 1) void mxfp4_gemm_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const uint8_t* __restrict__ b_codes, const uint8_t* __restrict__ b_scales,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K, int quad_base) {
  static_assert(kWT == 128 || kWT == 64 || kWT == 32, "wave tile edge");
  constexpr int kT = 2 * kWT;                // output tile edge (M and N)
  constexpr int kFr = kWT / 32;              // 32 x 32 MFMA tiles per wave edge
  constexpr int kStage = kT * kMxRowBytes;   // one operand, one stage
  constexpr int kGw = kT / 64;               // 16-row DMA groups per wave and operand
  constexpr int kDma = 2 * kGw;              // DMA instructions per wave and stage
  // one array per stage buffer and operand, so the compiler can tell the
  // buffer being filled by DMA from the one being read
  __shared__ __attribute__((aligned(1024))) uint8_t la0[kStage], la1[kStage],
      la2[kStage], la3[kStage];
  __shared__ __attribute__((aligned(1024))) uint8_t lb0[kStage], lb1[kStage],
      lb2[kStage], lb3[kStage];
  __shared__ uint32_t lsc[2][2][kT * kMxScaleStride];   // [group parity][operand][row, word]
  __shared__ uint16_t lbias[kT];
  uint8_t* const abuf[kMxBufs] = {la0, la1, la2, la3};
  uint8_t* const bbuf[kMxBufs] = {lb0, lb1, lb2, lb3};

  const int tiles_m = (int)((M + kT - 1) / kT);
  const int tiles_n = (int)((N + kT - 1) / kT);
  int tm, tn;
  if constexpr (kWT == 64) {
    if (quad_base >= 0) {
      // quadrant blockIdx % 4 of 256 x 256 tile quad_base + blockIdx / 4
      const int b = (int)blockIdx.x;
      tile_coords_at(quad_base + b / 4, (int)((M + 255) / 256), (int)((N + 255) / 256), tm, tn);
      tm = 2 * tm + ((b >> 1) & 1);
      tn = 2 * tn + (b & 1);
      if ((int64_t)tm * kT >= M || (int64_t)tn * kT >= N) return;   // quadrant outside the output
    } else {
      tile_coords(tiles_m, tiles_n, tm, tn);
    }
  } else {
    tile_coords(tiles_m, tiles_n, tm, tn);
  }
  const int64_t m0 = (int64_t)tm * kT;
  const int64_t n0 = (int64_t)tn * kT;

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int wm = wave >> 1;
  const int wn = wave & 1;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t kgroups = K / 32;
  const int64_t valid_a = min<int64_t>(M - m0, kT);
  const int64_t valid_b = min<int64_t>(N - n0, kT);
  const __amdgpu_buffer_rsrc_t rca = uniform_rsrc(a_codes + m0 * row_bytes, valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const uint32_t range_sa = (uint32_t)(valid_a * kgroups);
  const uint32_t range_sb = (uint32_t)(valid_b * kgroups);
  const __amdgpu_buffer_rsrc_t rsa = uniform_rsrc(a_scales + m0 * kgroups, range_sa);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * kgroups, range_sb);

  // Code DMA: wave w fills 16-row groups 4 w .. 4 w + 3 of each operand.  In
  // one instruction lane quad l/4 reads the 64 contiguous bytes of row l/4 of
  // the group (so the request coalesces), and the hardware stores lane l's 16
  // bytes at slot l of the group's 1 KB: the group holds [row][piece] x 16
  // bytes, with the piece order of row r swizzled to piece ^ ((r >> 2) & 3) so
  // that 16 lanes reading one piece of 16 consecutive rows for an MFMA
  // operand hit all 64 banks once.
  const int dma_r = lane >> 2;
  const int piece = (lane & 3) ^ ((dma_r >> 2) & 3);
  const uint32_t dma_off = (uint32_t)((16 * kGw * wave + dma_r) * row_bytes + 16 * piece);
  const uint32_t group_stride = (uint32_t)(16 * row_bytes);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any buffer range: loads read zero,
                                            // stores are dropped (N < 2^22, K < 2^24)
  // scale staging: thread t moves the scale group of tile row t of A and B
  const uint32_t sg_off = (uint32_t)(t * kgroups);
  // MFMA operand slots of this lane: row r of the tile lives in group r / 16
  // at byte (r % 16) * 64 + 16 * (piece ^ ((r % 16) >> 2)); lane (li, g) of
  // K-step st reads piece 2 st + g
  const int swz = ((li & 15) >> 2) & 3;
  const int rd_a = ((wm * kWT + li) >> 4) * 1024 + (li & 15) * 64;
  const int rd_b = ((wn * kWT + li) >> 4) * 1024 + (li & 15) * 64;
  const int q_off[2] = {16 * (g ^ swz), 16 * ((2 + g) ^ swz)};
  const int rs_a = (wm * kWT + li) * kMxScaleStride;
  const int rs_b = (wn * kWT + li) * kMxScaleStride;

  // the tile's bias (+0 without one: the accumulators start at +0 and never
  // hold -0, so adding +0 changes no result); parked in LDS once the
  // prologue's loads are out, so its latency overlaps theirs
  constexpr bool kAllRows = kT == kMxThreads;   // every thread stages one tile row
  const bool row_thread = kAllRows || t < kT;
  const uint16_t bias_v = bias && row_thread && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc[kFr][kFr];
#pragma unroll
  for (int i = 0; i < kFr; ++i)
#pragma unroll
    for (int j = 0; j < kFr; ++j) acc[i][j] = floatx16_t{};

  u32x4_t gsa, gsb;                      // scale group in flight
  uint32_t sca[2][kFr], scb[2][kFr];
  u32x4_t fa[2][kFr], fb[2][kFr];

  // 8 DMA instructions per wave: stage `stage` into buffer `buf`
  auto dma_stage = [&](int buf, int stage) {
    const bool ok = kFast || (int64_t)stage * kMxBK + 32 * piece < K;
    const uint32_t base = dma_off + (uint32_t)stage * kMxRowBytes;
#pragma unroll
    for (int j = 0; j < kGw; ++j) {
      const uint32_t off = ok ? base + j * group_stride : kDrop;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rca, (lds_ptr_t)(abuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rcb, (lds_ptr_t)(bbuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
    }
  };
  // half h of the DMA of `stage` (kGw / 2 groups, kDma / 2 instructions; with
  // one group per wave, the A group in half 0 and the B group in half 1)
  auto dma_half = [&](int buf, int stage, int h) {
    const bool ok = kFast || (int64_t)stage * kMxBK + 32 * piece < K;
    const uint32_t base = dma_off + (uint32_t)stage * kMxRowBytes;
    if constexpr (kGw == 1) {
      const uint32_t off = ok ? base : kDrop;
      if (h == 0)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(abuf[buf] + wave * 1024), 16, off, 0, 0, 1);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(bbuf[buf] + wave * 1024), 16, off, 0, 0, 1);
      return;
    }
#pragma unroll
    for (int jj = 0; jj < kGw / 2; ++jj) {
      const int j = h * (kGw / 2) + jj;
      const uint32_t off = ok ? base + j * group_stride : kDrop;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rca, (lds_ptr_t)(abuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rcb, (lds_ptr_t)(bbuf[buf] + (kGw * wave + j) * 1024), 16, off, 0, 0, 1);
    }
  };
  auto load_group = [&](int grp) {
    gsa = load_scale_group<kFast>(rsa, sg_off + 16 * grp, kgroups, grp, range_sa);
    gsb = load_scale_group<kFast>(rsb, sg_off + 16 * grp, kgroups, grp, range_sb);
  };
  auto store_group = [&](int set) {
    if (row_thread) {
      uint32_t* da = &lsc[set][0][t * kMxScaleStride];
      uint32_t* db = &lsc[set][1][t * kMxScaleStride];
      da[0] = gsa.x; da[1] = gsa.y; da[2] = gsa.z; da[3] = gsa.w;
      db[0] = gsb.x; db[1] = gsb.y; db[2] = gsb.z; db[3] = gsb.w;
    }
  };
  // this lane's scale words of `stage` (its 4 A rows and 4 B rows)
  auto read_scales = [&](uint32_t (&da)[kFr], uint32_t (&db)[kFr], int stage) {
    const int set = (stage / kMxGroup) & 1, w = stage % kMxGroup;
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      da[f] = lsc[set][0][rs_a + f * 32 * kMxScaleStride + w];
      db[f] = lsc[set][1][rs_b + f * 32 * kMxScaleStride + w];
    }
  };
  auto read_frags = [&](u32x4_t (&da)[kFr], u32x4_t (&db)[kFr], int buf, int st) {
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      da[f] = *reinterpret_cast<const u32x4_t*>(abuf[buf] + rd_a + f * 2048 + q_off[st]);
      db[f] = *reinterpret_cast<const u32x4_t*>(bbuf[buf] + rd_b + f * 2048 + q_off[st]);
    }
  };
  // one K-step: lane group g supplies kgroup 2 st + g of the stage, i.e.
  // byte 2 st + g of its scale words; after the shift by 8 g the byte
  // select is the constant 2 st for every lane
  auto mfma_step = [&](auto step, const u32x4_t (&xa)[kFr], const u32x4_t (&xb)[kFr],
                       const uint32_t (&ssa)[kFr], const uint32_t (&ssb)[kFr]) {
    constexpr int st = decltype(step)::value;
#pragma unroll
    for (int fn = 0; fn < kFr; ++fn)
#pragma unroll
      for (int fm = 0; fm < kFr; ++fm)
        acc[fn][fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            fp4_operand(xb[fn]), fp4_operand(xa[fm]), acc[fn][fm], 4, 4, 2 * st,
            (int)ssb[fn], 2 * st, (int)ssa[fm]);
  };

  const int nstages = (int)((K + kMxBK - 1) / kMxBK);
  // prologue: scale group 0, stages 0-2 in flight; once stages 0 and 1 have
  // landed (stage 2 may still be in flight) the scales are parked and the
  // first K-step's scales and operands read
  load_group(0);
  dma_stage(0, 0);
  dma_stage(1, 1);
  dma_stage(2, 2);
  if (row_thread) lbias[t] = bias_v;
  wait_counts<kDma, 15>();
  store_group(0);
  wait_counts<kDma, 0>();
  __builtin_amdgcn_s_barrier();
  read_scales(sca[0], scb[0], 0);
  read_frags(fa[0], fb[0], 0, 0);

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // Stage s with P = s % 4, computed from buffer P.  The DMA of stage s+3
  // goes to buffer (P + 3) % 4, last read in stage s-1, half in each K-step.
  // At P == 0 the scale group after the current one is fetched into
  // registers (before the DMA, so that the DMA is always the youngest
  // vector-memory work the stage-end wait counts), at P == 2 it is stored into the
  // LDS set of its parity (last read two stages earlier); it is first read
  // at P == 3, for the next stage.  The barrier ending stage s waits for this
  // wave's DMA of stage s+2, so in stage s+1 both its own buffer and the
  // next one (read ahead) are complete.
  auto run_stage = [&](auto phase, int s) {
    constexpr int P = decltype(phase)::value;
    constexpr int C = P & 1;               // scale-word register set of stage s
    uint32_t ssa[kFr], ssb[kFr];
#pragma unroll
    for (int f = 0; f < kFr; ++f) {
      ssa[f] = sca[C][f] >> (8 * g);
      ssb[f] = scb[C][f] >> (8 * g);
    }
    __builtin_amdgcn_sched_barrier(0);
    // K-step 0: the scale group goes out before the DMA, so the wait that
    // ends the stage can count the DMA alone (the compiler may merge the
    // scale loads into fewer instructions than written: counting them would
    // let older DMA still be in flight)
    if (P == 0) load_group(s / kMxGroup + 1);
    // the stage's DMA goes out half in each K-step: issued at once it filled
    // the texture addresser's queues (15% of the kernel's cycles) and held
    // up the MFMA issue behind it (3% slower)
    dma_half((P + 3) % kMxBufs, s + 3, 0);
    read_frags(fa[1], fb[1], P, 1);
    mfma_step(S0{}, fa[0], fb[0], ssa, ssb);
    if (P == 2) store_group((s / kMxGroup + 1) & 1);
    if constexpr (kFr == 4) {
#pragma unroll
      for (int i = 0; i < kFr * kFr; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // MFMA
        if (i < 8) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // DS read
        if (i < 8) __builtin_amdgcn_sched_group_barrier(0x020, P == 0 ? 2 : 1, 0);   // VMEM read
        if (P == 2 && i >= 8) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);   // DS write
      }
    } else {
      // 4 MFMAs share the step's 4 LDS reads, kDma (+ scale) loads and the
      // 8 scale stores
#pragma unroll
      for (int i = 0; i < kFr * kFr; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, P == 0 ? 4 : 1, 0);
        if (P == 2) __builtin_amdgcn_sched_group_barrier(0x200, 2, 0);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    // K-step 1, with the scales and operands of the next stage's first K-step
    dma_half((P + 3) % kMxBufs, s + 3, 1);
    read_scales(sca[C ^ 1], scb[C ^ 1], s + 1);
    read_frags(fa[0], fb[0], (P + 1) % kMxBufs, 0);
    mfma_step(S1{}, fa[1], fb[1], ssa, ssb);
#pragma unroll
    for (int i = 0; i < kFr * kFr; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 16 / (kFr * kFr), 0);
      if (i < 8) __builtin_amdgcn_sched_group_barrier(0x020, kFr == 4 ? 1 : 2, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // this stage's kDma DMA instructions, the last vector-memory operations
    // it issued, may stay in flight; everything older (the DMA of stage s+2
    // and any scale loads) is complete
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

  // epilogue: out = bf16(fp32(acc + bias)).  Lane (li, g) holds, per MFMA
  // tile, row m = li and the column runs 8k + 4g .. 8k + 4g + 3 (k = 0..3);
  // swapping halves with the lane 32 apart gives each lane two runs of 8
  // consecutive columns (16-byte stores).  Stores go through a buffer
  // resource covering the tile's valid rows, so rows past M are dropped by
  // the hardware range check; columns past N get an offset beyond the range.
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
#pragma unroll
  for (int fm = 0; fm < kFr; ++fm) {
    const uint32_t mrow = (uint32_t)((wm * kWT + fm * 32 + li) * N);
#pragma unroll
    for (int fn = 0; fn < kFr; ++fn) {
      const int nb = wn * kWT + fn * 32;
      float v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = acc[fn][fm][q];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint2 b2 = *reinterpret_cast<const uint2*>(&lbias[nb + 8 * k + 4 * g]);
        v[4 * k + 0] += __uint_as_float(b2.x << 16);
        v[4 * k + 1] += __uint_as_float(b2.x & 0xFFFF0000u);
        v[4 * k + 2] += __uint_as_float(b2.y << 16);
        v[4 * k + 3] += __uint_as_float(b2.y & 0xFFFF0000u);
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

// Few tokens, K a multiple of 128: one 32 x 32 output tile per workgroup
// of four waves, wave w running stages w, w + 4, w + 8, ... of K, each wave
// with a pipeline of its own (codes and scale bytes by DMA into four LDS
// stage buffers of its own, three of its stages ahead, waiting on its own
// loads only: no barrier in the main loop).  With 64 x 64 tiles one K loop
// per wave runs on as many CUs as there are tiles; here four times as many
// workgroups each run a quarter of it, and their 72 KB of LDS lets two
// share a CU.  Waves 1-3 park their sums in their own stage buffers and
// wave 0 adds them in wave order before the epilogue, so the FP32 sums are
// formed in a different order than in the other tile sizes: results agree
// with them to FP32 summation error, bit for bit where the sums are exact.
constexpr int kMxWKTile = 32;
constexpr int kMxWKWaves = kMxThreads / kWave;
constexpr int kMxWKCodes = kMxWKTile * kMxRowBytes;   // 2 KB per operand and stage
constexpr int kMxWKBuf = 2 * kMxWKCodes + 512;        // codes, then 256 B of scale words per operand
constexpr int kMxWKScales = 2 * kMxWKCodes;
static_assert(kMxWKWaves * kMxBufs * kMxWKBuf <= 80 * 1024 - 64, "two workgroups per CU");
static_assert(4 * kWave * (int)sizeof(floatx4_t) <= kMxBufs * kMxWKBuf, "partial sums fit a wave's buffers");

template <bool kVecOut>
__global__ __launch_bounds__(kMxThreads, 2) void mxfp4_gemm_wavek_kernel(
    const uint8_t* __restrict__ a_codes, const uint8_t* __restrict__ a_scales,
    const uint8_t* __restrict__ b_codes, const uint8_t* __restrict__ b_scales,
    const uint16_t* __restrict__ bias, uint16_t* __restrict__ out, int64_t M, int64_t N,
    int64_t K) {
  __shared__ __attribute__((aligned(1024))) uint8_t lbuf[kMxWKWaves][kMxBufs][kMxWKBuf];
  __shared__ uint16_t lbias[kMxWKTile];

  const int tiles_m = (int)((M + kMxWKTile - 1) / kMxWKTile);
  const int tiles_n = (int)((N + kMxWKTile - 1) / kMxWKTile);
  int tm, tn;
  tile_coords(tiles_m, tiles_n, tm, tn);
  const int64_t m0 = (int64_t)tm * kMxWKTile;
  const int64_t n0 = (int64_t)tn * kMxWKTile;
  const int nstages = (int)(K / kMxBK);

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int wave = t / kWave;
  const int li = lane & 31;
  const int g = lane >> 5;

  const int64_t row_bytes = K / 2;
  const int64_t kgroups = K / 32;
  const int64_t valid_a = min<int64_t>(M - m0, kMxWKTile);
  const int64_t valid_b = min<int64_t>(N - n0, kMxWKTile);
  const __amdgpu_buffer_rsrc_t rca = uniform_rsrc(a_codes + m0 * row_bytes, valid_a * row_bytes);
  const __amdgpu_buffer_rsrc_t rcb = uniform_rsrc(b_codes + n0 * row_bytes, valid_b * row_bytes);
  const __amdgpu_buffer_rsrc_t rsa = uniform_rsrc(a_scales + m0 * kgroups, valid_a * kgroups);
  const __amdgpu_buffer_rsrc_t rsb = uniform_rsrc(b_scales + n0 * kgroups, valid_b * kgroups);

  // this wave's stages: wave + 4 i for i < count
  const int count = nstages > wave ? (nstages - wave + kMxWKWaves - 1) / kMxWKWaves : 0;

  // code DMA as in the tiled kernel: lane quad l/4 reads the 64 bytes of row
  // l/4 of a 16-row group (rows past the operand read zero), lane l's 16
  // bytes land in slot l of the group's 1 KB, the piece order of row r
  // swizzled by (r >> 2) & 3
  const int dma_r = lane >> 2;
  const int piece = (lane & 3) ^ ((dma_r >> 2) & 3);
  const uint32_t dma_off = (uint32_t)(dma_r * row_bytes + 16 * piece);
  const uint32_t group_stride = (uint32_t)(16 * row_bytes);
  // operand slots of this lane (row li of A and of B): lane group g reads
  // piece 2 st + g in K-step st
  const int swz = ((li & 15) >> 2) & 3;
  const int rd = (li >> 4) * 1024 + (li & 15) * 64;
  const int q_off[2] = {16 * (g ^ swz), 16 * ((2 + g) ^ swz)};
  // scale DMA: lane l fetches the 4 scale bytes of row l % 32 for the stage
  // (kgroups 4 s .. 4 s + 3; lanes 32-63 repeat lanes 0-31), one
  // instruction per operand; rows past the operand read zero
  const uint32_t sc_off = (uint32_t)(li * kgroups);

  if (t < kMxWKTile) lbias[t] = bias && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc = floatx16_t{};

  // the loads of this wave's i-th stage into buffer B (6 instructions)
  auto issue = [&](auto buf, int i) {
    constexpr int B = decltype(buf)::value;
    const int stage = wave + kMxWKWaves * i;
    uint8_t* base = &lbuf[wave][B][0];
    const uint32_t off = dma_off + (uint32_t)stage * kMxRowBytes;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(base), 16, off, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rca, (lds_ptr_t)(base + 1024), 16, off + group_stride, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(base + kMxWKCodes), 16, off, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rcb, (lds_ptr_t)(base + kMxWKCodes + 1024), 16,
                                             off + group_stride, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, (lds_ptr_t)(base + kMxWKScales), 4,
                                             sc_off + 4 * stage, 0, 0, 1);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, (lds_ptr_t)(base + kMxWKScales + 256), 4,
                                             sc_off + 4 * stage, 0, 0, 1);
  };
  constexpr int kPerStage = 6;   // vector-memory instructions per stage

  // one stage from buffer B: per K-step st the lane's code pieces of A and
  // B and byte 2 st + g of its rows' scale words (brought to byte 2 st by a
  // shift of 8 g, so the byte select is a constant), then one MFMA
  auto compute = [&](auto buf) {
    constexpr int B = decltype(buf)::value;
    const uint8_t* base = &lbuf[wave][B][0];
    const u32x4_t xa0 = *reinterpret_cast<const u32x4_t*>(base + rd + q_off[0]);
    const u32x4_t xb0 = *reinterpret_cast<const u32x4_t*>(base + kMxWKCodes + rd + q_off[0]);
    const u32x4_t xa1 = *reinterpret_cast<const u32x4_t*>(base + rd + q_off[1]);
    const u32x4_t xb1 = *reinterpret_cast<const u32x4_t*>(base + kMxWKCodes + rd + q_off[1]);
    const uint32_t* sw = reinterpret_cast<const uint32_t*>(base + kMxWKScales);
    const int ssa = (int)(sw[li] >> (8 * g));
    const int ssb = (int)(sw[64 + li] >> (8 * g));
    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fp4_operand(xb0), fp4_operand(xa0), acc,
                                                          4, 4, 0, ssb, 0, ssa);
    acc = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fp4_operand(xb1), fp4_operand(xa1), acc,
                                                          4, 4, 2, ssb, 2, ssa);
  };

  // stage i (buffer i % 4): the loads of stage i+3 go into the buffer read
  // in stage i-1, whose LDS reads the wait at the end of that stage
  // completed; then wait until stage i's loads have landed
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using B2 = std::integral_constant<int, 2>;
  using B3 = std::integral_constant<int, 3>;
  auto run = [&](auto buf, int i) {
    constexpr int B = decltype(buf)::value;
    if (i + 3 < count) {
      issue(std::integral_constant<int, (B + 3) % kMxBufs>{}, i + 3);
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
  for (int w = 1; w < kMxWKWaves; ++w)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const floatx4_t p = reinterpret_cast<const floatx4_t*>(&lbuf[w][0][0])[q * kWave + lane];
      acc[4 * q] += p[0];
      acc[4 * q + 1] += p[1];
      acc[4 * q + 2] += p[2];
      acc[4 * q + 3] += p[3];
    }

  // epilogue: out = bf16(fp32(acc + bias)), stored as in the tiled kernel
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
  const uint32_t mrow = (uint32_t)(li * N);
  float v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) v[q] = acc[q];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint2 b2 = *reinterpret_cast<const uint2*>(&lbias[8 * k + 4 * g]);
    v[4 * k + 0] += __uint_as_float(b2.x << 16);
    v[4 * k + 1] += __uint_as_float(b2.x & 0xFFFF0000u);
    v[4 * k + 2] += __uint_as_float(b2.y << 16);
    v[4 * k + 3] += __uint_as_float(b2.y & 0xFFFF0000u);
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

hipError_t launch_mx_gemm_wavek(const uint8_t* a_codes, const uint8_t* a_scales,
                                const uint8_t* b_codes, const uint8_t* b_scales,
                                const uint16_t* bias, uint16_t* out, int64_t M, int64_t N,
                                int64_t K, hipStream_t stream) {
  const int64_t tiles = ((M + kMxWKTile - 1) / kMxWKTile) * ((N + kMxWKTile - 1) / kMxWKTile);
  const dim3 grid((unsigned)tiles), block(kMxThreads);
  return N % 8 == 0 ? launch_kernel(mxfp4_gemm_wavek_kernel<true>, grid, block, stream, a_codes,
                                    a_scales, b_codes, b_scales, bias, out, M, N, K)
                    : launch_kernel(mxfp4_gemm_wavek_kernel<false>, grid, block, stream, a_codes,
                                    a_scales, b_codes, b_scales, bias, out, M, N, K);
}

// The output tile edge: one workgroup holds one tile at a time on its CU, so
// a launch takes about ceil(tiles / CUs) rounds of one tile's time.  Between
// 256 x 256 and 128 x 128 tiles small_tiles_pay decides; a 64 x 64 tile costs
// SOLFP4_MX_TINY_TILE_COST of a 128 x 128 one (measured on 64 to 512 tokens:
// 64 x 64 tiles 1.13-1.61x faster where they take at most two rounds and
// 128 x 128 tiles one, 0.80x at three rounds against one).  Where 256 x 256
// tiles win, 64 x 64 ones cannot: that takes three or more rounds of
// 128 x 128 tiles, and 64 x 64 tiles then need about four times as many.
int mx_tile_edge(int64_t M, int64_t N) {
#ifndef SOLFP4_MX_TINY_TILE_COST
#define SOLFP4_MX_TINY_TILE_COST 0.46
#endif
  const int64_t t256 = ((M + 255) / 256) * ((N + 255) / 256);
  const int64_t t128 = ((M + 127) / 128) * ((N + 127) / 128);
  if (!small_tiles_pay(t256, t128)) return 256;
  const int64_t t64 = ((M + 63) / 64) * ((N + 63) / 64);
  const int64_t cus = device_cu_count();
  const double r128 = (double)((t128 + cus - 1) / cus);
  const double r64 = (double)((t64 + cus - 1) / cus);
  return r64 * SOLFP4_MX_TINY_TILE_COST < r128 ? 64 : 128;
}

// Few tokens: the wave-K kernel where its 32 x 32 tiles fit one workgroup
// per CU and its estimated time is below the 64 x 64 kernel's (which then
// runs one round).  Both are bound by how fast a CU moves codes into LDS:
// a second workgroup on a CU nearly doubles the wave-K kernel's time on
// long K, so past one tile per CU it lost to 64 x 64 tiles on most shapes
// measured (0.62-0.91x at 384 to 1024 tiles; 1.03-1.14x at 280 to 350).
// Costs in microseconds, fitted to measurements on one box (50 launches
// per timing): 64 x 64 tiles 2.70 + 0.158 per stage, wave-K 2.64 + 0.28 per
// stage of its longest wave (128 x 1152 x 1152 4.30 -> 3.43 us,
// 16 x 3072 x 3072 6.09 -> 4.61, 128 x 1152 x 4608 8.26 -> 5.14; a single
// stage, 7 x 33 x 128, stays on 64 x 64 tiles: 2.79 against 2.92).
bool use_mx_wavek(int64_t M, int64_t N, int64_t K) {
  if (K % kMxBK != 0 || K == 0 || M <= 0 || N <= 0 || mx_tile_edge(M, N) != 64) return false;
  const int64_t t32 = ((M + kMxWKTile - 1) / kMxWKTile) * ((N + kMxWKTile - 1) / kMxWKTile);
  if (t32 > device_cu_count()) return false;
  const int64_t stages = K / kMxBK;
  const double tiled = 2.70 + 0.158 * (double)stages;
  const double wavek = 2.64 + 0.28 * (double)((stages + kMxWKWaves - 1) / kMxWKWaves);
  return wavek < tiled;
}

// 256 x 256 tiles of the last round that run as 128 x 128 quadrants in a
// launch of their own: the remainder R of the tiles over the CU count when
// there are more tiles than CUs and 4R quadrants fit one round, else 0.
// Quadrants run the same MFMAs per output element in the same order as
// whole tiles, so the output is the same bit for bit.
int64_t mx_quad_tiles(int64_t M, int64_t N) {
  if (mx_tile_edge(M, N) != 256) return 0;
  const int64_t tiles = ((M + 255) / 256) * ((N + 255) / 256);
  const int64_t cus = device_cu_count();
  const int64_t rem = tiles % cus;
  return tiles > cus && 4 * rem <= cus ? rem : 0;
}

void describe_mx_gemm(int64_t M, int64_t N, int64_t K, int* kernel, int* tile, int64_t* workgroups) {
  if (use_mx_wavek(M, N, K)) {
    *kernel = SOLFP4_KERNEL_MXFP4_WAVEK;
    *tile = kMxWKTile;
    *workgroups = ((M + kMxWKTile - 1) / kMxWKTile) * ((N + kMxWKTile - 1) / kMxWKTile);
    return;
  }
  const int edge = mx_tile_edge(M, N);
  *kernel = SOLFP4_KERNEL_MXFP4;
  *tile = edge;
  *workgroups = ((M + edge - 1) / edge) * ((N + edge - 1) / edge) + 3 * mx_quad_tiles(M, N);
}

hipError_t launch_mx_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
                          const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M,
                          int64_t N, int64_t K, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  if (use_mx_wavek(M, N, K))
    return launch_mx_gemm_wavek(a_codes, a_scales, b_codes, b_scales, bias, out, M, N, K, stream);
  const int edge = mx_tile_edge(M, N);
  const int64_t tiles = ((M + edge - 1) / edge) * ((N + edge - 1) / edge);
  const int64_t quads = mx_quad_tiles(M, N);
  const dim3 block(kMxThreads);
  const bool fast = K % kMxBK == 0;
  const bool vec = N % 8 == 0;
#define SOLFP4_MX_LAUNCH(W, G, Q)                                                                \
  (fast ? (vec ? launch_kernel(mxfp4_gemm_kernel<true, true, W>, G, block, stream, a_codes,       \
                               a_scales, b_codes, b_scales, bias, out, M, N, K, Q)               \
               : launch_kernel(mxfp4_gemm_kernel<true, false, W>, G, block, stream, a_codes,      \
                               a_scales, b_codes, b_scales, bias, out, M, N, K, Q))              \
        : (vec ? launch_kernel(mxfp4_gemm_kernel<false, true, W>, G, block, stream, a_codes,      \
                               a_scales, b_codes, b_scales, bias, out, M, N, K, Q)               \
               : launch_kernel(mxfp4_gemm_kernel<false, false, W>, G, block, stream, a_codes,     \
                               a_scales, b_codes, b_scales, bias, out, M, N, K, Q)))
  hipError_t e;
  if (edge == 64) {
    e = SOLFP4_MX_LAUNCH(32, dim3((unsigned)tiles), -1);
  } else if (edge == 128) {
    e = SOLFP4_MX_LAUNCH(64, dim3((unsigned)tiles), -1);
  } else if (quads == 0) {
    e = SOLFP4_MX_LAUNCH(128, dim3((unsigned)tiles), -1);
  } else {
    // the whole tiles, then the last round's tiles as 128 x 128 quadrants
    e = SOLFP4_MX_LAUNCH(128, dim3((unsigned)(tiles - quads)), -1);
    if (e == hipSuccess)
      e = SOLFP4_MX_LAUNCH(64, dim3((unsigned)(4 * quads)), (int)(tiles - quads));
  }
#undef SOLFP4_MX_LAUNCH
  return e;
}

}  // namespace solfp4
