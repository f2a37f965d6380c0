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
// row reads and writes of 16 consecutive rows are bank-conflict free).
// Scale bytes are fetched 16 per row (four stages) by one thread per tile
// row with a single load, parked in LDS, and read by the lanes that use
// them: a lane needs the scale words of its own 8 rows, which would
// otherwise cost a 32-cache-line load per row and stage.
//
// Pipeline of stage s: the MFMAs read LDS buffer s%3; the codes of stage s+2,
// fetched during stage s-1, are stored to buffer (s+2)%3; the codes of stage
// s+3 are fetched; the scales and operands of the first K-step of stage s+1
// are read from LDS during the last K-step of stage s (that buffer was
// completed before the previous barrier), so the one barrier per stage does
// not expose LDS latency.
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
constexpr int kMxGroup = 4;                    // stages per scale group (16 scale bytes per row)
constexpr int kMxScaleStride = 5;              // words per row in LDS (4 + 1 pad: no bank conflicts)

struct MxSmem {
  uint8_t a[kMxBufs][kMxTile * kMxLdsRow];
  uint8_t b[kMxBufs][kMxTile * kMxLdsRow];
  uint32_t sc[2][2][kMxTile * kMxScaleStride];   // [group parity][operand][row, stage word]
  uint16_t bias[kMxTile];
};

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
// is kgroup i of stage 4 grp + j).  kFast: K % 128 == 0, so the bytes of every
// stage that is computed lie inside the row (a group reaching past K only
// covers stages that are never computed).  Otherwise byte loads, with kgroups
// past K zeroed (a stray 0xFF byte would be NaN).
template <bool kFast>
__device__ __forceinline__ u32x4_t load_scale_group(__amdgpu_buffer_rsrc_t src, uint32_t off,
                                                    int64_t kgroups, int grp) {
  if (kFast && kgroups % 16 == 0) return __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0);
  if (kFast) {
    u32x4_t v;
    v.x = __builtin_amdgcn_raw_buffer_load_b32(src, off, 0, 0);
    v.y = __builtin_amdgcn_raw_buffer_load_b32(src, off + 4, 0, 0);
    v.z = __builtin_amdgcn_raw_buffer_load_b32(src, off + 8, 0, 0);
    v.w = __builtin_amdgcn_raw_buffer_load_b32(src, off + 12, 0, 0);
    return v;
  }
  uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const uint32_t b = __builtin_amdgcn_raw_buffer_load_b8(src, off + i, 0, 0);
    w[i / 4] |= ((int64_t)grp * 16 + i < kgroups ? b : 0u) << (8 * (i % 4));
  }
  return u32x4_t{w[0], w[1], w[2], w[3]};
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
  // scale staging: thread t moves the scale group of tile row t of A and B
  const uint32_t sg_off = (uint32_t)(t * kgroups);
  // MFMA operand rows of this lane (LDS offsets)
  const int rd_a = (wm * kMxWaveTile + li) * kMxLdsRow + 16 * g;
  const int rd_b = (wn * kMxWaveTile + li) * kMxLdsRow + 16 * g;
  const int rs_a = (wm * kMxWaveTile + li) * kMxScaleStride;
  const int rs_b = (wn * kMxWaveTile + li) * kMxScaleStride;

  // the tile's bias (+0 without one: the accumulators start at +0 and never
  // hold -0, so adding +0 changes no result)
  smem.bias[t] = bias && n0 + t < N ? bias[n0 + t] : (uint16_t)0;

  floatx16_t acc[kMxFrags][kMxFrags];
#pragma unroll
  for (int i = 0; i < kMxFrags; ++i)
#pragma unroll
    for (int j = 0; j < kMxFrags; ++j) acc[i][j] = floatx16_t{};

  u32x4_t stg[2][2][kMxRounds];          // [set][operand][round]
  u32x4_t gsa, gsb;                      // scale group in flight
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
  auto load_group = [&](int grp) {
    gsa = load_scale_group<kFast>(rsa, sg_off + 16 * grp, kgroups, grp);
    gsb = load_scale_group<kFast>(rsb, sg_off + 16 * grp, kgroups, grp);
  };
  auto store_group = [&](int set) {
    uint32_t* da = &smem.sc[set][0][t * kMxScaleStride];
    uint32_t* db = &smem.sc[set][1][t * kMxScaleStride];
    da[0] = gsa.x; da[1] = gsa.y; da[2] = gsa.z; da[3] = gsa.w;
    db[0] = gsb.x; db[1] = gsb.y; db[2] = gsb.z; db[3] = gsb.w;
  };
  // this lane's scale words of `stage` (its 4 A rows and 4 B rows)
  auto read_scales = [&](uint32_t (&da)[kMxFrags], uint32_t (&db)[kMxFrags], int stage) {
    const int set = (stage / kMxGroup) & 1, w = stage % kMxGroup;
#pragma unroll
    for (int f = 0; f < kMxFrags; ++f) {
      da[f] = smem.sc[set][0][rs_a + f * 32 * kMxScaleStride + w];
      db[f] = smem.sc[set][1][rs_b + f * 32 * kMxScaleStride + w];
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
  // scale group 0 in LDS, the scales and operands of the first K-step
  load_group(0);
  load_codes(stg[0], 0);
  load_codes(stg[1], 1);
  store_group(0);
  store_codes(stg[0], 0);
  store_codes(stg[1], 1);
  load_codes(stg[0], 2);
  __syncthreads();
  read_scales(sca[0], scb[0], 0);
  read_frags(fa[0], fb[0], 0, 0);

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // Stage s with P = s % 4.  At P == 0 the scale group after the current one
  // is fetched into registers, at P == 2 it is stored into the LDS set of
  // its parity (last read two stages earlier); it is first read at P == 3,
  // for the next stage.
  auto run_stage = [&](auto phase, int s, int cur, int nxt, int wbuf) {
    constexpr int P = decltype(phase)::value;
    constexpr int C = P & 1;               // code and scale-word register set of stage s
    uint32_t ssa[kMxFrags], ssb[kMxFrags];
#pragma unroll
    for (int f = 0; f < kMxFrags; ++f) {
      ssa[f] = sca[C][f] >> (8 * g);
      ssb[f] = scb[C][f] >> (8 * g);
    }
    __builtin_amdgcn_sched_barrier(0);
    // K-step 0: fetch scales and codes ahead, read the operands of K-step 1,
    // store the codes of stage s+2
    if (P == 0) load_group(s / kMxGroup + 1);
    load_codes(stg[C ^ 1], s + 3);
    read_frags(fa[1], fb[1], cur, 1);
    mfma_step(S0{}, fa[0], fb[0], ssa, ssb);
    store_codes(stg[C], wbuf);
    if (P == 2) store_group((s / kMxGroup + 1) & 1);
#pragma unroll
    for (int i = 0; i < kMxFrags * kMxFrags; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // MFMA
      if (i < 8) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // DS read
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);                 // VMEM read
      if (i < 8) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      if (i >= 8) __builtin_amdgcn_sched_group_barrier(0x200, P == 2 ? 2 : 1, 0);   // DS write
    }
    __builtin_amdgcn_sched_barrier(0);
    // K-step 1, with the scales and operands of the next stage's first K-step
    read_scales(sca[C ^ 1], scb[C ^ 1], s + 1);
    read_frags(fa[0], fb[0], nxt, 0);
    mfma_step(S1{}, fa[1], fb[1], ssa, ssb);
#pragma unroll
    for (int i = 0; i < kMxFrags * kMxFrags; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
  };

  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  using P2 = std::integral_constant<int, 2>;
  using P3 = std::integral_constant<int, 3>;
  // LDS buffers rotate mod 3: stage s + j uses buffer (cur + j) % 3
  int s = 0, cur = 0;
  auto next3 = [](int b) { return b == 2 ? 0 : b + 1; };
  for (; s + 4 <= nstages; s += 4) {
    const int c1 = next3(cur), c2 = next3(c1);
    run_stage(P0{}, s, cur, c1, c2);
    run_stage(P1{}, s + 1, c1, c2, cur);
    run_stage(P2{}, s + 2, c2, cur, c1);
    run_stage(P3{}, s + 3, cur, c1, c2);
    cur = c1;   // (cur + 4) % 3
  }
  {
    const int rest = nstages - s;
    const int c1 = next3(cur), c2 = next3(c1);
    if (rest > 0) run_stage(P0{}, s, cur, c1, c2);
    if (rest > 1) run_stage(P1{}, s + 1, c1, c2, cur);
    if (rest > 2) run_stage(P2{}, s + 2, c2, cur, c1);
  }

  // epilogue: out = bf16(fp32(acc + bias)).  Lane (li, g) holds, per MFMA
  // tile, row m = li and the column runs 8k + 4g .. 8k + 4g + 3 (k = 0..3);
  // swapping halves with the lane 32 apart gives each lane two runs of 8
  // consecutive columns (16-byte stores).  Stores go through a buffer
  // resource covering the tile's valid rows, so rows past M are dropped by
  // the hardware range check; columns past N get an offset beyond the range.
  const __amdgpu_buffer_rsrc_t ro = uniform_rsrc(out + m0 * N, valid_a * N * 2);
  constexpr uint32_t kDrop = 0x80000000u;   // beyond any output range (N < 2^22)
#pragma unroll
  for (int fm = 0; fm < kMxFrags; ++fm) {
    const uint32_t mrow = (uint32_t)((wm * kMxWaveTile + fm * 32 + li) * N);
#pragma unroll
    for (int fn = 0; fn < kMxFrags; ++fn) {
      const int nb = wn * kMxWaveTile + fn * 32;
      float v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = acc[fn][fm][q];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const uint2 b2 = *reinterpret_cast<const uint2*>(&smem.bias[nb + 8 * k + 4 * g]);
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

hipError_t launch_mx_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
                          const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M,
                          int64_t N, int64_t K, hipStream_t stream) {
  if (M == 0 || N == 0) return hipSuccess;
  const int64_t tiles = ((M + kMxTile - 1) / kMxTile) * ((N + kMxTile - 1) / kMxTile);
  const dim3 grid((unsigned)tiles), block(kMxThreads);
  const bool fast = K % kMxBK == 0;
  const bool vec = N % 8 == 0;
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
