// Device-side types and helpers shared by the solfp4 kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace solfp4 {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));
typedef unsigned short ushort2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// An LDS address, as the LDS-destination buffer loads take it.
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// s_waitcnt with vmcnt(V) and lgkmcnt(L) (expcnt not waited on).
template <int V, int L>
__device__ __forceinline__ void wait_counts() {
  static_assert(V >= 0 && V < 64 && L >= 0 && L < 16, "counter range");
  __builtin_amdgcn_s_waitcnt((V & 15) | ((V >> 4) << 14) | (7 << 4) | (L << 8));
}

// Per-tensor scale divisor: largest E2M1 magnitude times largest E4M3 value.
constexpr float kAlphaDivisor = 6.0f * 448.0f;

__device__ __forceinline__ ushort2_t as_us2(uint32_t v) { return __builtin_bit_cast(ushort2_t, v); }
__device__ __forceinline__ uint32_t as_u32(ushort2_t v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ half2_t as_h2(uint32_t v) { return __builtin_bit_cast(half2_t, v); }
__device__ __forceinline__ uint32_t h2_as_u32(half2_t v) { return __builtin_bit_cast(uint32_t, v); }

// Largest BF16 magnitude (as its 15-bit pattern) among the two halves of
// each word, combined into a packed pair: |x| of non-negative floats orders
// like the integers of their bit patterns, so this max is exact.
__device__ __forceinline__ ushort2_t absmax_pair(ushort2_t acc, uint32_t w) {
  return __builtin_elementwise_max(acc, as_us2(w & 0x7FFF7FFFu));
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, off, kWave));
  return v;
}

// E4M3 (OCP E4M3FN) code of a non-negative binary32 value: nearest, ties to
// the even code, saturating at 448.  Normal range: round the binary32
// significand to 3 bits with the carry allowed into the exponent; subnormal
// range (< 2^-6): the E4M3 grid is k * 2^-9, so round s * 512 (exact) to an
// integer.  Branch free: both candidates are formed and one is selected.
__device__ __forceinline__ uint32_t e4m3_rne_sat(float s) {
  const uint32_t u = __float_as_uint(s);
  const uint32_t normal = ((u + 0x7FFFFu + ((u >> 20) & 1u)) >> 20) - (120u << 3);
  const uint32_t sub = (uint32_t)__builtin_rintf(s * 512.0f);
  const uint32_t code = s < 0x1p-6f ? sub : normal;
  return s < 448.0f ? code : 0x7Eu;
}

// Exact value of an E4M3 byte (finite codes 0x00..0x7E).
__device__ __forceinline__ float e4m3_value(uint32_t c) {
  return c < 8u ? (float)c * 0x1p-9f : __uint_as_float((c + (120u << 3)) << 20);
}

// Round binary32 to BF16 bits (nearest, ties to even).  Finite inputs.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// A buffer resource from wave-uniform values: readfirstlane pins the base
// and size to scalar registers, so loads through it need no per-lane
// descriptor handling.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t uniform_rsrc(const void* base, int64_t bytes) {
  const uint64_t p = (uint64_t)base;
  uint32_t lo = (uint32_t)p, hi = (uint32_t)(p >> 32);
  int n = (int)bytes;
  // The empty asm hides that the words are already uniform, so the compiler
  // cannot drop the readfirstlane: a uniform value that was computed by
  // vector instructions (64-bit min and multiply) and left in vector
  // registers would put a waterfall loop around every access through the
  // descriptor.
  asm volatile("" : "+v"(lo), "+v"(hi), "+v"(n));
  lo = __builtin_amdgcn_readfirstlane(lo);
  hi = __builtin_amdgcn_readfirstlane(hi);
  n = __builtin_amdgcn_readfirstlane(n);
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, n,
                                           0x00020000);
}

// Tile order: consecutive workgroups are dispatched round-robin over the 8
// XCDs, each with its own L2.  Remap so each XCD gets a contiguous range of
// tile ids, then walk tiles in groups of kGroupM row-tiles so the tiles an
// XCD runs together share A rows and B columns.
constexpr int kXcds = 8;
constexpr int kGroupM = 8;

// Tile b of that order (b in [0, tiles_m * tiles_n)).
__device__ __forceinline__ void tile_coords_at(int b, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int total = tiles_m * tiles_n;
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

__device__ __forceinline__ void tile_coords(int tiles_m, int tiles_n, int& tm, int& tn) {
  tile_coords_at(blockIdx.x, tiles_m, tiles_n, tm, tn);
}

}  // namespace solfp4
