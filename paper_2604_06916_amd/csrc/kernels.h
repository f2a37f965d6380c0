// Internal launch interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>
#include <utility>

namespace solfp4 {

// Launch `kernel` and return the status of this launch alone (the runtime's
// own, not whatever error an earlier, unrelated call may have left for
// hipGetLastError to report).  Arguments are converted to the kernel's
// parameter types first.
template <typename... P, size_t... I>
hipError_t launch_impl(void (*kernel)(P...), dim3 grid, dim3 block, hipStream_t stream,
                       std::index_sequence<I...>, std::tuple<P...>& args) {
  void* argv[] = {static_cast<void*>(&std::get<I>(args))..., nullptr};
  return hipLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, 0, stream);
}

template <typename... P, typename... A>
hipError_t launch_kernel(void (*kernel)(P...), dim3 grid, dim3 block, hipStream_t stream,
                         A&&... args) {
  static_assert(sizeof...(P) == sizeof...(A), "argument count");
  std::tuple<P...> t(std::forward<A>(args)...);
  return launch_impl(kernel, grid, block, stream, std::index_sequence_for<P...>{}, t);
}

// First quantize pass: at most this many partial maxima (workspace words).
constexpr int kMaxPartials = 1024;
// Encode pass: grid-stride loop over at most this many workgroups (eight
// per compute unit: more only adds per-workgroup set-up and an uneven tail).
constexpr int64_t kEncodeMaxGrid = 2048;
// MXFP4 quantize: grid-stride loop over at most this many workgroups.
constexpr int64_t kMxQuantMaxGrid = 8192;

int amax_partial_count(int64_t n_elems);

// The allocation-free quantize's scratch: a file-scope device array of
// kScratchWords words (the amax pass's partial maxima), one per device.
constexpr int kScratchWords = kMaxPartials;
static_assert(kScratchWords * 4 <= 4096, "scratch stays at 4 KiB");
// Device address of this device's scratch (looked up once per device).
hipError_t scratch_address(uint32_t** out);

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                           uint8_t* scales, float* global_scale, uint32_t* partial,
                           hipStream_t stream);

// Compute units of the current device, queried once per device (host only).
int device_cu_count();

// Whether a GEMM should run on 128 x 128 output tiles rather than 256 x 256
// ones, given the tile counts of both (host only).
bool small_tiles_pay(int64_t tiles256, int64_t tiles128);

// Output tile edge (256, 128 or 64) of the tiled MXFP4 GEMM kernel (host only).
int mx_tile_edge(int64_t M, int64_t N);

// 256 x 256 tiles of an MXFP4 GEMM's last round that run as 128 x 128
// quadrants in a second launch (0: none; host only).
int64_t mx_quad_tiles(int64_t M, int64_t N);

// Whether an MXFP4 GEMM runs on the wave-K kernel (32 x 32 tiles, each
// workgroup's K stages dealt to its four waves; host only).
bool use_mx_wavek(int64_t M, int64_t N, int64_t K);

// Split-K for the last, partial round of 256 x 256 tiles.  A GEMM with T
// tiles on C compute units runs about ceil(T / C) rounds of one tile's time;
// when the last round holds only R = T mod C tiles, most of the chip idles
// through it.  Instead, workgroups [0, dp_tiles) take whole tiles and each
// of the R remainder tiles is computed as two K halves, one workgroup each
// (when 2R <= C); each half parks its FP32 partial sums in a workspace, and
// the second of the two to finish adds the other's sums to its own and runs
// the epilogue.  Which one is second: each half swaps its own 64-bit token
// (a fixed pattern times the tile and half) into the tile's slot, and the
// one that gets the other half's token back is second and clears the slot.
// This works whatever the slot held before the launch (other than one of
// the two tokens), so the workspace needs no clearing between calls.
struct SplitK {
  float* part;          // two FP32 partial tiles per remainder tile (2 x 256 KB
                        // for 256 x 256 tiles, 2 x 64 KB for 128 x 128)
  uint64_t* slots;      // one per remainder tile: 0 after every launch, or
                        // the token of the half that finished first
  int dp_tiles;         // workgroups that take whole tiles (all of them: no split)
  int splits;           // K ranges per remainder tile: 2 (1: no split)
  int stages;           // K stages of the first half (the second may have fewer)
  int quad_base = -1;   // 128 x 128 tiles only: >= 0 when this launch covers the 256 x 256
                        // tiles from this index on (in tile order), each as four quadrants
};

struct SplitPlan {
  int64_t dp_tiles = 0, rem_tiles = 0, splits = 1, stages = 0;
  size_t bytes = 0;      // workspace: slots (256-byte aligned), then partial sums
  // the rem_tiles 256 x 256 tiles after the dp_tiles whole ones run in a
  // launch of their own as four 128 x 128 quadrants each (splits: K ranges
  // per quadrant)
  bool quad = false;
  bool active() const { return splits > 1; }
};

// The plan for `tiles` output tiles of `nstages` K stages each.  With
// quad_ok (256 x 256 tiles), a last round of at most a quarter of the CUs'
// worth of tiles runs as their 128 x 128 quadrants, and with at most an
// eighth and at least kQuadHalvesMinStages stages each quadrant as two K
// halves.  Otherwise the remainder tiles are split in two K halves when the
// estimated last round, ceil(nstages / 2) + fixed_cost + 2 part_cost stages
// (a half, then writing its partial tile and reading the other's), beats
// nstages + fixed_cost.  A tile's FP32 partial sums take part_tile_bytes.
SplitPlan plan_split(int64_t tiles, int64_t nstages, double fixed_cost, double part_cost,
                     size_t part_tile_bytes, bool quad_ok);
SplitK split_args(const SplitPlan& plan, void* workspace);
// token of half h of remainder tile r: kSplitToken ^ (2 r + h), never 0
constexpr uint64_t kSplitToken = 0xC6A4A7935BD1E995ull;

// Bytes of workspace launch_gemm uses to split this GEMM's last round (0:
// it runs unsplit).
size_t gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

// What launch_gemm runs for this shape (host only): kernel id (the
// SOLFP4_KERNEL_* values of solfp4.h), output tile edge, workgroups, and K
// ranges per remainder tile (1: no split).  `with_workspace`: a workspace of
// at least gemm_workspace_bytes(M, N, K) is passed.
void describe_gemm(int64_t M, int64_t N, int64_t K, bool with_workspace, int* kernel, int* tile,
                   int64_t* workgroups, int* splits);
void describe_mx_gemm(int64_t M, int64_t N, int64_t K, int* kernel, int* tile, int64_t* workgroups);

// The small-tile GEMM (64 x 64 output tiles, K % 128 == 0) and its fused
// variant, whose activations arrive as BF16 and are quantized in the kernel
// (bit-identical to nvfp4_quantize) after the amax pass has written its
// partial maxima.
struct SmallFuse {
  const uint16_t* x = nullptr;          // [M][K] BF16 activations
  const uint32_t* partial = nullptr;    // the amax pass's partial maxima
  int npartial = 0;
  uint8_t* codes_out = nullptr;         // [M][K/2], the activations' codes
  uint8_t* scales_out = nullptr;        // [M][K/16], their E4M3 scales
  float* alpha_out = nullptr;           // their alpha
};
// Whether a GEMM of this shape runs on the small-tile kernel (host only):
// K % 128 == 0 and its 64 x 64 tiles fit in one round on the device.
bool use_small_gemm(int64_t M, int64_t N, int64_t K);
// Whether a GEMM the small-tile kernel would take runs faster on the wave-K
// kernel (32 x 32 tiles, K dealt to the four waves of a workgroup; host
// only).
bool use_wavek_gemm(int64_t M, int64_t N, int64_t K);
hipError_t launch_gemm_wavek(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                             const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                             hipStream_t stream);
// nvfp4_linear quantizes the activations inside the small-tile kernel up to
// this K (where nvfp4_gemm takes that kernel, not the wave-K one); beyond it
// the amax and encode passes followed by the GEMM are faster (the in-kernel
// quantization costs as much VALU time as the encode pass, and saves only
// its launch).
constexpr int64_t kFusedMaxK = 512;
hipError_t launch_gemm_small(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                             const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                             const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                             const SmallFuse* fuse, hipStream_t stream);
// The amax pass alone (the first kernel of launch_quantize), and the encode
// pass alone (the second).
hipError_t launch_amax(const uint16_t* x, int64_t n_elems, uint32_t* partial, hipStream_t stream);
hipError_t launch_encode(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                         uint8_t* scales, float* global_scale, const uint32_t* partial,
                         hipStream_t stream);

// launch_gemm without the small-tile route (the 256 x 256 / 128 x 128 lane
// kernel or the workgroup-shared kernel, as gemm_plan chooses).
hipError_t launch_gemm_regular(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                               const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

hipError_t launch_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_gs,
                       const uint8_t* b_codes, const uint8_t* b_scales, const float* b_gs,
                       const uint16_t* bias, uint16_t* out, int64_t M, int64_t N, int64_t K,
                       void* workspace, size_t workspace_bytes, hipStream_t stream);

// MXFP4 (32-element blocks, E8M0 scales): one quantize pass, and the GEMM
// on the scaled FP4 matrix instructions.
hipError_t launch_mx_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                              uint8_t* scales, hipStream_t stream);

hipError_t launch_mx_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
                          const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M,
                          int64_t N, int64_t K, hipStream_t stream);

// The wave-K MXFP4 kernel alone (K % 128 == 0); launch_mx_gemm calls it
// where use_mx_wavek holds.
hipError_t launch_mx_gemm_wavek(const uint8_t* a_codes, const uint8_t* a_scales,
                                const uint8_t* b_codes, const uint8_t* b_scales,
                                const uint16_t* bias, uint16_t* out, int64_t M, int64_t N,
                                int64_t K, hipStream_t stream);

}  // namespace solfp4
