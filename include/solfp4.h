/*
 * solfp4 -- NVFP4 linear layer for AMD Instinct MI355X (gfx950).
 *
 * The hot path of the fast-rollout stage of Sol-RL (arXiv 2604.06916): every
 * linear layer of the diffusion-transformer denoiser runs on NVFP4 operands
 * (Sec. 3.4, Stage 1; Sec. 4.1 uses NVFP4 for the whole exploration model).
 * NVFP4 is defined in the Preliminaries ("FP4 Quantization and Hardware
 * Acceleration"): E2M1 elements (1 sign, 2 exponent, 1 mantissa bit), one
 * E4M3 scale per 16 contiguous elements, and Q(x) = S * Pi_FP4(x / S).
 *
 * Conventions shared by every call
 * --------------------------------
 * - All data pointers are DEVICE pointers (HIP global memory) owned by the
 *   caller; the library allocates and frees nothing and keeps no state
 *   between calls (workspaces are scratch for the duration of one call).
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   Calls only enqueue work and return; nothing synchronises the host.
 * - Matrices are row-major and contiguous.  BF16 values travel as their
 *   uint16_t bit patterns.  K, the reduction length, must be a multiple of
 *   16 (one NVFP4 block).
 * - Every pointer must be 16-byte aligned.
 * - Argument errors are detected on the host and returned BEFORE any kernel
 *   launch (the only HIP calls before that are device-attribute queries,
 *   which fall back to MI355X's values without a GPU), so they are safe to
 *   provoke on a machine without one.  Non-finite
 *   inputs (NaN, Inf) give unspecified codes but never fault.
 * - Return value: SOLFP4_OK (0) or one of the negative status codes below.
 *   Nothing throws across this boundary.
 *
 * NVFP4 encoding produced and consumed here (paper silent on these details;
 * this is the library's fixed reading):
 *   alpha = amax(|x|) / (6 * 448)                       FP32, per tensor
 *   s_b   = E4M3_RNE_SAT(amax_b / (6 * alpha))          per 16-element block
 *   q_i   = E2M1_RNE_SAT(x_i * (1 / (s_b * alpha)))     sign kept, also on 0
 *   decoded value = alpha * s_b * q_i
 * every step IEEE binary32 round-to-nearest-even in exactly this order.
 * Rounding to E4M3 and E2M1 is to nearest with ties to the even code and
 * saturates at 448 and 6.  amax == 0 gives alpha = 0, scales 0 and codes
 * sign<<3; a block whose scale rounds to 0 gets codes sign<<3.
 *
 * Layouts:
 *   codes  [rows][K/2]  uint8: element 2j in bits 3:0 of byte j, 2j+1 in 7:4
 *   scales [rows][K/16] uint8: E4M3 (OCP E4M3FN: bias 7, max 448, 0x7F NaN)
 *   global scale: one float (alpha) in device memory
 */
#ifndef SOLFP4_H
#define SOLFP4_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Every entry point below is exported from libsolfp4.so; nothing else is. */
#define SOLFP4_API __attribute__((visibility("default")))

#define SOLFP4_OK 0
#define SOLFP4_EINVAL (-1)     /* null pointer where data is needed, negative size */
#define SOLFP4_ESHAPE (-2)     /* K not a multiple of the block (16 NVFP4, 32 MXFP4), a size of
                                  2^31 or more, or a GEMM with K of 2^24 or more or N of 2^22
                                  or more */
#define SOLFP4_EALIGN (-3)     /* a pointer is not 16-byte aligned */
#define SOLFP4_EWORKSPACE (-4) /* workspace missing or smaller than the *_workspace_bytes query */
#define SOLFP4_EHIP (-5)       /* a HIP launch reported an error */

/* Static, human-readable text for a status code.  Host only; never NULL. */
SOLFP4_API const char* solfp4_strerror(int status);

/* Library version as 10000*major + 100*minor + patch.  Host only. */
SOLFP4_API int solfp4_version(void);

/*
 * Device workspace, in bytes, that nvfp4_quantize needs for a [rows, K]
 * input (room for the partial maxima of the first pass).  Host only; pure
 * function of its arguments; 0 for invalid sizes.
 */
SOLFP4_API size_t nvfp4_quantize_workspace_bytes(int64_t rows, int64_t K);

/*
 * NVFP4 quantization of a BF16 matrix (Preliminaries: 16-element blocks,
 * E4M3 block scales, E2M1 elements, plus the FP32 per-tensor scale above).
 *
 *   x            [rows][K] BF16, read only
 *   codes        [rows][K/2] uint8, written
 *   scales       [rows][K/16] uint8 (E4M3), written
 *   global_scale 1 float, written with alpha
 *   workspace    >= nvfp4_quantize_workspace_bytes(rows, K) bytes of device
 *                scratch, contents undefined on entry and on exit
 *
 * Two kernels run in stream order: a read of x for amax, then the encode
 * pass.  rows == 0 is valid and writes alpha = 0.  Codes, scales and alpha
 * are bit-identical to the encoding stated at the top of this header.
 */
SOLFP4_API int nvfp4_quantize(const uint16_t* x, int64_t rows, int64_t K,
                   uint8_t* codes, uint8_t* scales, float* global_scale,
                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * The two passes of nvfp4_quantize as separate calls, for callers that want
 * to schedule them apart (the amax pass of the next layer's input can run
 * on another stream, or be timed on its own).  nvfp4_quantize_amax(x, rows,
 * K, workspace, ...) reads x once and writes its partial maxima into the
 * workspace; nvfp4_quantize_encode(x, rows, K, codes, scales, global_scale,
 * workspace, ...) folds them into alpha and writes codes, scales and alpha.
 * The pair, in stream order, with the same x, sizes and workspace and
 * nothing writing x or the workspace in between, is exactly nvfp4_quantize
 * (same kernels, bit-identical results); the workspace must be at least
 * nvfp4_quantize_workspace_bytes(rows, K) bytes.  Argument checks and
 * errors as for nvfp4_quantize.
 */
SOLFP4_API int nvfp4_quantize_amax(const uint16_t* x, int64_t rows, int64_t K,
                   void* workspace, size_t workspace_bytes, void* stream);
SOLFP4_API int nvfp4_quantize_encode(const uint16_t* x, int64_t rows, int64_t K,
                   uint8_t* codes, uint8_t* scales, float* global_scale,
                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * nvfp4_quantize without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, kernels and results
 * as nvfp4_quantize (bit-identical codes, scales and alpha); the amax
 * pass's partial maxima go to a fixed 4 KiB device array of the library
 * instead (one per device, held until the process ends; looked up on the
 * first call on each device).  Allocates nothing, for any size: the amax
 * pass never runs more workgroups than the array has words, and a size
 * that needed more would be refused with SOLFP4_EWORKSPACE.
 *
 * Every call on one device shares that device's array: two calls that may
 * run at the same time on one device (on different streams, or from
 * different threads without ordering) race on it and may write a wrong
 * alpha.  Calls ordered on one stream, or separated by synchronisation, are
 * safe; the array's contents are rewritten by every call before they are
 * read, so nothing needs clearing.
 */
SOLFP4_API int nvfp4_quantize_noalloc(const uint16_t* x, int64_t rows, int64_t K,
                   uint8_t* codes, uint8_t* scales, float* global_scale, void* stream);

/*
 * Block-scaled NVFP4 GEMM with BF16 output (the "NVFP4 dense operations" of
 * Sec. 3.4, Stage 1):
 *
 *   out[m][n] = bf16_rne( a_gs * b_gs * sum_k (s_A q_A)[m][k] (s_B q_B)[n][k]
 *                         + bias[n] )
 *
 *   a_codes [M][K/2], a_scales [M][K/16], a_global_scale 1 float  (A = X)
 *   b_codes [N][K/2], b_scales [N][K/16], b_global_scale 1 float  (B = W,
 *            stored [N][K] as an nn.Linear weight)
 *   bias    [N] BF16 or NULL
 *   out     [M][N] BF16, written
 *
 * Each product (s q)(s q) is formed exactly (both factors are dequantized
 * exactly to FP16 and multiplied by the FP16 matrix cores); sums are FP32 in
 * an unspecified order; alpha = a_gs * b_gs is one FP32 multiply; the output
 * is bf16_rne(fp32(fma(alpha, acc, bias[n]))): one FP32 fused multiply-add,
 * then rounding to BF16.  Results may differ from a float64 evaluation by
 * the FP32 summation and FMA roundings plus the BF16 rounding.  M, N or K
 * equal to 0 are valid (K == 0 writes the bias, or zeros).  K must be below
 * 2^24 and N below 2^22.
 */
SOLFP4_API int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_global_scale,
               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_global_scale,
               const uint16_t* bias, uint16_t* out, void* workspace, size_t workspace_bytes,
               int64_t M, int64_t N, int64_t K, void* stream);

/*
 * Device workspace, in bytes, that nvfp4_gemm uses for an M x N x K product
 * on the current device (host only; 0 for invalid sizes).  The GEMM runs
 * one workgroup per 256 x 256 output tile (128 x 128 when there are too few
 * of those to fill the device), about ceil(tiles / CUs) rounds of one
 * tile's time.  A last round of at most a quarter of the CUs' worth of
 * 256 x 256 tiles runs after the others as four 128 x 128 quadrants per
 * tile (a second kernel launch, same results as whole tiles); with at most
 * an eighth and at least 16 K stages of 128 (K > 1920), each quadrant is
 * computed as two K halves by two workgroups.  Otherwise, when the last
 * round holds at most half the CUs' worth of tiles and K is long enough,
 * each of those tiles is computed as two K halves.  The halves add their
 * FP32 partial sums through this workspace (one partial tile per half:
 * 256 KB, or 64 KB for 128 x 128 tiles and quadrants; plus an 8-byte slot
 * per tile or quadrant that tells the second half to finish that it is
 * second).  0 means the shape runs without it,
 * which includes few-token shapes (K % 128 == 0 with at most one 64 x 64
 * tile per compute unit): they run on 64 x 64 tiles, or on 32 x 32 tiles
 * whose K stages the four waves of a workgroup share (their partial sums
 * added in LDS in wave order), whichever is estimated faster.
 *
 * nvfp4_gemm's workspace argument:
 *   NULL       no split (workspace_bytes is ignored)
 *   otherwise  16-byte aligned, at least nvfp4_gemm_workspace_bytes(M, N, K)
 *              bytes, else SOLFP4_EWORKSPACE; its contents on entry are
 *              ignored and undefined on return (it is scratch).  Calls that
 *              may run at the same time must not share one.
 * The split changes the order of the FP32 summation for the affected tiles
 * (two partial sums added once), so outputs with and without a workspace
 * may differ in their last bits; for a given choice results are
 * deterministic (the two halves are added by one commutative addition,
 * whichever finishes last).
 */
SOLFP4_API size_t nvfp4_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K);

/* Device workspace, in bytes, that nvfp4_linear needs for [M, K]
 * activations times an [N, K] weight: the activations' NVFP4 codes,
 * scales and alpha, the quantizer's scratch, then nvfp4_gemm's workspace.
 * Host only; 0 for invalid sizes. */
SOLFP4_API size_t nvfp4_linear_workspace_bytes(int64_t M, int64_t N, int64_t K);

/*
 * The NVFP4 linear layer of the denoiser (Sec. 4.1: the model's linears run
 * in NVFP4; Sec. 3.4: weights are quantized once per policy update, the
 * activations on the fly): quantize x exactly as nvfp4_quantize does, then
 * nvfp4_gemm against the pre-quantized weight, with bias.
 *
 *   x        [M][K] BF16
 *   w_codes  [N][K/2], w_scales [N][K/16], w_global_scale 1 float
 *            (the weight quantized with nvfp4_quantize)
 *   bias     [N] BF16 or NULL
 *   out      [M][N] BF16
 *   workspace >= nvfp4_linear_workspace_bytes(M, N, K) bytes; on return it
 *            holds the activation codes at offset 0, then their scales and
 *            alpha (offsets are an implementation detail).
 *
 * Launches: the amax pass, the encode pass and the GEMM; or, for few
 * tokens with K <= 512 where nvfp4_gemm runs on 64 x 64 tiles, the amax
 * pass and one GEMM kernel that quantizes the activations itself (with the
 * same tiles and summation order).  Either way the workspace
 * ends up holding the same codes, scales and alpha, and the result is
 * bit-identical to nvfp4_quantize followed by nvfp4_gemm with a workspace of
 * at least nvfp4_gemm_workspace_bytes(M, N, K) (the linear always splits
 * the last round where the GEMM would; nvfp4_gemm without a workspace runs
 * every tile whole, which may change the last bits of the affected
 * outputs).
 */
SOLFP4_API int nvfp4_linear(const uint16_t* x, const uint8_t* w_codes, const uint8_t* w_scales,
                 const float* w_global_scale, const uint16_t* bias, uint16_t* out,
                 void* workspace, size_t workspace_bytes,
                 int64_t M, int64_t N, int64_t K, void* stream);

/*
 * How a GEMM of this shape runs on the current device (host only; without a
 * GPU the device is taken to have MI355X's 256 compute units).  The kernel
 * choice depends only on the shape and the CU count, so callers (a
 * benchmark naming the kernel it times, a scheduler sizing its streams) can
 * ask instead of re-deriving it.
 *
 *   format          SOLFP4_FORMAT_NVFP4 (nvfp4_gemm) or SOLFP4_FORMAT_MXFP4
 *                   (mxfp4_gemm)
 *   with_workspace  nonzero: nvfp4_gemm gets a workspace of at least
 *                   nvfp4_gemm_workspace_bytes(M, N, K) (ignored for MXFP4)
 *   kernel          written: one of the SOLFP4_KERNEL_* ids below
 *   tile            written: output tile edge, 256, 128, 64 or 32
 *   workgroups      written: workgroups of the launch (of both launches
 *                   where the last round runs as 128 x 128 quadrants)
 *   splits          written: K ranges per tile of the last round, each on
 *                   a workgroup of its own (1: none; the wave-K kernel's
 *                   four K shares inside one workgroup are not counted)
 *
 * Returns SOLFP4_OK, SOLFP4_EINVAL for a null output pointer, a negative
 * size or an unknown format, or SOLFP4_ESHAPE for a shape the GEMM rejects.
 * M == 0 or N == 0 writes kernel 0 and workgroups 0 (nothing is launched).
 */
#define SOLFP4_FORMAT_NVFP4 0
#define SOLFP4_FORMAT_MXFP4 1
#define SOLFP4_KERNEL_NVFP4_LANE 1     /* codes to LDS by DMA, per-wave dequantization */
#define SOLFP4_KERNEL_NVFP4_SHARED 2   /* workgroup-shared dequantization into LDS */
#define SOLFP4_KERNEL_MXFP4 3          /* scaled FP4 matrix instructions (256 x 256,
                                          128 x 128 or, for few tokens, 64 x 64 tiles; a
                                          last round of at most a quarter of the CUs'
                                          worth of 256 x 256 tiles runs as their
                                          128 x 128 quadrants in a second launch) */
#define SOLFP4_KERNEL_NVFP4_SMALL 4    /* 64 x 64 tiles for few tokens (K % 128 == 0); in
                                          nvfp4_linear with K <= 512 it also quantizes the
                                          activations itself */
#define SOLFP4_KERNEL_NVFP4_WAVEK 5    /* 32 x 32 tiles for few tokens, each workgroup's
                                          K stages dealt to its four waves (K % 128 == 0) */
#define SOLFP4_KERNEL_MXFP4_WAVEK 6    /* MXFP4, 32 x 32 tiles for few tokens, each
                                          workgroup's K stages dealt to its four waves
                                          (K % 128 == 0) */
SOLFP4_API int solfp4_gemm_plan(int format, int64_t M, int64_t N, int64_t K, int with_workspace,
                     int* kernel, int* tile, int64_t* workgroups, int* splits);

/*
 * MXFP4 variant (Preliminaries: the OCP MX format, E2M1 elements with one
 * power-of-two E8M0 scale per 32 elements; this is the block format that
 * CDNA4's scaled FP4 matrix instructions consume natively).
 *
 * Encoding produced and consumed here (the OCP MX conversion rule):
 *   E     = floor(log2(amax_b)) - 2           per 32-element block (2 is the
 *                                             exponent of 6, the largest E2M1)
 *   scale = clamp(E + 127, 0, 254)            E8M0 byte; 0 for an all-zero block
 *   q_i   = E2M1_RNE_SAT(x_i / 2^(scale - 127))   exact division, ties to the
 *                                             even code, saturating at 6,
 *                                             sign kept on zero
 *   decoded value = 2^(scale - 127) * q_i
 * No per-tensor scale.  Layouts:
 *   codes  [rows][K/2]  uint8: as for NVFP4 (element 2j in bits 3:0 of byte j)
 *   scales [rows][K/32] uint8: E8M0, value 2^(byte - 127); 0xFF (NaN) is
 *          never produced and must not be passed in
 * K must be a multiple of 32.
 */

/*
 * MXFP4 quantization of a BF16 matrix: one pass over x.
 *
 *   x       [rows][K] BF16, read only
 *   codes   [rows][K/2] uint8, written
 *   scales  [rows][K/32] uint8 (E8M0), written
 *
 * Needs no workspace.  rows == 0 or K == 0 is valid and launches nothing.
 */
SOLFP4_API int mxfp4_quantize(const uint16_t* x, int64_t rows, int64_t K,
                   uint8_t* codes, uint8_t* scales, void* stream);

/*
 * MXFP4 GEMM with BF16 output on the scaled FP4 matrix instructions:
 *
 *   out[m][n] = bf16_rne( sum_k (X_A q_A)[m][k] (X_B q_B)[n][k] + bias[n] )
 *
 *   a_codes [M][K/2], a_scales [M][K/32]     (A = X, activations)
 *   b_codes [N][K/2], b_scales [N][K/32]     (B = W, stored [N][K])
 *   bias    [N] BF16 or NULL
 *   out     [M][N] BF16, written
 *
 * The matrix cores form each product of two decoded elements and sum them
 * into FP32 accumulators in an unspecified order; the bias is added in FP32
 * (one rounding), then the sum is rounded to BF16.  Products or sums outside
 * the FP32 range are unspecified.  M, N or K equal to 0 are valid (K == 0
 * writes the bias, or zeros).  K must be below 2^24 and N below 2^22.
 */
SOLFP4_API int mxfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales,
               const uint8_t* b_codes, const uint8_t* b_scales,
               const uint16_t* bias, uint16_t* out,
               int64_t M, int64_t N, int64_t K, void* stream);

/* Device workspace, in bytes, that mxfp4_linear needs for [M, K]
 * activations (their MXFP4 codes and scales).  Host only; 0 for invalid
 * sizes. */
SOLFP4_API size_t mxfp4_linear_workspace_bytes(int64_t M, int64_t K);

/*
 * MXFP4 linear layer: mxfp4_quantize of x into the workspace, then
 * mxfp4_gemm against the pre-quantized weight, with bias.
 *
 *   x        [M][K] BF16
 *   w_codes  [N][K/2], w_scales [N][K/32] (the weight quantized with
 *            mxfp4_quantize)
 *   bias     [N] BF16 or NULL
 *   out      [M][N] BF16
 *   workspace >= mxfp4_linear_workspace_bytes(M, K) bytes; on return it
 *            holds the activation codes at offset 0, then their scales.
 *
 * The result is bit-identical to mxfp4_quantize followed by mxfp4_gemm.
 */
SOLFP4_API int mxfp4_linear(const uint16_t* x, const uint8_t* w_codes, const uint8_t* w_scales,
                 const uint16_t* bias, uint16_t* out, void* workspace, size_t workspace_bytes,
                 int64_t M, int64_t N, int64_t K, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SOLFP4_H */
