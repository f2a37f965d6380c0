// C-ABI entry points of libsolfp4 (declared and documented in solfp4.h).
// Every argument check happens on the host before the first HIP call.
#include "solfp4.h"
#include "kernels.h"

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMaxDim = (int64_t)1 << 31;
// a GEMM addresses one 256-row operand tile through a 32-bit byte range
constexpr int64_t kMaxGemmK = (int64_t)1 << 24;
// the output of one 256-row tile is addressed through a 32-bit byte range
constexpr int64_t kMaxN = (int64_t)1 << 22;

size_t round_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int check_dims(int64_t a, int64_t b) {
  if (a < 0 || b < 0) return SOLFP4_EINVAL;
  if (a >= kMaxDim || b >= kMaxDim) return SOLFP4_ESHAPE;
  return SOLFP4_OK;
}

size_t quantize_scratch_bytes(int64_t rows, int64_t K) {
  return round_up((size_t)solfp4::amax_partial_count(rows * K) * sizeof(uint32_t));
}

struct LinearLayout {
  size_t codes, scales, alpha, partial, gemm, total;
};

LinearLayout linear_layout(int64_t M, int64_t N, int64_t K) {
  LinearLayout l;
  l.codes = 0;
  l.scales = round_up((size_t)(M * K / 2));
  l.alpha = l.scales + round_up((size_t)(M * K / 16));
  l.partial = l.alpha + kAlign;
  l.gemm = l.partial + quantize_scratch_bytes(M, K);
  l.total = l.gemm + round_up(solfp4::gemm_workspace_bytes(M, N, K));
  return l;
}

int quantize_checks(const uint16_t* x, int64_t rows, int64_t K, const uint8_t* codes,
                    const uint8_t* scales, const float* gs, const void* ws, size_t ws_bytes) {
  int rc = check_dims(rows, K);
  if (rc) return rc;
  if (K % 16) return SOLFP4_ESHAPE;
  const bool data = rows > 0 && K > 0;
  if (!gs || !ws || (data && (!x || !codes || !scales))) return SOLFP4_EINVAL;
  if (!aligned16(gs) || !aligned16(ws) ||
      (data && (!aligned16(x) || !aligned16(codes) || !aligned16(scales))))
    return SOLFP4_EALIGN;
  if (ws_bytes < quantize_scratch_bytes(rows, K)) return SOLFP4_EWORKSPACE;
  return SOLFP4_OK;
}

int gemm_checks(const uint8_t* ac, const uint8_t* as, const float* ags, const uint8_t* bc,
                const uint8_t* bs, const float* bgs, const uint16_t* bias, const uint16_t* out,
                const void* ws, size_t ws_bytes, int64_t M, int64_t N, int64_t K) {
  int rc = check_dims(M, N);
  if (rc) return rc;
  rc = check_dims(K, 0);
  if (rc) return rc;
  if (K % 16 || K >= kMaxGemmK || N >= kMaxN) return SOLFP4_ESHAPE;
  // the grid is one workgroup per 256 x 256 output tile
  if (((M + 255) / 256) * ((N + 255) / 256) >= kMaxDim) return SOLFP4_ESHAPE;
  const bool any_out = M > 0 && N > 0;
  if (!any_out) return SOLFP4_OK;
  if (!out || !ags || !bgs) return SOLFP4_EINVAL;
  if (K > 0 && (!ac || !as || !bc || !bs)) return SOLFP4_EINVAL;
  if (!aligned16(out) || !aligned16(ags) || !aligned16(bgs) || (bias && !aligned16(bias)))
    return SOLFP4_EALIGN;
  if (K > 0 && (!aligned16(ac) || !aligned16(as) || !aligned16(bc) || !aligned16(bs)))
    return SOLFP4_EALIGN;
  if (ws) {
    if (!aligned16(ws)) return SOLFP4_EALIGN;
    if (ws_bytes < solfp4::gemm_workspace_bytes(M, N, K)) return SOLFP4_EWORKSPACE;
  }
  return SOLFP4_OK;
}

struct MxLinearLayout {
  size_t codes, scales, total;
};

MxLinearLayout mx_linear_layout(int64_t M, int64_t K) {
  MxLinearLayout l;
  l.codes = 0;
  l.scales = round_up((size_t)(M * K / 2));
  l.total = l.scales + round_up((size_t)(M * K / 32));
  if (l.total == 0) l.total = kAlign;
  return l;
}

int mx_quantize_checks(const uint16_t* x, int64_t rows, int64_t K, const uint8_t* codes,
                       const uint8_t* scales) {
  int rc = check_dims(rows, K);
  if (rc) return rc;
  if (K % 32) return SOLFP4_ESHAPE;
  if (rows > 0 && K > 0) {
    if (!x || !codes || !scales) return SOLFP4_EINVAL;
    if (!aligned16(x) || !aligned16(codes) || !aligned16(scales)) return SOLFP4_EALIGN;
  }
  return SOLFP4_OK;
}

int mx_gemm_checks(const uint8_t* ac, const uint8_t* as, const uint8_t* bc, const uint8_t* bs,
                   const uint16_t* bias, const uint16_t* out, int64_t M, int64_t N, int64_t K) {
  int rc = check_dims(M, N);
  if (rc) return rc;
  rc = check_dims(K, 0);
  if (rc) return rc;
  if (K % 32 || K >= kMaxGemmK || N >= kMaxN) return SOLFP4_ESHAPE;
  if (((M + 255) / 256) * ((N + 255) / 256) >= kMaxDim) return SOLFP4_ESHAPE;
  if (M == 0 || N == 0) return SOLFP4_OK;
  if (!out) return SOLFP4_EINVAL;
  if (K > 0 && (!ac || !as || !bc || !bs)) return SOLFP4_EINVAL;
  if (!aligned16(out) || (bias && !aligned16(bias))) return SOLFP4_EALIGN;
  if (K > 0 && (!aligned16(ac) || !aligned16(as) || !aligned16(bc) || !aligned16(bs)))
    return SOLFP4_EALIGN;
  return SOLFP4_OK;
}

}  // namespace

extern "C" {

const char* solfp4_strerror(int status) {
  switch (status) {
    case SOLFP4_OK: return "success";
    case SOLFP4_EINVAL: return "invalid argument (null pointer or negative size)";
    case SOLFP4_ESHAPE:
      return "unsupported shape (K must be a multiple of 16, or of 32 for MXFP4; sizes below 2^31; "
             "GEMM K below 2^24 and N below 2^22)";
    case SOLFP4_EALIGN: return "pointer not 16-byte aligned";
    case SOLFP4_EWORKSPACE: return "workspace missing or too small";
    case SOLFP4_EHIP: return "HIP kernel launch failed";
    default: return "unknown status";
  }
}

int solfp4_version(void) { return 200; }

int solfp4_gemm_plan(int format, int64_t M, int64_t N, int64_t K, int with_workspace, int* kernel,
                     int* tile, int64_t* workgroups, int* splits) {
  if (!kernel || !tile || !workgroups || !splits) return SOLFP4_EINVAL;
  if (format != SOLFP4_FORMAT_NVFP4 && format != SOLFP4_FORMAT_MXFP4) return SOLFP4_EINVAL;
  int rc = check_dims(M, N);
  if (rc) return rc;
  rc = check_dims(K, 0);
  if (rc) return rc;
  const int64_t block = format == SOLFP4_FORMAT_NVFP4 ? 16 : 32;
  if (K % block || K >= kMaxGemmK || N >= kMaxN) return SOLFP4_ESHAPE;
  if (((M + 255) / 256) * ((N + 255) / 256) >= kMaxDim) return SOLFP4_ESHAPE;
  *kernel = 0;
  *tile = 256;
  *workgroups = 0;
  *splits = 1;
  if (M == 0 || N == 0) return SOLFP4_OK;
  if (format == SOLFP4_FORMAT_NVFP4)
    solfp4::describe_gemm(M, N, K, with_workspace != 0, kernel, tile, workgroups, splits);
  else
    solfp4::describe_mx_gemm(M, N, K, kernel, tile, workgroups);
  return SOLFP4_OK;
}

size_t nvfp4_quantize_workspace_bytes(int64_t rows, int64_t K) {
  if (check_dims(rows, K) || K % 16) return 0;
  return quantize_scratch_bytes(rows, K);
}

int nvfp4_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes, uint8_t* scales,
                   float* global_scale, void* workspace, size_t workspace_bytes, void* stream) {
  const int rc = quantize_checks(x, rows, K, codes, scales, global_scale, workspace, workspace_bytes);
  if (rc) return rc;
  const hipError_t e = solfp4::launch_quantize(x, rows, K, codes, scales, global_scale,
                                               static_cast<uint32_t*>(workspace),
                                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int nvfp4_quantize_amax(const uint16_t* x, int64_t rows, int64_t K, void* workspace,
                        size_t workspace_bytes, void* stream) {
  int rc = check_dims(rows, K);
  if (rc) return rc;
  if (K % 16) return SOLFP4_ESHAPE;
  if (!workspace || (rows > 0 && K > 0 && !x)) return SOLFP4_EINVAL;
  if (!aligned16(workspace) || (rows > 0 && K > 0 && !aligned16(x))) return SOLFP4_EALIGN;
  if (workspace_bytes < quantize_scratch_bytes(rows, K)) return SOLFP4_EWORKSPACE;
  const hipError_t e = solfp4::launch_amax(x, rows * K, static_cast<uint32_t*>(workspace),
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int nvfp4_quantize_encode(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                          uint8_t* scales, float* global_scale, void* workspace,
                          size_t workspace_bytes, void* stream) {
  const int rc = quantize_checks(x, rows, K, codes, scales, global_scale, workspace, workspace_bytes);
  if (rc) return rc;
  const hipError_t e = solfp4::launch_encode(x, rows, K, codes, scales, global_scale,
                                             static_cast<const uint32_t*>(workspace),
                                             static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int nvfp4_quantize_noalloc(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes,
                           uint8_t* scales, float* global_scale, void* stream) {
  int rc = check_dims(rows, K);
  if (rc) return rc;
  if (K % 16) return SOLFP4_ESHAPE;
  const bool data = rows > 0 && K > 0;
  if (!global_scale || (data && (!x || !codes || !scales))) return SOLFP4_EINVAL;
  if (!aligned16(global_scale) ||
      (data && (!aligned16(x) || !aligned16(codes) || !aligned16(scales))))
    return SOLFP4_EALIGN;
  // the partial maxima must fit the fixed scratch (they always do: the amax
  // pass never runs more than kMaxPartials workgroups)
  if (solfp4::amax_partial_count(rows * K) > solfp4::kScratchWords) return SOLFP4_EWORKSPACE;
  uint32_t* partial = nullptr;
  if (solfp4::scratch_address(&partial) != hipSuccess) return SOLFP4_EHIP;
  const hipError_t e = solfp4::launch_quantize(x, rows, K, codes, scales, global_scale, partial,
                                               static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int nvfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const float* a_global_scale,
               const uint8_t* b_codes, const uint8_t* b_scales, const float* b_global_scale,
               const uint16_t* bias, uint16_t* out, void* workspace, size_t workspace_bytes,
               int64_t M, int64_t N, int64_t K, void* stream) {
  const int rc = gemm_checks(a_codes, a_scales, a_global_scale, b_codes, b_scales, b_global_scale,
                             bias, out, workspace, workspace_bytes, M, N, K);
  if (rc) return rc;
  if (M == 0 || N == 0) return SOLFP4_OK;
  const hipError_t e = solfp4::launch_gemm(a_codes, a_scales, a_global_scale, b_codes, b_scales,
                                           b_global_scale, bias, out, M, N, K, workspace,
                                           workspace ? workspace_bytes : 0,
                                           static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

size_t nvfp4_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (check_dims(M, N) || check_dims(K, 0) || K % 16 || K >= kMaxGemmK || N >= kMaxN) return 0;
  return solfp4::gemm_workspace_bytes(M, N, K);
}

size_t nvfp4_linear_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (check_dims(M, N) || check_dims(K, 0) || K % 16 || K >= kMaxGemmK || N >= kMaxN) return 0;
  return linear_layout(M, N, K).total;
}

int nvfp4_linear(const uint16_t* x, const uint8_t* w_codes, const uint8_t* w_scales,
                 const float* w_global_scale, const uint16_t* bias, uint16_t* out,
                 void* workspace, size_t workspace_bytes, int64_t M, int64_t N, int64_t K,
                 void* stream) {
  int rc = check_dims(M, N);
  if (rc) return rc;
  rc = check_dims(K, 0);
  if (rc) return rc;
  if (K % 16 || K >= kMaxGemmK || N >= kMaxN) return SOLFP4_ESHAPE;
  if (!workspace) return SOLFP4_EINVAL;
  if (!aligned16(workspace)) return SOLFP4_EALIGN;
  const LinearLayout l = linear_layout(M, N, K);
  if (workspace_bytes < l.total) return SOLFP4_EWORKSPACE;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint8_t* xc = ws + l.codes;
  uint8_t* xs = ws + l.scales;
  float* xa = reinterpret_cast<float*>(ws + l.alpha);
  uint32_t* partial = reinterpret_cast<uint32_t*>(ws + l.partial);
  void* gws = ws + l.gemm;
  const size_t gws_bytes = l.total - l.gemm;
  rc = quantize_checks(x, M, K, xc, xs, xa, partial, l.gemm - l.partial);
  if (rc) return rc;
  rc = gemm_checks(xc, xs, xa, w_codes, w_scales, w_global_scale, bias, out, gws, gws_bytes, M,
                   N, K);
  if (rc) return rc;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (K <= solfp4::kFusedMaxK && solfp4::use_small_gemm(M, N, K) &&
      !solfp4::use_wavek_gemm(M, N, K)) {
    // few tokens and a short K, where nvfp4_gemm runs the small-tile kernel
    // too (so the FP32 sums are formed in the same order): the amax pass,
    // then the small-tile GEMM quantizing the activations itself (leaving
    // codes, scales and alpha in the workspace)
    solfp4::SmallFuse fuse;
    fuse.x = x;
    fuse.partial = partial;
    fuse.npartial = solfp4::amax_partial_count(M * K);
    fuse.codes_out = xc;
    fuse.scales_out = xs;
    fuse.alpha_out = xa;
    hipError_t e = solfp4::launch_amax(x, M * K, partial, s);
    if (e != hipSuccess) return SOLFP4_EHIP;
    e = solfp4::launch_gemm_small(nullptr, nullptr, nullptr, w_codes, w_scales, w_global_scale, bias,
                                  out, M, N, K, &fuse, s);
    return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
  }
  hipError_t e = solfp4::launch_quantize(x, M, K, xc, xs, xa, partial, s);
  if (e != hipSuccess) return SOLFP4_EHIP;
  if (M == 0 || N == 0) return SOLFP4_OK;
  e = solfp4::launch_gemm(xc, xs, xa, w_codes, w_scales, w_global_scale, bias, out, M, N, K, gws,
                          gws_bytes, s);
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int mxfp4_quantize(const uint16_t* x, int64_t rows, int64_t K, uint8_t* codes, uint8_t* scales,
                   void* stream) {
  const int rc = mx_quantize_checks(x, rows, K, codes, scales);
  if (rc) return rc;
  const hipError_t e =
      solfp4::launch_mx_quantize(x, rows, K, codes, scales, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

int mxfp4_gemm(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* b_codes,
               const uint8_t* b_scales, const uint16_t* bias, uint16_t* out, int64_t M, int64_t N,
               int64_t K, void* stream) {
  const int rc = mx_gemm_checks(a_codes, a_scales, b_codes, b_scales, bias, out, M, N, K);
  if (rc) return rc;
  const hipError_t e = solfp4::launch_mx_gemm(a_codes, a_scales, b_codes, b_scales, bias, out, M,
                                              N, K, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

size_t mxfp4_linear_workspace_bytes(int64_t M, int64_t K) {
  if (check_dims(M, K) || K % 32) return 0;
  return mx_linear_layout(M, K).total;
}

int mxfp4_linear(const uint16_t* x, const uint8_t* w_codes, const uint8_t* w_scales,
                 const uint16_t* bias, uint16_t* out, void* workspace, size_t workspace_bytes,
                 int64_t M, int64_t N, int64_t K, void* stream) {
  int rc = check_dims(M, N);
  if (rc) return rc;
  rc = check_dims(K, 0);
  if (rc) return rc;
  if (K % 32 || K >= kMaxGemmK || N >= kMaxN) return SOLFP4_ESHAPE;
  if (!workspace) return SOLFP4_EINVAL;
  if (!aligned16(workspace)) return SOLFP4_EALIGN;
  const MxLinearLayout l = mx_linear_layout(M, K);
  if (workspace_bytes < l.total) return SOLFP4_EWORKSPACE;
  uint8_t* ws = static_cast<uint8_t*>(workspace);
  uint8_t* xc = ws + l.codes;
  uint8_t* xs = ws + l.scales;
  rc = mx_quantize_checks(x, M, K, xc, xs);
  if (rc) return rc;
  rc = mx_gemm_checks(xc, xs, w_codes, w_scales, bias, out, M, N, K);
  if (rc) return rc;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = solfp4::launch_mx_quantize(x, M, K, xc, xs, s);
  if (e != hipSuccess) return SOLFP4_EHIP;
  e = solfp4::launch_mx_gemm(xc, xs, w_codes, w_scales, bias, out, M, N, K, s);
  return e == hipSuccess ? SOLFP4_OK : SOLFP4_EHIP;
}

}  // extern "C"
