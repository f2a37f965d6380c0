/* A plain C99 program against include/solfp4.h and libsolfp4.so: the
 * boundary used the way a C caller uses it, with no GPU.  Every call below
 * is rejected on the host before any kernel launch, or is a host-only
 * query, so the fake device addresses are never dereferenced.  Exit status
 * 0 when every check holds; each failed check prints its line. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "solfp4.h"

static int failures = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      printf("check failed at line %d: %s\n", __LINE__, #cond);      \
      ++failures;                                                    \
    }                                                                \
  } while (0)

int main(void) {
  uint8_t* const p = (uint8_t*)(uintptr_t)0x7F0000000000ull;   /* 256-byte aligned, never read */
  uint8_t* const mis = p + 8;                                  /* 8-byte aligned only */
  float* const fp = (float*)(uintptr_t)0x7F0000100000ull;
  uint16_t* const hp = (uint16_t*)(uintptr_t)0x7F0000200000ull;
  int kernel = -1, tile = -1, splits = -1;
  int64_t wgs = -1;

  CHECK(solfp4_version() >= 200);
  CHECK(strcmp(solfp4_strerror(SOLFP4_OK), "success") == 0);
  CHECK(solfp4_strerror(SOLFP4_ESHAPE) != NULL && solfp4_strerror(12345) != NULL);

  /* host-only queries */
  CHECK(nvfp4_quantize_workspace_bytes(128, 1152) >= 4);
  CHECK(nvfp4_quantize_workspace_bytes(128, 1000) == 0);            /* K % 16 != 0 */
  CHECK(nvfp4_gemm_workspace_bytes(18432, 9216, 3072) > 0);         /* last round split */
  CHECK(nvfp4_linear_workspace_bytes(128, 1152, 1152) >= (size_t)(128 * 1152 / 2 + 128 * 1152 / 16));
  CHECK(mxfp4_linear_workspace_bytes(128, 1152) >= (size_t)(128 * 1152 / 2 + 128 * 1152 / 32));
  CHECK(solfp4_gemm_plan(SOLFP4_FORMAT_NVFP4, 18432, 9216, 3072, 1, &kernel, &tile, &wgs, &splits) ==
        SOLFP4_OK);
  CHECK(kernel == SOLFP4_KERNEL_NVFP4_LANE && tile == 256 && splits == 2);
  CHECK(solfp4_gemm_plan(SOLFP4_FORMAT_MXFP4, 128, 1152, 1152, 0, &kernel, &tile, &wgs, &splits) ==
        SOLFP4_OK);
  CHECK(kernel == SOLFP4_KERNEL_MXFP4_WAVEK && tile == 32 && wgs == 144 && splits == 1);
  CHECK(solfp4_gemm_plan(7, 16, 16, 16, 0, &kernel, &tile, &wgs, &splits) == SOLFP4_EINVAL);

  /* argument errors, returned before any launch */
  CHECK(nvfp4_quantize(hp, 4, 24, p, p, fp, p, 4096, NULL) == SOLFP4_ESHAPE);    /* K % 16 */
  CHECK(nvfp4_quantize(hp, -1, 16, p, p, fp, p, 4096, NULL) == SOLFP4_EINVAL);
  CHECK(nvfp4_quantize(NULL, 4, 16, p, p, fp, p, 4096, NULL) == SOLFP4_EINVAL);
  CHECK(nvfp4_quantize(hp, 4, 16, mis, p, fp, p, 4096, NULL) == SOLFP4_EALIGN);
  CHECK(nvfp4_quantize(hp, 4, 16, p, p, fp, p, 0, NULL) == SOLFP4_EWORKSPACE);
  CHECK(nvfp4_gemm(p, p, fp, p, p, fp, NULL, hp, NULL, 0, 4, 4, 24, NULL) == SOLFP4_ESHAPE);
  CHECK(nvfp4_gemm(p, p, NULL, p, p, fp, NULL, hp, NULL, 0, 4, 4, 16, NULL) == SOLFP4_EINVAL);
  CHECK(nvfp4_gemm(mis, p, fp, p, p, fp, NULL, hp, NULL, 0, 4, 4, 16, NULL) == SOLFP4_EALIGN);
  CHECK(nvfp4_gemm(p, p, fp, p, p, fp, NULL, hp, p, 8, 18432, 9216, 3072, NULL) == SOLFP4_EWORKSPACE);
  CHECK(nvfp4_gemm(p, p, fp, p, p, fp, NULL, hp, NULL, 0, 4, (int64_t)1 << 22, 16, NULL) == SOLFP4_ESHAPE);
  CHECK(nvfp4_gemm(NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, 0, 16, 16, NULL) == SOLFP4_OK);
  CHECK(nvfp4_linear(hp, p, p, fp, NULL, hp, NULL, 0, 4, 4, 16, NULL) == SOLFP4_EINVAL);
  CHECK(nvfp4_linear(hp, p, p, fp, NULL, hp, p, 16, 4, 4, 16, NULL) == SOLFP4_EWORKSPACE);
  CHECK(nvfp4_quantize_noalloc(hp, 4, 24, p, p, fp, NULL) == SOLFP4_ESHAPE);
  CHECK(mxfp4_quantize(hp, 4, 48, p, p, NULL) == SOLFP4_ESHAPE);                /* K % 32 */
  CHECK(mxfp4_gemm(p, p, p, mis, NULL, hp, 4, 4, 32, NULL) == SOLFP4_EALIGN);
  CHECK(mxfp4_linear(hp, p, p, NULL, hp, p, 16, 4, 4, 32, NULL) == SOLFP4_EWORKSPACE);

  if (failures == 0) printf("all checks passed\n");
  return failures == 0 ? 0 : 1;
}
