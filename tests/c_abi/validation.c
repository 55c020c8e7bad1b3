/*
 * Plain C99 client of include/fp4attn.h: compiled with gcc, linked against the
 * library, and run without a GPU.  It calls only argument combinations the
 * header documents as errors, which the library rejects on the host before any
 * HIP call, and checks the status codes and strings.  Exit status 0 = all
 * checks held; otherwise the number of the first failed check.
 */
#include <stdio.h>
#include <string.h>

#include "fp4attn.h"

#define CHECK(n, cond)                                  \
  do {                                                  \
    if (!(cond)) {                                      \
      fprintf(stderr, "check %d failed: %s\n", n, #cond); \
      return n;                                         \
    }                                                   \
  } while (0)

int main(void) {
  /* aligned, never dereferenced: every call below is refused before it could be */
  uint8_t* p = (uint8_t*)(uintptr_t)4096;
  void* out = (void*)(uintptr_t)8192;
  fp4attn_forward_options o;

  CHECK(1, fp4attn_abi_version() >> 16 == 2);
  CHECK(2, strcmp(fp4attn_status_string(FP4ATTN_OK), "ok") == 0);
  CHECK(3, fp4attn_forward_mxfp4(NULL, p, p, p, p, p, 1, 1, 128, 64, 0.125f, 1.5f, 1.2f, out, FP4ATTN_F32, NULL) ==
               FP4ATTN_ERR_INVALID_ARG);
  CHECK(4, strstr(fp4attn_last_error(), "q_codes") != NULL);
  CHECK(5, fp4attn_forward_mxfp4(p, p, p, p, p, p, 1, 1, 100, 64, 0.125f, 1.5f, 1.2f, out, FP4ATTN_F32, NULL) ==
               FP4ATTN_ERR_INVALID_ARG);                                         /* N not a multiple of 128 */
  CHECK(6, fp4attn_forward_mxfp4(p, p, p, p, p, p, 1, 1, 128, 96, 0.125f, 1.5f, 1.2f, out, FP4ATTN_F32, NULL) ==
               FP4ATTN_ERR_UNSUPPORTED);                                         /* d = 96 */
  CHECK(7, fp4attn_forward_bf16(p, p, NULL, 1, 1, 128, 64, 0.125f, out, FP4ATTN_F32, NULL) ==
               FP4ATTN_ERR_INVALID_ARG);                                         /* null v */
  CHECK(8, fp4attn_quantize_mxfp4(p, FP4ATTN_BF16, 1, 4, 48, 1, p, p, NULL) == FP4ATTN_ERR_INVALID_ARG);
  fp4attn_forward_options_init(&o);
  CHECK(9, o.struct_size == sizeof(o) && o.ex2_pairs == 0 && o.lse == NULL);
  o.ex2_pairs = 3;
  CHECK(10, fp4attn_forward_mxfp4_ex(p, p, p, p, p, p, 1, 1, 128, 64, 0.125f, &o, out, FP4ATTN_F32, NULL) ==
                FP4ATTN_ERR_INVALID_ARG);                                        /* 3 pairs of 16 */
  printf("c-abi validation: all checks held\n");
  return 0;
}
