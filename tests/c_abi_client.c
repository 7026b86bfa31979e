/* A plain C99 client of the library: it includes the public header and links
 * against libtfm.so with the host C compiler, then calls the entry points that
 * need no GPU (queries and argument validation, which returns before anything
 * is enqueued).  Built and run by tests/test_abi.py; prints one line per check
 * and exits non-zero on the first failure. */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "tfm.h"

#define CHECK(cond)                                             \
  do {                                                          \
    if (!(cond)) {                                              \
      printf("FAIL line %d: %s\n", __LINE__, #cond);            \
      return 1;                                                 \
    }                                                           \
    printf("ok: %s\n", #cond);                                  \
  } while (0)

int main(void) {
  tfm_icl_options opts;
  void* p = malloc(64); /* a 16-byte aligned non-NULL pointer; never dereferenced by these calls */
  if (!p) return 1;
  memset(&opts, 0, sizeof(opts));
  CHECK(strcmp(tfm_status_string(TFM_OK), "TFM_OK") == 0);
  CHECK(tfm_version() > 0);
  CHECK(tfm_icl_attention_fp8_block_kv(64) == 128);
  CHECK(tfm_icl_attention_fp8_workspace_bytes(2, 6, 64, 65536, 16384) > 0);
  CHECK(tfm_icl_attention_fp8_workspace_bytes(2, 6, 64, 65536, 16384) >=
        tfm_icl_attention_fp8_workspace_bytes(2, 6, 64, 65536, 0));
  /* validation: bad shapes, dtypes, head dims and missing pointers are refused */
  CHECK(tfm_icl_attention_fp8(TFM_BF16, TFM_BF16, &opts, 0, 6, 64, 1024, 0, 0.125f, p, p, p, NULL, p, NULL, p,
                              1 << 20, NULL) == TFM_ERR_BAD_SHAPE);
  CHECK(tfm_icl_attention_fp8(7, TFM_BF16, NULL, 1, 6, 64, 1024, 0, 0.125f, p, p, p, NULL, p, NULL, p, 1 << 20,
                              NULL) == TFM_ERR_BAD_DTYPE);
  CHECK(tfm_icl_attention_fp8(TFM_BF16, TFM_BF16, NULL, 1, 6, 96, 1024, 0, 0.125f, p, p, p, NULL, p, NULL, p,
                              1 << 20, NULL) == TFM_ERR_UNSUPPORTED_HEAD_DIM);
  CHECK(tfm_icl_attention_fp8(TFM_BF16, TFM_BF16, NULL, 1, 6, 64, 1024, 0, 0.125f, NULL, p, p, NULL, p, NULL, p,
                              1 << 20, NULL) == TFM_ERR_NULL_PTR);
  CHECK(tfm_icl_attention_fp8_noalloc(TFM_BF16, TFM_BF16, NULL, 8, 8, 64, 65536, 0, 0.125f, p, p, p, NULL, p, NULL,
                                      NULL) == TFM_ERR_WORKSPACE_TOO_SMALL);
  CHECK(tfm_icl_attention_bf16(TFM_BF16, TFM_F32, NULL, 1, 1, 64, 16, 0, -1.0f, p, p, p, NULL, p, NULL, NULL) !=
        TFM_OK);
  free(p);
  printf("c client: all checks passed\n");
  return 0;
}
