/* A plain C11 program against libsgemmcube: the header compiles as C and the
 * entry points link and run from C.  Only calls that return before any device
 * work (queries and argument validation), so it runs without a GPU.  Prints
 * the number of failed checks and exits with it. */
#include <stdio.h>
#include <string.h>

#include "sgemm_cube.h"

#define CHECK(x)                                              \
  do {                                                        \
    if (!(x)) {                                               \
      fprintf(stderr, "%s:%d: failed: %s\n", __FILE__, __LINE__, #x); \
      ++bad;                                                  \
    }                                                         \
  } while (0)

int main(void) {
  int bad = 0;
  const float* A = (const float*)(uintptr_t)(1ull << 40);
  const float* B = (const float*)(uintptr_t)((1ull << 40) + (1ull << 30));
  float* C = (float*)(uintptr_t)((1ull << 40) + (2ull << 30));
  CHECK(sgemm_cube_block_k() == 32);
  CHECK(strcmp(sgemm_cube_status_string(SGEMM_CUBE_ERR_INVALID_VALUE),
               "SGEMM_CUBE_ERR_INVALID_VALUE") == 0);
  CHECK(sgemm_cube_workspace_size(8192, 8192, 8192, SGEMM_CUBE_ELEMENTWISE) ==
        256 + (size_t)4 * 8192 * 8192 * 2);
  CHECK(sgemm_cube_ex_workspace_size(300, 200, 128, SGEMM_CUBE_TERMWISE,
                                     SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM) ==
        sgemm_cube_workspace_size(300, 200, 128, SGEMM_CUBE_TERMWISE));
  /* Validation only. */
  CHECK(sgemm_cube(0, 4, 4, NULL, 4, B, 4, NULL, 4, 2048.0f, SGEMM_CUBE_TERMWISE, NULL) ==
        SGEMM_CUBE_OK);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 4, 3.0f, SGEMM_CUBE_ELEMENTWISE, NULL) ==
        SGEMM_CUBE_ERR_INVALID_VALUE);
  CHECK(sgemm_cube(4, 4, 4, A, 3, B, 4, C, 4, 2048.0f, SGEMM_CUBE_ELEMENTWISE, NULL) ==
        SGEMM_CUBE_ERR_INVALID_VALUE);
  CHECK(sgemm_cube_splits_a_in_gemm(1024, 1024, 1024, A, 1024, 2048.0f,
                                    SGEMM_CUBE_ELEMENTWISE) == 1);
  CHECK(sgemm_cube_splits_a_in_gemm(1024, 8192, 1024, A, 1024, 2048.0f,
                                    SGEMM_CUBE_ELEMENTWISE) == 0);
  printf("%d\n", bad);
  return bad;
}
