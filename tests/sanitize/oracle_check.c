/*
 * Drives the CPU oracle (oracle/oracle.c, test infrastructure) under the host
 * AddressSanitizer and UndefinedBehaviorSanitizer: every exported function on
 * small and degenerate inputs, padded leading dimensions, one and several
 * OpenMP threads, and the argument errors.  The values are checked loosely
 * (the oracle's exact pins live in the Python tests); what this program is
 * for is that no call reads or writes outside its buffers or hits undefined
 * behaviour.  Exit status 0 = all checks passed; the sanitizers abort on
 * their first report.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

uint16_t oracle_f32_to_f16_bits(uint32_t x);
uint32_t oracle_f16_to_f32_bits(uint16_t h);
void oracle_convert_range(uint64_t start, uint64_t count, uint16_t* out);
void oracle_convert_array(int64_t n, const float* x, uint16_t* out);
void oracle_widen_array(int64_t n, const uint16_t* h, float* out);
int oracle_split(int64_t rows, int64_t cols, const float* X, int64_t ldx, uint16_t* hi,
                 uint16_t* lo, int64_t ldh, float scale);
int oracle_sgemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                 int64_t ldb, float* C, int64_t ldc, float scale, int order, int64_t kb,
                 int nthreads);
int oracle_max_threads(void);

static int failures = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                    \
    }                                                                \
  } while (0)

static uint32_t bits(float x) {
  uint32_t u;
  memcpy(&u, &x, 4);
  return u;
}

static float from_bits(uint32_t u) {
  float x;
  memcpy(&x, &u, 4);
  return x;
}

/* Deterministic values in [-1, 1) from a 64-bit LCG (Knuth's MMIX constants). */
static uint64_t lcg_state = 12345;
static float next_value(void) {
  lcg_state = lcg_state * 6364136223846793005ULL + 1442695040888963407ULL;
  return (float)((double)(lcg_state >> 11) / 9007199254740992.0 * 2.0 - 1.0);
}

static void check_conversions(void) {
  CHECK(oracle_f32_to_f16_bits(bits(1.0f)) == 0x3c00);
  CHECK(oracle_f32_to_f16_bits(bits(-2.0f)) == 0xc000);
  CHECK(oracle_f32_to_f16_bits(bits(65520.0f)) == 0x7c00);
  CHECK(oracle_f32_to_f16_bits(bits(65504.0f)) == 0x7bff);
  CHECK(oracle_f32_to_f16_bits(bits(ldexpf(1.0f, -24))) == 0x0001);
  CHECK(oracle_f32_to_f16_bits(bits(ldexpf(1.0f, -25))) == 0x0000);
  CHECK((oracle_f32_to_f16_bits(0x7fc00000u) & 0x7c00) == 0x7c00);
  CHECK(oracle_f16_to_f32_bits(0x3c00) == bits(1.0f));
  CHECK(oracle_f16_to_f32_bits(0x0001) == bits(ldexpf(1.0f, -24)));
  /* A strided walk over all 2^32 patterns, through the range converter. */
  enum { kChunk = 4096 };
  uint16_t* out = malloc(kChunk * sizeof(uint16_t));
  for (uint64_t start = 0; start < (1ULL << 32); start += 1ULL << 22) {
    oracle_convert_range(start, kChunk, out);
    for (int i = 0; i < kChunk; ++i)
      CHECK(out[i] == oracle_f32_to_f16_bits((uint32_t)(start + (uint64_t)i)));
  }
  oracle_convert_range(0xffffffffULL - kChunk + 1, kChunk, out);
  free(out);
  /* Round trip of every FP16 pattern through the array converters. */
  uint16_t* h = malloc(65536 * sizeof(uint16_t));
  uint16_t* h2 = malloc(65536 * sizeof(uint16_t));
  float* w = malloc(65536 * sizeof(float));
  for (int i = 0; i < 65536; ++i) h[i] = (uint16_t)i;
  oracle_widen_array(65536, h, w);
  oracle_convert_array(65536, w, h2);
  for (int i = 0; i < 65536; ++i) {
    const int nan = (i & 0x7c00) == 0x7c00 && (i & 0x3ff);
    CHECK(nan ? (h2[i] & 0x7c00) == 0x7c00 && (h2[i] & 0x3ff) : h2[i] == h[i]);
  }
  oracle_convert_array(0, w, h2);
  oracle_widen_array(0, h, w);
  free(h);
  free(h2);
  free(w);
}

static void check_split(void) {
  const int64_t rows = 33, cols = 47, ldx = 50, ldh = 49;
  float* X = malloc(sizeof(float) * rows * ldx);
  uint16_t* hi = malloc(sizeof(uint16_t) * rows * ldh);
  uint16_t* lo = malloc(sizeof(uint16_t) * rows * ldh);
  for (int64_t i = 0; i < rows * ldx; ++i) X[i] = next_value() * 100.0f;
  X[0] = 1.0f;
  X[1] = from_bits(0x7f800000u);
  CHECK(oracle_split(rows, cols, X, ldx, hi, lo, ldh, 2048.0f) == 0);
  CHECK(hi[0] == 0x3c00 && lo[0] == 0);
  CHECK(hi[1] == 0x7c00);
  for (int64_t i = 0; i < rows; ++i)
    for (int64_t j = 0; j < cols; ++j) {
      const float a = X[i * ldx + j];
      if (!isfinite(a)) continue;
      const float h = from_bits(oracle_f16_to_f32_bits(hi[i * ldh + j]));
      const float l = from_bits(oracle_f16_to_f32_bits(lo[i * ldh + j]));
      CHECK(fabs((double)h + (double)l / 2048.0 - (double)a) <= fabs((double)a) * 1e-6 + 1e-9);
    }
  CHECK(oracle_split(0, cols, X, ldx, hi, lo, ldh, 2048.0f) == 0);
  CHECK(oracle_split(rows, 0, X, ldx, hi, lo, ldh, 2048.0f) == 0);
  free(X);
  free(hi);
  free(lo);
}

/* C against an FP64 GEMM of the same FP32 inputs: within 2K u32 |A||B| plus
 * the dropped lo*lo term, far inside the check for values in [-1, 1). */
static void check_gemm_case(int64_t M, int64_t N, int64_t K, int64_t pad, int order, int64_t kb,
                            int threads) {
  const int64_t lda = K + pad, ldb = N + pad, ldc = N + pad;
  float* A = malloc(sizeof(float) * (size_t)(M * lda + 1));
  float* B = malloc(sizeof(float) * (size_t)(K * ldb + 1));
  float* C = malloc(sizeof(float) * (size_t)(M * ldc + 1));
  for (int64_t i = 0; i < M * lda; ++i) A[i] = next_value();
  for (int64_t i = 0; i < K * ldb; ++i) B[i] = next_value();
  for (int64_t i = 0; i < M * ldc; ++i) C[i] = NAN;
  CHECK(oracle_sgemm(M, N, K, A, lda, B, ldb, C, ldc, 2048.0f, order, kb, threads) == 0);
  for (int64_t i = 0; i < M; ++i)
    for (int64_t j = 0; j < N; ++j) {
      double ref = 0.0, mag = 0.0;
      for (int64_t k = 0; k < K; ++k) {
        ref += (double)A[i * lda + k] * (double)B[k * ldb + j];
        mag += fabs((double)A[i * lda + k] * (double)B[k * ldb + j]);
      }
      const double tol = (order == 2 ? 1e-3 : 4.0 * (double)K * ldexp(1.0, -24)) * mag + 1e-30;
      CHECK(fabs((double)C[i * ldc + j] - ref) <= tol);
    }
  free(A);
  free(B);
  free(C);
}

static void check_gemm(void) {
  const int threads = oracle_max_threads();
  CHECK(threads >= 1);
  for (int order = 0; order <= 3; ++order) {
    check_gemm_case(17, 19, 70, 3, order, 32, 1);
    check_gemm_case(9, 33, 64, 0, order, 64, threads);
    check_gemm_case(1, 1, 1, 0, order, 1, 2);
    check_gemm_case(5, 7, 100, 1, order, 7, 0);
  }
  /* K = 0 writes zeros; M = 0 or N = 0 touches nothing. */
  float A[4] = {1, 2, 3, 4}, B[4] = {1, 2, 3, 4}, C[4] = {NAN, NAN, NAN, NAN};
  CHECK(oracle_sgemm(2, 2, 0, A, 1, B, 2, C, 2, 2048.0f, 0, 32, 1) == 0);
  CHECK(C[0] == 0.0f && C[3] == 0.0f);
  CHECK(oracle_sgemm(0, 2, 2, A, 2, B, 2, C, 2, 2048.0f, 0, 32, 1) == 0);
  CHECK(oracle_sgemm(2, 0, 2, A, 2, B, 2, C, 2, 2048.0f, 1, 32, 1) == 0);
  /* Argument errors. */
  CHECK(oracle_sgemm(-1, 2, 2, A, 2, B, 2, C, 2, 2048.0f, 0, 32, 1) == -1);
  CHECK(oracle_sgemm(2, 2, 2, A, 2, B, 2, C, 2, 2048.0f, 4, 32, 1) == -1);
  CHECK(oracle_sgemm(2, 2, 2, A, 2, B, 2, C, 2, 2048.0f, 0, 0, 1) == -1);
}

int main(void) {
  check_conversions();
  check_split();
  check_gemm();
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("oracle_check: all checks passed\n");
  return 0;
}
