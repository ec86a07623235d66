/*
 * SGEMM-cube CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct CPU implementation of what the FP32-accuracy
 * GEMM of arXiv 2507.23387 ("SGEMM-cube") computes.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load this library.
 * The HIP product path never links, loads or calls it, and it shares no code,
 * header, table or helper with that path.
 *
 * What it follows (paper sections / equation labels):
 *   - fl16 is round-to-nearest, ties-to-even, with gradual underflow
 *     (Sec. 3.2 notation table; Sec. 4.1, the 2^-25 halfway threshold).
 *   - The two-component split (Sec. 3.3 and Eq. recover_eqn, Sec. 4.3):
 *       hi = fl16(a),  r = a - hi  (exact in FP32),  lo = fl16(r * s_f).
 *   - Three FP16 products per k-block, FP32 accumulation, lo*lo dropped
 *     (Eq. recover_eqn).
 *   - Block structure g = 0..G of the contraction dimension and the two
 *     accumulation orders, Eq. elementwise and Eq. termwise (Sec. 4.5).
 *   - The per-block "cross terms first" order suggested at the end of
 *     Sec. 4.5 (the improved elementwise order).
 *
 * Arithmetic: every FP16 value is widened exactly to FP32; a product of two
 * FP16 values is exact in FP32 (at most 22 significant bits, magnitude within
 * [2^-48, 2^32]); every sum is one IEEE binary32 round-to-nearest addition,
 * in ascending k inside a block and ascending g across blocks.  Built without
 * -ffast-math and with -ffp-contract=off; FTZ/DAZ are never enabled.
 *
 * Parity status of each entry point is recorded in oracle/__init__.py.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Order codes (the same integers the product's C-ABI uses; written here
 * independently). */
#define ORACLE_ELEMENTWISE 0
#define ORACLE_TERMWISE 1
#define ORACLE_HI_ONLY 2
#define ORACLE_ELEMENTWISE_CROSS_FIRST 3

static uint32_t f32_bits(float x) {
  uint32_t u;
  memcpy(&u, &x, sizeof u);
  return u;
}

static float bits_f32(uint32_t u) {
  float x;
  memcpy(&x, &u, sizeof x);
  return x;
}

/*
 * fl16: binary32 -> binary16, round to nearest, ties to even, gradual
 * underflow (Sec. 3.2 notation table; Sec. 4.1 for the subnormal and
 * halfway-to-zero behaviour).  Done on the bit pattern so no host FP16
 * hardware or library conversion is involved.
 *
 *   |x| >= 65520           -> +-inf   (65520 is the halfway point between the
 *                                      largest finite FP16, 65504, and 2^16)
 *   2^-14 <= |x| < 65520   -> normal FP16, 10 stored mantissa bits
 *   |x| < 2^-14            -> FP16 subnormal: round(|x| / 2^-24) units of
 *                             2^-24; 2^-25 exactly is a tie and goes to 0
 *   NaN                    -> quiet NaN (payload not specified)
 */
uint16_t oracle_f32_to_f16_bits(uint32_t x) {
  uint32_t sign = (x >> 16) & 0x8000u;
  uint32_t ax = x & 0x7fffffffu;
  if (ax > 0x7f800000u) /* NaN */
    return (uint16_t)(sign | 0x7e00u | ((ax >> 13) & 0x1ffu));
  if (ax >= 0x477ff000u) /* >= 65520, includes inf */
    return (uint16_t)(sign | 0x7c00u);
  if (ax >= 0x38800000u) { /* >= 2^-14: result is a normal FP16 */
    /* Re-bias the exponent (127 -> 15) in place, then round away the low 13
     * mantissa bits.  A mantissa carry rolls into the exponent, which is the
     * correct next binade (and 65504 < |x| < 65520 cannot carry to inf). */
    uint32_t m = ax - (112u << 23);
    uint32_t keep = m >> 13;
    uint32_t rest = m & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (keep & 1u))) keep += 1u;
    return (uint16_t)(sign | keep);
  }
  if (ax < 0x33000000u) /* < 2^-25: below half the smallest subnormal */
    return (uint16_t)sign;
  {
    /* 2^-25 <= |x| < 2^-14, |x| normal in FP32.  |x| = M * 2^(e-150) with
     * the 24-bit significand M; in units of 2^-24 that is M / 2^(126-e). */
    uint32_t e = ax >> 23;
    uint32_t M = (ax & 0x7fffffu) | 0x800000u;
    uint32_t sh = 126u - e; /* in [14, 24] */
    uint32_t q = M >> sh;
    uint32_t rem = M & ((1u << sh) - 1u);
    uint32_t half = 1u << (sh - 1u);
    if (rem > half || (rem == half && (q & 1u))) q += 1u;
    return (uint16_t)(sign | q); /* q == 0x400 is the smallest normal */
  }
}

/* Exact widening binary16 -> binary32 (every FP16 value is an FP32 value). */
uint32_t oracle_f16_to_f32_bits(uint16_t h) {
  uint32_t sign = ((uint32_t)h & 0x8000u) << 16;
  uint32_t e = ((uint32_t)h >> 10) & 0x1fu;
  uint32_t m = (uint32_t)h & 0x3ffu;
  if (e == 0x1fu) return sign | 0x7f800000u | (m << 13); /* inf / NaN */
  if (e != 0u) return sign | ((e + 112u) << 23) | (m << 13);
  if (m == 0u) return sign;
  /* subnormal: m * 2^-24, m < 2^10, exactly representable */
  return f32_bits((float)m * 0x1p-24f) | sign;
}

static float widen(uint16_t h) { return bits_f32(oracle_f16_to_f32_bits(h)); }

/* Convert `count` consecutive FP32 bit patterns starting at `start` (used by
 * the exhaustive 2^32 check). */
void oracle_convert_range(uint64_t start, uint64_t count, uint16_t* out) {
#ifdef _OPENMP
#pragma omp parallel for schedule(static)
#endif
  for (uint64_t i = 0; i < count; ++i)
    out[i] = oracle_f32_to_f16_bits((uint32_t)(start + i));
}

void oracle_convert_array(int64_t n, const float* x, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = oracle_f32_to_f16_bits(f32_bits(x[i]));
}

void oracle_widen_array(int64_t n, const uint16_t* h, float* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = widen(h[i]);
}

/*
 * Two-component split of one FP32 value (Sec. 3.3; Eq. recover_eqn):
 *   hi = fl16(a)
 *   r  = a - hi          exact in FP32 (needs at most 24 significant bits)
 *   lo = fl16(r * s_f)   s_f a power of two, so r * s_f is exact
 */
static void split_one(float a, float scale, uint16_t* hi, uint16_t* lo) {
  uint16_t h = oracle_f32_to_f16_bits(f32_bits(a));
  float r = a - widen(h);
  float rs = r * scale;
  *hi = h;
  *lo = oracle_f32_to_f16_bits(f32_bits(rs));
}

/* Split a rows x cols row-major FP32 matrix (leading dimension ldx) into
 * row-major FP16 hi / lo planes (leading dimension ldh).  Returns 0. */
int oracle_split(int64_t rows, int64_t cols, const float* X, int64_t ldx, uint16_t* hi,
                 uint16_t* lo, int64_t ldh, float scale) {
#ifdef _OPENMP
#pragma omp parallel for schedule(static) if (rows * cols > 65536)
#endif
  for (int64_t i = 0; i < rows; ++i)
    for (int64_t j = 0; j < cols; ++j)
      split_one(X[i * ldx + j], scale, &hi[i * ldh + j], &lo[i * ldh + j]);
  return 0;
}

/*
 * C = SGEMM-cube(A, B) for row-major A (M x K, lda), B (K x N, ldb),
 * C (M x N, ldc), residual scale s_f, accumulation order, and k-block size kb
 * (blocks g = 0..G of the contraction dimension, the last one possibly
 * short).  nthreads <= 0 means "all available".
 *
 * Per output row i and block g, with the split planes widened to FP32:
 *   hh_g[j] = sum_{k in g} Ahi[i,k] Bhi[k,j]
 *   xa_g[j] = sum_{k in g} Alo[i,k] Bhi[k,j]     (R_A^[g] B^[g])
 *   xb_g[j] = sum_{k in g} Ahi[i,k] Blo[k,j]     (A^[g] R_B^[g])
 * each a sequential FP32 sum from +0 in ascending k.  Then
 *   ELEMENTWISE (Eq. elementwise):
 *       acc = ((acc + hh_g) + xa_g / s_f) + xb_g / s_f,   C = acc
 *   TERMWISE (Eq. termwise):
 *       HH += hh_g, XA += xa_g, XB += xb_g over g,  C = (HH + XA/s_f) + XB/s_f
 *   HI_ONLY (plain FP16 GEMM with FP32 accumulation, the HGEMM baseline):
 *       HH += hh_g, C = HH
 *   ELEMENTWISE_CROSS_FIRST (the reordering proposed at the end of Sec. 4.5):
 *       acc = acc + ((xa_g + xb_g) / s_f + hh_g),        C = acc
 * Division by s_f is multiplication by the exact power of two 1/s_f; it
 * cannot underflow because a nonzero block sum of FP16 x FP16 products is at
 * least 2^-48 in magnitude.
 *
 * Returns 0 on success, -1 on bad arguments, -2 if out of memory.
 */
int oracle_sgemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                 int64_t ldb, float* C, int64_t ldc, float scale, int order, int64_t kb,
                 int nthreads) {
  if (M < 0 || N < 0 || K < 0 || kb <= 0) return -1;
  if (order < ORACLE_ELEMENTWISE || order > ORACLE_ELEMENTWISE_CROSS_FIRST) return -1;
  if (M == 0 || N == 0) return 0;
  const float inv_s = 1.0f / scale;

  /* Split and widen the operands once. */
  float* ah = (float*)malloc(sizeof(float) * (size_t)(M * K + 1));
  float* al = (float*)malloc(sizeof(float) * (size_t)(M * K + 1));
  float* bh = (float*)malloc(sizeof(float) * (size_t)(K * N + 1));
  float* bl = (float*)malloc(sizeof(float) * (size_t)(K * N + 1));
  if (!ah || !al || !bh || !bl) {
    free(ah); free(al); free(bh); free(bl);
    return -2;
  }
  for (int64_t i = 0; i < M; ++i)
    for (int64_t k = 0; k < K; ++k) {
      uint16_t h, l;
      split_one(A[i * lda + k], scale, &h, &l);
      ah[i * K + k] = widen(h);
      al[i * K + k] = widen(l);
    }
  for (int64_t k = 0; k < K; ++k)
    for (int64_t j = 0; j < N; ++j) {
      uint16_t h, l;
      split_one(B[k * ldb + j], scale, &h, &l);
      bh[k * N + j] = widen(h);
      bl[k * N + j] = widen(l);
    }

  int failed = 0;
#ifdef _OPENMP
  if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel num_threads(nthreads) reduction(| : failed)
#endif
  {
    /* Per-thread row buffers: block partial sums and the running sums. */
    float* hh = (float*)malloc(sizeof(float) * (size_t)N);
    float* xa = (float*)malloc(sizeof(float) * (size_t)N);
    float* xb = (float*)malloc(sizeof(float) * (size_t)N);
    float* HH = (float*)malloc(sizeof(float) * (size_t)N);
    float* XA = (float*)malloc(sizeof(float) * (size_t)N);
    float* XB = (float*)malloc(sizeof(float) * (size_t)N);
    if (!hh || !xa || !xb || !HH || !XA || !XB) {
      failed = 1;
    } else {
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
      for (int64_t i = 0; i < M; ++i) {
        for (int64_t j = 0; j < N; ++j) HH[j] = XA[j] = XB[j] = 0.0f;
        for (int64_t k0 = 0; k0 < K; k0 += kb) {
          int64_t k1 = k0 + kb < K ? k0 + kb : K;
          for (int64_t j = 0; j < N; ++j) hh[j] = xa[j] = xb[j] = 0.0f;
          for (int64_t k = k0; k < k1; ++k) {
            const float a_h = ah[i * K + k], a_l = al[i * K + k];
            const float* bh_k = bh + k * N;
            const float* bl_k = bl + k * N;
            for (int64_t j = 0; j < N; ++j) {
              hh[j] = hh[j] + a_h * bh_k[j];
              xa[j] = xa[j] + a_l * bh_k[j];
              xb[j] = xb[j] + a_h * bl_k[j];
            }
          }
          switch (order) {
            case ORACLE_ELEMENTWISE:
              for (int64_t j = 0; j < N; ++j) {
                float t = HH[j] + hh[j];
                t = t + xa[j] * inv_s;
                HH[j] = t + xb[j] * inv_s;
              }
              break;
            case ORACLE_TERMWISE:
              for (int64_t j = 0; j < N; ++j) {
                HH[j] = HH[j] + hh[j];
                XA[j] = XA[j] + xa[j];
                XB[j] = XB[j] + xb[j];
              }
              break;
            case ORACLE_HI_ONLY:
              for (int64_t j = 0; j < N; ++j) HH[j] = HH[j] + hh[j];
              break;
            default: /* ORACLE_ELEMENTWISE_CROSS_FIRST */
              for (int64_t j = 0; j < N; ++j) {
                float cross = xa[j] + xb[j];
                float blk = cross * inv_s + hh[j];
                HH[j] = HH[j] + blk;
              }
              break;
          }
        }
        if (order == ORACLE_TERMWISE) {
          for (int64_t j = 0; j < N; ++j) {
            float t = HH[j] + XA[j] * inv_s;
            C[i * ldc + j] = t + XB[j] * inv_s;
          }
        } else {
          for (int64_t j = 0; j < N; ++j) C[i * ldc + j] = HH[j];
        }
      }
    }
    free(hh); free(xa); free(xb); free(HH); free(XA); free(XB);
  }
  free(ah); free(al); free(bh); free(bl);
  return failed ? -2 : 0;
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
