// Range extensions around the split (the exponent management and overflow
// detection that Sec. 4.2 leaves out of scope and Sec. 7 and 8 list as the way
// to widen the method's range):
//   - power-of-two pre-scaling: the largest finite magnitude of every row of A
//     and every column of B is measured, the splits multiply the row (column)
//     by the power of two that brings it to a fixed exponent, and the product
//     is scaled back entry by entry, C_ij = 2^-(p_i + q_j) C'_ij (exact unless
//     C_ij is FP32-subnormal);
//   - the range report: the OR of the range classes the splits stamped.
#include "internal.h"

namespace sgc {
namespace {

// Largest finite |A[i, :]| per row, one workgroup per row; as a side job the
// grid also clears the column maxima that absmax_cols_kernel raises next.
__global__ __launch_bounds__(256) void absmax_rows_kernel(int64_t M, int64_t K,
                                                          const float* __restrict__ A,
                                                          int64_t lda,
                                                          uint32_t* __restrict__ row_max,
                                                          uint32_t* __restrict__ col_max,
                                                          int64_t Np) {
  __shared__ float part[4];
  const int t = threadIdx.x;
  for (int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + t; j < Np;
       j += static_cast<int64_t>(gridDim.x) * 256)
    col_max[j] = 0u;
  for (int64_t i = blockIdx.x; i < M; i += gridDim.x) {
    float m = 0.0f;
    for (int64_t k = t; k < K; k += 256) {
      const float a = __builtin_fabsf(A[i * lda + k]);
      if (a <= 3.4028235e38f) m = __builtin_fmaxf(m, a);  // skips inf and NaN
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = __builtin_fmaxf(m, __shfl_xor(m, off));
    if ((t & 63) == 0) part[t >> 6] = m;
    __syncthreads();
    if (t == 0)
      row_max[i] = __builtin_bit_cast(
          uint32_t, __builtin_fmaxf(__builtin_fmaxf(part[0], part[1]),
                                    __builtin_fmaxf(part[2], part[3])));
    __syncthreads();
  }
}

// Largest finite |B[:, j]| per column: workgroup (column block, row block)
// reduces 64 rows of 256 columns and raises the column maxima atomically
// (non-negative floats order like their bit patterns).
__global__ __launch_bounds__(256) void absmax_cols_kernel(int64_t K, int64_t N,
                                                          const float* __restrict__ B,
                                                          int64_t ldb,
                                                          uint32_t* __restrict__ col_max) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= N) return;
  const int64_t k0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int64_t k1 = k0 + 64 < K ? k0 + 64 : K;
  float m = 0.0f;
  for (int64_t k = k0; k < k1; ++k) {
    const float b = __builtin_fabsf(B[k * ldb + j]);
    if (b <= 3.4028235e38f) m = __builtin_fmaxf(m, b);
  }
  if (m > 0.0f) atomicMax(col_max + j, __builtin_bit_cast(uint32_t, m));
}

// C_ij := 2^-(p_i + q_j) C_ij, one rounding (ldexp).
__global__ __launch_bounds__(256) void unscale_kernel(int64_t M, int64_t N, float* __restrict__ C,
                                                      int64_t ldc,
                                                      const uint32_t* __restrict__ row_max,
                                                      const uint32_t* __restrict__ col_max,
                                                      int exp_a, int exp_b) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (j >= N) return;
  const int q = prescale_shift(col_max[j], exp_b);
  for (int64_t i = blockIdx.y; i < M; i += gridDim.y) {
    const int p = prescale_shift(row_max[i], exp_a);
    C[i * ldc + j] = __builtin_ldexpf(C[i * ldc + j], -(p + q));
  }
}

// *out = OR of the range classes stamped by the last split of each operand.
__global__ void range_report_kernel(const uint32_t* __restrict__ range, int empty,
                                    uint32_t* __restrict__ out) {
  uint32_t bits = 0;
  if (!empty) {
    for (int b = 0; b < kRangeClasses; ++b) {
      if (range[kWordAClass + b] == range[kWordAStamp]) bits |= 1u << b;
      if (range[kWordBClass + b] == range[kWordBStamp]) bits |= 1u << b;
    }
  }
  *out = bits;
}

inline unsigned grid_y(int64_t rows) {
  return static_cast<unsigned>(rows < 65535 ? (rows > 0 ? rows : 1) : 65535);
}

}  // namespace

hipError_t launch_absmax(const Planes& p, int64_t M, int64_t N, int64_t K, const float* A,
                         int64_t lda, const float* B, int64_t ldb, hipStream_t stream) {
  const int64_t rows_grid = M < (int64_t{1} << 30) ? (M > 0 ? M : 1) : (int64_t{1} << 30);
  hipLaunchKernelGGL(absmax_rows_kernel, dim3(static_cast<unsigned>(rows_grid)), dim3(256), 0,
                     stream, M, K, A, lda, p.row_max, p.col_max, p.Np);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 grid(static_cast<unsigned>((N + 255) / 256), static_cast<unsigned>((K + 63) / 64));
  hipLaunchKernelGGL(absmax_cols_kernel, grid, dim3(256), 0, stream, K, N, B, ldb, p.col_max);
  return hipGetLastError();
}

hipError_t launch_unscale(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                          const RangeOpts& opt, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((N + 255) / 256), grid_y(M));
  hipLaunchKernelGGL(unscale_kernel, grid, dim3(256), 0, stream, M, N, C, ldc, p.row_max,
                     p.col_max, opt.exp_a, opt.exp_b);
  return hipGetLastError();
}

hipError_t launch_range_report(const Planes& p, bool empty, uint32_t* out, hipStream_t stream) {
  hipLaunchKernelGGL(range_report_kernel, dim3(1), dim3(1), 0, stream, p.range, empty ? 1 : 0,
                     out);
  return hipGetLastError();
}

}  // namespace sgc
