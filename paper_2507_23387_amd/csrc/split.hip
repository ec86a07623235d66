// Split kernels: FP32 -> (FP16 high word, FP16 scaled residual).
//
// Sec. 3.3 and Eq. recover_eqn of arXiv 2507.23387:
//   hi = fl16(a); r = a - hi (exact in FP32); lo = fl16(r * s)
// with fl16 = round to nearest even and gradual underflow.  On gfx950:
//   - v_cvt_f16_f32 rounds with the MODE register's round mode (RNE by
//     default) and keeps FP16 denormals (the kernels are built with the
//     default float_denorm_mode_16_64 = 3, never with flush-to-zero);
//   - the FP32 subtraction keeps FP32 denormals (float_denorm_mode_32 = 3);
//   - the compiler may fuse r * s and the conversion into v_fma_mixlo_f16,
//     which rounds once; r * s is exact because s is a power of two (checked
//     by the C-ABI), so this equals the two-step definition bit for bit.
// Both kernels are HBM-bound elementwise passes: 4 B read and 4 B written
// (hi + lo) per element.
#include "internal.h"

namespace sgc {
namespace {

__device__ __forceinline__ void split_value(float a, float s, uint16_t& hi, uint16_t& lo) {
  const _Float16 h = static_cast<_Float16>(a);
  const float r = a - static_cast<float>(h);
  const _Float16 l = static_cast<_Float16>(r * s);
  hi = __builtin_bit_cast(uint16_t, h);
  lo = __builtin_bit_cast(uint16_t, l);
}

// Row-major split.  Thread = 4 consecutive columns of one row; blockIdx.y
// strides over rows.  kVec: X rows are 16-byte aligned and hi/lo rows 8-byte
// aligned, so whole quads move as float4 / 8-byte stores.
template <bool kVec>
__global__ __launch_bounds__(256) void split_rows_kernel(
    int64_t rows, int64_t cols, const float* __restrict__ X, int64_t ldx,
    uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int64_t ldh, int64_t rows_pad,
    int64_t cols_pad, float s) {
  const int64_t c0 = (static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x) * 4;
  if (c0 >= cols_pad) return;
  for (int64_t i = blockIdx.y; i < rows_pad; i += gridDim.y) {
    float v[4];
    if (kVec && i < rows && c0 + 3 < cols) {
      const float4 f = *reinterpret_cast<const float4*>(X + i * ldx + c0);
      v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = (i < rows && c0 + e < cols) ? X[i * ldx + c0 + e] : 0.0f;
    }
    uint16_t h[4], l[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) split_value(v[e], s, h[e], l[e]);
    uint16_t* hrow = hi + i * ldh + c0;
    uint16_t* lrow = lo + i * ldh + c0;
    if (kVec && c0 + 3 < cols_pad) {
      const uint2 hv = {static_cast<uint32_t>(h[0]) | (static_cast<uint32_t>(h[1]) << 16),
                        static_cast<uint32_t>(h[2]) | (static_cast<uint32_t>(h[3]) << 16)};
      const uint2 lv = {static_cast<uint32_t>(l[0]) | (static_cast<uint32_t>(l[1]) << 16),
                        static_cast<uint32_t>(l[2]) | (static_cast<uint32_t>(l[3]) << 16)};
      *reinterpret_cast<uint2*>(hrow) = hv;
      *reinterpret_cast<uint2*>(lrow) = lv;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (c0 + e < cols_pad) {
          hrow[e] = h[e];
          lrow[e] = l[e];
        }
    }
  }
}

// Transposing split of B (K x N row-major) into Np x Kp k-contiguous planes.
// A 64 (k) x 64 (n) tile per workgroup: coalesced row reads along n, split in
// registers, transpose through LDS, coalesced 32-byte row writes along k.
__global__ __launch_bounds__(256) void split_cols_t_kernel(
    int64_t K, int64_t N, const float* __restrict__ B, int64_t ldb,
    uint16_t* __restrict__ hi_t, uint16_t* __restrict__ lo_t, int64_t Kp, float s) {
  constexpr int kPitch = 66;  // halves per LDS row (64 + 2): spreads banks
  __shared__ uint16_t sh[64 * kPitch];
  __shared__ uint16_t sl[64 * kPitch];
  const int64_t k0 = static_cast<int64_t>(blockIdx.x) * 64;
  const int64_t n0 = static_cast<int64_t>(blockIdx.y) * 64;
  const int t = threadIdx.x;
  {
    const int n = t & 63;
    const int kq = t >> 6;
    const int64_t gn = n0 + n;
#pragma unroll 4
    for (int r = 0; r < 16; ++r) {
      const int k = kq + 4 * r;
      const int64_t gk = k0 + k;
      const float a = (gk < K && gn < N) ? B[gk * ldb + gn] : 0.0f;
      uint16_t h, l;
      split_value(a, s, h, l);
      sh[n * kPitch + k] = h;
      sl[n * kPitch + k] = l;
    }
  }
  __syncthreads();
  {
    const int n = t >> 2;
    const int kc = (t & 3) * 16;
    uint32_t hv[8], lv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      hv[e] = static_cast<uint32_t>(sh[n * kPitch + kc + 2 * e]) |
              (static_cast<uint32_t>(sh[n * kPitch + kc + 2 * e + 1]) << 16);
      lv[e] = static_cast<uint32_t>(sl[n * kPitch + kc + 2 * e]) |
              (static_cast<uint32_t>(sl[n * kPitch + kc + 2 * e + 1]) << 16);
    }
    uint4* hdst = reinterpret_cast<uint4*>(hi_t + (n0 + n) * Kp + k0 + kc);
    uint4* ldst = reinterpret_cast<uint4*>(lo_t + (n0 + n) * Kp + k0 + kc);
    hdst[0] = uint4{hv[0], hv[1], hv[2], hv[3]};
    hdst[1] = uint4{hv[4], hv[5], hv[6], hv[7]};
    ldst[0] = uint4{lv[0], lv[1], lv[2], lv[3]};
    ldst[1] = uint4{lv[4], lv[5], lv[6], lv[7]};
  }
}

__global__ __launch_bounds__(256) void zero_kernel(int64_t M, int64_t N, float* __restrict__ C,
                                                   int64_t ldc) {
  const int64_t j = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (j >= N) return;
  for (int64_t i = blockIdx.y; i < M; i += gridDim.y) C[i * ldc + j] = 0.0f;
}

inline unsigned grid_rows(int64_t rows) {
  return static_cast<unsigned>(rows < 65535 ? (rows > 0 ? rows : 1) : 65535);
}

}  // namespace

hipError_t launch_split_rows(int64_t rows, int64_t cols, const float* X, int64_t ldx,
                             uint16_t* hi, uint16_t* lo, int64_t ldh, int64_t rows_pad,
                             int64_t cols_pad, float scale, hipStream_t stream) {
  if (rows_pad <= 0 || cols_pad <= 0) return hipSuccess;
  const int64_t quads = (cols_pad + 3) / 4;
  const dim3 grid(static_cast<unsigned>((quads + 255) / 256), grid_rows(rows_pad));
  const bool vec = (reinterpret_cast<uintptr_t>(X) % 16 == 0) && (ldx % 4 == 0) &&
                   (reinterpret_cast<uintptr_t>(hi) % 8 == 0) &&
                   (reinterpret_cast<uintptr_t>(lo) % 8 == 0) && (ldh % 4 == 0);
  if (vec)
    hipLaunchKernelGGL(split_rows_kernel<true>, grid, dim3(256), 0, stream, rows, cols, X, ldx,
                       hi, lo, ldh, rows_pad, cols_pad, scale);
  else
    hipLaunchKernelGGL(split_rows_kernel<false>, grid, dim3(256), 0, stream, rows, cols, X, ldx,
                       hi, lo, ldh, rows_pad, cols_pad, scale);
  return hipGetLastError();
}

hipError_t launch_split_cols_transposed(int64_t K, int64_t N, const float* B, int64_t ldb,
                                        uint16_t* hi_t, uint16_t* lo_t, int64_t Np,
                                        int64_t Kp, float scale, hipStream_t stream) {
  // Np and Kp are multiples of 64 (plan_planes pads them to the GEMM tiles).
  const dim3 grid(static_cast<unsigned>(Kp / 64), static_cast<unsigned>(Np / 64));
  hipLaunchKernelGGL(split_cols_t_kernel, grid, dim3(256), 0, stream, K, N, B, ldb, hi_t, lo_t,
                     Kp, scale);
  return hipGetLastError();
}

hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((N + 255) / 256), grid_rows(M));
  hipLaunchKernelGGL(zero_kernel, grid, dim3(256), 0, stream, M, N, C, ldc);
  return hipGetLastError();
}

}  // namespace sgc
