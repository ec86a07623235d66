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
// All split kernels are HBM-bound elementwise passes: 4 B read and 4 B
// written (hi + lo) per element.
#include "internal.h"

namespace sgc {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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

// Split of A into the tiled planes.  Thread = 8 consecutive k of one row (one
// 16-byte chunk of each output plane); a workgroup covers 4 rows x 512 k, so
// each wave reads 2 KiB of one row contiguously and the four rows of a
// workgroup complete every 128-byte line they write.  blockIdx.y strides
// over row quads.
template <bool kVec>
__global__ __launch_bounds__(256) void split_a_tiled_kernel(
    int64_t M, int64_t K, const float* __restrict__ X, int64_t ldx, uint16_t* __restrict__ hi,
    uint16_t* __restrict__ lo, int64_t Mp, int64_t Kp, float s) {
  const int64_t k0 = (static_cast<int64_t>(blockIdx.x) * 64 + (threadIdx.x & 63)) * 8;
  if (k0 >= Kp) return;
  for (int64_t m = static_cast<int64_t>(blockIdx.y) * 4 + (threadIdx.x >> 6); m < Mp;
       m += static_cast<int64_t>(gridDim.y) * 4) {
    float v[8];
    if (kVec && m < M && k0 + 7 < K) {
      const float4* src = reinterpret_cast<const float4*>(X + m * ldx + k0);
      const float4 f0 = src[0], f1 = src[1];
      v[0] = f0.x; v[1] = f0.y; v[2] = f0.z; v[3] = f0.w;
      v[4] = f1.x; v[5] = f1.y; v[6] = f1.z; v[7] = f1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (m < M && k0 + e < K) ? X[m * ldx + k0 + e] : 0.0f;
    }
    u32x4 hv, lv;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint16_t h0, l0, h1, l1;
      split_value(v[2 * e], s, h0, l0);
      split_value(v[2 * e + 1], s, h1, l1);
      hv[e] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
      lv[e] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
    }
    const int64_t idx = tiled_index(m, k0, Kp);
    *reinterpret_cast<u32x4*>(hi + idx) = hv;
    *reinterpret_cast<u32x4*>(lo + idx) = lv;
  }
}

// Split of B (K x N row-major) into the tiled planes of B transposed.  One
// workgroup = one 128 (n) x 16 (k) tile: thread t reads 8 consecutive n of
// row k = t / 16 (each wave reads four 512-byte row pieces), the split values
// are transposed through LDS, and thread t writes 16-byte chunk t of the 4 KiB
// tile of each plane.  It also raises the range flag when some
// |B_hi| * s > 65504 (the largest finite FP16 value).
template <bool kVec>
__global__ __launch_bounds__(256) void split_b_tiled_kernel(
    int64_t K, int64_t N, const float* __restrict__ B, int64_t ldb, uint16_t* __restrict__ hi,
    uint16_t* __restrict__ lo, int64_t Kp, float s, int* __restrict__ range_flag) {
  constexpr int kPitch = kSlice + 2;  // halves per LDS row: 36 bytes spread the banks
  __shared__ uint16_t sh[kPanel * kPitch];
  __shared__ uint16_t sl[kPanel * kPitch];
  const int t = threadIdx.x;
  const int64_t slice = blockIdx.x;
  const int64_t panel = blockIdx.y;
  {
    const int kl = t >> 4;
    const int nl = (t & 15) * 8;
    const int64_t k = slice * kSlice + kl;
    const int64_t n = panel * kPanel + nl;
    float v[8];
    if (kVec && k < K && n + 7 < N) {
      const float4* src = reinterpret_cast<const float4*>(B + k * ldb + n);
      const float4 f0 = src[0], f1 = src[1];
      v[0] = f0.x; v[1] = f0.y; v[2] = f0.z; v[3] = f0.w;
      v[4] = f1.x; v[5] = f1.y; v[6] = f1.z; v[7] = f1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = (k < K && n + e < N) ? B[k * ldb + n + e] : 0.0f;
    }
    bool big = false;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint16_t h, l;
      split_value(v[e], s, h, l);
      big |= __builtin_fabsf(static_cast<float>(__builtin_bit_cast(_Float16, h))) * s > 65504.0f;
      sh[(nl + e) * kPitch + kl] = h;
      sl[(nl + e) * kPitch + kl] = l;
    }
    if (big) *range_flag = 1;
  }
  __syncthreads();
  {
    const int r = t >> 1;
    const int c = (t & 1) ^ tile_swizzle(r);  // logical chunk stored at position t & 1
    const uint16_t* hrow = sh + r * kPitch + c * 8;
    const uint16_t* lrow = sl + r * kPitch + c * 8;
    u32x4 hv, lv;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      hv[e] = static_cast<uint32_t>(hrow[2 * e]) | (static_cast<uint32_t>(hrow[2 * e + 1]) << 16);
      lv[e] = static_cast<uint32_t>(lrow[2 * e]) | (static_cast<uint32_t>(lrow[2 * e + 1]) << 16);
    }
    const int64_t base = (panel * (Kp / kSlice) + slice) * kTileHalves + t * 8;
    *reinterpret_cast<u32x4*>(hi + base) = hv;
    *reinterpret_cast<u32x4*>(lo + base) = lv;
  }
}

__global__ void flag_reset_kernel(int* range_flag) { *range_flag = 0; }

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
                             uint16_t* hi, uint16_t* lo, int64_t ldh, float scale,
                             hipStream_t stream) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  const int64_t quads = (cols + 3) / 4;
  const dim3 grid(static_cast<unsigned>((quads + 255) / 256), grid_rows(rows));
  const bool vec = (reinterpret_cast<uintptr_t>(X) % 16 == 0) && (ldx % 4 == 0) &&
                   (reinterpret_cast<uintptr_t>(hi) % 8 == 0) &&
                   (reinterpret_cast<uintptr_t>(lo) % 8 == 0) && (ldh % 4 == 0);
  if (vec)
    hipLaunchKernelGGL(split_rows_kernel<true>, grid, dim3(256), 0, stream, rows, cols, X, ldx,
                       hi, lo, ldh, rows, cols, scale);
  else
    hipLaunchKernelGGL(split_rows_kernel<false>, grid, dim3(256), 0, stream, rows, cols, X, ldx,
                       hi, lo, ldh, rows, cols, scale);
  return hipGetLastError();
}

hipError_t launch_split_a(const Planes& p, int64_t M, int64_t K, const float* A, int64_t lda,
                          float scale, hipStream_t stream) {
  // Mp is a multiple of 256 and Kp of 64 (plan_planes).
  const dim3 grid(static_cast<unsigned>((p.Kp + 511) / 512), grid_rows(p.Mp / 4));
  const bool vec = (reinterpret_cast<uintptr_t>(A) % 16 == 0) && (lda % 4 == 0);
  if (vec)
    hipLaunchKernelGGL(split_a_tiled_kernel<true>, grid, dim3(256), 0, stream, M, K, A, lda,
                       p.a_hi, p.a_lo, p.Mp, p.Kp, scale);
  else
    hipLaunchKernelGGL(split_a_tiled_kernel<false>, grid, dim3(256), 0, stream, M, K, A, lda,
                       p.a_hi, p.a_lo, p.Mp, p.Kp, scale);
  return hipGetLastError();
}

hipError_t launch_split_b(const Planes& p, int64_t K, int64_t N, const float* B, int64_t ldb,
                          float scale, hipStream_t stream) {
  hipLaunchKernelGGL(flag_reset_kernel, dim3(1), dim3(1), 0, stream, p.range_flag);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // One workgroup per tile: Kp / 16 slices x Np / 128 panels (Np / 128 <= 65535
  // is checked by the C-ABI).
  const dim3 grid(static_cast<unsigned>(p.Kp / kSlice), static_cast<unsigned>(p.Np / kPanel));
  const bool vec = (reinterpret_cast<uintptr_t>(B) % 16 == 0) && (ldb % 4 == 0);
  if (vec)
    hipLaunchKernelGGL(split_b_tiled_kernel<true>, grid, dim3(256), 0, stream, K, N, B, ldb,
                       p.b_hi, p.b_lo, p.Kp, scale, p.range_flag);
  else
    hipLaunchKernelGGL(split_b_tiled_kernel<false>, grid, dim3(256), 0, stream, K, N, B, ldb,
                       p.b_hi, p.b_lo, p.Kp, scale, p.range_flag);
  return hipGetLastError();
}

hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((N + 255) / 256), grid_rows(M));
  hipLaunchKernelGGL(zero_kernel, grid, dim3(256), 0, stream, M, N, C, ldc);
  return hipGetLastError();
}

}  // namespace sgc
