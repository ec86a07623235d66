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

// Range classes of one split entry a -> (hi, lo), after any pre-scaling:
//   1  a is inf or NaN
//   2  a is finite but fl16(a) is infinite (|a| >= 65520, Sec. 3.1)
//   4  hi is finite but the scaled residual overflows FP16 (Rule 2, Sec. 4.2)
//   8  hi is a nonzero FP16 subnormal (the 22-bit guarantee of Sec. 4.2 is lost)
__device__ __forceinline__ uint32_t range_class(float a, uint16_t h, uint16_t l) {
  const bool fin = __builtin_isfinite(a);
  const bool h_fin = (h & 0x7c00) != 0x7c00;
  uint32_t c = fin ? 0u : 1u;
  if (fin && !h_fin) c |= 2u;
  if (h_fin && (l & 0x7fff) == 0x7c00) c |= 4u;
  if ((h & 0x7c00) == 0 && (h & 0x03ff) != 0) c |= 8u;
  return c;
}

// Stamp the classes any lane of the wave saw into header words word..word+3
// (one store per class and wave).
__device__ __forceinline__ void report_classes(uint32_t cls, uint32_t* range, int word,
                                               uint32_t stamp) {
#pragma unroll
  for (int b = 0; b < kRangeClasses; ++b) {
    const unsigned long long m = __ballot((cls >> b) & 1u);
    if (m && static_cast<int>(threadIdx.x & 63) == __ffsll(static_cast<long long>(m)) - 1)
      range[word + b] = stamp;
  }
}

// Split of A into the tiled planes.  A workgroup covers 16 rows x 128 k and a
// wave 4 rows x 128 k: lane l takes 8 consecutive k of row l / 16, so each row
// is read as one 512-byte piece, and the 16-byte chunks a store instruction
// writes fill 8 whole 128-byte lines (4 rows x 32 bytes of one tile each).
// blockIdx.y strides over row blocks.
template <bool kVec, bool kPre, bool kReport>
__global__ __launch_bounds__(256) void split_a_tiled_kernel(
    int64_t M, int64_t K, const float* __restrict__ X, int64_t ldx, uint16_t* __restrict__ hi,
    uint16_t* __restrict__ lo, int64_t Mp, int64_t Kp, float s,
    const uint32_t* __restrict__ row_max, int exp_a, uint32_t* __restrict__ range,
    uint32_t stamp) {
  const int lane = threadIdx.x & 63;
  const int64_t k0 = static_cast<int64_t>(blockIdx.x) * 128 + (lane & 15) * 8;
  if (kReport && threadIdx.x == 0) range[kWordAStamp] = stamp;
  if (k0 >= Kp) return;
  uint32_t cls = 0;
  for (int64_t m = static_cast<int64_t>(blockIdx.y) * 16 + (threadIdx.x >> 6) * 4 + (lane >> 4);
       m < Mp; m += static_cast<int64_t>(gridDim.y) * 16) {
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
    if constexpr (kPre) {
      const int shift = m < M ? prescale_shift(row_max[m], exp_a) : 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = __builtin_ldexpf(v[e], shift);
    }
    u32x4 hv, lv;
    split8(v, s, hv, lv);
    if constexpr (kReport) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        cls |= range_class(v[2 * e], hv[e] & 0xffff, lv[e] & 0xffff);
        cls |= range_class(v[2 * e + 1], hv[e] >> 16, lv[e] >> 16);
      }
    }
    const int64_t idx = tiled_index(m, k0, Kp);
    store_stream(hi + idx, hv);
    store_stream(lo + idx, lv);
  }
  if constexpr (kReport) report_classes(cls, range, kWordAClass, stamp);
}

// Split of B (K x N row-major) into the tiled planes of B transposed.  One
// workgroup = 32 k x 128 n (two tiles): thread t splits rows k and k+1
// (k = 2 (t / 16)) at 8 consecutive n, each wave reading eight 512-byte row
// pieces.  The (k, k+1) pairs of hi and of lo go to LDS as 32-bit words, n-major,
// so each 16-byte chunk of a tile row is one LDS read; thread t then writes
// chunk t of both tiles of both planes (4 KiB contiguous per tile).  It also
// stamps the range flag (see launch_split_b) when some |B_hi| s > 65504, the
// largest finite FP16 value.
template <bool kVec, bool kPre, bool kReport>
__global__ __launch_bounds__(256) void split_b_tiled_kernel(
    int64_t K, int64_t N, const float* __restrict__ B, int64_t ldb, uint16_t* __restrict__ hi,
    uint16_t* __restrict__ lo, int64_t Kp, float s, const uint32_t* __restrict__ col_max,
    int exp_b, uint32_t* __restrict__ range, uint32_t stamp) {
  constexpr int kK = 2 * kSlice;
  constexpr int kPitch = kK / 2 + 4;  // words per n row; 16-byte aligned rows
  __shared__ __align__(16) uint32_t ph[kPanel * kPitch];
  __shared__ __align__(16) uint32_t pl[kPanel * kPitch];
  const int t = threadIdx.x;
  const int64_t kblock = blockIdx.x;
  const int64_t panel = blockIdx.y;
  const int nl = (t & 15) * 8;
  const int kp = t >> 4;  // k pair
  const int64_t k = kblock * kK + 2 * kp;
  const int64_t n = panel * kPanel + nl;
  float v0[8], v1[8];
  if (kVec && k + 1 < K && n + 7 < N) {
    const float4* r0 = reinterpret_cast<const float4*>(B + k * ldb + n);
    const float4* r1 = reinterpret_cast<const float4*>(B + (k + 1) * ldb + n);
    const float4 a0 = r0[0], a1 = r0[1], c0 = r1[0], c1 = r1[1];
    v0[0] = a0.x; v0[1] = a0.y; v0[2] = a0.z; v0[3] = a0.w;
    v0[4] = a1.x; v0[5] = a1.y; v0[6] = a1.z; v0[7] = a1.w;
    v1[0] = c0.x; v1[1] = c0.y; v1[2] = c0.z; v1[3] = c0.w;
    v1[4] = c1.x; v1[5] = c1.y; v1[6] = c1.z; v1[7] = c1.w;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      v0[e] = (k < K && n + e < N) ? B[k * ldb + n + e] : 0.0f;
      v1[e] = (k + 1 < K && n + e < N) ? B[(k + 1) * ldb + n + e] : 0.0f;
    }
  }
  if constexpr (kPre) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int shift = n + e < N ? prescale_shift(col_max[n + e], exp_b) : 0;
      v0[e] = __builtin_ldexpf(v0[e], shift);
      v1[e] = __builtin_ldexpf(v1[e], shift);
    }
  }
  bool big = false;
  uint32_t cls = 0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint16_t h0, l0, h1, l1;
    split_value(v0[e], s, h0, l0);
    split_value(v1[e], s, h1, l1);
    big |= __builtin_fabsf(static_cast<float>(__builtin_bit_cast(_Float16, h0))) * s > 65504.0f;
    big |= __builtin_fabsf(static_cast<float>(__builtin_bit_cast(_Float16, h1))) * s > 65504.0f;
    if constexpr (kReport) cls |= range_class(v0[e], h0, l0) | range_class(v1[e], h1, l1);
    ph[(nl + e) * kPitch + kp] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
    pl[(nl + e) * kPitch + kp] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
  }
  if (big) range[kWordBOverflow] = stamp;
  if (t == 0) range[kWordBStamp] = stamp;
  if constexpr (kReport) report_classes(cls, range, kWordBClass, stamp);
  __syncthreads();
  const int r = t >> 1;
  const int c = (t & 1) ^ tile_swizzle(r);  // logical chunk stored at position t & 1
#pragma unroll
  for (int sl = 0; sl < kK / kSlice; ++sl) {
    const u32x4 hv = *reinterpret_cast<const u32x4*>(ph + r * kPitch + sl * 8 + c * 4);
    const u32x4 lv = *reinterpret_cast<const u32x4*>(pl + r * kPitch + sl * 8 + c * 4);
    const int64_t base = (panel * (Kp / kSlice) + kblock * (kK / kSlice) + sl) * kTileHalves + t * 8;
    store_stream(hi + base, hv);
    store_stream(lo + base, lv);
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

namespace {

template <bool kPre, bool kReport>
void enqueue_split_a(const Planes& p, int64_t M, int64_t K, const float* A, int64_t lda,
                     float scale, const RangeOpts& opt, uint32_t stamp, hipStream_t stream) {
  // Mp is a multiple of 256 and Kp of 64 (plan_planes).
  const dim3 grid(static_cast<unsigned>((p.Kp + 127) / 128), grid_rows(p.Mp / 16));
  const bool vec = (reinterpret_cast<uintptr_t>(A) % 16 == 0) && (lda % 4 == 0);
  if (vec)
    hipLaunchKernelGGL((split_a_tiled_kernel<true, kPre, kReport>), grid, dim3(256), 0, stream,
                       M, K, A, lda, p.a_hi, p.a_lo, p.Mp, p.Kp, scale, p.row_max, opt.exp_a,
                       p.range, stamp);
  else
    hipLaunchKernelGGL((split_a_tiled_kernel<false, kPre, kReport>), grid, dim3(256), 0, stream,
                       M, K, A, lda, p.a_hi, p.a_lo, p.Mp, p.Kp, scale, p.row_max, opt.exp_a,
                       p.range, stamp);
}

template <bool kPre, bool kReport>
void enqueue_split_b(const Planes& p, int64_t K, int64_t N, const float* B, int64_t ldb,
                     float scale, const RangeOpts& opt, uint32_t stamp, hipStream_t stream) {
  // One workgroup per two tiles: Kp / 32 k blocks x Np / 128 panels (Np / 128
  // <= 65535 is checked by the C-ABI).
  const dim3 grid(static_cast<unsigned>(p.Kp / (2 * kSlice)), static_cast<unsigned>(p.Np / kPanel));
  const bool vec = (reinterpret_cast<uintptr_t>(B) % 16 == 0) && (ldb % 4 == 0);
  if (vec)
    hipLaunchKernelGGL((split_b_tiled_kernel<true, kPre, kReport>), grid, dim3(256), 0, stream,
                       K, N, B, ldb, p.b_hi, p.b_lo, p.Kp, scale, p.col_max, opt.exp_b, p.range,
                       stamp);
  else
    hipLaunchKernelGGL((split_b_tiled_kernel<false, kPre, kReport>), grid, dim3(256), 0, stream,
                       K, N, B, ldb, p.b_hi, p.b_lo, p.Kp, scale, p.col_max, opt.exp_b, p.range,
                       stamp);
}

}  // namespace

hipError_t launch_split_a(const Planes& p, int64_t M, int64_t K, const float* A, int64_t lda,
                          float scale, const RangeOpts& opt, uint32_t stamp, hipStream_t stream) {
  if (opt.prescale && opt.report) enqueue_split_a<true, true>(p, M, K, A, lda, scale, opt, stamp, stream);
  else if (opt.prescale) enqueue_split_a<true, false>(p, M, K, A, lda, scale, opt, stamp, stream);
  else if (opt.report) enqueue_split_a<false, true>(p, M, K, A, lda, scale, opt, stamp, stream);
  else enqueue_split_a<false, false>(p, M, K, A, lda, scale, opt, stamp, stream);
  return hipGetLastError();
}

hipError_t launch_split_b(const Planes& p, int64_t K, int64_t N, const float* B, int64_t ldb,
                          float scale, const RangeOpts& opt, uint32_t stamp,
                          hipStream_t stream) {
  // Every workgroup writes range[kWordBStamp] = stamp and the ones that see
  // an FP16 overflow of s B_hi write range[kWordBOverflow] = stamp, so the two
  // words are equal afterwards exactly when this split found one; a fresh
  // stamp per call makes a reset pass unnecessary.
  if (opt.prescale && opt.report) enqueue_split_b<true, true>(p, K, N, B, ldb, scale, opt, stamp, stream);
  else if (opt.prescale) enqueue_split_b<true, false>(p, K, N, B, ldb, scale, opt, stamp, stream);
  else if (opt.report) enqueue_split_b<false, true>(p, K, N, B, ldb, scale, opt, stamp, stream);
  else enqueue_split_b<false, false>(p, K, N, B, ldb, scale, opt, stamp, stream);
  return hipGetLastError();
}

hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream) {
  if (M <= 0 || N <= 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((N + 255) / 256), grid_rows(M));
  hipLaunchKernelGGL(zero_kernel, grid, dim3(256), 0, stream, M, N, C, ldc);
  return hipGetLastError();
}

}  // namespace sgc
