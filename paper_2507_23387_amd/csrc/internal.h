// Internal declarations shared by the split kernels, the GEMM kernels and the
// C-ABI layer of libsgemmcube.  Not installed; the public interface is
// include/sgemm_cube.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sgc {

// Internal accumulation variants: the public orders plus the high-high-only
// baseline.
enum Variant : int { kElementwise = 0, kTermwise = 1, kHiOnly = 2, kCrossFirst = 3 };

// Plane layout in the workspace ("panel tiles").  Every FP16 plane (A_hi,
// A_lo, and B_hi, B_lo of B transposed) is cut into panels of kPanel rows and
// slices of kSlice values of k; the kPanel x kSlice tile of (panel, slice) is
// stored contiguously (4 KiB) at tile index panel * (Kp / kSlice) + slice, so
// one k-step of a GEMM stage is a handful of contiguous 4 KiB blocks and the
// DMA into LDS reads whole cache lines.  Inside a tile, row r holds its 16
// values as two 16-byte chunks; chunk c is stored at position c ^ tile_swizzle(r)
// with tile_swizzle(r) = bit 4 of r.  With that swap the 16-byte fragment reads
// of the GEMM kernels from LDS (16 rows x 4 chunks of a 32-wide k-step for
// v_mfma_f32_16x16x32_f16) are free of bank conflicts on gfx950 (measured with
// the LDS bank-conflict counter).  The GEMM copies tiles into LDS verbatim.
constexpr int kPanel = 128;                     // rows per panel
constexpr int kSlice = 16;                      // k per tile
constexpr int kTileHalves = kPanel * kSlice;    // 2048 halves = 4 KiB
constexpr int kRowPad = 256;                    // M and N are padded to this
constexpr int kKPad = 64;                       // K is padded to this
constexpr int kFlagBytes = 256;                 // workspace header

__host__ __device__ inline int tile_swizzle(int row) { return (row >> 4) & 1; }

// Index (in halves) of element (row, k) of a tiled plane with Kp columns.
__host__ __device__ inline int64_t tiled_index(int64_t row, int64_t k, int64_t Kp) {
  const int64_t tile = (row / kPanel) * (Kp / kSlice) + k / kSlice;
  const int r = static_cast<int>(row % kPanel);
  const int kk = static_cast<int>(k % kSlice);
  return tile * kTileHalves + r * kSlice + (((kk >> 3) ^ tile_swizzle(r)) << 3) + (kk & 7);
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// The two-component split of one value (Sec. 3.3, Eq. recover_eqn):
// hi = fl16(a), r = a - hi (exact in FP32), lo = fl16(r * s), RN-even with
// gradual underflow.  Shared by the split kernels and the GEMM that splits A
// in registers, so both produce the same bits.
__device__ __forceinline__ void split_value(float a, float s, uint16_t& hi, uint16_t& lo) {
  const _Float16 h = static_cast<_Float16>(a);
  const float r = a - static_cast<float>(h);
  const _Float16 l = static_cast<_Float16>(r * s);
  hi = __builtin_bit_cast(uint16_t, h);
  lo = __builtin_bit_cast(uint16_t, l);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte store that bypasses the caches' retention (the planes are streamed
// out once and read back by the GEMM much later).
__device__ __forceinline__ void store_stream(uint16_t* p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}

// The split of eight consecutive values into packed hi and lo words.
__device__ __forceinline__ void split8(const float (&v)[8], float s, u32x4& hv, u32x4& lv) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint16_t h0, l0, h1, l1;
    split_value(v[2 * e], s, h0, l0);
    split_value(v[2 * e + 1], s, h1, l1);
    hv[e] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
    lv[e] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
  }
}

// Pre-scaling shift of a row (column) whose largest finite magnitude has the
// bits `max_bits`: the power of two that brings that magnitude into
// [2^target, 2^(target+1)); 0 for an all-zero (or all non-finite) line.
__device__ inline int prescale_shift(uint32_t max_bits, int target) {
  const float m = __builtin_bit_cast(float, max_bits);
  if (!(m > 0.0f) || !(m <= 3.4028235e38f)) return 0;
  int e = 0;
  (void)__builtin_frexpf(m, &e);
  return target - (e - 1);
}

// Workspace: a header holding the range flag, then the four planes.  A planes
// are Mp x Kp, B planes Np x Kp (B transposed), all tiled.  The range flag is
// two words: range[0] == range[1] after the split of B exactly when some
// |B_hi| * s exceeds the largest finite FP16 value, so that the scaled
// elementwise kernel cannot be used.
struct Planes {
  int64_t Mp, Np, Kp;
  uint32_t* range;
  uint32_t* row_max;  // pre-scaling only: bits of each row's largest |A| (else null)
  uint32_t* col_max;  // pre-scaling only: bits of each column's largest |B| (else null)
  uint16_t* a_hi;
  uint16_t* a_lo;
  uint16_t* b_hi;
  uint16_t* b_lo;
  size_t bytes;  // total workspace bytes
};

// Workspace header words (uint32).  Words 3..6 (A) and 7..10 (B) hold the
// stamp of the split that saw an entry of range class 1, 2, 4, 8 (see
// range_class in split.hip); compared with the split's own stamp word they
// give the range report of the last split of each operand.
constexpr int kWordBOverflow = 0;  // range flag: |B_hi| s > 65504 (stamped)
constexpr int kWordBStamp = 1;
constexpr int kWordAStamp = 2;
constexpr int kWordAClass = 3;
constexpr int kWordBClass = 7;
constexpr int kRangeClasses = 4;

// Options of one call: power-of-two pre-scaling of rows of A and columns of B
// (target exponents of their largest magnitudes), and the range report.
struct RangeOpts {
  bool prescale = false;
  bool report = false;
  int exp_a = 0;
  int exp_b = 0;
};

// Workspace layout for an M x N x K problem carved from `base`.  With base
// null only the sizes (Mp, Np, Kp, bytes) are filled and every pointer is null.
Planes plan_planes(int64_t M, int64_t N, int64_t K, void* base, bool prescale = false);

// Enqueue the split of a rows x cols row-major FP32 matrix into row-major
// hi/lo planes with leading dimension ldh (the public split entry point).
hipError_t launch_split_rows(int64_t rows, int64_t cols, const float* X, int64_t ldx,
                             uint16_t* hi, uint16_t* lo, int64_t ldh, float scale,
                             hipStream_t stream);

// Enqueue the split of A (M x K row-major) into the tiled A planes,
// zero-filling the padding up to Mp x Kp; with opt.prescale row i is first
// multiplied by its power of two (p.row_max), with opt.report the range
// classes are stamped (`stamp`) into the workspace header.
hipError_t launch_split_a(const Planes& p, int64_t M, int64_t K, const float* A, int64_t lda,
                          float scale, const RangeOpts& opt, uint32_t stamp, hipStream_t stream);

// Enqueue the split of B (K x N row-major) into the tiled, transposed B
// planes (Np x Kp), zero-filling the padding, and recompute the range flag.
// `stamp` must differ from the stamp of the previous split into the same
// workspace (the C-ABI draws a fresh one per call).
hipError_t launch_split_b(const Planes& p, int64_t K, int64_t N, const float* B, int64_t ldb,
                          float scale, const RangeOpts& opt, uint32_t stamp,
                          hipStream_t stream);

// Pre-scaling: enqueue the row maxima of |A| and column maxima of |B| (finite
// entries only) into p.row_max / p.col_max.
hipError_t launch_absmax(const Planes& p, int64_t M, int64_t N, int64_t K, const float* A,
                         int64_t lda, const float* B, int64_t ldb, hipStream_t stream);

// Pre-scaling: C_ij := 2^-(p_i + q_j) C_ij with the powers of two the splits
// applied.
hipError_t launch_unscale(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                          const RangeOpts& opt, hipStream_t stream);

// Range report: *out := OR of the classes the last splits of A and B saw
// (0 when `empty`, i.e. no split ran).
hipError_t launch_range_report(const Planes& p, bool empty, uint32_t* out, hipStream_t stream);

// Enqueue the MFMA GEMM on prepared planes.
hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float scale, int variant, hipStream_t stream);

// The elementwise GEMM with the copies of the 256 x 256 kernel overlapped
// with its MFMAs (stages = 2, the library's default) or issued and waited for
// at the end of each step (stages = 1), for the pipeline ablation.  The
// fallback kernel (range flag set) keeps its own pipeline.
hipError_t launch_gemm_stages(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                              float scale, int stages, hipStream_t stream);

// The unscaled elementwise kernel alone (only = true: it computes C whatever
// the range flag says) or after a scaled kernel (only = false: it computes C
// when the range flag is set and returns at once otherwise).
hipError_t launch_gemm_unscaled(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                                float scale, bool only, hipStream_t stream);

// The tile-shape and k-depth sweep of the scaled elementwise kernel
// (gemm_tile.hip): tile_m x tile_n tiles of C with block_k of k per pipeline
// stage, computed by workgroups of `waves` waves, one of the configurations
// tile_config_ok accepts; the same bits as launch_gemm's elementwise order.
// Scales above 2^15 and a set range flag take the unscaled kernel, as there.
bool tile_config_ok(int tile_m, int tile_n, int block_k, int waves);
hipError_t launch_gemm_tile(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                            float scale, int tile_m, int tile_n, int block_k, int waves,
                            hipStream_t stream);

// True when the order (kElementwise or kTermwise) can split A inside its GEMM
// kernel: A is 16-byte aligned, lda is a multiple of 4 (16-byte chunks), K a
// multiple of 64 (the copies never read past a row) and 256 rows of A span
// less than 4 GiB (per-lane 32-bit copy offsets); for the elementwise order
// also s <= 2^15 (its kernel keeps the s-scaled accumulator).
bool fused_split_ok(const float* A, int64_t lda, int64_t K, float scale, int variant);

// GEMM that reads A as FP32 and splits it in registers, on a workspace whose B
// planes (and range flag) were written by launch_split_b; requires
// fused_split_ok.  Elementwise: the 256 x 256 kernel; when the range flag is
// set (some |B_hi| s > 65504) it writes the A planes instead and the unscaled
// elementwise kernel, launched after it, computes C.  Termwise: the 256 x 128
// kernel.
hipError_t launch_gemm_fused_a(const Planes& p, int64_t M, int64_t N, int64_t K,
                               const float* A, int64_t lda, float* C, int64_t ldc, float scale,
                               int variant, hipStream_t stream);

// True when the termwise kernel can split B inside itself: B is 16-byte
// aligned, ldb and N are multiples of 4 (16-byte chunks of whole columns), K
// a multiple of 64 and 32 rows of B span less than 4 GiB.
bool fused_split_b_ok(const float* B, int64_t ldb, int64_t N, int64_t K);

// Termwise GEMM that reads B as FP32 and splits it in the kernel (requires
// fused_split_b_ok); A is split in the kernel too when split_a_in_gemm
// (requires fused_split_ok), else read from the A planes of the workspace.
// The result is that of launch_gemm's termwise order on planes, bit for bit.
hipError_t launch_gemm_fused_b(const Planes& p, int64_t M, int64_t N, int64_t K,
                               const float* A, int64_t lda, bool split_a_in_gemm,
                               const float* B, int64_t ldb, float* C, int64_t ldc, float scale,
                               hipStream_t stream);

// Enqueue C := 0 for an M x N block with leading dimension ldc (a fill
// kernel, so the call stays safe under stream capture).
hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream);

// The scaled elementwise kernels form s * B_hi in FP16, which needs s itself
// to be a finite FP16 value: s <= 2^15 (2^16 rounds to +inf).  Larger scales,
// which the C-ABI accepts up to 2^24, always take the unscaled elementwise
// kernel; the host decides this before any launch.
constexpr float kMaxScaledScale = 32768.0f;
inline bool scaled_kernel_ok(float scale) { return scale <= kMaxScaledScale; }

// The elementwise k-block of the scaled kernel, of the fallback kernel used
// when the range flag is set and of the cross-terms-first order: one
// 16 x 16 x 32 MFMA k-step.
constexpr int kBlockScaled = 2 * kSlice;
constexpr int kBlockFallback = 2 * kSlice;

}  // namespace sgc
