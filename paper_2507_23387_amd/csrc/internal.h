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
// so that the MFMA fragment reads from LDS (32 rows, one chunk each) spread
// over all banks.  The GEMM copies tiles into LDS verbatim.
constexpr int kPanel = 128;                     // rows per panel
constexpr int kSlice = 16;                      // k per tile = one MFMA k-step
constexpr int kTileHalves = kPanel * kSlice;    // 2048 halves = 4 KiB
constexpr int kRowPad = 256;                    // M and N are padded to this
constexpr int kKPad = 64;                       // K is padded to this
constexpr int kFlagBytes = 256;                 // workspace header

__host__ __device__ inline int tile_swizzle(int row) { return (row >> 3) & 1; }

// Index (in halves) of element (row, k) of a tiled plane with Kp columns.
__host__ __device__ inline int64_t tiled_index(int64_t row, int64_t k, int64_t Kp) {
  const int64_t tile = (row / kPanel) * (Kp / kSlice) + k / kSlice;
  const int r = static_cast<int>(row % kPanel);
  const int kk = static_cast<int>(k % kSlice);
  return tile * kTileHalves + r * kSlice + (((kk >> 3) ^ tile_swizzle(r)) << 3) + (kk & 7);
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Workspace: a header holding the range flag, then the four planes.  A planes
// are Mp x Kp, B planes Np x Kp (B transposed), all tiled.  The range flag is
// two words: range[0] == range[1] after the split of B exactly when some
// |B_hi| * s exceeds the largest finite FP16 value, so that the scaled
// elementwise kernel cannot be used.
struct Planes {
  int64_t Mp, Np, Kp;
  uint32_t* range;
  uint16_t* a_hi;
  uint16_t* a_lo;
  uint16_t* b_hi;
  uint16_t* b_lo;
  size_t bytes;  // total workspace bytes
};

Planes plan_planes(int64_t M, int64_t N, int64_t K, void* base);

// Enqueue the split of a rows x cols row-major FP32 matrix into row-major
// hi/lo planes with leading dimension ldh (the public split entry point).
hipError_t launch_split_rows(int64_t rows, int64_t cols, const float* X, int64_t ldx,
                             uint16_t* hi, uint16_t* lo, int64_t ldh, float scale,
                             hipStream_t stream);

// Enqueue the split of A (M x K row-major) into the tiled A planes,
// zero-filling the padding up to Mp x Kp.
hipError_t launch_split_a(const Planes& p, int64_t M, int64_t K, const float* A, int64_t lda,
                          float scale, hipStream_t stream);

// Enqueue the split of B (K x N row-major) into the tiled, transposed B
// planes (Np x Kp), zero-filling the padding, and recompute the range flag.
// `stamp` must differ from the stamp of the previous split into the same
// workspace (the C-ABI draws a fresh one per call).
hipError_t launch_split_b(const Planes& p, int64_t K, int64_t N, const float* B, int64_t ldb,
                          float scale, uint32_t stamp, hipStream_t stream);

// Enqueue the MFMA GEMM on prepared planes.  `cus` is the device's compute
// unit count (sizes the persistent grid of the 256 x 128 kernel).
hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float scale, int variant, int cus, hipStream_t stream);

// Enqueue C := 0 for an M x N block with leading dimension ldc (a fill
// kernel, so the call stays safe under stream capture).
hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream);

// The elementwise k-block of the scaled kernel (one MFMA k-step), and of the
// fallback kernel used when the range flag is set and of the cross-terms-first
// order (two k-steps).
constexpr int kBlockScaled = kSlice;
constexpr int kBlockFallback = 2 * kSlice;

}  // namespace sgc
