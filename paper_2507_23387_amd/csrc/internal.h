// Internal declarations shared by the split kernels, the GEMM kernels and the
// C-ABI layer of libsgemmcube.  Not installed; the public interface is
// include/sgemm_cube.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sgc {

// Internal accumulation variants: the two public orders plus the
// high-high-only baseline.
enum Variant : int { kElementwise = 0, kTermwise = 1, kHiOnly = 2 };

// GEMM tiling.  The split planes are padded to these multiples so the GEMM's
// main loop needs no bounds checks; only the C store is masked.
constexpr int kBM = 256;     // rows of C per workgroup
constexpr int kBN = 128;     // columns of C per workgroup
constexpr int kBK = 32;      // k per LDS stage; also the elementwise k-block
constexpr int kKPad = 64;    // K is padded to a multiple of this (an even number of stages)
constexpr int kThreads = 512;

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Layout of the split planes in the workspace.  A_hi/A_lo are Mp x Kp,
// k-contiguous (row-major).  B_hi/B_lo hold B transposed, Np x Kp,
// k-contiguous, so both MFMA operands read 8 consecutive k per lane.
struct Planes {
  int64_t Mp, Np, Kp;
  uint16_t* a_hi;
  uint16_t* a_lo;
  uint16_t* b_hi;
  uint16_t* b_lo;
  size_t bytes;  // total workspace bytes
};

Planes plan_planes(int64_t M, int64_t N, int64_t K, void* base);

// Enqueue the split of a rows x cols row-major FP32 matrix into row-major
// hi/lo planes with leading dimension ldh, writing zeros in the padding
// [rows, rows_pad) x [0, cols_pad) and [0, rows) x [cols, cols_pad).
hipError_t launch_split_rows(int64_t rows, int64_t cols, const float* X, int64_t ldx,
                             uint16_t* hi, uint16_t* lo, int64_t ldh, int64_t rows_pad,
                             int64_t cols_pad, float scale, hipStream_t stream);

// Enqueue the split of a K x N row-major FP32 matrix B into TRANSPOSED
// planes (Np x Kp, k-contiguous), zero-padded.
hipError_t launch_split_cols_transposed(int64_t K, int64_t N, const float* B, int64_t ldb,
                                        uint16_t* hi_t, uint16_t* lo_t, int64_t Np,
                                        int64_t Kp, float scale, hipStream_t stream);

// Enqueue the three-product MFMA GEMM on prepared planes.
hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float inv_scale, int variant, hipStream_t stream);

// Enqueue C := 0 for an M x N block with leading dimension ldc (a fill
// kernel, so the call stays safe under stream capture).
hipError_t launch_zero(int64_t M, int64_t N, float* C, int64_t ldc, hipStream_t stream);

}  // namespace sgc
