// Elementwise GEMM that splits A in registers (gfx950).
//
// Same computation as the 256 x 256 elementwise kernel of gemm.hip (three
// v_mfma_f32_16x16x32_f16 products per block into one accumulator that holds
// s * acc, Eq. elementwise of arXiv 2507.23387), but A is read as FP32 from
// its row-major storage and split (Sec. 3.3, Eq. recover_eqn) by the
// workgroup that uses it, with the same arithmetic as the split kernels
// (split_value), so the A planes never go through HBM.  B still comes from
// the tiled planes of the split of B.
//
// Data path per 32-wide k-step (stage), 256 threads:
//   A: eight 16-byte global loads per lane (8 lanes cover the 128 bytes of
//      one row's 32 values, 8 rows per instruction), issued two steps ahead
//      into one of two register sets; split in registers and written to the
//      LDS stage with 8-byte stores (hi and lo planes, same tile layout and
//      swizzle as the planes the split kernels write).
//   B: LDS DMA of the two B planes, as in gemm.hip.
// Schedule ("row-fused"): for each row i of 16 x 16 blocks the wave issues
// HH(i, .), XA(i, .), XB(i, .), so every accumulator sees the block terms in
// the order HH, XA, XB.  The B fragments of a step stay in registers; A
// fragments are read one row ahead.  In step kt: rows 0-1 issue the B DMAs of
// stage kt+1 into LDS slot (kt+1) % 2, rows 2-5 issue the A loads of stage
// kt+3, one barrier before row 7 publishes stage kt+1 (whose A was split into
// the slot at the end of step kt-1) and retires slot kt % 2, and row 7 then
// splits stage kt+2's A (loaded during step kt-1) into that slot.  The A loads
// are ordinary loads, so the compiler's own waits cover them (conservatively:
// the DMAs are invisible to it, and a wait counted without them only waits
// longer; it never waits on a DMA that the barrier did not already retire,
// because the split happens right after the barrier).
//
// When some |B_hi| s exceeds 65504 (the range flag set by the split of B) the
// scaled accumulator cannot be used: the kernel then splits A into the tiled
// A planes instead (each workgroup a share of the slices of its row panel),
// and the 256 x 128 kernel that runs next computes the unscaled elementwise
// order from the planes.
#include "gemm_common.h"

namespace sgc {
namespace {

constexpr int kFTile = 256;
constexpr int kFThreads = 256;
constexpr int kFStages = 2;
constexpr int kFStep = 2 * kSlice;                        // 32
constexpr int kFPlaneHalves = kFTile * kFStep;            // 8192 halves per plane per stage
constexpr int kFStageHalves = 4 * kFPlaneHalves;          // A_hi, B_hi, A_lo, B_lo
constexpr size_t kFLdsBytes = static_cast<size_t>(kFStages) * kFStageHalves * 2;  // 128 KiB
constexpr int kFBDma = 8;                                 // B DMAs per wave per stage
constexpr int kFALoads = 8;                               // A loads per lane per stage

typedef float floatv4 __attribute__((ext_vector_type(4)));

// Split of A into the tiled planes, used when the scaled kernel cannot run:
// workgroup (tm, tn) takes slices tn, tn + tiles_n, ... of row panel pair tm;
// thread t splits row t's 16 values of a slice.
__device__ void split_a_share(const float* __restrict__ A, int64_t lda, int M, int K, int Kp,
                              int tm, int tn, int tiles_n, uint16_t* __restrict__ a_hi,
                              uint16_t* __restrict__ a_lo, float s) {
  const int t = threadIdx.x;
  const int64_t row = static_cast<int64_t>(tm) * kFTile + t;
  for (int sl = tn; sl < Kp / kSlice; sl += tiles_n) {
    uint32_t hw[8], lw[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int k0 = sl * kSlice + 2 * e;
      const float v0 = (row < M && k0 < K) ? A[row * lda + k0] : 0.0f;
      const float v1 = (row < M && k0 + 1 < K) ? A[row * lda + k0 + 1] : 0.0f;
      uint16_t h0, l0, h1, l1;
      split_value(v0, s, h0, l0);
      split_value(v1, s, h1, l1);
      hw[e] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
      lw[e] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
    }
    // Chunk c (k 8c .. 8c+7) of the row goes to position c ^ tile_swizzle(r).
    const int64_t base = tiled_index(row, static_cast<int64_t>(sl) * kSlice, Kp) -
                         (tile_swizzle(static_cast<int>(row % kPanel)) << 3);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const int64_t at = base + ((c ^ tile_swizzle(static_cast<int>(row % kPanel))) << 3);
      const uint4 hv = {hw[4 * c], hw[4 * c + 1], hw[4 * c + 2], hw[4 * c + 3]};
      const uint4 lv = {lw[4 * c], lw[4 * c + 1], lw[4 * c + 2], lw[4 * c + 3]};
      *reinterpret_cast<uint4*>(a_hi + at) = hv;
      *reinterpret_cast<uint4*>(a_lo + at) = lv;
    }
  }
}

__global__ __launch_bounds__(kFThreads, 1) void gemm_fused_a_kernel(
    const float* __restrict__ A, int64_t lda, int M, int K,
    uint16_t* __restrict__ a_hi, uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int N, float s, float inv_s) {
  constexpr int S = kFStages;
  constexpr int kSub = 8;  // 16 x 16 MFMA tiles per wave side
  int tm, tn;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn))
    tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  if (range[0] == range[1]) {
    // s B_hi overflows FP16: provide the A planes for the unscaled kernel.
    split_a_share(A, lda, M, K, Kp, tm, tn, tiles_n, a_hi, a_lo, s);
    return;
  }
  extern __shared__ __align__(16) uint16_t lds[];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int64_t slices = Kp / kSlice;
  const int ksteps = static_cast<int>(slices / 2);
  constexpr int kAH = 0, kBH = 1, kAL = 2, kBL = 3;

  // --- B: LDS DMA of the tiled planes (as in gemm.hip) ----------------------
  const int64_t panel_stride = slices * kTileHalves;
  const uint16_t* bsrc[2] = {b_hi + 2 * tn * panel_stride, b_lo + 2 * tn * panel_stride};
  const int64_t lane_off = w * 512 + lane * 8;
  const unsigned lds_base = lds_address(lds);
  auto dma_b = [&](int kt, int n) {  // n-th B DMA of stage kt, n < kFBDma
    const int ktc = min(kt, ksteps - 1);
    const int q = n >> 2, ph = (n >> 1) & 1, sl = n & 1;
    const int plane = q ? kBL : kBH;
    const unsigned dst = lds_base + ((kt % S) * kFStageHalves + plane * kFPlaneHalves +
                                     (2 * ph + sl) * kTileHalves + w * 512) * 2;
    dma16(bsrc[q] + ph * panel_stride + static_cast<int64_t>(2 * ktc + sl) * kTileHalves +
              lane_off, dst);
  };

  // --- A: FP32 loads, split in registers, 8-byte LDS stores -----------------
  // Lane l of wave w handles rows R = 64 w + 8 q + l/8 (q = 0..7) of the tile
  // and the 4 values k = 4 (l % 8) .. +3 of the step.  In the LDS tile layout
  // row R is row r = R % 128 of panel R / 128 = w / 2; its k values sit in
  // slice (l % 8) / 4, chunk ((l % 8) / 2) % 2, at offset 4 (l % 2) in the
  // chunk; bit 4 of r (the chunk swap) is bit 1 of q.
  const int arow0 = tm * kFTile + 64 * w + (lane >> 3);
  const int ak = 4 * (lane & 7);
  const float* const abase = A + static_cast<int64_t>(arow0) * lda + ak;
  const int a_lds0 = (2 * (w >> 1) + ((lane & 7) >> 2)) * kTileHalves +
                     (64 * (w & 1) + (lane >> 3)) * kSlice + 4 * (lane & 1);
  const int a_chunk = ((lane & 7) >> 1) & 1;
  floatv4 st0[kFALoads], st1[kFALoads];
  // K is a multiple of 4 (checked by the caller), so each 16-byte load is
  // wholly inside or wholly outside the row's K values.  Out-of-range loads
  // read A's first 16 bytes instead (always valid) and are replaced by zeros
  // when the registers are split (not here, which would make the wave wait for
  // the load at once), so the loop has no branches.
  auto a_ok = [&](int kt, int q) { return arow0 + 8 * q < M && kt * kFStep + ak < K; };
  auto load_a = [&](int kt, floatv4 (&st)[kFALoads], int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      const float* p =
          a_ok(kt, q) ? abase + static_cast<int64_t>(8 * q) * lda + kt * kFStep : A;
      st[q] = *reinterpret_cast<const floatv4*>(p);
    }
  };
  auto store_a = [&](int kt, const floatv4 (&st)[kFALoads], int q0, int q1) {
    uint16_t* const slot = lds + (kt % S) * kFStageHalves;
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      const floatv4 v = a_ok(kt, q) ? st[q] : floatv4{0.0f, 0.0f, 0.0f, 0.0f};
      uint16_t h[4], l[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) split_value(v[e], s, h[e], l[e]);
      const uint2 hv = {static_cast<uint32_t>(h[0]) | (static_cast<uint32_t>(h[1]) << 16),
                        static_cast<uint32_t>(h[2]) | (static_cast<uint32_t>(h[3]) << 16)};
      const uint2 lv = {static_cast<uint32_t>(l[0]) | (static_cast<uint32_t>(l[1]) << 16),
                        static_cast<uint32_t>(l[2]) | (static_cast<uint32_t>(l[3]) << 16)};
      const int off = a_lds0 + 8 * q * kSlice + ((a_chunk ^ ((q >> 1) & 1)) << 3);
      *reinterpret_cast<uint2*>(slot + kAH * kFPlaneHalves + off) = hv;
      *reinterpret_cast<uint2*>(slot + kAL * kFPlaneHalves + off) = lv;
    }
  };

  // --- fragments -------------------------------------------------------------
  const int fr = lane & 15, fc = lane >> 4;
  int a_off[2], b_off[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int row_off = fr * kSlice + (((fc & 1) ^ tile_swizzle(16 * par + fr)) << 3);
    a_off[par] = (2 * wm + (fc >> 1)) * kTileHalves + row_off;
    b_off[par] = (2 * wn + (fc >> 1)) * kTileHalves + row_off;
  }
  auto rd = [&](int kt, int plane, int i) -> half8 {
    const int off = (plane == kAH || plane == kAL) ? a_off[i & 1] : b_off[i & 1];
    return *reinterpret_cast<const half8*>(lds + (kt % S) * kFStageHalves +
                                           plane * kFPlaneHalves + off + i * 16 * kSlice);
  };
  const _Float16 s16 = static_cast<_Float16>(s);

  floatx4 acc[kSub][kSub];
#pragma unroll
  for (int i = 0; i < kSub; ++i)
#pragma unroll
    for (int j = 0; j < kSub; ++j) acc[i][j] = floatx4{};

  // --- prologue: stages 0 and 1 of A split into LDS, stage 2 in registers ----
  load_a(0, st0, 0, kFALoads);
#pragma unroll
  for (int n = 0; n < kFBDma; ++n) dma_b(0, n);
  store_a(0, st0, 0, kFALoads);
  load_a(1, st1, 0, kFALoads);
  load_a(2, st0, 0, kFALoads);  // split at the end of step 0
  store_a(1, st1, 0, kFALoads);
  wait_vmcnt<kFALoads>();       // all but the stage-2 loads: the B DMAs of stage 0
  lds_barrier();

  half8 bx[kSub], by[kSub], bl[kSub], a_h[2], a_l[2];
#pragma unroll
  for (int j = 0; j < kSub; ++j) {
    by[j] = rd(0, kBH, j);
    bl[j] = rd(0, kBL, j);
  }
#pragma unroll
  for (int j = 0; j < kSub; ++j) bx[j] = by[j] * s16;
  a_h[0] = rd(0, kAH, 0);
  a_l[0] = rd(0, kAL, 0);

  // One step.  bs: s B_hi of this step, bh: B_hi of this step (the two sets
  // swap roles every step).  ld: the A register set that receives stage kt+3
  // (its stage kt+1 was split at the end of step kt-1); sp: the set holding
  // stage kt+2, split into LDS slot kt % 2 right after the barrier.  Splitting
  // only right after a barrier that waited for every older DMA keeps the
  // compiler's own waits for these loads from stalling on a DMA.
  auto step = [&](int kt, half8 (&bs)[kSub], half8 (&bh)[kSub], floatv4 (&ld)[kFALoads],
                  floatv4 (&sp)[kFALoads]) {
    const int nk = kt + 1;
#pragma unroll
    for (int i = 0; i < kSub; ++i) {
      const int c = i & 1;
      if (i == kSub - 1) {
        // The B DMAs of stage kt+1 are done (only the A loads of this step,
        // the youngest kFALoads memory operations, may still be in flight),
        // then all waves meet: stage kt+1 is published, slot kt % 2 retired.
        wait_vmcnt<kFALoads>();
        lds_barrier();
        a_h[c ^ 1] = rd(nk, kAH, 0);
        a_l[c ^ 1] = rd(nk, kAL, 0);
      } else {
        a_h[c ^ 1] = rd(kt, kAH, i + 1);
        a_l[c ^ 1] = rd(kt, kAL, i + 1);
      }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_h[c], bs[j], acc[i][j]);
      SCHED_FENCE();
      if (i < 2) {
        dma_b(nk, 4 * i);
        dma_b(nk, 4 * i + 1);
      } else if (i < 6) {
        load_a(kt + 3, ld, 2 * (i - 2), 2 * (i - 2) + 1);
      } else if (i == kSub - 1) {
        store_a(kt + 2, sp, 0, 3);
#pragma unroll
        for (int j = 0; j < kSub; ++j) bs[j] = rd(nk, kBH, j);
      }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_l[c], bh[j], acc[i][j]);
      SCHED_FENCE();
      if (i < 2) {
        dma_b(nk, 4 * i + 2);
        dma_b(nk, 4 * i + 3);
      } else if (i < 6) {
        load_a(kt + 3, ld, 2 * (i - 2) + 1, 2 * (i - 2) + 2);
      } else if (i == kSub - 1) {
        store_a(kt + 2, sp, 3, 6);
#pragma unroll
        for (int j = 0; j < kSub; ++j) bh[j] = bs[j] * s16;
      }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_h[c], bl[j], acc[i][j]);
      SCHED_FENCE();
      if (i == kSub - 1) {
        store_a(kt + 2, sp, 6, kFALoads);
#pragma unroll
        for (int j = 0; j < kSub; ++j) bl[j] = rd(nk, kBL, j);
      }
      SCHED_FENCE();
    }
  };
  for (int kt = 0; kt < ksteps; kt += 2) {
    step(kt, bx, by, st1, st0);
    step(kt + 1, by, bx, st0, st1);
  }
  // No DMA or load may still be in flight when the workgroup retires.
  wait_vmcnt<0>();

  const int col0 = tn * kFTile + wn * 128 + (lane & 15);
  const int row0 = tm * kFTile + wm * 128 + (lane >> 4) * 4;
  const bool full = (tm + 1) * kFTile <= M && (tn + 1) * kFTile <= N;
  store_tile16<kSub, kSub>(C, ldc, M, N, row0, col0, full,
                           [&](int i, int j, int r) { return acc[i][j][r] * inv_s; });
}

}  // namespace

hipError_t launch_gemm_fused_a(const Planes& p, int64_t M, int64_t N, int64_t K,
                               const float* A, int64_t lda, float* C, int64_t ldc, float scale,
                               hipStream_t stream) {
  if (!scaled_kernel_ok(scale)) return hipErrorInvalidValue;  // s must be a finite FP16 value
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_fused_a_kernel, kFLdsBytes, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kFTile);
  const int tiles_n = static_cast<int>(p.Np / kFTile);
  hipLaunchKernelGGL(gemm_fused_a_kernel, dim3(tiles_m * tiles_n), dim3(kFThreads), kFLdsBytes,
                     stream, A, lda, static_cast<int>(M), static_cast<int>(K), p.a_hi, p.a_lo,
                     p.b_hi, p.b_lo, p.range, static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc,
                     static_cast<int>(N), scale, 1.0f / scale);
  return hipGetLastError();
}

}  // namespace sgc
