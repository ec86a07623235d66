// Three-product MFMA GEMM on prepared FP16 planes (gfx950).
//
// For each tile of C it forms (Eq. recover_eqn of arXiv 2507.23387)
//   HH = A_hi B_hi,  XA = A_lo B_hi,  XB = A_hi B_lo
// with v_mfma_f32_32x32x16_f16 (FP16 x FP16 products are exact; the MFMA adds
// the 16 products of a k-step to its C operand in one fused, once-rounded FP32
// operation) and reconstructs C in the accumulation order asked for.
//
// Two kernels share one data path:
//
// gemm_wide_kernel, 256 x 256 tiles, 4 waves of 128 x 128 (one per SIMD, the
// 256-register accumulator in AGPRs):
//   kElementwise (Eq. elementwise, Sec. 4.5) with the contraction cut into
//     blocks g of one k-step (16).  The accumulator holds s * acc, so that the
//     three per-block additions of the equation become three chained MFMAs:
//       s*acc <- fl(s*acc + A_hi (s B_hi))   = s * fl(acc + HH_g)
//       s*acc <- fl(s*acc + A_lo B_hi)       = s * fl(acc + XA_g / s)
//       s*acc <- fl(s*acc + A_hi B_lo)       = s * fl(acc + XB_g / s)
//     and C = (s*acc) / s at the end.  s B_hi is formed in registers with
//     v_pk_mul_f16; it is exact because s is a power of two, provided
//     |B_hi| s <= 65504, which the split of B checks (the range flag).  Each
//     block term is summed by the MFMA together with the accumulator, with
//     one rounding, instead of being rounded to FP32 on its own first.
//   kHiOnly: C = HH, the native-FP16 GEMM baseline.
//
// gemm_narrow_kernel, 256 x 128 tiles, 8 waves of 64 x 64 (two per SIMD):
//   kTermwise (Eq. termwise): three FP32 accumulators over all of K,
//     C = (HH + XA / s) + XB / s in the epilogue.
//   kCrossFirst (the reordered elementwise accumulation proposed at the end
//     of Sec. 4.5): per block g of two k-steps the cross products are summed
//     first, X_g = XA_g + XB_g (one MFMA chain), HH_g separately, and
//     acc = acc + (X_g / s + HH_g) with one v_fma_f32 and one add.
//   kElementwise when the range flag is set: unscaled, blocks of two k-steps
//     (32): HH goes straight into the accumulator, XA_g and XB_g into block
//     sums started from zero, and acc = (acc + XA_g / s) + XB_g / s with two
//     v_fma_f32 at the end of each block (1/s is exact).
// Both elementwise kernels are launched; each reads the range flag first and
// the one that does not apply returns at once.
//
// Data path.  The planes are stored as 4 KiB tiles of 128 rows x 16 k in the
// order and swizzle the LDS wants (internal.h), so one pipeline stage (one
// k-step of every plane the kernel needs) is a few contiguous 4 KiB blocks,
// copied from global memory straight into LDS with global_load_lds_dwordx4 (no
// VGPR staging).  Stages go into a ring of kStages slots.  In k-step kt the
// fragments of step kt+1 are read while the MFMAs of step kt run: each
// fragment register is reloaded as soon as its last MFMA of the step has been
// issued (a rolling schedule; it fits the register file where double
// buffering does not), and the DMAs for stage kt+kStages are spread between
// the MFMA groups so the in-order wave never stalls on a burst of memory
// instructions.  One s_barrier per step both publishes stage kt+1 and retires
// the slot of stage kt before it is refilled.  Past the last stage the loads
// repeat the last stage, so every wait count is a compile-time constant.
#include <algorithm>
#include <atomic>

#include "gemm_common.h"

namespace sgc {
namespace {

constexpr int kKSteps = kSlice / 16;  // MFMA k-steps per tile slice (1)
static_assert(kKSteps == 1, "one MFMA k-step per slice");
static_assert(kKPad % (2 * kSlice) == 0, "the main loops take two slices per iteration");

// ---------------------------------------------------------------------------
// 256 x 256 tiles: scaled elementwise and hi-only, on v_mfma_f32_16x16x32_f16.
//
// The 16 x 16 x 32 form is used here because under the board's power limit it
// sustains a higher FP16 rate on random operands than the 32 x 32 x 16 form
// (less energy per product, so a higher shader clock at the same power).
constexpr int kWide = 256;
constexpr int kWideThreads = 256;
constexpr int kWideStages = 2;
constexpr int kStep = 2 * kSlice;  // k per MFMA step of the wide kernel (32): two slices


template <int V>
constexpr int wide_planes() { return V == kElementwise ? 4 : 2; }

template <int V, int S>
constexpr size_t wide_lds_bytes() {
  return static_cast<size_t>(S) * wide_planes<V>() * kWide * kStep * 2;
}


// S = number of LDS stage slots, one 32-k step each (64 KiB with four planes).
// S = 2: the DMAs of stage kt+2 are in flight while step kt+1 computes.
// S = 1 (no prefetch, for the pipeline ablation): the next stage is copied and
// waited for inside each step.
template <int V, int S>
__global__ __launch_bounds__(kWideThreads, 1) void gemm_wide_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int M, int N, float s, float inv_s) {
  static_assert(V == kElementwise || V == kHiOnly, "wide kernel variants");
  static_assert((S == 1 && V == kElementwise) || S == 2, "stage count");
  constexpr bool kEl = V == kElementwise;
  constexpr int kPlanes = wide_planes<V>();       // LDS slots: A_hi, B_hi, A_lo, B_lo
  constexpr int kPlaneHalves = kWide * kStep;     // two panels x two slices: four tiles
  constexpr int kStageHalves = kPlanes * kPlaneHalves;
  constexpr int kDma = kPlanes * 4;               // 1 KiB DMAs per wave per stage
  constexpr int kSub = 8;                         // 16 x 16 MFMA tiles per wave side
  if constexpr (kEl) {
    if (range[0] == range[1]) return;  // s B_hi overflows FP16: the narrow kernel runs instead
  }
  extern __shared__ __align__(16) uint16_t lds[];

  int tm, tn;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn))
    tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int64_t slices = Kp / kSlice;
  const int ksteps = static_cast<int>(slices / 2);

  // A stage holds, per plane, the tiles (panel ph, slice sl) of the tile's two
  // panels and the step's two slices at tile position 2*ph + sl.  Wave w copies
  // 1 KiB block w of each of those four tiles.
  const int64_t panel_stride = slices * kTileHalves;
  const uint16_t* src[4] = {a_hi + 2 * tm * panel_stride, b_hi + 2 * tn * panel_stride,
                            kEl ? a_lo + 2 * tm * panel_stride : nullptr,
                            kEl ? b_lo + 2 * tn * panel_stride : nullptr};
  const int64_t lane_off = w * 512 + lane * 8;
  const unsigned lds_base = lds_address(lds);
  auto dma_one = [&](int kt, int n) {  // n-th DMA of stage kt, n < kDma
    const int ktc = min(kt, ksteps - 1);
    const int p = n >> 2, ph = (n >> 1) & 1, sl = n & 1;
    const unsigned dst = lds_base + ((kt % S) * kStageHalves + p * kPlaneHalves +
                                     (2 * ph + sl) * kTileHalves + w * 512) * 2;
    dma16(src[p] + ph * panel_stride + static_cast<int64_t>(2 * ktc + sl) * kTileHalves +
              lane_off, dst);
  };

  // Fragment of block i (rows 16 i .. 16 i + 15 of this wave's 128 rows, which
  // are panel wm of A / panel wn of B): lane l reads row 16 i + l%16, k chunk
  // c = l/16 of the step, i.e. chunk c%2 of slice c/2.  The chunk swap of the
  // tile layout depends on bit 4 of the row, i.e. on the parity of i.
  const int fr = lane & 15, fc = lane >> 4;
  int a_off[2], b_off[2];
#pragma unroll
  for (int par = 0; par < 2; ++par) {
    const int row_off = fr * kSlice + (((fc & 1) ^ tile_swizzle(16 * par + fr)) << 3);
    a_off[par] = (2 * wm + (fc >> 1)) * kTileHalves + row_off;
    b_off[par] = (2 * wn + (fc >> 1)) * kTileHalves + row_off;
  }
  constexpr int kAH = 0, kBH = 1, kAL = 2, kBL = 3;
  auto rd = [&](int kt, int plane, int i) -> half8 {
    const int off = (plane == kAH || plane == kAL) ? a_off[i & 1] : b_off[i & 1];
    return *reinterpret_cast<const half8*>(lds + (kt % S) * kStageHalves + plane * kPlaneHalves +
                                           off + i * 16 * kSlice);
  };
  const _Float16 s16 = static_cast<_Float16>(s);

  floatx4 acc[kSub][kSub];
#pragma unroll
  for (int i = 0; i < kSub; ++i)
#pragma unroll
    for (int j = 0; j < kSub; ++j) acc[i][j] = floatx4{};

  // Prologue: stage 0 (each step copies the next stage).
#pragma unroll
  for (int n = 0; n < kDma; ++n) dma_one(0, n);
  wait_vmcnt<0>();
  lds_barrier();

  if constexpr (kEl) {
    // Row-fused schedule: for each row i of 16 x 16 blocks the wave issues
    // HH(i, .), then XA(i, .), then XB(i, .), so every accumulator still sees
    // the block terms in the order HH, XA, XB.  The B fragments of the whole
    // step stay in registers (s B_hi, B_hi, B_lo); A fragments are needed one
    // row at a time and are read one row ahead.  The two B_hi register sets
    // swap roles every step: after HH of row 7 the set that held s B_hi
    // receives the next step's B_hi, and after XA of row 7 the other set
    // receives s times it.  One barrier per step, before row 7, publishes
    // stage kt+1 (row 7 reads the next step's fragments from it) and retires
    // the slot of stage kt; the DMAs of stage kt+1 are issued in rows 0-5 of
    // step kt.
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

    // bs: s B_hi of this step, bh: B_hi of this step.
    auto step = [&](int kt, half8 (&bs)[kSub], half8 (&bh)[kSub]) {
      const int nk = kt + 1;
      int dn = 0;
      auto dma_some = [&](int n) {
        if constexpr (S > 1) {
#pragma unroll
          for (int q = 0; q < n; ++q)
            if (dn < kDma) dma_one(nk, dn++);
        }
      };
#pragma unroll
      for (int i = 0; i < kSub; ++i) {
        const int c = i & 1;
        if (i == kSub - 1) {
          if constexpr (S == 1) {
            // Retire the single slot, copy stage kt+1 into it and wait.
            lds_barrier();
#pragma unroll
            for (int n = 0; n < kDma; ++n) dma_one(nk, n);
            wait_vmcnt<0>();
            lds_barrier();
          } else {
            wait_vmcnt<0>();
            lds_barrier();
          }
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
        if (i == kSub - 1) {
#pragma unroll
          for (int j = 0; j < kSub; ++j) bs[j] = rd(nk, kBH, j);
        } else if (i < 6) {
          dma_some((kDma + 5) / 6 - (kDma + 5) / 12);
        }
        SCHED_FENCE();
#pragma unroll
        for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_l[c], bh[j], acc[i][j]);
        SCHED_FENCE();
        if (i == kSub - 1) {
#pragma unroll
          for (int j = 0; j < kSub; ++j) bh[j] = bs[j] * s16;
        } else if (i < 6) {
          dma_some((kDma + 5) / 12);
        }
        SCHED_FENCE();
#pragma unroll
        for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_h[c], bl[j], acc[i][j]);
        SCHED_FENCE();
        if (i == kSub - 1) {
#pragma unroll
          for (int j = 0; j < kSub; ++j) bl[j] = rd(nk, kBL, j);
        }
        SCHED_FENCE();
      }
      if constexpr (S > 1) dma_some(kDma);  // any DMA of stage kt+1 not issued yet
    };
    for (int kt = 0; kt < ksteps; kt += 2) {
      step(kt, bx, by);
      step(kt + 1, by, bx);
    }
  } else {
    // Hi-only, the same row schedule with one product: the B_hi fragments of
    // the next step go to the other register set right after the barrier.
    half8 b0[kSub], b1[kSub], a_h[2];
#pragma unroll
    for (int j = 0; j < kSub; ++j) b0[j] = rd(0, kBH, j);
    a_h[0] = rd(0, kAH, 0);
    auto step = [&](int kt, half8 (&bc)[kSub], half8 (&bn)[kSub]) {
      const int nk = kt + 1;
      int dn = 0;
#pragma unroll
      for (int i = 0; i < kSub; ++i) {
        const int c = i & 1;
        if (i == kSub - 1) {
          wait_vmcnt<0>();
          lds_barrier();
          a_h[c ^ 1] = rd(nk, kAH, 0);
#pragma unroll
          for (int j = 0; j < kSub; ++j) bn[j] = rd(nk, kBH, j);
        } else {
          a_h[c ^ 1] = rd(kt, kAH, i + 1);
          if (i < 6) {
#pragma unroll
            for (int q = 0; q < 2; ++q)
              if (dn < kDma) dma_one(nk, dn++);
          }
        }
        SCHED_FENCE();
#pragma unroll
        for (int j = 0; j < kSub; ++j) acc[i][j] = mfma16(a_h[c], bc[j], acc[i][j]);
        SCHED_FENCE();
      }
    };
    for (int kt = 0; kt < ksteps; kt += 2) {
      step(kt, b0, b1);
      step(kt + 1, b1, b0);
    }
  }
  // No LDS DMA may still be writing when the workgroup retires.
  wait_vmcnt<0>();

  const float out_scale = kEl ? inv_s : 1.0f;
  const int col0 = tn * kWide + wn * 128 + (lane & 15);
  const int row0 = tm * kWide + wm * 128 + (lane >> 4) * 4;
  const bool full = (tm + 1) * kWide <= M && (tn + 1) * kWide <= N;
  store_tile16<kSub, kSub>(C, ldc, M, N, row0, col0, full,
                           [&](int i, int j, int r) { return acc[i][j][r] * out_scale; });
}
// ---------------------------------------------------------------------------
// 256 x 128 tiles: termwise and the unscaled elementwise fallback.
constexpr int kNarrowM = 256;
constexpr int kNarrowN = 128;
constexpr int kNarrowThreads = 512;
constexpr int kNarrowStages = 4;
constexpr size_t kNarrowLdsBytes =
    static_cast<size_t>(kNarrowStages) * 2 * (kNarrowM + kNarrowN) * kSlice * 2;

template <int V>
__global__ __launch_bounds__(kNarrowThreads, 1) void gemm_narrow_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int M, int N, float s, float inv_s) {
  static_assert(V == kElementwise || V == kTermwise || V == kCrossFirst, "narrow kernel variants");
  constexpr int S = kNarrowStages;
  constexpr int kAHalves = kNarrowM * kSlice;  // A plane slot: two tiles
  constexpr int kBHalves = kNarrowN * kSlice;  // B plane slot: one tile
  constexpr int kAH = 0, kAL = kAHalves, kBH = 2 * kAHalves, kBL = 2 * kAHalves + kBHalves;
  constexpr int kStageHalves = 2 * (kAHalves + kBHalves);
  constexpr int kDma = 3;  // 24 blocks of 1 KiB per stage over 8 waves
  constexpr int kSub = 2;
  if constexpr (V == kElementwise) {
    if (range[0] != range[1]) return;  // the scaled wide kernel handles this case
  }
  extern __shared__ __align__(16) uint16_t lds[];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  // Persistent grid: each workgroup walks tiles blockIdx.x, + gridDim.x, ...
  for (int tile = blockIdx.x; tile < tiles_m * tiles_n; tile += gridDim.x) {
    int tm, tn;
    tile_of<8>(tile, tiles_m, tiles_n, tm, tn);
    // Every wave is done with the previous tile's LDS before it is refilled.
    lds_barrier();
    const int64_t slices = Kp / kSlice;
    const int ktiles = static_cast<int>(slices);
    const int64_t panel_stride = slices * kTileHalves;

    // Wave w copies block w of A_hi and of A_lo (8 blocks each: two tiles of
    // four) and block w of the eight blocks of B_hi and B_lo.
    const uint16_t* src[3] = {
        a_hi + (2 * tm + (w >> 2)) * panel_stride + (w & 3) * 512 + lane * 8,
        a_lo + (2 * tm + (w >> 2)) * panel_stride + (w & 3) * 512 + lane * 8,
        (w < 4 ? b_hi : b_lo) + tn * panel_stride + (w & 3) * 512 + lane * 8};
    const int dst_off[3] = {kAH + w * 512, kAL + w * 512, (w < 4 ? kBH : kBL) + (w & 3) * 512};
    const unsigned lds_base = lds_address(lds);
    auto dma_one = [&](int kt, int n) {
      const int ktc = min(kt, ktiles - 1);
      dma16(src[n] + static_cast<int64_t>(ktc) * kTileHalves,
            lds_base + ((kt % S) * kStageHalves + dst_off[n]) * 2);
    };

    const int fr = lane & 31, fk = lane >> 5;
    int aoff[kSub], boff[kSub];
  #pragma unroll
    for (int i = 0; i < kSub; ++i) {
      aoff[i] = frag_offset(wm * 64 + i * 32 + fr, fk);
      boff[i] = frag_offset(wn * 64 + i * 32 + fr, fk);
    }
    auto rd = [&](int kt, int slot, int off) -> half8 {
      return *reinterpret_cast<const half8*>(lds + (kt % S) * kStageHalves + slot + off);
    };
    const floatx16 zero = {};
    floatx16 acc[kSub][kSub], xa[kSub][kSub], xb[kSub][kSub];
  #pragma unroll
    for (int i = 0; i < kSub; ++i)
  #pragma unroll
      for (int j = 0; j < kSub; ++j) acc[i][j] = xa[i][j] = xb[i][j] = zero;
    half8 ah[kSub], al[kSub], bh[kSub], bl[kSub];

  #pragma unroll
    for (int st = 0; st < S; ++st)
  #pragma unroll
      for (int n = 0; n < kDma; ++n) dma_one(st, n);
    wait_vmcnt<(S - 1) * kDma>();
    lds_barrier();
  #pragma unroll
    for (int i = 0; i < kSub; ++i) {
      ah[i] = rd(0, kAH, aoff[i]);
      al[i] = rd(0, kAL, aoff[i]);
      bh[i] = rd(0, kBH, boff[i]);
      bl[i] = rd(0, kBL, boff[i]);
    }

    // One k-step: XA, then HH, then XB; each fragment is reloaded with step
    // kt+1 once its last MFMA of the step is issued.  `first` marks the first
    // step of a block (block sums restart), `last` its end (fold).  Register
    // sets: termwise acc = HH, xa = XA, xb = XB; elementwise fallback acc =
    // running sum, xa = XA_g, xb = XB_g; cross-first acc = running sum, xa =
    // X_g = XA_g + XB_g, xb = HH_g.
    constexpr bool kBlocks = V != kTermwise;
    auto step = [&](int kt, bool first, bool last) {
      const int nk = kt + 1;
#pragma unroll
      for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j)
          xa[i][j] = mfma32(al[i], bh[j], (kBlocks && first) ? zero : xa[i][j]);
      SCHED_FENCE();
      wait_vmcnt<(S - 2) * kDma>();
      lds_barrier();
#pragma unroll
      for (int i = 0; i < kSub; ++i) al[i] = rd(nk, kAL, aoff[i]);
      dma_one(kt + S, 0);
      SCHED_FENCE();
#pragma unroll
      for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
          if constexpr (V == kCrossFirst)
            xb[i][j] = mfma32(ah[i], bh[j], first ? zero : xb[i][j]);
          else
            acc[i][j] = mfma32(ah[i], bh[j], acc[i][j]);
        }
      SCHED_FENCE();
#pragma unroll
      for (int j = 0; j < kSub; ++j) bh[j] = rd(nk, kBH, boff[j]);
      dma_one(kt + S, 1);
      SCHED_FENCE();
#pragma unroll
      for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
          if constexpr (V == kCrossFirst)
            xa[i][j] = mfma32(ah[i], bl[j], xa[i][j]);
          else
            xb[i][j] = mfma32(ah[i], bl[j], (kBlocks && first) ? zero : xb[i][j]);
        }
      SCHED_FENCE();
#pragma unroll
      for (int i = 0; i < kSub; ++i) {
        ah[i] = rd(nk, kAH, aoff[i]);
        bl[i] = rd(nk, kBL, boff[i]);
      }
      dma_one(kt + S, 2);
      SCHED_FENCE();
      if constexpr (V == kElementwise) {
        if (last) {
          // End of block g: acc = (acc + XA_g / s) + XB_g / s.
#pragma unroll
          for (int i = 0; i < kSub; ++i)
#pragma unroll
            for (int j = 0; j < kSub; ++j)
#pragma unroll
              for (int e = 0; e < 16; ++e) {
                acc[i][j][e] = __builtin_fmaf(xa[i][j][e], inv_s, acc[i][j][e]);
                acc[i][j][e] = __builtin_fmaf(xb[i][j][e], inv_s, acc[i][j][e]);
              }
        }
      } else if constexpr (V == kCrossFirst) {
        if (last) {
          // End of block g: acc = acc + (X_g / s + HH_g).
#pragma unroll
          for (int i = 0; i < kSub; ++i)
#pragma unroll
            for (int j = 0; j < kSub; ++j)
#pragma unroll
              for (int e = 0; e < 16; ++e)
                acc[i][j][e] += __builtin_fmaf(xa[i][j][e], inv_s, xb[i][j][e]);
        }
      }
    };
    for (int kt = 0; kt < ktiles; kt += 2) {
      step(kt, true, false);
      step(kt + 1, false, true);
    }
    wait_vmcnt<0>();

    const int col0 = tn * kNarrowN + wn * 64 + (lane & 31);
    const int row0 = tm * kNarrowM + wm * 64 + (lane >> 5) * 4;
    const bool full = (tm + 1) * kNarrowM <= M && (tn + 1) * kNarrowN <= N;
    store_tile<kSub, kSub>(C, ldc, M, N, row0, col0, full, [&](int i, int j, int r) {
      float v = acc[i][j][r];
      if constexpr (V == kTermwise) {
        v = __builtin_fmaf(xa[i][j][r], inv_s, v);
        v = __builtin_fmaf(xb[i][j][r], inv_s, v);
      }
      return v;
    });
  }
}


template <int V, int S = kWideStages>
hipError_t launch_wide(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc, float s,
                       hipStream_t stream) {
  constexpr size_t lds = wide_lds_bytes<V, S>();
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_wide_kernel<V, S>, lds, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kWide);
  const int tiles_n = static_cast<int>(p.Np / kWide);
  hipLaunchKernelGGL((gemm_wide_kernel<V, S>), dim3(tiles_m * tiles_n), dim3(kWideThreads), lds,
                     stream, p.a_hi, p.a_lo, p.b_hi, p.b_lo, p.range,
                     static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc, static_cast<int>(M),
                     static_cast<int>(N), s, 1.0f / s);
  return hipGetLastError();
}

template <int V>
hipError_t launch_narrow(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc, float s,
                         int cus, hipStream_t stream) {
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_narrow_kernel<V>, kNarrowLdsBytes, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kNarrowM);
  const int tiles_n = static_cast<int>(p.Np / kNarrowN);
  // One workgroup per compute unit (the kernel's occupancy), rounded to the
  // 8 XCDs; fewer when there are fewer tiles.
  const int grid = static_cast<int>(
      std::min<int64_t>(static_cast<int64_t>(tiles_m) * tiles_n, std::max(8, cus / 8 * 8)));
  hipLaunchKernelGGL(gemm_narrow_kernel<V>, dim3(grid), dim3(kNarrowThreads),
                     kNarrowLdsBytes, stream, p.a_hi, p.a_lo, p.b_hi, p.b_lo, p.range,
                     static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc, static_cast<int>(M),
                     static_cast<int>(N), s, 1.0f / s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float scale, int variant, int cus, hipStream_t stream) {
  switch (variant) {
    case kElementwise: {
      const hipError_t e = launch_wide<kElementwise>(p, M, N, C, ldc, scale, stream);
      if (e != hipSuccess) return e;
      return launch_narrow<kElementwise>(p, M, N, C, ldc, scale, cus, stream);
    }
    case kTermwise: return launch_narrow<kTermwise>(p, M, N, C, ldc, scale, cus, stream);
    case kCrossFirst: return launch_narrow<kCrossFirst>(p, M, N, C, ldc, scale, cus, stream);
    case kHiOnly: return launch_wide<kHiOnly>(p, M, N, C, ldc, scale, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_fallback(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                                float scale, int cus, hipStream_t stream) {
  return launch_narrow<kElementwise>(p, M, N, C, ldc, scale, cus, stream);
}

hipError_t launch_gemm_stages(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                              float scale, int stages, int cus, hipStream_t stream) {
  hipError_t e = hipSuccess;
  switch (stages) {
    case 1: e = launch_wide<kElementwise, 1>(p, M, N, C, ldc, scale, stream); break;
    case 2: e = launch_wide<kElementwise, 2>(p, M, N, C, ldc, scale, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  return launch_narrow<kElementwise>(p, M, N, C, ldc, scale, cus, stream);
}

}  // namespace sgc
