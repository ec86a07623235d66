// Three-product MFMA GEMM on prepared FP16 planes (gfx950).
//
// For each tile of C it forms (Eq. recover_eqn of arXiv 2507.23387)
//   HH = A_hi B_hi,  XA = A_lo B_hi,  XB = A_hi B_lo
// (FP16 x FP16 products are exact; an MFMA adds the products of a k-step to
// its C operand in one fused, once-rounded FP32 operation) and reconstructs
// C in the accumulation order asked for.
//
// Kernels:
//   gemm_el_kernel   256 x 256 tiles, v_mfma_f32_16x16x32_f16: the scaled
//                    elementwise order (Eq. elementwise, Sec. 4.5), one
//                    accumulator holding s * acc, blocks of one 32-wide
//                    k-step; on the A planes, or (kFusedA) on FP32 A that it
//                    splits in registers (Sec. 3.3).
//   gemm_n128_kernel 256 x 128 tiles, v_mfma_f32_16x16x32_f16: the orders
//                    that need more than one register set -- termwise (Eq.
//                    termwise), the unscaled elementwise fallback (range
//                    flag set) and the cross-terms-first order (end of
//                    Sec. 4.5), scaled and unscaled; termwise also on FP32
//                    A split in registers (kFusedA) and on FP32 B that the
//                    workgroup splits into its LDS planes (kFusedB).
//   gemm_hi_kernel   256 x 256 tiles: HH only, the native-FP16 baseline.
// The tile-shape sweep of the scaled elementwise order is in gemm_tile.hip.
// For the elementwise and cross-terms-first orders with s <= 2^15 both the
// scaled and the unscaled kernel of the order are launched; each reads the
// range flag first and the one that does not apply returns at once.  For s >
// 2^15, which is not a finite FP16 value, the host launches the unscaled
// kernel alone.
//
// Data path.  The planes are stored as 4 KiB tiles of 128 rows x 16 k in the
// order and swizzle the LDS wants (internal.h), so one pipeline stage (one
// k-step of a plane) is a few contiguous 4 KiB blocks, copied from global
// memory straight into LDS with global_load_lds_dwordx4 (no VGPR staging).
// Every wait count is a compile-time constant: past the last stage the loads
// repeat the last stage.  Each kernel's comment describes its schedule.
#include <algorithm>
#include <atomic>

#include "gemm_common.h"

namespace sgc {
namespace {

constexpr int kKSteps = kSlice / 16;  // MFMA k-steps per tile slice (1)
static_assert(kKSteps == 1, "one MFMA k-step per slice");
static_assert(kKPad % (2 * kSlice) == 0, "the main loops take two slices per iteration");

// ---------------------------------------------------------------------------
// 256 x 256 tiles on v_mfma_f32_16x16x32_f16: the scaled elementwise kernel
// and the hi-only baseline.
//
// The 16 x 16 x 32 form is used here because under the board's power limit it
// sustains a higher FP16 rate on random operands than the 32 x 32 x 16 form
// (less energy per product, so a higher shader clock at the same power).
constexpr int kWide = 256;
constexpr int kWideThreads = 256;
constexpr int kStep = 2 * kSlice;                  // k per MFMA step (32): two slices
constexpr int kWSub = 8;                           // 16 x 16 MFMA tiles per wave side
constexpr int kStepPlaneHalves = kWide * kStep;    // one plane of one step: 16 KiB
constexpr int kSlotHalves = 2 * kStepPlaneHalves;  // hi and lo planes of one operand
constexpr size_t kElLdsBytes = static_cast<size_t>(4) * kSlotHalves * 2;  // 128 KiB
constexpr size_t kHiLdsBytes = static_cast<size_t>(2) * 2 * kStepPlaneHalves * 2;  // 64 KiB

// Fragment offsets (halves, within one plane of one step) of this lane for a
// wave whose rows are panel `panel` of the tile: block i (rows 16 i .. 16 i
// + 15 of the panel) is at off[i & 1] + 16 i * kSlice.  Lane l reads row
// 16 i + l%16 and k chunk c = l/16 of the step, i.e. chunk c%2 of slice c/2;
// the chunk swap of the tile layout depends on bit 4 of the row, i.e. on the
// parity of i.
__device__ __forceinline__ void wide_frag_offsets(int lane, int panel, int (&off)[2]) {
  const int fr = lane & 15, fc = lane >> 4;
#pragma unroll
  for (int par = 0; par < 2; ++par)
    off[par] = (2 * panel + (fc >> 1)) * kTileHalves + fr * kSlice +
               (((fc & 1) ^ tile_swizzle(16 * par + fr)) << 3);
}

// Split of A into the tiled planes, used when the scaled kernel cannot run
// and the unscaled kernel that follows needs them: the blocking of the split
// kernel of A (a block of 16 rows x 128 k; lane l of wave w splits 8
// consecutive k of row 4w + l / 16, so each row is read as one 512-byte piece
// and each store fills whole 128-byte lines), the blocks taken in turn by the
// workgroups of the GEMM grid.  The GEMM's LDS allows one workgroup per
// compute unit, so each pass of the loop loads four blocks before it splits
// and stores them, to keep enough reads in flight.  A is 16-byte aligned with
// lda a multiple of 4 here; rows past M and k past K are written as zeros.
__device__ void split_a_planes(const float* __restrict__ A, int64_t lda, int M, int K, int Mp,
                               int Kp, uint16_t* __restrict__ a_hi, uint16_t* __restrict__ a_lo,
                               float s) {
  constexpr int kUnroll = 4;
  const int lane = threadIdx.x & 63;
  const int kblocks = (Kp + 127) / 128;
  const int64_t blocks = static_cast<int64_t>(Mp / 16) * kblocks;
  const int64_t stride = gridDim.x;
  for (int64_t b0 = blockIdx.x; b0 < blocks; b0 += stride * kUnroll) {
    float v[kUnroll][8];
    int64_t m[kUnroll], k0[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t b = b0 + u * stride;
      m[u] = (b / kblocks) * 16 + (threadIdx.x >> 6) * 4 + (lane >> 4);
      k0[u] = (b % kblocks) * 128 + (lane & 15) * 8;
      if (b < blocks && m[u] < M && k0[u] + 7 < K) {
        const float4* src = reinterpret_cast<const float4*>(A + m[u] * lda + k0[u]);
        const float4 f0 = src[0], f1 = src[1];
        v[u][0] = f0.x; v[u][1] = f0.y; v[u][2] = f0.z; v[u][3] = f0.w;
        v[u][4] = f1.x; v[u][5] = f1.y; v[u][6] = f1.z; v[u][7] = f1.w;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          v[u][e] = (b < blocks && m[u] < M && k0[u] + e < K) ? A[m[u] * lda + k0[u] + e] : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (b0 + u * stride >= blocks || k0[u] >= Kp) continue;
      u32x4 hv, lv;
      split8(v[u], s, hv, lv);
      const int64_t idx = tiled_index(m[u], k0[u], Kp);
      store_stream(a_hi + idx, hv);
      store_stream(a_lo + idx, lv);
    }
  }
}

// Scaled elementwise kernel (Eq. elementwise, Sec. 4.5), one 256 x 256 tile
// of C per workgroup, 4 waves of 128 x 128 (one per SIMD; 64 accumulators of
// 16 x 16 in the 256 AGPRs).  The contraction is cut into blocks g of one
// MFMA k-step (32), and the accumulator holds s * acc, so the three
// per-block additions of the equation are three chained MFMAs:
//   s*acc <- fl(s*acc + A_hi (s B_hi))   = s * fl(acc + HH_g)
//   s*acc <- fl(s*acc + A_lo B_hi)       = s * fl(acc + XA_g / s)
//   s*acc <- fl(s*acc + A_hi B_lo)       = s * fl(acc + XB_g / s)
// and C = (s*acc) / s at the end.  s B_hi is formed in registers with
// v_pk_mul_f16 from s converted to FP16; it is exact because s is a power of
// two, provided s <= 2^15 (checked on the host, which otherwise never launches
// this kernel) and |B_hi| s <= 65504, which the split of B checks (the range
// flag; when it is set this kernel returns at once and gemm_n128_kernel
// computes C).  Each
// block term is summed by the MFMA together with the accumulator, with one
// rounding, instead of being rounded to FP32 on its own first.
//
// Data path.  LDS holds two A slots and two B slots (32 KiB each: the hi and
// lo planes of one operand for one step, copied verbatim from the tiled planes
// by LDS DMA).  A wave keeps the A fragments of the whole step in registers
// (A_hi, A_lo of its 128 rows) and streams B one 16-column block at a time,
// read from LDS one block ahead.  During step kt it
//   - reads the A fragments of step kt+1 into a second register set, two or
//     three per column block (blocks 0-6), the two sets swapping roles each
//     step;
//   - copies B stage kt+1 and A stage kt+2 into LDS with 16 DMAs, four in
//     each of column blocks 0-3 (bursts of DMAs stall the wave's issue);
// and every LDS read, DMA and VALU instruction sits between two MFMAs.  One
// barrier per step, before the last column block, publishes B stage kt+1 and
// A stage kt+2 and retires the slots of B stage kt and A stage kt+1.  Stages
// past the end repeat the last stage, so every wait count is a constant.
// kPrefetch = false (pipeline ablation): the 16 DMAs of a step are issued
// right before its barrier, so no copy overlaps the MFMAs.
template <bool kPrefetch, bool kFusedA>
__global__ __launch_bounds__(kWideThreads, 1) void gemm_el_kernel(
    uint16_t* __restrict__ a_hi, uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int M, int N, float s, float inv_s,
    const float* __restrict__ af, int64_t lda, int K) {
  static_assert(kPrefetch || !kFusedA, "the fused split runs with the overlapped copies only");
  constexpr int kBBase = 2 * kSlotHalves;     // the B slots follow the two A slots
  // The furthest DMA targets: plane tile 3 of the lo plane of B slot 1, and
  // of A slot 1 (FP32 rows of the fused split: 4 KiB group 7 of slot 1).
  static_assert(dma_end_bytes(kBBase + kSlotHalves + kStepPlaneHalves + 3 * kTileHalves) <=
                    kElLdsBytes && kElLdsBytes <= kMaxLdsBytes, "B DMAs stay in LDS");
  static_assert(dma_end_bytes(kSlotHalves + kStepPlaneHalves + 3 * kTileHalves) <=
                    static_cast<size_t>(kBBase) * 2, "A DMAs stay in the A slots");
  static_assert(static_cast<size_t>(kSlotHalves) * 2 + 7 * 4096 + 4096 <=
                    static_cast<size_t>(kBBase) * 2, "FP32 A DMAs stay in the A slots");
  constexpr int kDmaCols = 4;                 // column blocks that issue the DMAs
  constexpr int kDmaPerCol = 16 / kDmaCols;   // after MFMAs 2, 8, 14, 20 of a block
  int tm, tn;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn))
    tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  if (range[0] == range[1]) {
    // s B_hi overflows FP16: gemm_n128_kernel runs instead.  Without planes
    // of A (fused split), this kernel first writes them for it.
    if constexpr (kFusedA) split_a_planes(af, lda, M, K, tiles_m * kWide, Kp, a_hi, a_lo, s);
    return;
  }
  extern __shared__ __align__(16) uint16_t lds[];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int64_t slices = Kp / kSlice;
  const int ksteps = static_cast<int>(slices / 2);

  // One plane of one stage is the four 4 KiB tiles (panel ph, slice sl) of
  // the tile's two panels and the step's two slices, at tile position
  // 2*ph + sl of the slot; wave w copies 1 KiB block w of each.
  const int64_t panel_stride = slices * kTileHalves;
  const unsigned lane_off = static_cast<unsigned>(w * 512 + lane * 8) * 2;  // bytes
  const uint16_t* const src_a[2] = {a_hi + 2 * tm * panel_stride, a_lo + 2 * tm * panel_stride};
  const uint16_t* const src_b[2] = {b_hi + 2 * tn * panel_stride, b_lo + 2 * tn * panel_stride};
  const unsigned lds_base = lds_address(lds) + w * 1024;
  // n-th DMA (n < 8) of the A or B stage t.
  auto dma_stage = [&](const uint16_t* const (&src)[2], int base, int t, int n) {
    const int tc = min(t, ksteps - 1);
    const int p = n >> 2, ph = (n >> 1) & 1, sl = n & 1;
    dma16s(src[p] + ph * panel_stride + static_cast<int64_t>(2 * tc + sl) * kTileHalves,
           lane_off,
           lds_base + (base + (t & 1) * kSlotHalves + p * kStepPlaneHalves +
                       (2 * ph + sl) * kTileHalves) * 2);
  };
  // Fused split: an A slot holds the FP32 rows of the stage, 256 rows x 32 k
  // (32 KiB).  Row r's eight 16-byte chunks (k 4q .. 4q+3) sit at chunk
  // positions q ^ g(r) of its 128 bytes, g(r) = (r & 3) << 1 | bit 3 of r.
  // Measured with the LDS bank-conflict counter on gfx950: the fragment
  // reads below (16 rows x 4 chunks per instruction) have no bank conflicts
  // with this swap, while swaps that leave rows 8 apart (1 KiB) on the same
  // chunk positions conflict (4-12 extra cycles per read).  DMA n (0-31)
  // fills rows 8n .. 8n+7, wave w issuing n = w + 4d, d = 0-7: lane l copies
  // chunk (l & 7) ^ g(r) of row r = 8n + (l >> 3), and
  // g(r) = ((l >> 3) & 3) << 1 | (w & 1) for every d.  Rows past M repeat row
  // M - 1 (their results are never stored).  K is a multiple of 64 here, so
  // no copy reads past a row of A.
  unsigned a_voff[kFusedA ? 8 : 1];
  const float* a_tile = nullptr;
  if constexpr (kFusedA) {
    const int row0 = tm * kWide;
    const int q = (lane & 7) ^ ((((lane >> 3) & 3) << 1) | (w & 1));
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const int r = min(row0 + 8 * (w + 4 * d) + (lane >> 3), M - 1) - row0;
      a_voff[d] = static_cast<unsigned>(r * lda * 4 + q * 16);
    }
    a_tile = af + static_cast<int64_t>(row0) * lda;
  }
  auto dma_af = [&](int t, int d) {
    const int tc = min(t, ksteps - 1);
    dma16s(a_tile + static_cast<int64_t>(tc) * kStep, a_voff[d],
           lds_base + (t & 1) * kSlotHalves * 2 + d * 4096);
  };
  // The d-th of the 16 DMAs of step kt: B stage kt+1, then A stage kt+2.
  auto dma = [&](int kt, int d) {
    if (d < 8)
      dma_stage(src_b, kBBase, kt + 1, d);
    else if constexpr (kFusedA)
      dma_af(kt + 2, d - 8);
    else
      dma_stage(src_a, 0, kt + 2, d - 8);
  };
  // Fused split: lane l's A fragment of row block i is row 16 i + l % 16 of
  // the wave's 128 rows, k 8c .. 8c + 7 (c = l / 16), i.e. chunks 2c and
  // 2c + 1 of the row; with the swap above (bits 0, 1 and 3 of the row are
  // those of l), two 16-byte reads.
  int af_off[2];
  const int af_swap = ((lane & 3) << 1) | ((lane >> 3) & 1);
#pragma unroll
  for (int h = 0; h < 2; ++h)
    af_off[h] = ((lane & 15) * 8 + ((2 * (lane >> 4) + h) ^ af_swap)) * 16;
  auto rd_af = [&](int t, int i, int h) -> floatx4 {
    const char* base = reinterpret_cast<const char*>(lds) + (t & 1) * kSlotHalves * 2;
    return *reinterpret_cast<const floatx4*>(base + (128 * wm + 16 * i) * 128 + af_off[h]);
  };
  const float s_sgpr = __builtin_bit_cast(
      float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, s)));
  // Instruction k (0-19) of the split of one row block's eight values f
  // (f[0]: k 8c .. 8c+3, f[1]: 8c+4 .. 8c+7) into the A_hi and A_lo
  // fragments h, l: the four high words first (k 0-3), then for pairs 0-1
  // and then 2-3 the residuals and the scaled residual words (k 4-11,
  // 12-19), five instructions per pair.
  auto split_k = [&](auto Kc, half8& h, half8& l, const floatx4 (&f)[2], float (&r)[2][2]) {
    constexpr int k = decltype(Kc)::value;
    constexpr int pair = k < 4 ? k : 2 * ((k - 4) / 8) + ((k - 4) % 8 < 4 ? ((k - 4) % 8) / 2
                                                                          : ((k - 4) % 8 - 4) / 2);
    constexpr int op = k < 4 ? 0 : ((k - 4) % 8 < 4 ? 1 + (k - 4) % 2 : 3 + (k - 4) % 2);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 hv = __builtin_bit_cast(u32x4, h), lv = __builtin_bit_cast(u32x4, l);
    uint32_t hw = hv[pair], lw = lv[pair];
    const float a0 = f[pair / 2][2 * (pair % 2)], a1 = f[pair / 2][2 * (pair % 2) + 1];
    split_op<op>(hw, lw, r[pair % 2], a0, a1, s_sgpr);
    if constexpr (op == 0) {
      hv[pair] = hw;
      h = __builtin_bit_cast(half8, hv);
    }
    if constexpr (op >= 3) {
      lv[pair] = lw;
      l = __builtin_bit_cast(half8, lv);
    }
  };

  int a_off[2], b_off[2];
  wide_frag_offsets(lane, wm, a_off);
  wide_frag_offsets(lane, wn, b_off);
  auto rd_a = [&](int t, int p, int i) -> half8 {
    return *reinterpret_cast<const half8*>(lds + (t & 1) * kSlotHalves + p * kStepPlaneHalves +
                                           a_off[i & 1] + i * 16 * kSlice);
  };
  auto rd_b = [&](int t, int p, int j) -> half8 {
    return *reinterpret_cast<const half8*>(lds + kBBase + (t & 1) * kSlotHalves +
                                           p * kStepPlaneHalves + b_off[j & 1] + j * 16 * kSlice);
  };
  // (s, s) as a packed FP16 pair, wave-uniform.
  const uint16_t s_bits = __builtin_bit_cast(uint16_t, static_cast<_Float16>(s));
  const uint32_t s2 = static_cast<uint32_t>(
      __builtin_amdgcn_readfirstlane(static_cast<int>(s_bits * 0x10001u)));

  floatx4 acc[kWSub][kWSub];
#pragma unroll
  for (int i = 0; i < kWSub; ++i)
#pragma unroll
    for (int j = 0; j < kWSub; ++j) acc[i][j] = floatx4{};

  // Prologue: A stages 0 and 1 and B stage 0; A stage 0 goes to registers.
  if constexpr (kFusedA) {
    static_for<8>([&](auto n) { dma_af(0, decltype(n)::value); });
    static_for<8>([&](auto n) { dma_af(1, decltype(n)::value); });
  } else {
    static_for<8>([&](auto n) { dma_stage(src_a, 0, 0, decltype(n)::value); });
    static_for<8>([&](auto n) { dma_stage(src_a, 0, 1, decltype(n)::value); });
  }
  static_for<8>([&](auto n) { dma_stage(src_b, kBBase, 0, decltype(n)::value); });
  wait_vmcnt<0>();
  lds_barrier();
  // (AH, AL) and (NH, NL): A_hi, A_lo of the current and of the next step.
  // bh, bl, bs: B_hi, B_lo, s B_hi of a column block, double-buffered by the
  // parity of the block.  Fused split: F[i & 1] holds the FP32 fragment of
  // row block i of the next stage from its reads (one column block before
  // its split) to its split; rr holds the residuals of two pairs.
  half8 AH[kWSub], AL[kWSub], NH[kWSub], NL[kWSub], bh[2], bl[2], bs[2];
  floatx4 F[2][2];
  float rr[2][2];
  if constexpr (kFusedA) {
#pragma unroll
    for (int i = 0; i < kWSub; ++i) {
      AH[i] = AL[i] = half8{};
      F[0][0] = rd_af(0, i, 0);
      F[0][1] = rd_af(0, i, 1);
      static_for<20>([&](auto Kc) { split_k(Kc, AH[i], AL[i], F[0], rr); });
    }
    // Row block 0 of stage 1, split during step 0.
    F[0][0] = rd_af(1, 0, 0);
    F[0][1] = rd_af(1, 0, 1);
  } else {
#pragma unroll
    for (int i = 0; i < kWSub; ++i) {
      AH[i] = rd_a(0, 0, i);
      AL[i] = rd_a(0, 1, i);
    }
  }
  bh[0] = rd_b(0, 0, 0);
  bl[0] = rd_b(0, 1, 0);
  bs[0] = pk_scale(bh[0], s2);
  lds_barrier();  // A slot 0 is refilled (stage 2) during step 0

  // One step.  Column block j issues HH(., j), XA(., j), XB(., j), so every
  // accumulator sees the block terms in the order HH, XA, XB, and the three
  // MFMAs of one accumulator are 8 MFMAs apart.  After MFMA m of a block:
  // m = 1, 9, 17 read the next A fragments, m = 2, 8, 14, 20 of blocks 0-3
  // issue the DMAs, m = 12 and 14 form the next block's s B_hi (two halves:
  // two VALU instructions overlap an MFMA for free, four do not).
  auto step = [&](int kt, half8 (&ah)[kWSub], half8 (&al)[kWSub], half8 (&nh)[kWSub],
                  half8 (&nl)[kWSub]) {
    static_for<kWSub>([&](auto J) {
      constexpr int j = decltype(J)::value, c = j & 1;
      if constexpr (j == kWSub - 1) {
        if constexpr (!kPrefetch) static_for<16>([&](auto d) { dma(kt, decltype(d)::value); });
        wait_vmcnt<0>();
        lds_barrier();
        bh[c ^ 1] = rd_b(kt + 1, 0, 0);
        bl[c ^ 1] = rd_b(kt + 1, 1, 0);
      } else {
        bh[c ^ 1] = rd_b(kt, 0, j + 1);
        bl[c ^ 1] = rd_b(kt, 1, j + 1);
      }
      SCHED_FENCE();
      // A fragments rb .. re-1 of the 16 (A_hi rows 0-7, then A_lo) in block j.
      constexpr int rb = (16 * j + 6) / 7, re = (16 * (j + 1) + 6) / 7;
      static_for<3 * kWSub>([&](auto Mc) {
        constexpr int m = decltype(Mc)::value, g = m / kWSub, i = m % kWSub;
        if constexpr (g == 0)
          mfma16_acc(acc[i][j], ah[i], bs[c]);
        else if constexpr (g == 1)
          mfma16_acc(acc[i][j], al[i], bh[c]);
        else
          mfma16_acc(acc[i][j], ah[i], bl[c]);
        SCHED_FENCE();
        if constexpr (kFusedA) {
          // One VALU instruction after every MFMA: s B_hi of the next block
          // one word at a time after MFMAs 12-15, and the 20 instructions of
          // the split after MFMAs 0-11 and 16-23.  Column block j reads row
          // block j + 1 of stage kt+1 (block 7, after its barrier: row block
          // 0 of stage kt+2) and splits row block j, read one block earlier,
          // into the next step's fragments; the last instruction for row
          // block 7 comes 16 MFMAs before the next step's first use of it.
          if constexpr (m >= 12 && m <= 15) pk_scale_word<m - 12>(bs[c ^ 1], bh[c ^ 1], s2);
          constexpr int nxt = (j + 1) % kWSub;
          if constexpr (m == 1) F[nxt & 1][0] = rd_af(j == kWSub - 1 ? kt + 2 : kt + 1, nxt, 0);
          if constexpr (m == 3) F[nxt & 1][1] = rd_af(j == kWSub - 1 ? kt + 2 : kt + 1, nxt, 1);
          constexpr int k = m < 12 ? m : m >= 16 ? m - 4 : -1;
          if constexpr (k >= 0)
            split_k(std::integral_constant<int, k>{}, nh[j], nl[j], F[j & 1], rr);
        } else {
          if constexpr (m == 12) pk_scale_half<0>(bs[c ^ 1], bh[c ^ 1], s2);
          if constexpr (m == 14) pk_scale_half<1>(bs[c ^ 1], bh[c ^ 1], s2);
        }
        if constexpr (!kFusedA && j < kWSub - 1 && m % kWSub == 1) {
          constexpr int r = rb + m / kWSub;
          if constexpr (r < re) {
            if constexpr (r < kWSub)
              nh[r] = rd_a(kt + 1, 0, r);
            else
              nl[r - kWSub] = rd_a(kt + 1, 1, r - kWSub);
          }
        }
        if constexpr (kPrefetch && j < kDmaCols && m % 6 == 2) dma(kt, j * kDmaPerCol + m / 6);
        SCHED_FENCE();
      });
    });
  };
  for (int kt = 0; kt < ksteps; kt += 2) {
    step(kt, AH, AL, NH, NL);
    step(kt + 1, NH, NL, AH, AL);
  }
  // No LDS DMA may still be writing when the workgroup retires.
  wait_vmcnt<0>();
  mfma_drain();

  const int col0 = tn * kWide + wn * 128 + (lane & 15);
  const int row0 = tm * kWide + wm * 128 + (lane >> 4) * 4;
  const bool full = (tm + 1) * kWide <= M && (tn + 1) * kWide <= N;
  store_tile16<kWSub, kWSub>(C, ldc, M, N, row0, col0, full,
                             [&](int i, int j, int r) { return acc[i][j][r] * inv_s; });
}

// Hi-only kernel: C = A_hi B_hi, the native-FP16 GEMM baseline (Sec. 6.2),
// with the tile, wave split and LDS layout of the elementwise kernel minus
// the lo planes: a two-slot ring of (A_hi, B_hi) stages; each wave walks its
// rows of 16 x 16 blocks, B fragments of the step in registers, A fragments
// read one row ahead; one barrier per step publishes stage kt+1.
__global__ __launch_bounds__(kWideThreads, 1) void gemm_hi_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ b_hi, int Kp, int tiles_m,
    int tiles_n, float* __restrict__ C, int64_t ldc, int M, int N) {
  constexpr int kStageHalves = 2 * kStepPlaneHalves;  // A_hi, B_hi
  constexpr int kDma = 8;                             // 1 KiB DMAs per wave per stage
  static_assert(dma_end_bytes(kStageHalves + kStepPlaneHalves + 3 * kTileHalves) <=
                    kHiLdsBytes && kHiLdsBytes <= kMaxLdsBytes, "DMAs stay in LDS");
  extern __shared__ __align__(16) uint16_t lds[];

  int tm, tn;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn))
    tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int64_t slices = Kp / kSlice;
  const int ksteps = static_cast<int>(slices / 2);
  const int64_t panel_stride = slices * kTileHalves;
  const unsigned lane_off = static_cast<unsigned>(w * 512 + lane * 8) * 2;
  const uint16_t* const src[2] = {a_hi + 2 * tm * panel_stride, b_hi + 2 * tn * panel_stride};
  const unsigned lds_base = lds_address(lds) + w * 1024;
  auto dma_one = [&](int kt, int n) {  // n-th DMA of stage kt, n < kDma
    const int ktc = min(kt, ksteps - 1);
    const int p = n >> 2, ph = (n >> 1) & 1, sl = n & 1;
    dma16s(src[p] + ph * panel_stride + static_cast<int64_t>(2 * ktc + sl) * kTileHalves,
           lane_off,
           lds_base + ((kt & 1) * kStageHalves + p * kStepPlaneHalves +
                       (2 * ph + sl) * kTileHalves) * 2);
  };
  int a_off[2], b_off[2];
  wide_frag_offsets(lane, wm, a_off);
  wide_frag_offsets(lane, wn, b_off);
  auto rd = [&](int kt, int p, int i) -> half8 {
    return *reinterpret_cast<const half8*>(lds + (kt & 1) * kStageHalves + p * kStepPlaneHalves +
                                           (p == 0 ? a_off[i & 1] : b_off[i & 1]) +
                                           i * 16 * kSlice);
  };

  floatx4 acc[kWSub][kWSub];
#pragma unroll
  for (int i = 0; i < kWSub; ++i)
#pragma unroll
    for (int j = 0; j < kWSub; ++j) acc[i][j] = floatx4{};

  static_for<kDma>([&](auto n) { dma_one(0, decltype(n)::value); });
  wait_vmcnt<0>();
  lds_barrier();
  half8 b0[kWSub], b1[kWSub], a_h[2];
#pragma unroll
  for (int j = 0; j < kWSub; ++j) b0[j] = rd(0, 1, j);
  a_h[0] = rd(0, 0, 0);
  auto step = [&](int kt, half8 (&bc)[kWSub], half8 (&bn)[kWSub]) {
    static_for<kWSub>([&](auto I) {
      constexpr int i = decltype(I)::value, c = i & 1;
      if constexpr (i == kWSub - 1) {
        wait_vmcnt<0>();
        lds_barrier();
        a_h[c ^ 1] = rd(kt + 1, 0, 0);
#pragma unroll
        for (int j = 0; j < kWSub; ++j) bn[j] = rd(kt + 1, 1, j);
      } else {
        a_h[c ^ 1] = rd(kt, 0, i + 1);
        if constexpr (i < 4) {
          dma_one(kt + 1, 2 * i);
          dma_one(kt + 1, 2 * i + 1);
        }
      }
      SCHED_FENCE();
      static_for<kWSub>([&](auto J) {
        constexpr int j = decltype(J)::value;
        mfma16_acc(acc[i][j], a_h[c], bc[j]);
      });
      SCHED_FENCE();
    });
  };
  for (int kt = 0; kt < ksteps; kt += 2) {
    step(kt, b0, b1);
    step(kt + 1, b1, b0);
  }
  wait_vmcnt<0>();
  mfma_drain();

  const int col0 = tn * kWide + wn * 128 + (lane & 15);
  const int row0 = tm * kWide + wm * 128 + (lane >> 4) * 4;
  const bool full = (tm + 1) * kWide <= M && (tn + 1) * kWide <= N;
  store_tile16<kWSub, kWSub>(C, ldc, M, N, row0, col0, full,
                             [&](int i, int j, int r) { return acc[i][j][r]; });
}

// ---------------------------------------------------------------------------
// 256 x 128 tiles on v_mfma_f32_16x16x32_f16 for the orders that need three
// accumulator sets: one tile of C per workgroup, 4 waves of 64 x 128 (one
// per SIMD).
//   kTermwise (Eq. termwise): HH = A_hi B_hi, XA = A_lo B_hi, XB = A_hi B_lo
//     accumulate over all of K (HH and XA in AGPRs, XB in VGPRs, each
//     updated once per step) and the epilogue forms C = (HH + XA / s) + XB / s.
//   kElementwise when the range flag is set (s B_hi overflows FP16, so the
//     scaled 256 x 256 kernel cannot run): unscaled, blocks of one 32-wide
//     k-step.  HH goes straight into the accumulator (VGPRs) and XA_g, XB_g
//     into block sums started from zero; one column block later,
//     acc = (acc + XA_g / s) + XB_g / s with two v_fma_f32 (1/s is exact).
//   kCrossScaled (the reordered elementwise accumulation proposed at the end
//     of Sec. 4.5), the scaled kernel of that order: per block one MFMA
//     chain started from zero, XA_g, then XB_g, then A_hi (s B_hi), gives
//     fl(X_g + s HH_g) = s fl(X_g / s + HH_g) (s a power of two, s B_hi exact
//     under the same conditions as for the scaled elementwise kernel: s <=
//     2^15, range flag clear; when it is set this kernel returns at once);
//     one column block later the accumulator, which holds s * acc, adds it
//     with one v_add_f32, and C = (s * acc) / s.
//   kCrossFirst, its unscaled fallback (range flag set, or s > 2^15): per
//     block X_g = XA_g + XB_g (one MFMA chain started from zero) and HH_g
//     (started from zero); one column block later acc = acc + (X_g / s +
//     HH_g) with one v_fma_f32 and one add.
// In the block-fold orders the A fragments live in AGPRs (the MFMA reads its
// A operand from there) so that the accumulators and block sums fit the
// VGPRs; the fold of column block j runs between the MFMAs of block j+1, at
// least 8 MFMAs after the results it reads.
//
// The data path is the elementwise kernel's at half the width: LDS holds two
// A slots (A_hi, A_lo of 256 rows x 32 k: 32 KiB) and two B slots (B_hi,
// B_lo of 128 columns: 16 KiB).  A wave keeps its 64 rows of A for the step
// in registers and streams B one 16-column block at a time, one block ahead;
// during step kt it issues 12 DMAs (B stage kt+1, then A stage kt+2; three in
// each of blocks 0-3: spread two per block over blocks 0-5 they left the
// block-fold orders 5-6 % slower) and reads the A fragments of step kt+1 into
// a second set (one or two per block, blocks 2-6).  Two barriers per step:
// before block 2, A stage kt+1 (copied during step kt-1) has landed; before
// block 7, B stage kt+1 has, and B stage kt is retired.  The A copies so get
// a step and two blocks to land, not five blocks: with planes larger than the
// last-level cache (K = 16384) the single barrier that waited for all copies
// of the step left termwise 18 % slower.
//
// kFusedA (termwise only): the A slots hold the stage's FP32 rows instead of
// the A planes (256 rows x 32 k, 32 KiB, copied and swizzled as in the fused
// elementwise kernel), and each wave splits its 64 rows in registers (Sec.
// 3.3): it waits for A stage kt+1 before block 1 instead of block 2, and
// during blocks 1-7 of step kt it reads the FP32 fragments of that stage
// (two 16-byte reads per 16-row block, all before the barrier of block 7,
// which the DMAs of step kt+1 into that slot wait behind) and runs the 80
// vector instructions of the split, one between consecutive MFMAs (two once),
// into the register set of step kt+1.  The last of them comes 10 MFMAs
// before that set's first use.  The bits are those of the planes path.
//
// kFusedB (termwise only; with or without kFusedA): no B planes are read.
// Two more LDS slots (16 KiB each, 128 KiB in all) hold the FP32 rows of B
// for the stage, 32 k-rows x 128 columns, copied verbatim by LDS DMA one
// stage ahead as A is (columns past N repeat the last four; N is a multiple
// of 4 here).  The workgroup splits them into the B plane slots itself (Sec.
// 3.3): during blocks 2-6 of step kt, each thread splits one column, k
// 16 (t / 128) .. + 15 of stage kt+1, reading its 16 values from the FP32
// slot (each read has the 64 lanes of a wave on 64 consecutive words) and
// writing the high and the scaled residual words as the 16-byte chunks of
// the tiled plane layout, so everything after that is the planes path: the
// same fragments, the same MFMAs, the same bits.  The barrier before block 7,
// which publishes B stage kt+1, also publishes these writes; the FP32 slot
// is refilled (stage kt+3) only after it.
// The scaled cross-terms-first kernel: an n128 variant of the kernel only
// (the host's order code stays kCrossFirst).
constexpr int kCrossScaled = 4;
constexpr int kTwM = 256;
constexpr int kTwN = 128;
constexpr int kTwASlot = 2 * kTwM * kStep;        // halves: A_hi, A_lo of one step
constexpr int kTwBSlot = 2 * kTwN * kStep;        // halves: B_hi, B_lo of one step
constexpr int kTwBfSlotBytes = kTwN * kStep * 4;  // FP32 B rows of one step: 16 KiB
constexpr size_t kTwLdsBytes = static_cast<size_t>(2) * (kTwASlot + kTwBSlot) * 2;  // 96 KiB
constexpr size_t kTwFusedBLdsBytes = kTwLdsBytes + 2 * kTwBfSlotBytes;             // 128 KiB

// Slot (the MFMA of a step, 12 per column block, after which it is issued)
// of split instruction q (0-79: 16-row block q / 20, instruction q % 20) in
// the fused termwise kernel: 80 instructions over slots 15-93 (one slot holds
// two), so that the first comes three slots after the first fragment read
// (the reads start after the barrier before block 1, slot 12) and the last 10
// MFMAs before the next step's first use.
constexpr int kTwSplitFirst = 15, kTwSplitLast = 93;
constexpr int tw_split_slot(int q) {
  return kTwSplitFirst + q * (kTwSplitLast - kTwSplitFirst + 1) / 80;
}

template <int V, bool kFusedA = false, bool kFusedB = false>
__global__ __launch_bounds__(kWideThreads, 1) void gemm_n128_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int M, int N, float inv_s, int unscaled_only,
    const float* __restrict__ af, int64_t lda, float s, const float* __restrict__ bf,
    int64_t ldb) {
  static_assert(V == kTermwise || V == kElementwise || V == kCrossFirst || V == kCrossScaled,
                "n128 variants");
  static_assert(!kFusedA || V == kTermwise, "the fused split of A is built for termwise only");
  static_assert(!kFusedB || V == kTermwise, "the fused split of B is built for termwise only");
  constexpr bool kFold = V != kTermwise;
  constexpr int kRows = 4;                   // 16-row blocks per wave
  constexpr int kCols = 8;                   // 16-column blocks per wave
  constexpr int kAPlane = kTwM * kStep;      // one A plane of one step: 16 KiB
  constexpr int kBPlane = kTwN * kStep;      // one B plane of one step: 8 KiB
  constexpr int kBBase = 2 * kTwASlot;       // the B slots follow the two A slots
  static_assert(dma_end_bytes(kTwASlot + kAPlane + 3 * kTileHalves) <=
                    static_cast<size_t>(kBBase) * 2, "A DMAs stay in the A slots");
  static_assert(dma_end_bytes(kBBase + kTwBSlot + kBPlane + kTileHalves) <= kTwLdsBytes &&
                    kTwLdsBytes <= kMaxLdsBytes, "B DMAs stay in LDS");
  // Fused split of B: the FP32 slots follow the B plane slots; DMA d (0-3) of
  // wave w fills 1 KiB block w + 4 d of a slot.
  constexpr int kBfBase = 2 * kBBase + 2 * kTwBSlot * 2;  // bytes
  static_assert(kBfBase == static_cast<int>(kTwLdsBytes), "FP32 B slots follow the planes");
  static_assert(kBfBase + kTwBfSlotBytes + 3 * 4096 + 4096 <= static_cast<int>(kTwFusedBLdsBytes) &&
                    kTwFusedBLdsBytes <= kMaxLdsBytes, "FP32 B DMAs stay in LDS");
  if constexpr (V == kElementwise || V == kCrossFirst) {
    // Unless the host routed the call here (unscaled_only: s is not a finite
    // FP16 value), the scaled kernel of the order (256 x 256 elementwise,
    // kCrossScaled) handles the case where the range flag is clear.
    if (!unscaled_only && range[0] != range[1]) return;
  }
  if constexpr (V == kCrossScaled) {
    if (range[0] == range[1]) return;  // s B_hi overflows FP16: kCrossFirst runs
  }
  extern __shared__ __align__(16) uint16_t lds[];

  int tm, tn;
  if (!tile_of_block(blockIdx.x, tiles_m, tiles_n, tm, tn))
    tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t slices = Kp / kSlice;
  const int ksteps = static_cast<int>(slices / 2);

  // A stage: tiles (panel ph, slice sl) of the tile's two A panels at
  // position 2*ph + sl of each plane; B stage: tiles (slice sl) of its one B
  // panel at position sl.  Wave w copies 1 KiB block w of every tile.
  const int64_t panel_stride = slices * kTileHalves;
  const unsigned lane_off = static_cast<unsigned>(w * 512 + lane * 8) * 2;  // bytes
  const uint16_t* const src_a[2] = {a_hi + 2 * tm * panel_stride, a_lo + 2 * tm * panel_stride};
  const uint16_t* const src_b[2] = {b_hi + tn * panel_stride, b_lo + tn * panel_stride};
  const unsigned lds_base = lds_address(lds) + w * 1024;
  auto dma_a = [&](int t, int n) {  // n < 8
    const int tc = min(t, ksteps - 1);
    const int p = n >> 2, ph = (n >> 1) & 1, sl = n & 1;
    dma16s(src_a[p] + ph * panel_stride + static_cast<int64_t>(2 * tc + sl) * kTileHalves,
           lane_off,
           lds_base + ((t & 1) * kTwASlot + p * kAPlane + (2 * ph + sl) * kTileHalves) * 2);
  };
  auto dma_b = [&](int t, int n) {  // n < 4
    const int tc = min(t, ksteps - 1);
    const int p = n >> 1, sl = n & 1;
    dma16s(src_b[p] + static_cast<int64_t>(2 * tc + sl) * kTileHalves, lane_off,
           lds_base + (kBBase + (t & 1) * kTwBSlot + p * kBPlane + sl * kTileHalves) * 2);
  };
  // Fused split: an A slot holds the FP32 rows of the stage with the layout
  // of gemm_el_kernel's (row r's 16-byte chunks at positions q ^ g(r),
  // g(r) = (r & 3) << 1 | bit 3 of r; DMA n = w + 4d fills rows 8n .. 8n+7;
  // rows past M repeat row M - 1).
  unsigned a_voff[kFusedA ? 8 : 1];
  const float* a_tile = nullptr;
  if constexpr (kFusedA) {
    const int row0 = tm * kTwM;
    const int q = (lane & 7) ^ ((((lane >> 3) & 3) << 1) | (w & 1));
#pragma unroll
    for (int d = 0; d < 8; ++d) {
      const int r = min(row0 + 8 * (w + 4 * d) + (lane >> 3), M - 1) - row0;
      a_voff[d] = static_cast<unsigned>(r * lda * 4 + q * 16);
    }
    a_tile = af + static_cast<int64_t>(row0) * lda;
  }
  auto dma_af = [&](int t, int d) {
    const int tc = min(t, ksteps - 1);
    dma16s(a_tile + static_cast<int64_t>(tc) * kStep, a_voff[d],
           lds_base + (t & 1) * kTwASlot * 2 + d * 4096);
  };
  // Fused split of B: lane l of DMA d of wave w copies k-row
  // 2 (w + 4 d) + l / 32 of the stage, columns 4 (l % 32) .. + 3 of the tile
  // (clamped to the last four columns of B), to byte 512 k-row + 16 (l % 32)
  // of the slot.  K is a multiple of 64 here, so no copy reads past row K - 1.
  unsigned b_voff[kFusedB ? 4 : 1];
  const float* b_tile = nullptr;
  if constexpr (kFusedB) {
    const int col = min(tn * kTwN + 4 * (lane & 31), N - 4);
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const int row = 2 * (w + 4 * d) + (lane >> 5);
      b_voff[d] = static_cast<unsigned>((row * ldb + col) * 4);
    }
    b_tile = bf;
  }
  auto dma_bf = [&](int t, int d) {
    const int tc = min(t, ksteps - 1);
    dma16s(b_tile + static_cast<int64_t>(tc) * kStep * ldb, b_voff[d],
           lds_base + kBfBase + (t & 1) * kTwBfSlotBytes + d * 4096);
  };
  // The d-th of the 12 DMAs of step kt: B stage kt+1 (FP32 B: stage kt+2),
  // then A stage kt+2.
  auto dma = [&](int kt, int d) {
    if (d < 4) {
      if constexpr (kFusedB)
        dma_bf(kt + 2, d);
      else
        dma_b(kt + 1, d);
    } else if constexpr (kFusedA)
      dma_af(kt + 2, d - 4);
    else
      dma_a(kt + 2, d - 4);
  };

  // Wave w's rows are rows 64 (w & 1) .. 64 (w & 1) + 63 of A panel w >> 1;
  // block i (16 rows) of them and column block j of the B panel are read as
  // in the elementwise kernel (row bit 4 = parity of the block).
  int a_off[2], b_off[2];
  wide_frag_offsets(lane, w >> 1, a_off);
  wide_frag_offsets(lane, 0, b_off);
  const int a_row = 64 * (w & 1) * kSlice;
  auto rd_a = [&](int t, int p, int i) -> half8 {
    return *reinterpret_cast<const half8*>(lds + (t & 1) * kTwASlot + p * kAPlane + a_off[i & 1] +
                                           a_row + i * 16 * kSlice);
  };
  auto rd_b = [&](int t, int p, int j) -> half8 {
    return *reinterpret_cast<const half8*>(lds + kBBase + (t & 1) * kTwBSlot + p * kBPlane +
                                           b_off[j & 1] + j * 16 * kSlice);
  };
  // Fused split: lane l's FP32 fragment of 16-row block i is row
  // 64 w + 16 i + l % 16 of the tile, k 8c .. 8c + 7 (c = l / 16): chunks 2c
  // and 2c + 1 of the row, two 16-byte reads (bits 0, 1 and 3 of the row are
  // those of l, so the swap is the elementwise kernel's).
  int af_off[2];
  const int af_swap = ((lane & 3) << 1) | ((lane >> 3) & 1);
#pragma unroll
  for (int h = 0; h < 2; ++h)
    af_off[h] = ((lane & 15) * 8 + ((2 * (lane >> 4) + h) ^ af_swap)) * 16;
  auto rd_af = [&](int t, int i, int h) -> floatx4 {
    const char* base = reinterpret_cast<const char*>(lds) + (t & 1) * kTwASlot * 2;
    return *reinterpret_cast<const floatx4*>(base + (64 * w + 16 * i) * 128 + af_off[h]);
  };
  const float s_sgpr = __builtin_bit_cast(
      float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, s)));
  // Instruction k (0-19) of the split of one 16-row block's eight values f
  // (f[0]: k 8c .. 8c+3, f[1]: 8c+4 .. 8c+7) into the A_hi and A_lo
  // fragments h, l, in the order that finishes with f[0] first: the high
  // words of pairs 0-1, their residuals and scaled residual words (k 2-9),
  // then the same for pairs 2-3 (k 10-19).
  auto split_k = [&](auto Kc, half8& h, half8& l, const floatx4 (&f)[2], float (&r)[2][2]) {
    constexpr int k = decltype(Kc)::value;
    constexpr int grp = k / 10, kk = k % 10;  // pairs 2 grp, 2 grp + 1
    constexpr int pair = 2 * grp + (kk < 2 ? kk : ((kk - 2) % 4) / 2);
    constexpr int op = kk < 2 ? 0 : ((kk - 2) < 4 ? 1 + (kk - 2) % 2 : 3 + (kk - 2) % 2);
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    u32x4 hv = __builtin_bit_cast(u32x4, h), lv = __builtin_bit_cast(u32x4, l);
    uint32_t hw = hv[pair], lw = lv[pair];
    const float a0 = f[pair / 2][2 * (pair % 2)], a1 = f[pair / 2][2 * (pair % 2) + 1];
    split_op<op>(hw, lw, r[pair % 2], a0, a1, s_sgpr);
    if constexpr (op == 0) {
      hv[pair] = hw;
      h = __builtin_bit_cast(half8, hv);
    }
    if constexpr (op >= 3) {
      lv[pair] = lw;
      l = __builtin_bit_cast(half8, lv);
    }
  };

  // Fused split of B: thread t splits column bn = t % 128 of the tile, k
  // 16 bs .. 16 bs + 15 of a stage (bs = t / 128: slice bs of the stage),
  // as two chunks of eight k.  Chunk ch: bsplit_read loads its eight FP32
  // values from the stage's FP32 slot (k-row r at byte 512 r, column bn at
  // 4 bn; the 64 lanes of a wave read 64 consecutive words), bsplit_op<q> is
  // instruction q (0-19) of their split (pair q / 5, step q % 5 of
  // split_op), and bsplit_write stores the four high words and the four
  // scaled residual words as chunk ch of row bn of the slice's plane tiles,
  // at chunk position ch ^ tile_swizzle(bn), as the split kernel of B lays
  // them out.
  const int bn = threadIdx.x & (kTwN - 1), bs = threadIdx.x >> 7;
  float bfv[8], brr[2];
  uint32_t bhw[4], blw[4];
  auto bsplit_read = [&](int t, int ch) {
    const float* src = reinterpret_cast<const float*>(reinterpret_cast<const char*>(lds) +
                                                      kBfBase + (t & 1) * kTwBfSlotBytes);
#pragma unroll
    for (int e = 0; e < 8; ++e) bfv[e] = src[(16 * bs + 8 * ch + e) * kTwN + bn];
  };
  auto bsplit_op = [&](auto Qc) {
    constexpr int q = decltype(Qc)::value, pr = q / 5, op = q % 5;
    split_op<op>(bhw[pr], blw[pr], brr, bfv[2 * pr], bfv[2 * pr + 1], s_sgpr);
  };
  auto bsplit_write = [&](int t, int ch) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const int off = kBBase + (t & 1) * kTwBSlot + bs * kTileHalves + bn * kSlice +
                    ((ch ^ tile_swizzle(bn)) << 3);
    *reinterpret_cast<u32x4*>(lds + off) = u32x4{bhw[0], bhw[1], bhw[2], bhw[3]};
    *reinterpret_cast<u32x4*>(lds + off + kBPlane) = u32x4{blw[0], blw[1], blw[2], blw[3]};
  };

  // Termwise: hh, xa, xb.  Block folds: acc (= hh) and the block sums t1, t2
  // of the current and the previous column block (index: block parity).
  floatx4 hh[kRows][kCols], xa[kFold ? 1 : kRows][kFold ? 1 : kCols],
      xb[kFold ? 1 : kRows][kFold ? 1 : kCols], t1[2][kRows], t2[2][kRows];
#pragma unroll
  for (int i = 0; i < kRows; ++i) {
#pragma unroll
    for (int j = 0; j < kCols; ++j) hh[i][j] = floatx4{};
    t1[0][i] = t1[1][i] = t2[0][i] = t2[1][i] = floatx4{};
  }
  if constexpr (!kFold) {
#pragma unroll
    for (int i = 0; i < kRows; ++i)
#pragma unroll
      for (int j = 0; j < kCols; ++j) xa[i][j] = xb[i][j] = floatx4{};
  }

  if constexpr (kFusedA) {
    static_for<8>([&](auto n) { dma_af(0, decltype(n)::value); });
    static_for<8>([&](auto n) { dma_af(1, decltype(n)::value); });
  } else {
    static_for<8>([&](auto n) { dma_a(0, decltype(n)::value); });
    static_for<8>([&](auto n) { dma_a(1, decltype(n)::value); });
  }
  if constexpr (kFusedB) {
    // FP32 B stages 0 and 1; stage 0 is split here, stage 1 during step 0.
    static_for<4>([&](auto n) { dma_bf(0, decltype(n)::value); });
    static_for<4>([&](auto n) { dma_bf(1, decltype(n)::value); });
    wait_vmcnt<0>();
    lds_barrier();
#pragma unroll
    for (int ch = 0; ch < 2; ++ch) {
      bsplit_read(0, ch);
      static_for<20>([&](auto q) { bsplit_op(q); });
      bsplit_write(0, ch);
    }
  } else {
    static_for<4>([&](auto n) { dma_b(0, decltype(n)::value); });
  }
  wait_vmcnt<0>();
  lds_barrier();
  half8 AH[kRows], AL[kRows], NH[kRows], NL[kRows], bh[2], bl[2], bsh[2];
  // kCrossScaled: bsh holds s B_hi of a column block (parity-indexed as bh),
  // formed from (s, s) as a packed FP16 pair, wave-uniform.
  const uint16_t s_bits = __builtin_bit_cast(uint16_t, static_cast<_Float16>(s));
  const uint32_t s2 = static_cast<uint32_t>(
      __builtin_amdgcn_readfirstlane(static_cast<int>(s_bits * 0x10001u)));
  // Fused split: F holds the FP32 fragment of one 16-row block from its reads
  // to the last split instruction that uses it; rr the residuals of two pairs.
  floatx4 F[2];
  float rr[2][2];
  if constexpr (kFusedA) {
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
      AH[i] = AL[i] = NH[i] = NL[i] = half8{};
      F[0] = rd_af(0, i, 0);
      F[1] = rd_af(0, i, 1);
      static_for<20>([&](auto Kc) { split_k(Kc, AH[i], AL[i], F, rr); });
    }
  } else {
#pragma unroll
    for (int i = 0; i < kRows; ++i) {
      AH[i] = rd_a(0, 0, i);
      AL[i] = rd_a(0, 1, i);
    }
  }
  bh[0] = rd_b(0, 0, 0);
  bl[0] = rd_b(0, 1, 0);
  if constexpr (V == kCrossScaled) bsh[0] = pk_scale(bh[0], s2);
  lds_barrier();  // A slot 0 is refilled (stage 2) during step 0

  // The fold of column block jp (block sums of parity cp) in two halves, for
  // rows and elements q = 4 i + e in [q0, q1):
  //   elementwise   first  acc = fl(acc + XA_g / s)       (acc holds acc + HH_g)
  //                 second acc = fl(acc + XB_g / s)
  //   cross-first   first  HH_g <- fl(X_g / s + HH_g)
  //                 second acc = fl(acc + HH_g)
  //   cross-scaled  second s acc = fl(s acc + T_g), T_g = fl(X_g + s HH_g)
  //                 (first: nothing)
  // One v_fma_f32 or v_add_f32 per element and half (1/s is exact).
  auto fold_first = [&](int jp, int cp, int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      const int i = q >> 2, e = q & 3;
      if constexpr (V == kElementwise)
        hh[i][jp][e] = __builtin_fmaf(t1[cp][i][e], inv_s, hh[i][jp][e]);
      else
        t2[cp][i][e] = __builtin_fmaf(t1[cp][i][e], inv_s, t2[cp][i][e]);
    }
  };
  auto fold_second = [&](int jp, int cp, int q0, int q1) {
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      const int i = q >> 2, e = q & 3;
      if constexpr (V == kElementwise)
        hh[i][jp][e] = __builtin_fmaf(t2[cp][i][e], inv_s, hh[i][jp][e]);
      else if constexpr (V == kCrossScaled)
        hh[i][jp][e] += t1[cp][i][e];
      else
        hh[i][jp][e] += t2[cp][i][e];
    }
  };

  // Column block j issues its 12 MFMAs: termwise HH(., j), XA(., j),
  // XB(., j); elementwise HH into acc, XA_g, XB_g; cross-first HH_g, XA_g,
  // then XB_g chained onto XA_g.  After MFMA m of a block: m = 1, 7 of blocks
  // 2-6 read the next A fragments, m = 2, 6, 10 of blocks 0-3 issue the DMAs
  // (the 4 of B first), and in the block-fold orders MFMAs 3-11 are each
  // followed by 1-2 of the 16 folds of the previous column block.  DMAs
  // complete in issue order, so a vmcnt wait retires all but the newest.
  constexpr int kDmaPerBlock = 3, kBDmas = 4, kADmas = 8;
  // The block before which A stage kt+1 (copied during step kt-1) is waited
  // for: block 2, or block 1 with the fused split, whose reads of that stage
  // then start one block earlier and leave room for one split instruction per
  // MFMA.
  constexpr int kAWaitBlock = kFusedA ? 1 : 2;
  static_assert(kBDmas + kADmas == 4 * kDmaPerBlock && kBDmas <= 2 * kDmaPerBlock,
                "the B DMAs of a step are issued in blocks 0-1, before its A DMAs");
  auto step = [&](int kt, half8 (&ah)[kRows], half8 (&al)[kRows], half8 (&nh)[kRows],
                  half8 (&nl)[kRows]) {
    static_for<kCols>([&](auto J) {
      constexpr int j = decltype(J)::value, c = j & 1;
      constexpr int jp = (j + kCols - 1) % kCols;  // the block folded now
      if constexpr (j == kAWaitBlock) {
        // All but the DMAs of this step's blocks before it: A stage kt+1 is in.
        wait_vmcnt<kAWaitBlock * kDmaPerBlock>();
        lds_barrier();
      }
      if constexpr (j == kCols - 1) {
        // All but this step's A DMAs: B stage kt+1 is in.  With the fused
        // split of B the barrier publishes the split's writes of that stage
        // instead, and every DMA of the step is for stage kt+2.
        if constexpr (!kFusedB) wait_vmcnt<kADmas>();
        lds_barrier();
        bh[c ^ 1] = rd_b(kt + 1, 0, 0);
        bl[c ^ 1] = rd_b(kt + 1, 1, 0);
      } else {
        bh[c ^ 1] = rd_b(kt, 0, j + 1);
        bl[c ^ 1] = rd_b(kt, 1, j + 1);
      }
      SCHED_FENCE();
      // A fragments rb .. re-1 of the 8 (A_hi blocks 0-3, then A_lo), read in
      // blocks 2-6.
      constexpr int rb = j < 2 ? 0 : (8 * (j - 2) + 4) / 5;
      constexpr int re = j < 2 ? 0 : (8 * (j - 1) + 4) / 5;
      static_for<3 * kRows>([&](auto Mc) {
        constexpr int m = decltype(Mc)::value, g = m / kRows, i = m % kRows;
        if constexpr (V == kTermwise) {
          if constexpr (g == 0)
            mfma16_acc(hh[i][j], ah[i], bh[c]);
          else if constexpr (g == 1)
            mfma16_acc(xa[i][j], al[i], bh[c]);
          else
            mfma16_vacc(xb[i][j], ah[i], bl[c]);
        } else if constexpr (V == kElementwise) {
          if constexpr (g == 0)
            mfma16_va_acc(hh[i][j], ah[i], bh[c]);
          else if constexpr (g == 1)
            mfma16_va_new(t1[c][i], al[i], bh[c]);
          else
            mfma16_va_new(t2[c][i], ah[i], bl[c]);
        } else if constexpr (V == kCrossScaled) {
          if constexpr (g == 0)
            mfma16_va_new(t1[c][i], al[i], bh[c]);
          else if constexpr (g == 1)
            mfma16_va_acc(t1[c][i], ah[i], bl[c]);
          else
            mfma16_va_acc(t1[c][i], ah[i], bsh[c]);
        } else {
          if constexpr (g == 0)
            mfma16_va_new(t2[c][i], ah[i], bh[c]);
          else if constexpr (g == 1)
            mfma16_va_new(t1[c][i], al[i], bh[c]);
          else
            mfma16_va_acc(t1[c][i], ah[i], bl[c]);
        }
        SCHED_FENCE();
        // Folds: at most three VALU operations after any MFMA (up to two
        // overlap an MFMA for free; each further one costs its issue time).
        // Every block sum is read at least 8 MFMAs after the MFMA that wrote
        // it, and before the MFMA of a later block that overwrites it.
        if constexpr (V == kElementwise) {
          // Block jp: XA_g of row i written by its MFMA 4 + i, XB_g by 8 + i,
          // so the first half of row i may run after MFMA m >= i here and
          // the second after m >= 4 + i.  Both halves of the 16 elements:
          // 3,3,3,3,2,2 per MFMA over MFMAs 0-5, then 2,2,3,3,3,3 over 6-11.
          constexpr int f1[7] = {0, 3, 6, 9, 12, 14, 16};
          constexpr int f2[7] = {0, 2, 4, 7, 10, 13, 16};
          if constexpr (m < 6) fold_first(jp, c ^ 1, f1[m], f1[m + 1]);
          else fold_second(jp, c ^ 1, f2[m - 6], f2[m - 5]);
        } else if constexpr (V == kCrossFirst) {
          // Block jp: X_g of row i complete after its MFMA 8 + i, HH_g after
          // MFMA i, so the first half of row i may run after m >= 4 + i.  The
          // second half of rows 2-3 spills into the next block's MFMAs 0-2:
          // that block (parity cp) overwrites HH_g of row i with its MFMA i.
          constexpr int f1[7] = {0, 3, 6, 9, 12, 15, 16};  // after MFMAs 4-9
          constexpr int f2[6] = {0, 2, 5, 8, 11, 14};      // after MFMAs 9-11, next 0-1
          if constexpr (m >= 4 && m <= 9) fold_first(jp, c ^ 1, f1[m - 4], f1[m - 3]);
          if constexpr (m >= 9) fold_second(jp, c ^ 1, f2[m - 9], f2[m - 8]);
          // The spill of block j - 2 (the same parity as this block).
          constexpr int jpp = (j + kCols - 2) % kCols;
          if constexpr (m == 0) fold_second(jpp, c, 8, 11);
          if constexpr (m == 1) fold_second(jpp, c, 11, 14);
          if constexpr (m == 2) fold_second(jpp, c, 14, 16);
        } else if constexpr (V == kCrossScaled) {
          // Block jp: T_g of row i is complete after its MFMA 8 + i, so its
          // fold may run after m >= 4 + i: rows 0-2 fold two elements after
          // each of MFMAs 4-9, and row 3 spills into the next block's MFMAs
          // 0-1 (that block, of parity cp, overwrites T_g of row 3 with its
          // MFMA 3).  s B_hi of the next block: two v_pk_mul_f16 after each
          // of MFMAs 10 and 11, 9 MFMAs ahead of its first use.
          if constexpr (m >= 4 && m <= 9) fold_second(jp, c ^ 1, 2 * (m - 4), 2 * (m - 3));
          constexpr int jpp = (j + kCols - 2) % kCols;
          if constexpr (m <= 1) fold_second(jpp, c, 12 + 2 * m, 14 + 2 * m);
          if constexpr (m == 10) pk_scale_half<0>(bsh[c ^ 1], bh[c ^ 1], s2);
          if constexpr (m == 11) pk_scale_half<1>(bsh[c ^ 1], bh[c ^ 1], s2);
        }
        if constexpr (kFusedA) {
          // Slot P of the step: the reads of 16-row block r's two FP32
          // halves come after the last use of the previous block's half
          // (F[0] after its instruction 9, F[1] after 19; block 0 right
          // after the barrier before block 1), and each split instruction
          // after the MFMA of its slot.
          constexpr int P = kRows * 3 * j + m;
          constexpr int kFirstRead = kRows * 3 * kAWaitBlock;
          static_for<kRows>([&](auto Rc) {
            constexpr int r = decltype(Rc)::value;
            constexpr int f0 = r == 0 ? kFirstRead : tw_split_slot(20 * (r - 1) + 9) + 1;
            constexpr int f1 = r == 0 ? kFirstRead + 1 : tw_split_slot(20 * (r - 1) + 19) + 1;
            static_assert(f0 >= kFirstRead && f1 >= kFirstRead && f1 < kRows * 3 * (kCols - 1) &&
                              f0 < tw_split_slot(20 * r) && f1 < tw_split_slot(20 * r + 10),
                          "fragment reads after the barrier of block 1, before that of block 7");
            if constexpr (P == f0) F[0] = rd_af(kt + 1, r, 0);
            if constexpr (P == f1) F[1] = rd_af(kt + 1, r, 1);
          });
          static_for<80>([&](auto Qc) {
            constexpr int q = decltype(Qc)::value;
            if constexpr (tw_split_slot(q) == P)
              split_k(std::integral_constant<int, q % 20>{}, nh[q / 20], nl[q / 20], F, rr);
          });
        } else if constexpr (j < kCols - 1 && (m == 1 || m == 7)) {
          constexpr int r = rb + m / 6;
          if constexpr (r < re) {
            if constexpr (r < kRows)
              nh[r] = rd_a(kt + 1, 0, r);
            else
              nl[r - kRows] = rd_a(kt + 1, 1, r - kRows);
          }
        }
        if constexpr (kFusedB) {
          // Split of B stage kt+1 (landed at the barrier of block
          // kAWaitBlock <= 2) into its plane slot, in slots 24-81 (blocks
          // 2-6): chunk ch reads at slot 24 + 29 ch, issues one instruction
          // per slot from eight slots later (the reads' latency, so the
          // wave does not stall on them), and writes after the last.
          constexpr int P = kRows * 3 * j + m;
          static_assert(kRows * 3 * 2 >= kRows * 3 * kAWaitBlock &&
                            kRows * 3 * 2 + 29 + 28 < kRows * 3 * (kCols - 1),
                        "the split of B runs between the barriers of blocks 2 and 7");
          static_for<2>([&](auto Ch) {
            constexpr int ch = decltype(Ch)::value, P0 = kRows * 3 * 2 + 29 * ch;
            if constexpr (P == P0) bsplit_read(kt + 1, ch);
            if constexpr (P >= P0 + 8 && P < P0 + 28)
              bsplit_op(std::integral_constant<int, P - P0 - 8>{});
            if constexpr (P == P0 + 28) bsplit_write(kt + 1, ch);
          });
        }
        if constexpr (j < 4 && m % 4 == 2) dma(kt, kDmaPerBlock * j + m / 4);
        SCHED_FENCE();
      });
    });
  };
  for (int kt = 0; kt < ksteps; kt += 2) {
    step(kt, AH, AL, NH, NL);
    step(kt + 1, NH, NL, AH, AL);
  }
  wait_vmcnt<0>();
  mfma_drain();
  if constexpr (V == kElementwise) {
    fold_first(kCols - 1, 1, 0, 4 * kRows);
    fold_second(kCols - 1, 1, 0, 4 * kRows);
  } else if constexpr (V == kCrossFirst) {
    fold_second(kCols - 2, 0, 8, 4 * kRows);  // the spill of block 6
    fold_first(kCols - 1, 1, 0, 4 * kRows);
    fold_second(kCols - 1, 1, 0, 4 * kRows);
  } else if constexpr (V == kCrossScaled) {
    fold_second(kCols - 2, 0, 12, 4 * kRows);  // the spill of block 6 (row 3)
    fold_second(kCols - 1, 1, 0, 4 * kRows);
  }

  const int col0 = tn * kTwN + (lane & 15);
  const int row0 = tm * kTwM + w * 64 + (lane >> 4) * 4;
  const bool full = (tm + 1) * kTwM <= M && (tn + 1) * kTwN <= N;
  store_tile16<kRows, kCols>(C, ldc, M, N, row0, col0, full, [&](int i, int j, int r) {
    if constexpr (V == kCrossScaled) {
      return hh[i][j][r] * inv_s;
    } else if constexpr (kFold) {
      return hh[i][j][r];
    } else {
      return __builtin_fmaf(xb[i][j][r], inv_s, __builtin_fmaf(xa[i][j][r], inv_s, hh[i][j][r]));
    }
  });
}

template <bool kPrefetch, bool kFusedA>
hipError_t launch_el(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc, float s,
                     hipStream_t stream, const float* A = nullptr, int64_t lda = 0,
                     int64_t K = 0) {
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_el_kernel<kPrefetch, kFusedA>, kElLdsBytes, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kWide);
  const int tiles_n = static_cast<int>(p.Np / kWide);
  hipLaunchKernelGGL((gemm_el_kernel<kPrefetch, kFusedA>), dim3(tiles_m * tiles_n),
                     dim3(kWideThreads), kElLdsBytes, stream, p.a_hi, p.a_lo, p.b_hi, p.b_lo,
                     p.range, static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc,
                     static_cast<int>(M), static_cast<int>(N), s, 1.0f / s, A, lda,
                     static_cast<int>(K));
  return hipGetLastError();
}

hipError_t launch_hi(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                     hipStream_t stream) {
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_hi_kernel, kHiLdsBytes, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kWide);
  const int tiles_n = static_cast<int>(p.Np / kWide);
  hipLaunchKernelGGL(gemm_hi_kernel, dim3(tiles_m * tiles_n), dim3(kWideThreads), kHiLdsBytes,
                     stream, p.a_hi, p.b_hi, static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc,
                     static_cast<int>(M), static_cast<int>(N));
  return hipGetLastError();
}

template <int V, bool kFusedA = false, bool kFusedB = false>
hipError_t launch_n128(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc, float s,
                       hipStream_t stream, bool unscaled_only = false,
                       const float* A = nullptr, int64_t lda = 0, const float* B = nullptr,
                       int64_t ldb = 0) {
  constexpr size_t kLds = kFusedB ? kTwFusedBLdsBytes : kTwLdsBytes;
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr = set_lds(&gemm_n128_kernel<V, kFusedA, kFusedB>, kLds, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kTwM);
  const int tiles_n = static_cast<int>(p.Np / kTwN);
  hipLaunchKernelGGL((gemm_n128_kernel<V, kFusedA, kFusedB>), dim3(tiles_m * tiles_n),
                     dim3(kWideThreads), kLds, stream, p.a_hi, p.a_lo, p.b_hi, p.b_lo,
                     p.range, static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc,
                     static_cast<int>(M), static_cast<int>(N), 1.0f / s, unscaled_only ? 1 : 0,
                     A, lda, s, B, ldb);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float scale, int variant, hipStream_t stream) {
  switch (variant) {
    case kElementwise: {
      if (!scaled_kernel_ok(scale))
        return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream, true);
      const hipError_t e = launch_el<true, false>(p, M, N, C, ldc, scale, stream);
      if (e != hipSuccess) return e;
      return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream);
    }
    case kTermwise: return launch_n128<kTermwise>(p, M, N, C, ldc, scale, stream);
    case kCrossFirst: {
      if (!scaled_kernel_ok(scale))
        return launch_n128<kCrossFirst>(p, M, N, C, ldc, scale, stream, true);
      const hipError_t e = launch_n128<kCrossScaled>(p, M, N, C, ldc, scale, stream);
      if (e != hipSuccess) return e;
      return launch_n128<kCrossFirst>(p, M, N, C, ldc, scale, stream);
    }
    case kHiOnly: return launch_hi(p, M, N, C, ldc, stream);
    default: return hipErrorInvalidValue;
  }
}

bool fused_split_ok(const float* A, int64_t lda, int64_t K, float scale, int variant) {
  const bool layout = reinterpret_cast<uintptr_t>(A) % 16 == 0 && lda % 4 == 0 &&
                      K % kKPad == 0 && lda < (int64_t{1} << 22);
  if (variant == kElementwise) return layout && scaled_kernel_ok(scale);
  return layout && variant == kTermwise;
}

hipError_t launch_gemm_fused_a(const Planes& p, int64_t M, int64_t N, int64_t K,
                               const float* A, int64_t lda, float* C, int64_t ldc, float scale,
                               int variant, hipStream_t stream) {
  if (!fused_split_ok(A, lda, K, scale, variant)) return hipErrorInvalidValue;
  if (variant == kTermwise)
    return launch_n128<kTermwise, true>(p, M, N, C, ldc, scale, stream, false, A, lda);
  const hipError_t e = launch_el<true, true>(p, M, N, C, ldc, scale, stream, A, lda, K);
  if (e != hipSuccess) return e;
  return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream);
}

bool fused_split_b_ok(const float* B, int64_t ldb, int64_t N, int64_t K) {
  return reinterpret_cast<uintptr_t>(B) % 16 == 0 && ldb % 4 == 0 && N % 4 == 0 &&
         K % kKPad == 0 && ldb < (int64_t{1} << 22);
}

hipError_t launch_gemm_fused_b(const Planes& p, int64_t M, int64_t N, int64_t K,
                               const float* A, int64_t lda, bool split_a_in_gemm,
                               const float* B, int64_t ldb, float* C, int64_t ldc, float scale,
                               hipStream_t stream) {
  if (!fused_split_b_ok(B, ldb, N, K)) return hipErrorInvalidValue;
  if (split_a_in_gemm) {
    if (!fused_split_ok(A, lda, K, scale, kTermwise)) return hipErrorInvalidValue;
    return launch_n128<kTermwise, true, true>(p, M, N, C, ldc, scale, stream, false, A, lda, B,
                                              ldb);
  }
  return launch_n128<kTermwise, false, true>(p, M, N, C, ldc, scale, stream, false, nullptr, 0,
                                             B, ldb);
}

hipError_t launch_gemm_unscaled(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                                float scale, bool only, hipStream_t stream) {
  return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream, only);
}

hipError_t launch_gemm_stages(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                              float scale, int stages, hipStream_t stream) {
  if (stages < 1 || stages > 2) return hipErrorInvalidValue;
  if (!scaled_kernel_ok(scale))
    return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream, true);
  hipError_t e = hipSuccess;
  switch (stages) {
    case 1: e = launch_el<false, false>(p, M, N, C, ldc, scale, stream); break;
    case 2: e = launch_el<true, false>(p, M, N, C, ldc, scale, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  return launch_n128<kElementwise>(p, M, N, C, ldc, scale, stream);
}

}  // namespace sgc
