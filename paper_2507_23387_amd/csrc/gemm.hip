// Three-product MFMA GEMM on prepared FP16 planes (gfx950).
//
// For each 256 x 128 tile of C it computes (Eq. recover_eqn of arXiv
// 2507.23387)
//   HH = A_hi B_hi,  XA = A_lo B_hi,  XB = A_hi B_lo
// with v_mfma_f32_32x32x16_f16 (FP16 x FP16 products are exact; the MFMA sums
// them with its C operand in one fused, once-rounded FP32 operation), and
// reconstructs C in one of three ways:
//   kElementwise (Eq. elementwise, Sec. 4.5): the contraction dimension is cut
//     into blocks g of kBK = 32.  Per block the high-high products go straight
//     into the running FP32 accumulator (its MFMA C operand -- the matrix-unit
//     "C_blk <- A_blk B_blk + C_blk" of Alg. 1), the two cross products go into
//     separate FP32 block sums started from zero, and at the end of the block
//       acc = (acc + XA_g / s) + XB_g / s
//     with two v_fma_f32 (1/s is an exact power of two, so each fma is exactly
//     one rounded FP32 addition).
//   kTermwise (Eq. termwise): three FP32 accumulators over all of K, combined
//     once in the epilogue as C = (HH + XA / s) + XB / s.
//   kHiOnly: C = HH, the native-FP16 GEMM baseline.
//
// Data path.  A planes are Mp x Kp and B planes Np x Kp (B transposed), both
// k-contiguous and zero-padded, so the main loop has no bounds checks.  Each
// k-stage of 32 brings the workgroup's 256 + 128 rows x 32 k of every plane
// (48 KiB) from global memory straight into LDS with global_load_lds_dwordx4
// (no VGPR staging), into a ring of kStages stages, so the loads for stage
// kt+2 are in flight while stage kt feeds the MFMAs (the double buffering of
// Sec. 5.4 taken one step deeper).  Rows are 64 B; their four 16-byte chunks
// are XOR-swizzled by (row >> 2) & 3 so that the MFMA fragment reads (16
// consecutive rows at one chunk per LDS cycle) hit 16 distinct bank groups.
// The loop body is branch-free (past the end it re-loads the last stage into
// the free slot) so the vmcnt waits stay exact, and one s_barrier per stage
// both publishes the landed stage and retires the stage being overwritten.
//
// Workgroup: 512 threads = 8 waves (2 per SIMD) in a 4 x 2 grid; each wave owns
// a 64 x 64 sub-tile = 2 x 2 MFMA tiles of 32 x 32, so 2 waves share each SIMD
// and hide each other's LDS latency.  Accumulators: 64 (hi-only), 192
// (termwise) or 64 + 128 block temporaries (elementwise) registers per lane.
#include "internal.h"

namespace sgc {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kWaves = kThreads / 64;  // 8
constexpr int kWavesM = 4;
constexpr int kWavesN = 2;
constexpr int kWaveM = kBM / kWavesM;  // 64 rows per wave
constexpr int kWaveN = kBN / kWavesN;  // 64 columns per wave
constexpr int kSubM = kWaveM / 32;     // 2 MFMA tiles per wave along M
constexpr int kSubN = kWaveN / 32;     // 2 along N
constexpr int kStages = 3;
constexpr int kChunksPerRow = kBK / 8;  // 16-byte chunks per LDS row (4)
static_assert(kWavesM * kWavesN == kWaves, "wave grid");
static_assert(kKPad % kBK == 0, "whole stages per padded K");

// D(32x32) = A(32x16) B(16x32) + C.  Lane l supplies A row l%32 and B column
// l%32 with the 8 consecutive k values 8*(l/32) .. 8*(l/32)+7 of the 16-wide
// step; D element (row 8*(r/4) + 4*(l/32) + r%4, column l%32) is in register r.
__device__ __forceinline__ floatx16 mfma32(const half8& a, const half8& b, const floatx16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Physical 16-byte chunk of logical chunk c in LDS row `row` (64-byte rows).
__device__ __forceinline__ int swizzle(int row, int c) { return c ^ ((row >> 2) & 3); }

// One 64-lane LDS DMA: lane l copies 16 bytes from g into LDS byte address
// lds_addr + 16 * l.  Issued as inline asm so the compiler does not add its
// own conservative vmcnt(0) waits before every later LDS read; the kernel
// waits explicitly with wait_vmcnt<>() before the barrier that publishes a
// stage.
__device__ __forceinline__ void dma16(const void* g, unsigned lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr)
               : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// This wave's LDS reads are complete, then all waves meet.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Map the hardware workgroup id to a (tile_m, tile_n) pair.  Workgroups are
// dispatched round-robin over the 8 XCDs; renumbering gives each XCD a
// contiguous range of logical tiles, and grouping 8 tile-rows keeps the A
// and B panels a group touches resident in that XCD's L2.
__device__ __forceinline__ void tile_of(int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  int wg = blockIdx.x;
  if ((nwg & 7) == 0) wg = (wg & 7) * (nwg >> 3) + (wg >> 3);
  constexpr int kGroup = 8;
  const int per_group = kGroup * tiles_n;
  const int group = wg / per_group;
  const int first_m = group * kGroup;
  const int gsize = min(tiles_m - first_m, kGroup);
  const int in_group = wg - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

template <int V>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo, int Kp, int tiles_m,
    int tiles_n, float* __restrict__ C, int64_t ldc, int M, int N, float inv_s) {
  // Planes staged per stage: A_hi, B_hi [, A_lo, B_lo].
  constexpr int kPairs = (V == kHiOnly) ? 1 : 2;
  constexpr int kABlocks = kBM * kChunksPerRow / 64;  // 64-chunk DMA blocks per A plane tile
  constexpr int kBBlocks = kBN * kChunksPerRow / 64;
  static_assert(kABlocks % kWaves == 0 && kBBlocks % kWaves == 0, "DMA blocks per wave");
  constexpr int kDmaPerStage = kPairs * (kABlocks + kBBlocks) / kWaves;  // per wave
  constexpr int kAPlane = kBM * kBK;  // halves
  constexpr int kBPlane = kBN * kBK;
  constexpr int kStage = kPairs * (kAPlane + kBPlane);
  constexpr int kOffAH = 0, kOffBH = kAPlane, kOffAL = kAPlane + kBPlane,
                kOffBL = 2 * kAPlane + kBPlane;
  constexpr int kSteps = kBK / 16;  // MFMA k-steps per stage
  extern __shared__ __align__(16) uint16_t lds[];

  int tm, tn;
  tile_of(tiles_m, tiles_n, tm, tn);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / kWavesN;
  const int wn = wave % kWavesN;

  const uint16_t* const ga[2] = {a_hi + static_cast<size_t>(tm) * kBM * Kp,
                                 a_lo + static_cast<size_t>(tm) * kBM * Kp};
  const uint16_t* const gb[2] = {b_hi + static_cast<size_t>(tn) * kBN * Kp,
                                 b_lo + static_cast<size_t>(tn) * kBN * Kp};
  // LDS byte address of the dynamic shared-memory base (the M0 operand of the
  // DMA): cast the generic pointer to the LDS address space, then to int.
  const unsigned lds_base = static_cast<unsigned>(
      (uintptr_t)((__attribute__((address_space(3))) uint16_t*)lds));

  // DMA the k-stage kt into ring slot `slot`.  LDS slot q of a plane tile holds
  // logical chunk swizzle(row, q % 4) of row q / 4; lane l of DMA block b
  // fills slot 64 b + l, so each instruction writes 1 KiB contiguously.
  auto issue = [&](int kt, int slot) {
    const unsigned base = lds_base + slot * kStage * 2;
    const int k0 = kt * kBK;
#pragma unroll
    for (int p = 0; p < kPairs; ++p) {
#pragma unroll
      for (int i = 0; i < kABlocks / kWaves; ++i) {
        const int blk = i * kWaves + wave;
        const int q = blk * 64 + lane;
        const int row = q / kChunksPerRow;
        const int c = swizzle(row, q % kChunksPerRow);
        dma16(ga[p] + static_cast<size_t>(row) * Kp + k0 + c * 8,
              base + ((p ? kOffAL : kOffAH) + blk * 512) * 2);
      }
#pragma unroll
      for (int i = 0; i < kBBlocks / kWaves; ++i) {
        const int blk = i * kWaves + wave;
        const int q = blk * 64 + lane;
        const int row = q / kChunksPerRow;
        const int c = swizzle(row, q % kChunksPerRow);
        dma16(gb[p] + static_cast<size_t>(row) * Kp + k0 + c * 8,
              base + ((p ? kOffBL : kOffBH) + blk * 512) * 2);
      }
    }
  };

  const floatx16 zero = {};
  floatx16 acc[kSubM][kSubN];  // running accumulator (elementwise) or HH
  floatx16 xa[kSubM][kSubN];   // termwise XA, or elementwise block sum XA_g
  floatx16 xb[kSubM][kSubN];   // termwise XB, or elementwise block sum XB_g
#pragma unroll
  for (int i = 0; i < kSubM; ++i)
#pragma unroll
    for (int j = 0; j < kSubN; ++j) acc[i][j] = xa[i][j] = xb[i][j] = zero;

  const int ktiles = Kp / kBK;
#pragma unroll
  for (int s = 0; s < kStages - 1; ++s) issue(min(s, ktiles - 1), s);

  const int frag_row = lane & 31;  // row (A) / column (B) inside a 32 x 32 tile
  const int frag_kc = lane >> 5;   // which 8-wide k chunk of the 16-wide step
  for (int kt = 0; kt < ktiles; ++kt) {
    // Stage kt has landed for this wave once at most the (kStages - 2) later
    // stages' DMAs are outstanding; the barrier makes it so for every wave and
    // guarantees that no wave still reads the slot refilled just below.
    wait_vmcnt<(kStages - 2) * kDmaPerStage>();
    lds_barrier();
    issue(min(kt + kStages - 1, ktiles - 1), (kt + kStages - 1) % kStages);
    const uint16_t* s = lds + (kt % kStages) * kStage;
#pragma unroll
    for (int ks = 0; ks < kSteps; ++ks) {
      const int kc = ks * 2 + frag_kc;
      half8 ah[kSubM], al[kSubM], bh[kSubN], bl[kSubN];
#pragma unroll
      for (int i = 0; i < kSubM; ++i) {
        const int r = wm * kWaveM + i * 32 + frag_row;
        const int o = r * kBK + (swizzle(r, kc) << 3);
        ah[i] = *reinterpret_cast<const half8*>(s + kOffAH + o);
        if constexpr (kPairs == 2) al[i] = *reinterpret_cast<const half8*>(s + kOffAL + o);
      }
#pragma unroll
      for (int j = 0; j < kSubN; ++j) {
        const int r = wn * kWaveN + j * 32 + frag_row;
        const int o = r * kBK + (swizzle(r, kc) << 3);
        bh[j] = *reinterpret_cast<const half8*>(s + kOffBH + o);
        if constexpr (kPairs == 2) bl[j] = *reinterpret_cast<const half8*>(s + kOffBL + o);
      }
#pragma unroll
      for (int i = 0; i < kSubM; ++i)
#pragma unroll
        for (int j = 0; j < kSubN; ++j) {
          acc[i][j] = mfma32(ah[i], bh[j], acc[i][j]);
          if constexpr (V == kTermwise) {
            xa[i][j] = mfma32(al[i], bh[j], xa[i][j]);
            xb[i][j] = mfma32(ah[i], bl[j], xb[i][j]);
          } else if constexpr (V == kElementwise) {
            xa[i][j] = mfma32(al[i], bh[j], ks == 0 ? zero : xa[i][j]);
            xb[i][j] = mfma32(ah[i], bl[j], ks == 0 ? zero : xb[i][j]);
          }
        }
    }
    if constexpr (V == kElementwise) {
      // End of block g: acc = (acc + XA_g / s) + XB_g / s.
#pragma unroll
      for (int i = 0; i < kSubM; ++i)
#pragma unroll
        for (int j = 0; j < kSubN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            acc[i][j][e] = __builtin_fmaf(xa[i][j][e], inv_s, acc[i][j][e]);
            acc[i][j][e] = __builtin_fmaf(xb[i][j][e], inv_s, acc[i][j][e]);
          }
    }
  }
  // No LDS DMA may still be writing when the workgroup retires.
  wait_vmcnt<0>();

  // Epilogue: register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4 and
  // column l%32 of its 32 x 32 tile.
  const int col0 = tn * kBN + wn * kWaveN + (lane & 31);
  const int row0 = tm * kBM + wm * kWaveM + (lane >> 5) * 4;
#pragma unroll
  for (int i = 0; i < kSubM; ++i)
#pragma unroll
    for (int j = 0; j < kSubN; ++j) {
      const int col = col0 + j * 32;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = row0 + i * 32 + (r >> 2) * 8 + (r & 3);
        float v = acc[i][j][r];
        if constexpr (V == kTermwise) {
          v = __builtin_fmaf(xa[i][j][r], inv_s, v);
          v = __builtin_fmaf(xb[i][j][r], inv_s, v);
        }
        if (row < M && col < N) C[static_cast<size_t>(row) * ldc + col] = v;
      }
    }
}

template <int V>
hipError_t launch_variant(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                          float inv_s, hipStream_t stream) {
  constexpr int kPairs = (V == kHiOnly) ? 1 : 2;
  constexpr size_t lds_bytes =
      static_cast<size_t>(kStages) * kPairs * (kBM + kBN) * kBK * sizeof(uint16_t);
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&gemm_kernel<V>),
      hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds_bytes));
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>(p.Mp / kBM);
  const int tiles_n = static_cast<int>(p.Np / kBN);
  hipLaunchKernelGGL(gemm_kernel<V>, dim3(tiles_m * tiles_n), dim3(kThreads), lds_bytes, stream,
                     p.a_hi, p.a_lo, p.b_hi, p.b_lo, static_cast<int>(p.Kp), tiles_m, tiles_n, C,
                     ldc, static_cast<int>(M), static_cast<int>(N), inv_s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                       float inv_scale, int variant, hipStream_t stream) {
  switch (variant) {
    case kElementwise: return launch_variant<kElementwise>(p, M, N, C, ldc, inv_scale, stream);
    case kTermwise: return launch_variant<kTermwise>(p, M, N, C, ldc, inv_scale, stream);
    case kHiOnly: return launch_variant<kHiOnly>(p, M, N, C, ldc, inv_scale, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sgc
