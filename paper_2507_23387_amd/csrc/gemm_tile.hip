// Tile-shape and k-depth sweep of the scaled elementwise GEMM (gfx950), the
// measurement behind sgemm_cube_compute_tile: the analogue on this GPU of
// the block-size study of Sec. 6.3 (which sweeps b_m, b_k, b_n of the
// double-buffered pipeline of Sec. 5.4).
//
// gemm_tile_kernel<kBM, kBN, kBK, kOcc, kWM, kWN> computes a kBM x kBN tile of
// C per workgroup of kWM x kWN waves (each (kBM/kWM) x (kBN/kWN) in 16 x 16
// MFMA tiles), taking kBK of k per pipeline stage, with kOcc workgroups per
// compute unit.  Eight waves put two waves on each SIMD, so one wave's MFMAs
// can run while the other waits on its LDS reads or its DMA issue.
// Its data path is the library's: the tiled planes (internal.h) copied into a
// two-slot LDS ring by LDS DMA, one 4 KiB plane tile per DMA group, and the
// arithmetic is that of gemm_el_kernel: per 32-wide MFMA k-step and 16 x 16
// accumulator the three chained MFMAs A_hi (s B_hi), A_lo B_hi, A_hi B_lo into
// an accumulator holding s * acc, C = acc / s.  Every accumulator therefore
// sees the same MFMAs in the same order as in gemm_el_kernel, whatever the
// tile, and the results are identical bit for bit.
//
// The schedule is generic, one shape of code for every tile: at the start
// of each 32-wide k-step a wave reads the A fragments of its rows, then per
// 16-column block it reads the B fragments of the next block and issues
// that block's MFMAs; the DMAs of the next stage are spread over the first
// half of the column blocks of the stage's first k-step (as in
// gemm_el_kernel: a copy issued late in a stage would not land before the
// stage's barrier), and one barrier per stage publishes it.  The MFMAs are
// the compiler's builtins, so the compiler keeps every hazard.  The
// hand-placed schedule of gemm_el_kernel (A fragments of the next step
// prefetched into a second register set, every LDS read, DMA and VALU
// instruction between two MFMAs) is not reproduced: the sweep measures what
// the tile shape, the stage depth and the number of waves change, on one
// code shape.
#include <atomic>

#include "gemm_common.h"

namespace sgc {
namespace {

constexpr int kTileStep = 2 * kSlice;  // k per MFMA step (32)

template <int kBM, int kBN, int kBK, int kWM = 2, int kWN = 2>
struct TileShape {
  static constexpr int kWaves = kWM * kWN;
  static constexpr int kThreads = 64 * kWaves;
  // A 4 KiB plane tile is four 1 KiB wave DMAs; with eight waves the two
  // groups of four copy one plane each (group 0 the high planes, group 1 the
  // low planes).
  static constexpr int kGroups = kWaves / 4;
  static constexpr int kPlanesPerGroup = 2 / kGroups;
  static constexpr int kPA = kBM / kPanel;             // 128-row panels of A per tile
  static constexpr int kPB = kBN / kPanel;
  static constexpr int kSL = kBK / kSlice;             // plane tiles along k per stage
  static constexpr int kKS = kBK / kTileStep;          // MFMA k-steps per stage
  static constexpr int kWRows = kBM / kWM;            // rows and columns per wave
  static constexpr int kWCols = kBN / kWN;
  static constexpr int kRT = kWRows / 16;              // 16-row blocks per wave
  static constexpr int kCT = kWCols / 16;              // 16-column blocks per wave
  static constexpr int kAPlane = kPA * kSL * kTileHalves;  // halves
  static constexpr int kBPlane = kPB * kSL * kTileHalves;
  static constexpr int kASlot = 2 * kAPlane;           // hi and lo
  static constexpr int kBSlot = 2 * kBPlane;
  static constexpr int kBBase = 2 * kASlot;            // B slots follow the two A slots
  static constexpr int kTiles = 2 * kSL * (kPA + kPB); // plane tiles per stage
  static constexpr int kGroupTiles = kTiles / kGroups; // plane tiles per wave group
  // The next stage's DMAs go out over the first kSpread column blocks of a
  // stage, so the last of them has half a stage to land.
  static constexpr int kSpread = kCT >= 2 ? kCT / 2 : 1;
  static constexpr size_t kLdsBytes = static_cast<size_t>(2) * (kASlot + kBSlot) * 2;
  static_assert(kBM % kPanel == 0 && kBN % kPanel == 0, "tiles are whole 128-row panels");
  static_assert(kWaves == 4 || kWaves == 8, "one or two waves per SIMD");
  static_assert(kWRows % 16 == 0 && kWCols % 16 == 0, "whole MFMA tiles per wave");
  static_assert(kBK % kTileStep == 0 && kKPad % kBK == 0, "stages divide the padded K");
  static_assert(kLdsBytes <= kMaxLdsBytes, "LDS of every kernel stays within 128 KiB");
  // The furthest DMA targets: the last tile of the lo plane of slot 1 of A
  // (before the B slots) and of B (the end of LDS).
  static_assert(dma_end_bytes(kASlot + kAPlane + (kPA * kSL - 1) * kTileHalves) <=
                    static_cast<size_t>(kBBase) * 2, "A DMAs stay in the A slots");
  static_assert(dma_end_bytes(kBBase + kBSlot + kBPlane + (kPB * kSL - 1) * kTileHalves) <=
                    kLdsBytes, "B DMAs stay in LDS");
};

// Halves offset, within one plane of one stage, of this lane's fragment of
// the 16-row block starting at row `r0` (a multiple of 16) of the tile, for
// k-step 0 of the stage: lane l reads row r0 + l%16 and k chunk l/16 of the
// 32-wide step (slice (l/16)/2, chunk (l/16)%2, stored at position
// chunk ^ tile_swizzle(row)).  k-step ks adds 2 ks tiles.
template <int kSL>
__device__ __forceinline__ int tile_frag_offset(int lane, int r0) {
  const int r = r0 + (lane & 15), fc = lane >> 4;
  const int panel = r / kPanel, rp = r % kPanel;
  return (panel * kSL + (fc >> 1)) * kTileHalves + rp * kSlice +
         (((fc & 1) ^ tile_swizzle(rp)) << 3);
}

template <int kBM, int kBN, int kBK, int kOcc, int kWM, int kWN>
__global__ __launch_bounds__(64 * kWM * kWN, kOcc) void gemm_tile_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo,
    const uint32_t* __restrict__ range, int Kp, int tiles_m, int tiles_n,
    float* __restrict__ C, int64_t ldc, int M, int N, float s, float inv_s) {
  using T = TileShape<kBM, kBN, kBK, kWM, kWN>;
  if (range[0] == range[1]) return;  // s B_hi overflows FP16: the unscaled kernel runs
  int tm, tn;
  tile_of<4>(blockIdx.x, tiles_m, tiles_n, tm, tn);
  extern __shared__ __align__(16) uint16_t lds[];

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w / kWN, wn = w % kWN;
  const int64_t slices = Kp / kSlice;
  const int stages = Kp / kBK;
  const int64_t panel_stride = slices * kTileHalves;

  // DMA n (0 .. kGroupTiles-1) of a stage copies plane tile n of the wave's
  // group: the A tiles (plane, panel, slice) first, then the B tiles, the
  // planes being both (four waves) or the group's one (eight waves); wave w
  // copies 1 KiB block w % 4 of every tile of group w / 4.
  const int part = w & 3, group = w >> 2;
  const unsigned lane_off = static_cast<unsigned>(part * 512 + lane * 8) * 2;  // bytes
  const unsigned lds_base = lds_address(lds) + part * 1024;
  auto dma = [&](int t, int n) {
    constexpr int kA = T::kPlanesPerGroup * T::kPA * T::kSL;
    const bool is_a = n < kA;
    const int m = is_a ? n : n - kA;
    const int per_plane = (is_a ? T::kPA : T::kPB) * T::kSL;
    const int p = m / per_plane + group, rem = m % per_plane, ph = rem / T::kSL,
              sl = rem % T::kSL;
    const uint16_t* plane = is_a ? (p ? a_lo : a_hi) : (p ? b_lo : b_hi);
    const int first_panel = is_a ? tm * T::kPA : tn * T::kPB;
    const uint16_t* src = plane + static_cast<int64_t>(first_panel + ph) * panel_stride +
                          static_cast<int64_t>(t * T::kSL + sl) * kTileHalves;
    const int dst = (is_a ? 0 : T::kBBase) + (t & 1) * (is_a ? T::kASlot : T::kBSlot) +
                    p * (is_a ? T::kAPlane : T::kBPlane) + (ph * T::kSL + sl) * kTileHalves;
    dma16s(src, lane_off, lds_base + static_cast<unsigned>(dst) * 2);
  };

  int a_off[T::kRT], b_off[T::kCT];
#pragma unroll
  for (int i = 0; i < T::kRT; ++i) a_off[i] = tile_frag_offset<T::kSL>(lane, wm * T::kWRows + 16 * i);
#pragma unroll
  for (int j = 0; j < T::kCT; ++j) b_off[j] = tile_frag_offset<T::kSL>(lane, wn * T::kWCols + 16 * j);
  auto rd_a = [&](int t, int p, int i, int ks) -> half8 {
    return *reinterpret_cast<const half8*>(lds + (t & 1) * T::kASlot + p * T::kAPlane + a_off[i] +
                                           2 * ks * kTileHalves);
  };
  auto rd_b = [&](int t, int p, int j, int ks) -> half8 {
    return *reinterpret_cast<const half8*>(lds + T::kBBase + (t & 1) * T::kBSlot +
                                           p * T::kBPlane + b_off[j] + 2 * ks * kTileHalves);
  };
  // s as eight FP16 values: s B_hi is exact (s a power of two <= 2^15 and
  // |B_hi| s <= 65504, both checked before this kernel runs).
  const _Float16 s16 = static_cast<_Float16>(s);
  const half8 s8 = {s16, s16, s16, s16, s16, s16, s16, s16};

  floatx4 acc[T::kRT][T::kCT];
#pragma unroll
  for (int i = 0; i < T::kRT; ++i)
#pragma unroll
    for (int j = 0; j < T::kCT; ++j) acc[i][j] = floatx4{};

  static_for<T::kGroupTiles>([&](auto n) { dma(0, decltype(n)::value); });
  wait_vmcnt<0>();
  lds_barrier();

  for (int t = 0; t < stages; ++t) {
    const bool more = t + 1 < stages;
    static_for<T::kKS>([&](auto KSc) {
      constexpr int ks = decltype(KSc)::value;
      half8 ah[T::kRT], al[T::kRT], bh[2], bl[2], bs[2];
#pragma unroll
      for (int i = 0; i < T::kRT; ++i) {
        ah[i] = rd_a(t, 0, i, ks);
        al[i] = rd_a(t, 1, i, ks);
      }
      bh[0] = rd_b(t, 0, 0, ks);
      bl[0] = rd_b(t, 1, 0, ks);
      bs[0] = bh[0] * s8;
      static_for<T::kCT>([&](auto J) {
        constexpr int j = decltype(J)::value, c = j & 1;
        if constexpr (j + 1 < T::kCT) {
          bh[c ^ 1] = rd_b(t, 0, j + 1, ks);
          bl[c ^ 1] = rd_b(t, 1, j + 1, ks);
          bs[c ^ 1] = bh[c ^ 1] * s8;
        }
        if constexpr (ks == 0) {
          // DMAs [j kGroupTiles / kSpread, (j + 1) kGroupTiles / kSpread) of
          // stage t + 1.
          if constexpr (j < T::kSpread) {
            constexpr int d0 = j * T::kGroupTiles / T::kSpread;
            constexpr int d1 = (j + 1) * T::kGroupTiles / T::kSpread;
            if (more) static_for<d1 - d0>([&](auto d) { dma(t + 1, d0 + decltype(d)::value); });
          }
        }
        SCHED_FENCE();
#pragma unroll
        for (int i = 0; i < T::kRT; ++i) acc[i][j] = mfma16(ah[i], bs[c], acc[i][j]);
#pragma unroll
        for (int i = 0; i < T::kRT; ++i) acc[i][j] = mfma16(al[i], bh[c], acc[i][j]);
#pragma unroll
        for (int i = 0; i < T::kRT; ++i) acc[i][j] = mfma16(ah[i], bl[c], acc[i][j]);
        SCHED_FENCE();
      });
    });
    // Stage t + 1 has landed and every wave is done with stage t's slots.
    wait_vmcnt<0>();
    lds_barrier();
  }

  const int col0 = tn * kBN + wn * T::kWCols + (lane & 15);
  const int row0 = tm * kBM + wm * T::kWRows + (lane >> 4) * 4;
  const bool full = (tm + 1) * kBM <= M && (tn + 1) * kBN <= N;
  store_tile16<T::kRT, T::kCT>(C, ldc, M, N, row0, col0, full,
                               [&](int i, int j, int r) { return acc[i][j][r] * inv_s; });
}

template <int kBM, int kBN, int kBK, int kOcc, int kWM = 2, int kWN = 2>
hipError_t launch_tile(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc, float s,
                       hipStream_t stream) {
  using T = TileShape<kBM, kBN, kBK, kWM, kWN>;
  static std::atomic<bool> done[kMaxDevices];
  const hipError_t attr =
      set_lds(&gemm_tile_kernel<kBM, kBN, kBK, kOcc, kWM, kWN>, T::kLdsBytes, done);
  if (attr != hipSuccess) return attr;
  const int tiles_m = static_cast<int>((M + kBM - 1) / kBM);
  const int tiles_n = static_cast<int>((N + kBN - 1) / kBN);
  hipLaunchKernelGGL((gemm_tile_kernel<kBM, kBN, kBK, kOcc, kWM, kWN>), dim3(tiles_m * tiles_n),
                     dim3(T::kThreads), T::kLdsBytes, stream, p.a_hi, p.a_lo, p.b_hi, p.b_lo,
                     p.range, static_cast<int>(p.Kp), tiles_m, tiles_n, C, ldc,
                     static_cast<int>(M), static_cast<int>(N), s, 1.0f / s);
  return hipGetLastError();
}

}  // namespace

bool tile_config_ok(int tile_m, int tile_n, int block_k, int waves) {
  if (waves == 8) return tile_m == 256 && tile_n == 256 && block_k == 32;
  return waves == 4 && ((tile_m == 256 && tile_n == 256 && block_k == 32) ||
                        (tile_m == 256 && tile_n == 128 && block_k == 32) ||
                        (tile_m == 128 && tile_n == 256 && block_k == 32) ||
                        (tile_m == 128 && tile_n == 128 && block_k == 32) ||
                        (tile_m == 128 && tile_n == 128 && block_k == 64));
}

hipError_t launch_gemm_tile(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                            float scale, int tile_m, int tile_n, int block_k, int waves,
                            hipStream_t stream) {
  if (!tile_config_ok(tile_m, tile_n, block_k, waves)) return hipErrorInvalidValue;
  if (!scaled_kernel_ok(scale)) return launch_gemm_unscaled(p, M, N, C, ldc, scale, true, stream);
  hipError_t e = hipSuccess;
  if (waves == 8)
    e = launch_tile<256, 256, 32, 1, 2, 4>(p, M, N, C, ldc, scale, stream);
  else if (tile_m == 256 && tile_n == 256)
    e = launch_tile<256, 256, 32, 1>(p, M, N, C, ldc, scale, stream);
  else if (tile_m == 256)
    e = launch_tile<256, 128, 32, 1>(p, M, N, C, ldc, scale, stream);
  else if (tile_n == 256)
    e = launch_tile<128, 256, 32, 1>(p, M, N, C, ldc, scale, stream);
  else if (block_k == 32)
    e = launch_tile<128, 128, 32, 2>(p, M, N, C, ldc, scale, stream);
  else
    e = launch_tile<128, 128, 64, 1>(p, M, N, C, ldc, scale, stream);
  if (e != hipSuccess) return e;
  return launch_gemm_unscaled(p, M, N, C, ldc, scale, false, stream);
}

}  // namespace sgc
