// Three-product MFMA GEMM on prepared FP16 planes (gfx950).
//
// Computes, for each 128 x 128 tile of C (Eq. recover_eqn of arXiv
// 2507.23387):
//   HH = A_hi B_hi,  XA = A_lo B_hi,  XB = A_hi B_lo
// with v_mfma_f32_16x16x32_f16 (FP16 x FP16 products are exact in FP32 and
// are accumulated in FP32), and reconstructs C in one of three ways:
//   kElementwise (Eq. elementwise, Sec. 4.5): the contraction dimension is cut
//     into blocks g of kBK = 64.  Per block, the high-high products are
//     accumulated straight into the running FP32 accumulator (the MFMA's
//     C operand, as the matrix unit does "C_blk <- A_blk B_blk + C_blk" in
//     Alg. 1), the two cross products of the block are accumulated in
//     separate FP32 temporaries from zero, and then folded in order:
//       acc = (acc + XA_g / s) + XB_g / s.
//     Division by s is multiplication by the power of two 1/s, exact, so each
//     fold is one rounded FP32 addition (one v_fma_f32).
//   kTermwise (Eq. termwise): three FP32 accumulators over all of K, combined
//     once in the epilogue as C = (HH + XA / s) + XB / s.
//   kHiOnly: C = HH, the native-FP16 GEMM baseline.
//
// Layout: A planes are Mp x Kp and B planes Np x Kp (B transposed), both
// k-contiguous, zero-padded to the tile multiples, so the main loop has no
// bounds checks.  Per stage, each of the (2 or 4) plane tiles is 128 rows x
// 64 k of FP16 = 16 KiB in LDS, rows of 128 bytes whose 16-byte chunks are
// XOR-swizzled by (row & 7) so that both the 16-byte stores and the MFMA
// fragment reads (8 consecutive k of 16 consecutive rows) are bank-conflict
// free.  Two stages: the next k-tile's global loads are in flight in
// registers while the current stage feeds the MFMAs (double buffering,
// Sec. 5.4), one barrier per k-tile.
//
// Workgroup: 256 threads = 4 waves in a 2 x 2 grid; each wave owns a 64 x 64
// sub-tile = 4 x 4 MFMA tiles of 16 x 16.
#include "internal.h"

namespace sgc {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kTileHalves = kBM * kBK;  // halves per plane tile per stage

__device__ __forceinline__ floatx4 mfma16(const half8& a, const half8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
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

// Global -> registers: the 128 x 64 k-tile kt of each plane, 16 B per chunk,
// 4 chunks per thread per plane (chunk c: row c / 8, k-chunk c % 8).
template <int NP>
__device__ __forceinline__ void global_load(const uint16_t* const (&src)[4], int Kp, int kt,
                                            int t, u32x4 (&stg)[NP][4]) {
  const int k0 = kt * kBK;
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = i * kThreads + t;
      const int row = c >> 3;
      const int kc = c & 7;
      stg[p][i] = *reinterpret_cast<const u32x4*>(src[p] + static_cast<size_t>(row) * Kp + k0 +
                                                  kc * 8);
    }
}

// Registers -> LDS stage, 16-byte chunks XOR-swizzled by (row & 7).
template <int NP>
__device__ __forceinline__ void lds_store(uint16_t* lds, int stage, int t,
                                          const u32x4 (&stg)[NP][4]) {
  uint16_t* base = lds + stage * NP * kTileHalves;
#pragma unroll
  for (int p = 0; p < NP; ++p)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = i * kThreads + t;
      const int row = c >> 3;
      const int kc = c & 7;
      *reinterpret_cast<u32x4*>(base + p * kTileHalves + row * kBK + ((kc ^ (row & 7)) << 3)) =
          stg[p][i];
    }
}

template <int V>
__global__ __launch_bounds__(kThreads, 1) void gemm_kernel(
    const uint16_t* __restrict__ a_hi, const uint16_t* __restrict__ a_lo,
    const uint16_t* __restrict__ b_hi, const uint16_t* __restrict__ b_lo, int Kp, int tiles_m,
    int tiles_n, float* __restrict__ C, int64_t ldc, int M, int N, float inv_s) {
  constexpr int NP = (V == kHiOnly) ? 2 : 4;  // staged planes: a_hi, b_hi[, a_lo, b_lo]
  extern __shared__ __align__(16) uint16_t lds[];

  int tm, tn;
  tile_of(tiles_m, tiles_n, tm, tn);
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  const int wm = wave >> 1;
  const int wn = wave & 1;

  const size_t a_off = static_cast<size_t>(tm) * kBM * Kp;
  const size_t b_off = static_cast<size_t>(tn) * kBN * Kp;
  const uint16_t* const gsrc[4] = {a_hi + a_off, b_hi + b_off, (NP == 4) ? a_lo + a_off : nullptr,
                             (NP == 4) ? b_lo + b_off : nullptr};

  // Staging registers: each plane tile is 1024 chunks of 16 B, 4 per thread.
  u32x4 stg[NP][4];

  const floatx4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
  floatx4 acc[4][4];  // running accumulator (elementwise) or HH (termwise, hi-only)
  floatx4 xa[4][4];   // termwise XA, or elementwise per-block XA_g
  floatx4 xb[4][4];   // termwise XB, or elementwise per-block XB_g
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = xa[i][j] = xb[i][j] = zero;

  const int ktiles = Kp / kBK;
  global_load<NP>(gsrc, Kp, 0, t, stg);
  lds_store<NP>(lds, 0, t, stg);
  __syncthreads();

  const int frag_row = lane & 15;          // row (A) / column (B) inside a 16 x 16 tile
  const int frag_kc = lane >> 4;           // which 8-wide k chunk of the 32-wide step
  for (int kt = 0; kt < ktiles; ++kt) {
    const bool more = kt + 1 < ktiles;
    if (more) global_load<NP>(gsrc, Kp, kt + 1, t, stg);
    const uint16_t* s = lds + (kt & 1) * NP * kTileHalves;
#pragma unroll
    for (int ks = 0; ks < kBK / 32; ++ks) {
      const int kc = ks * 4 + frag_kc;
      half8 ah[4], bh[4], al[4], bl[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ra = wm * 64 + i * 16 + frag_row;
        const int oa = ra * kBK + ((kc ^ (ra & 7)) << 3);
        ah[i] = *reinterpret_cast<const half8*>(s + 0 * kTileHalves + oa);
        const int rb = wn * 64 + i * 16 + frag_row;
        const int ob = rb * kBK + ((kc ^ (rb & 7)) << 3);
        bh[i] = *reinterpret_cast<const half8*>(s + 1 * kTileHalves + ob);
        if constexpr (NP == 4) {
          al[i] = *reinterpret_cast<const half8*>(s + 2 * kTileHalves + oa);
          bl[i] = *reinterpret_cast<const half8*>(s + 3 * kTileHalves + ob);
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[i][j] = mfma16(ah[i], bh[j], acc[i][j]);
          if constexpr (V == kTermwise) {
            xa[i][j] = mfma16(al[i], bh[j], xa[i][j]);
            xb[i][j] = mfma16(ah[i], bl[j], xb[i][j]);
          } else if constexpr (V == kElementwise) {
            xa[i][j] = mfma16(al[i], bh[j], ks == 0 ? zero : xa[i][j]);
            xb[i][j] = mfma16(ah[i], bl[j], ks == 0 ? zero : xb[i][j]);
          }
        }
    }
    if constexpr (V == kElementwise) {
      // End of block g: acc = (acc + XA_g / s) + XB_g / s.
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            acc[i][j][e] = __builtin_fmaf(xa[i][j][e], inv_s, acc[i][j][e]);
            acc[i][j][e] = __builtin_fmaf(xb[i][j][e], inv_s, acc[i][j][e]);
          }
    }
    if (more) lds_store<NP>(lds, (kt + 1) & 1, t, stg);
    __syncthreads();
  }

  // Epilogue.  MFMA 16x16 output layout: lane holds rows 4*(lane/16)+e,
  // column lane%16 of its tile.
  const int col0 = tn * kBN + wn * 64 + (lane & 15);
  const int row0 = tm * kBM + wm * 64 + (lane >> 4) * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = col0 + j * 16;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = row0 + i * 16 + e;
        float v = acc[i][j][e];
        if constexpr (V == kTermwise) {
          v = __builtin_fmaf(xa[i][j][e], inv_s, v);
          v = __builtin_fmaf(xb[i][j][e], inv_s, v);
        }
        if (row < M && col < N) C[static_cast<size_t>(row) * ldc + col] = v;
      }
    }
}

template <int V>
hipError_t launch_variant(const Planes& p, int64_t M, int64_t N, float* C, int64_t ldc,
                          float inv_s, hipStream_t stream) {
  constexpr int NP = (V == kHiOnly) ? 2 : 4;
  constexpr size_t lds_bytes = 2 * NP * kTileHalves * sizeof(uint16_t);
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
