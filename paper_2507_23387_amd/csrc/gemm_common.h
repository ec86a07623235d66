// Building blocks shared by the GEMM kernels of libsgemmcube (gfx950): MFMA
// wrappers, the LDS DMA, explicit waits and barriers, the XCD-aware tile maps
// and the accumulator stores.  Internal; every function has internal linkage.
#pragma once

#include <atomic>
#include <utility>

#include "internal.h"

namespace sgc {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// One 64-lane LDS DMA: lane l copies 16 bytes from g into LDS byte address
// lds_addr + 16 * l (the instruction takes the LDS base from M0, which the
// "{m0}" operand has the compiler load).  Inline asm, so the compiler adds no
// conservative vmcnt(0) before later LDS reads; the kernels wait explicitly
// with wait_vmcnt<>() before the barrier that publishes a stage.
__device__ __forceinline__ void dma16(const void* g, unsigned lds_addr) {
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(lds_addr) : "memory");
}

// The same DMA with the global base in an SGPR pair and a per-lane 32-bit
// byte offset (the saddr form): the wave-uniform part of the address costs
// scalar instructions only.  `base` must be wave-uniform; readfirstlane makes
// the compiler keep it in SGPRs.
__device__ __forceinline__ void dma16s(const void* base, unsigned voff, unsigned lds_addr) {
  // readfirstlane returns a signed int: take both words as uint32_t before
  // widening, so the low word is zero-extended.
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b)));
  const uint64_t sb = (static_cast<uint64_t>(hi) << 32) | lo;
  asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sb), "{m0}"(lds_addr) : "memory");
}

// Byte just past the furthest LDS DMA target of a kernel whose DMAs write
// 4 KiB plane tiles (each wave of four copying its 1 KiB block of the tile)
// at LDS halves offsets up to `last_tile_halves`.  The kernels check this
// against their dynamic LDS size, and against the 128 KiB that every DMA
// target stays below, at compile time.
constexpr size_t dma_end_bytes(int last_tile_halves) {
  return static_cast<size_t>(last_tile_halves) * 2 + static_cast<size_t>(kTileHalves) * 2;
}
constexpr size_t kMaxLdsBytes = 128 * 1024;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// This wave's LDS reads are complete, then all waves meet.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Keeps the instruction groups of the schedule in program order.
#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

// LDS byte address of the dynamic shared-memory base (the M0 operand of the
// DMA): cast the generic pointer to the LDS address space, then to int.
__device__ __forceinline__ unsigned lds_address(const uint16_t* p) {
  return static_cast<unsigned>((uintptr_t)((__attribute__((address_space(3))) const uint16_t*)p));
}

// Map a tile index to a (tile_m, tile_n) pair.  Workgroups are dispatched
// round-robin over the 8 XCDs, so index i runs on XCD i % 8 (also for the
// persistent grid, whose size is a multiple of 8); renumbering gives each XCD
// a contiguous range of logical tiles, and grouping kGroup tile-rows keeps the
// A and B panels a group touches resident in that XCD's L2.
template <int kGroup>
__device__ __forceinline__ void tile_of(int index, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int nwg = tiles_m * tiles_n;
  int wg = index;
  if ((nwg & 7) == 0) wg = (wg & 7) * (nwg >> 3) + (wg >> 3);
  const int per_group = kGroup * tiles_n;
  const int group = wg / per_group;
  const int first_m = group * kGroup;
  const int gsize = min(tiles_m - first_m, kGroup);
  const int in_group = wg - group * per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// Tile map for grids made of whole 16 x 16 blocks of 256 x 256 tiles (both
// tile counts multiples of 16): the 256 workgroups of one dispatch round
// (index / 256, one workgroup per compute unit) cover one 16 x 16 block, the
// blocks in snake order along block rows; inside a block, XCD x (index % 8)
// takes the 4 x 8 sub-block (x / 2, x % 2).  So in a round each A panel is
// read by two XCDs and each B panel by four, and consecutive rounds share a
// row (or column) of panels, which the last-level cache can serve.  Returns
// false (and leaves tm, tn alone) when the grid is not made of such blocks.
__device__ __forceinline__ bool tile_of_block(int index, int tiles_m, int tiles_n, int& tm,
                                              int& tn) {
  if ((tiles_m & 15) != 0 || (tiles_n & 15) != 0) return false;
  const int round = index >> 8, x = index & 7, j = (index & 255) >> 3;
  const int per_row = tiles_n >> 4;
  const int br = round / per_row;
  const int in_row = round - br * per_row;
  const int bc = (br & 1) ? per_row - 1 - in_row : in_row;
  tm = br * 16 + (x >> 1) * 4 + (j & 3);
  tn = bc * 16 + (x & 1) * 8 + (j >> 2);
  return true;
}

// D(16x16) = A(16x32) B(32x16) + C.  Lane l supplies A row l%16 and B column
// l%16 with the 8 consecutive k values 8*(l/16) .. 8*(l/16)+7 of the 32-wide
// step; D element (row 4*(l/16) + r, column l%16) is in register r.
__device__ __forceinline__ floatx4 mfma16(const half8& a, const half8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// acc += A B on v_mfma_f32_16x16x32_f16 (operands as for mfma16), with the
// accumulator tied to one AGPR quad ("+a") so that the register allocator
// keeps every accumulator in place across the main loop.  The compiler does
// not see an MFMA here, so the callers keep the MFMA hazards themselves, by
// distance in the instruction stream (one of these MFMAs occupies the
// matrix pipe 16 cycles): an MFMA that reads another's result as its C
// operand comes at least 4 MFMAs after it (8 in the 256 x 256 kernels); a
// VALU instruction that reads an MFMA result comes at least 8 MFMAs after
// it, or after mfma_drain(); VALU results an MFMA reads are written at
// least 8 MFMAs before it; and an operand register is rewritten (by an LDS
// read) no earlier than one MFMA after its last reader was issued.
__device__ __forceinline__ void mfma16_acc(floatx4& acc, const half8& a, const half8& b) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// x * s for the eight halves of x, s given as a packed pair (s, s): four
// v_pk_mul_f16 issued as volatile asm, so that the compiler neither moves nor
// rematerializes them next to an mfma16_acc that reads the result (it would
// not see that hazard); the callers place them at least 8 MFMAs ahead.
__device__ __forceinline__ half8 pk_scale(const half8& x, uint32_t s2) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_bit_cast(u32x4, x);
  uint32_t r0, r1, r2, r3;
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r0) : "s"(s2), "v"(v.x));
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r1) : "s"(s2), "v"(v.y));
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r2) : "s"(s2), "v"(v.z));
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r3) : "s"(s2), "v"(v.w));
  return __builtin_bit_cast(half8, u32x4{r0, r1, r2, r3});
}

// Half of pk_scale: words 2 * kPart and 2 * kPart + 1 of out = x * s (four
// halves).  Two VALU instructions overlap one MFMA for free, four do not, so
// the kernels form s * B_hi in two halves after different MFMAs.
template <int kPart>
__device__ __forceinline__ void pk_scale_half(half8& out, const half8& x, uint32_t s2) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_bit_cast(u32x4, x);
  u32x4 o = __builtin_bit_cast(u32x4, out);
  uint32_t r0, r1;
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r0) : "s"(s2), "v"(v[2 * kPart]));
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r1) : "s"(s2), "v"(v[2 * kPart + 1]));
  o[2 * kPart] = r0;
  o[2 * kPart + 1] = r1;
  out = __builtin_bit_cast(half8, o);
}

// The split of Sec. 3.3 (hi = fl16(a), r = a - hi exactly, lo = fl16(r s)) of
// two FP32 values a0, a1 into one packed word of high halves and one of scaled
// residuals, five VALU instructions:
//   kOp 0  v_cvt_pk_f16_f32      hi = fl16(a0), fl16(a1)
//   kOp 1  v_fma_mix_f32         r[0] = hi.lo * (-1) + a0   (exact: a - hi
//   kOp 2  v_fma_mix_f32         r[1] = hi.hi * (-1) + a1    fits FP32)
//   kOp 3  v_fma_mixlo_f16       lo.lo = fl16(r[0] * s + 0)  (r s exact, s a
//   kOp 4  v_fma_mixhi_f16       lo.hi = fl16(r[1] * s + 0)   power of two; r
//                                                             is never -0)
// Each result is one round-to-nearest-even conversion of an exact value with
// FP16 and FP32 denormals kept, so the words equal those of split_value.
// One instruction per call (volatile asm), so that the kernels can place each
// between two MFMAs; `s` is the wave-uniform scale.  kOp 3 defines the whole
// register (its other half is written by kOp 4), so no earlier value of lo
// has to be kept.
template <int kOp>
__device__ __forceinline__ void split_op(uint32_t& hi, uint32_t& lo, float (&r)[2], float a0,
                                         float a1, float s) {
  if constexpr (kOp == 0)
    asm volatile("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(hi) : "v"(a0), "v"(a1));
  else if constexpr (kOp == 1)
    asm volatile("v_fma_mix_f32 %0, %1, -1.0, %2 op_sel_hi:[1,0,0]"
                 : "=v"(r[0]) : "v"(hi), "v"(a0));
  else if constexpr (kOp == 2)
    asm volatile("v_fma_mix_f32 %0, %1, -1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
                 : "=v"(r[1]) : "v"(hi), "v"(a1));
  else if constexpr (kOp == 3)
    asm volatile("v_fma_mixlo_f16 %0, %1, %2, 0" : "=v"(lo) : "v"(r[0]), "s"(s));
  else
    asm volatile("v_fma_mixhi_f16 %0, %1, %2, 0" : "+v"(lo) : "v"(r[1]), "s"(s));
}

// The same split with the five instructions issued back to back.
__device__ __forceinline__ void split_pair_all(uint32_t& hi, uint32_t& lo, float a0, float a1,
                                               float s) {
  float r[2];
  split_op<0>(hi, lo, r, a0, a1, s);
  split_op<1>(hi, lo, r, a0, a1, s);
  split_op<2>(hi, lo, r, a0, a1, s);
  split_op<3>(hi, lo, r, a0, a1, s);
  split_op<4>(hi, lo, r, a0, a1, s);
}

// s * x for four of the eight halves of x (words 2 kPart and 2 kPart + 1 of
// pk_scale), one v_pk_mul_f16 per word: kWord selects the word.
template <int kWord>
__device__ __forceinline__ void pk_scale_word(half8& out, const half8& x, uint32_t s2) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_bit_cast(u32x4, x);
  u32x4 o = __builtin_bit_cast(u32x4, out);
  uint32_t r;
  asm volatile("v_pk_mul_f16 %0, %1, %2" : "=v"(r) : "s"(s2), "v"(v[kWord]));
  o[kWord] = r;
  out = __builtin_bit_cast(half8, o);
}

// The same with the accumulator tied to a VGPR quad.
__device__ __forceinline__ void mfma16_vacc(floatx4& acc, const half8& a, const half8& b) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(acc) : "v"(a), "v"(b));
}

// acc += A B with the accumulator tied to a VGPR quad and the A operand read
// from AGPRs (the block-fold kernels keep their A fragments there).
__device__ __forceinline__ void mfma16_va_acc(floatx4& acc, const half8& a, const half8& b) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, %0" : "+v"(acc) : "a"(a), "v"(b));
}

// out = A B (accumulator input zero) into a fresh VGPR quad, A from AGPRs.
__device__ __forceinline__ void mfma16_va_new(floatx4& out, const half8& a, const half8& b) {
  asm volatile("v_mfma_f32_16x16x32_f16 %0, %1, %2, 0" : "=&v"(out) : "a"(a), "v"(b));
}

// Wait states after the last mfma16_acc before its accumulators are read.
__device__ __forceinline__ void mfma_drain() {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// Compile-time loop: f(std::integral_constant<int, I>{}) for I = 0 .. N-1, so
// every index in the body is a constant expression (no reliance on unrolling).
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Store a wave's 16 x 16 accumulators: register r of MFMA tile (i, j) holds
// row 4*(l/16) + r and column l%16 of that tile.  `value` maps (i, j, r) to
// the float to store.  Tiles entirely inside C take the unmasked path.
template <int kSubM, int kSubN, typename F>
__device__ __forceinline__ void store_tile16(float* __restrict__ C, int64_t ldc, int M, int N,
                                             int row0, int col0, bool full, F value) {
  float* const base = C + static_cast<int64_t>(row0) * ldc + col0;
#pragma unroll
  for (int i = 0; i < kSubM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int rr = i * 16 + r;
      float* const p = base + static_cast<int64_t>(rr) * ldc;
#pragma unroll
      for (int j = 0; j < kSubN; ++j)
        if (full || (row0 + rr < M && col0 + j * 16 < N)) p[j * 16] = value(i, j, r);
    }
}

// Raise a kernel's dynamic-LDS limit on the current device, once per device
// and kernel (each instantiation calls this with its own `done` table).
constexpr int kMaxDevices = 64;
template <typename Kern>
hipError_t set_lds(Kern kernel, size_t bytes, std::atomic<bool> (&done)[kMaxDevices]) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kMaxDevices && done[dev].load(std::memory_order_acquire))
    return hipSuccess;
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                          hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
  if (e == hipSuccess && dev >= 0 && dev < kMaxDevices)
    done[dev].store(true, std::memory_order_release);
  return e;
}

}  // namespace
}  // namespace sgc
