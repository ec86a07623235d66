// Register-only MFMA loop (gfx950): the sustained rate of the instruction the
// GEMM kernels are built from, v_mfma_f32_16x16x32_f16, with its operands held
// in registers and no memory traffic inside the loop.  It measures what the
// matrix units deliver under the board's power limit for given operand data,
// the practical ceiling for the GEMM kernels' roofline fraction.  Not part of
// the method.
//
// Each wave holds 8 A and 8 B fragments (16 x 32 FP16 each) and 64
// accumulators of 16 x 16 (256 AGPRs, tied to their registers as in the GEMM
// kernels); one iteration issues the 64 MFMAs acc[i][j] += A_i B_(i+j)%8, so
// dependent MFMAs on one accumulator are 64 apart.  Thread t of every
// workgroup reads fragments 16 t .. 16 t + 15 of the 4096-fragment operand
// block and writes the sum of its 256 accumulator values to out[256 b + t].
#include "ceiling.h"
#include "gemm_common.h"

namespace sgc {
namespace {

constexpr int kLoopThreads = 256;
constexpr int kLoopFrags = 16;  // half8 operand fragments per thread

__global__ __launch_bounds__(kLoopThreads, 1) void mfma_loop_kernel(
    const half8* __restrict__ operands, float* __restrict__ out, int iters) {
  const int t = threadIdx.x;
  half8 a[8], b[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    a[q] = operands[t * kLoopFrags + q];
    b[q] = operands[t * kLoopFrags + 8 + q];
  }
  floatx4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = floatx4{};
  mfma_drain();  // the zeroed accumulators are read by the first MFMAs
  for (int it = 0; it < iters; ++it) {
    static_for<64>([&](auto M) {
      constexpr int i = decltype(M)::value / 8, j = decltype(M)::value % 8;
      mfma16_acc(acc[i][j], a[i], b[(i + j) & 7]);
    });
  }
  mfma_drain();
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) s += acc[i][j][e];
  out[static_cast<int64_t>(blockIdx.x) * kLoopThreads + t] = s;
}

}  // namespace

hipError_t launch_mfma_loop(int64_t workgroups, int64_t iters, const uint16_t* operands,
                            float* out, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_loop_kernel, dim3(static_cast<unsigned>(workgroups)),
                     dim3(kLoopThreads), 0, stream, reinterpret_cast<const half8*>(operands),
                     out, static_cast<int>(iters));
  return hipGetLastError();
}

}  // namespace sgc
