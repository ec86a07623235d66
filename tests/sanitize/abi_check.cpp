// Drives every entry point of include/sgemm_cube.h from a host program built
// with the host AddressSanitizer and UndefinedBehaviorSanitizer (the library's
// sources compiled with the sanitizers on their host pass only; the kernels
// are the production ones).
//
//   abi_check cpu   argument validation, sizes, names and the split query:
//                   paths that return before any device work (no GPU needed)
//   abi_check gpu   the above, then small problems through every entry point
//                   on the current device, results checked against an FP64
//                   GEMM of the same FP32 inputs within 4 K 2^-24 (|A||B|)_ij
//
// Exit status 0 = every check passed; the sanitizers abort on their first
// report.  What this program is for is the host code (validation, workspace
// carving, the memory pool, the fixed workspace's address lookup); the
// numerics have their own tests.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "sgemm_cube.h"

namespace {

int failures = 0;
#define CHECK(cond)                                                               \
  do {                                                                            \
    if (!(cond)) {                                                                \
      std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                                 \
    }                                                                             \
  } while (0)

// Addresses that are never dereferenced: validation rejects the call first.
const uintptr_t kFake = uintptr_t{1} << 40;
template <typename T>
T* fake(uintptr_t off = 0) {
  return reinterpret_cast<T*>(kFake + off);
}

void check_validation() {
  const float* A = fake<float>();
  const float* B = fake<float>(1u << 30);
  float* C = fake<float>(uintptr_t{2} << 30);
  void* ws = fake<void>(uintptr_t{3} << 30);
  const int INV = SGEMM_CUBE_ERR_INVALID_VALUE, NS = SGEMM_CUBE_ERR_NOT_SUPPORTED;
  // sgemm_cube: every rejected argument class.
  CHECK(sgemm_cube(-1, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 3, B, 4, C, 4, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 3, C, 4, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 3, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, nullptr, 4, B, 4, C, 4, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 4, 3.f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 4, NAN, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 4, 0x1p25f, 0, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 3, nullptr) == INV);
  CHECK(sgemm_cube(4, 4, 4, A, 4, B, 4, fake<float>(8), 4, 2048.f, 0, nullptr) == INV);
  CHECK(sgemm_cube((int64_t{1} << 30) + 1, 4, 4, A, 4, fake<float>(uintptr_t{1} << 44), 4,
                   fake<float>(uintptr_t{1} << 45), 4, 2048.f, 0, nullptr) == NS);
  CHECK(sgemm_cube(0, 4, 4, nullptr, 4, B, 4, nullptr, 4, 2048.f, 0, nullptr) == 0);
  CHECK(sgemm_cube(4, 0, 4, A, 4, B, 1, C, 1, 2048.f, 1, nullptr) == 0);
  // _ws and _noalloc.
  const size_t need = sgemm_cube_workspace_size(4, 4, 4, 0);
  CHECK(need > 0);
  CHECK(sgemm_cube_ws(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, nullptr, need, nullptr) == INV);
  CHECK(sgemm_cube_ws(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, ws, need - 1, nullptr) == INV);
  CHECK(sgemm_cube_ws(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, fake<void>((uintptr_t{3} << 30) + 16),
                      need, nullptr) == INV);
  CHECK(sgemm_cube_ws(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, fake<void>(), need, nullptr) == INV);
  CHECK(sgemm_cube_noalloc(4, 4, 4, A, 4, B, 4, C, 4, 5.f, 0, nullptr) == INV);
  CHECK(sgemm_cube_noalloc(8192, 8192, 8192, A, 8192, fake<float>(uintptr_t{1} << 38), 8192,
                           fake<float>(uintptr_t{1} << 39), 8192, 2048.f, 0, nullptr) == NS);
  // _ex.
  uint32_t* rep = fake<uint32_t>((uintptr_t{3} << 30) + 64);
  CHECK(sgemm_cube_ex(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, 4, ws, 1 << 20, nullptr, nullptr) ==
        INV);
  // The split of B in the GEMM: termwise only, on its layouts.
  CHECK(sgemm_cube_ex(4, 4, 64, A, 64, B, 4, C, 4, 2048.f, 0, 2, ws, 1 << 20, nullptr, nullptr) ==
        NS);
  CHECK(sgemm_cube_ex(4, 6, 64, A, 64, B, 6, C, 6, 2048.f, 1, 2, ws, 1 << 20, nullptr, nullptr) ==
        NS);
  CHECK(sgemm_cube_ex(0, 4, 64, A, 64, B, 4, C, 4, 2048.f, 1, 2, ws, 1 << 20, nullptr, nullptr) ==
        0);
  CHECK(sgemm_cube_ex(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, 0, ws, 1 << 20, rep, nullptr) == INV);
  CHECK(sgemm_cube_ex(4, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, 0, ws, 1 << 20,
                      fake<uint32_t>((uintptr_t{5} << 30) + 2), nullptr) == INV);
  CHECK(sgemm_cube_ex(0, 4, 4, A, 4, B, 4, C, 4, 2048.f, 0, 1, ws, 1 << 20, nullptr, nullptr) ==
        0);
  CHECK(sgemm_cube_ex_workspace_size(300, 200, 100, 0, 0) ==
        sgemm_cube_workspace_size(300, 200, 100, 0));
  CHECK(sgemm_cube_ex_workspace_size(300, 200, 100, 0, 4) == 0);
  CHECK(sgemm_cube_ex_workspace_size(300, 200, 128, 1, 2) ==
        sgemm_cube_ex_workspace_size(300, 200, 128, 1, 0));
  // prepare / compute / compute_a / compute_stages.
  CHECK(sgemm_cube_prepare(4, 4, 4, A, 4, B, 4, 3.f, ws, need, nullptr) == INV);
  CHECK(sgemm_cube_prepare(4, 4, 4, A, 4, B, 4, 2048.f, ws, need - 1, nullptr) == INV);
  CHECK(sgemm_cube_compute(4, 4, 4, C, 4, 2048.f, 5, ws, need, nullptr) == INV);
  CHECK(sgemm_cube_compute(4, 4, 4, fake<float>((uintptr_t{3} << 30) + 64), 4, 2048.f, 0, ws,
                           need, nullptr) == INV);
  CHECK(sgemm_cube_compute_a(4, 4, 4, A, 3, C, 4, 2048.f, 0, ws, need, nullptr) == INV);
  CHECK(sgemm_cube_compute_a(4, 4, 4, A, 4, fake<float>(8), 4, 2048.f, 0, ws, need, nullptr) ==
        INV);
  CHECK(sgemm_cube_compute_b(4, 4, 64, B, 3, C, 4, 2048.f, 1, ws, need, nullptr) == INV);
  CHECK(sgemm_cube_compute_b(4, 4, 64, B, 4, C, 4, 2048.f, 0, ws, need, nullptr) == NS);
  CHECK(sgemm_cube_compute_b(4, 4, 96, B, 4, C, 4, 2048.f, 1, ws, need, nullptr) == NS);
  CHECK(sgemm_cube_compute_b(0, 4, 64, B, 4, C, 4, 2048.f, 1, ws, need, nullptr) == 0);
  CHECK(sgemm_cube_compute_stages(4, 4, 4, C, 4, 2048.f, 0, 3, ws, need, nullptr) == INV);
  CHECK(sgemm_cube_compute_stages(4, 4, 4, C, 4, 2048.f, 1, 2, ws, need, nullptr) == NS);
  // split, hgemm.
  uint16_t* H = fake<uint16_t>(uintptr_t{1} << 30);
  uint16_t* L = fake<uint16_t>(uintptr_t{2} << 30);
  CHECK(sgemm_cube_split(4, 4, A, 3, H, L, 4, 2048.f, nullptr) == INV);
  CHECK(sgemm_cube_split(4, 4, A, 4, H, H + 2, 4, 2048.f, nullptr) == INV);
  CHECK(sgemm_cube_split(0, 4, nullptr, 4, nullptr, nullptr, 4, 2048.f, nullptr) == 0);
  CHECK(sgemm_cube_hgemm(4, 4, 4, A, 3, B, 4, C, 4, nullptr) == INV);
  CHECK(sgemm_cube_hgemm(0, 4, 4, A, 4, B, 4, C, 4, nullptr) == 0);
  // Queries.
  CHECK(sgemm_cube_splits_a_in_gemm(512, 4096, 1024, A, 1024, 2048.f, 0) == 1);
  CHECK(sgemm_cube_splits_a_in_gemm(512, 4097, 1024, A, 1024, 2048.f, 0) == 0);
  CHECK(sgemm_cube_splits_a_in_gemm(512, 4096, 1024, fake<float>(4), 1024, 2048.f, 0) == 0);
  CHECK(sgemm_cube_block_k() == 32);
  for (int st = -1; st <= 5; ++st) CHECK(sgemm_cube_status_string(st) != nullptr);
  CHECK(std::string(sgemm_cube_status_string(SGEMM_CUBE_ERR_ALLOC)) == "SGEMM_CUBE_ERR_ALLOC");
  CHECK(sgemm_cube_workspace_size(0, 4, 4, 0) == 0);
}

// ---------------------------------------------------------------- GPU part

uint64_t g_lcg = 0x9e3779b97f4a7c15ULL;
float next_value() {  // deterministic values in [-1, 1)
  g_lcg = g_lcg * 6364136223846793005ULL + 1442695040888963407ULL;
  return static_cast<float>(static_cast<double>(g_lcg >> 11) / 9007199254740992.0 * 2.0 - 1.0);
}

#define HIP_OK(expr) CHECK((expr) == hipSuccess)

struct Problem {
  int64_t M, N, K, lda, ldb, ldc;
  std::vector<float> A, B;
  float *dA = nullptr, *dB = nullptr, *dC = nullptr;
  Problem(int64_t m, int64_t n, int64_t k, int64_t pad)
      : M(m), N(n), K(k), lda(k + pad), ldb(n + pad), ldc(n + pad) {
    A.resize(static_cast<size_t>(std::max<int64_t>(M * lda, 1)));
    B.resize(static_cast<size_t>(std::max<int64_t>(K * ldb, 1)));
    for (float& x : A) x = next_value();
    for (float& x : B) x = next_value();
    HIP_OK(hipMalloc(&dA, A.size() * 4));
    HIP_OK(hipMalloc(&dB, B.size() * 4));
    HIP_OK(hipMalloc(&dC, static_cast<size_t>(std::max<int64_t>(M * ldc, 1)) * 4));
    HIP_OK(hipMemcpy(dA, A.data(), A.size() * 4, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(dB, B.data(), B.size() * 4, hipMemcpyHostToDevice));
  }
  ~Problem() {
    (void)hipFree(dA);
    (void)hipFree(dB);
    (void)hipFree(dC);
  }
  void poison_c(hipStream_t s) {  // NaN bytes, so an unwritten entry fails the check
    HIP_OK(hipMemsetAsync(dC, 0xff, static_cast<size_t>(std::max<int64_t>(M * ldc, 1)) * 4, s));
  }
  // |C - AB| <= rel * (|A||B|)_ij for every entry (FP64 reference).
  bool check_c(hipStream_t s, double rel, const char* what) {
    HIP_OK(hipStreamSynchronize(s));
    std::vector<float> C(static_cast<size_t>(std::max<int64_t>(M * ldc, 1)));
    HIP_OK(hipMemcpy(C.data(), dC, C.size() * 4, hipMemcpyDeviceToHost));
    for (int64_t i = 0; i < M; ++i)
      for (int64_t j = 0; j < N; ++j) {
        double ref = 0, mag = 0;
        for (int64_t k = 0; k < K; ++k) {
          const double p = static_cast<double>(A[i * lda + k]) * B[k * ldb + j];
          ref += p;
          mag += std::fabs(p);
        }
        const double c = C[i * ldc + j];
        if (!(std::fabs(c - ref) <= rel * mag) || (K == 0 && std::signbit(c))) {
          std::fprintf(stderr, "%s: %lldx%lldx%lld C[%lld,%lld] = %.9g, FP64 %.9g\n", what,
                       (long long)M, (long long)N, (long long)K, (long long)i, (long long)j, c,
                       ref);
          ++failures;
          return false;
        }
      }
    return true;
  }
};

void check_gpu(hipStream_t s) {
  const int64_t shapes[][4] = {{70, 130, 200, 5}, {1, 1, 1, 0},   {257, 300, 64, 0},
                               {8, 4100, 64, 0},  {33, 17, 0, 1}, {130, 140, 256, 4}};
  for (const auto& sh : shapes) {
    Problem p(sh[0], sh[1], sh[2], sh[3]);
    const double rel = 4.0 * static_cast<double>(std::max<int64_t>(p.K, 1)) * 0x1p-24;
    const size_t need = sgemm_cube_workspace_size(p.M, p.N, p.K, 0);
    void* ws = nullptr;
    if (need) HIP_OK(hipMalloc(&ws, need));
    for (int order = 0; order <= 2; ++order) {
      p.poison_c(s);
      CHECK(sgemm_cube(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, p.dC, p.ldc, 2048.f, order, s) ==
            0);
      p.check_c(s, rel, "sgemm_cube");
      p.poison_c(s);
      CHECK(sgemm_cube_ws(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, p.dC, p.ldc, 2048.f, order, ws,
                          need, s) == 0);
      p.check_c(s, rel, "sgemm_cube_ws");
      p.poison_c(s);
      CHECK(sgemm_cube_noalloc(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, p.dC, p.ldc, 2048.f,
                               order, s) == 0);
      p.check_c(s, rel, "sgemm_cube_noalloc");
      if (p.K > 0) {
        p.poison_c(s);
        CHECK(sgemm_cube_prepare(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, 2048.f, ws, need, s) ==
              0);
        CHECK(sgemm_cube_compute(p.M, p.N, p.K, p.dC, p.ldc, 2048.f, order, ws, need, s) == 0);
        p.check_c(s, rel, "prepare + compute");
        p.poison_c(s);
        CHECK(sgemm_cube_prepare(p.M, p.N, p.K, nullptr, p.lda, p.dB, p.ldb, 2048.f, ws, need,
                                 s) == 0);
        CHECK(sgemm_cube_compute_a(p.M, p.N, p.K, p.dA, p.lda, p.dC, p.ldc, 2048.f, order, ws,
                                   need, s) == 0);
        p.check_c(s, rel, "prepare(B) + compute_a");
      }
    }
    // Pre-scaling and the range report.
    const size_t need_ex = sgemm_cube_ex_workspace_size(p.M, p.N, p.K, 1, 1);
    void* ws_ex = nullptr;
    uint32_t* rep = nullptr;
    if (need_ex) HIP_OK(hipMalloc(&ws_ex, need_ex));
    HIP_OK(hipMalloc(&rep, 4));
    p.poison_c(s);
    CHECK(sgemm_cube_ex(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, p.dC, p.ldc, 2048.f, 1, 1, ws_ex,
                        need_ex, rep, s) == 0);
    p.check_c(s, rel, "sgemm_cube_ex prescaled termwise");
    uint32_t classes = 0xffffffffu;
    HIP_OK(hipMemcpy(&classes, rep, 4, hipMemcpyDeviceToHost));
    CHECK((classes & (SGEMM_CUBE_RANGE_NONFINITE | SGEMM_CUBE_RANGE_HI_OVERFLOW |
                      SGEMM_CUBE_RANGE_LO_OVERFLOW)) == 0);
    if (p.K > 0) {
      for (int stages = 1; stages <= 2; ++stages) {
        p.poison_c(s);
        CHECK(sgemm_cube_prepare(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, 2048.f, ws, need, s) ==
              0);
        CHECK(sgemm_cube_compute_stages(p.M, p.N, p.K, p.dC, p.ldc, 2048.f, 0, stages, ws, need,
                                        s) == 0);
        p.check_c(s, rel, "compute_stages");
      }
      p.poison_c(s);
      CHECK(sgemm_cube_hgemm(p.M, p.N, p.K, p.dA, p.lda, p.dB, p.ldb, p.dC, p.ldc, s) == 0);
      p.check_c(s, 1e-3, "sgemm_cube_hgemm");
      // Row-major split of A: hi + lo/s reproduces A to ~2^-22 relative, or to
      // 2^-36 absolute where lo is FP16-subnormal.
      const int64_t ldh = p.K + 3;
      uint16_t *hi = nullptr, *lo = nullptr;
      HIP_OK(hipMalloc(&hi, static_cast<size_t>(p.M * ldh) * 2));
      HIP_OK(hipMalloc(&lo, static_cast<size_t>(p.M * ldh) * 2));
      CHECK(sgemm_cube_split(p.M, p.K, p.dA, p.lda, hi, lo, ldh, 2048.f, s) == 0);
      HIP_OK(hipStreamSynchronize(s));
      std::vector<_Float16> h(static_cast<size_t>(p.M * ldh)), l(h.size());
      HIP_OK(hipMemcpy(h.data(), hi, h.size() * 2, hipMemcpyDeviceToHost));
      HIP_OK(hipMemcpy(l.data(), lo, l.size() * 2, hipMemcpyDeviceToHost));
      for (int64_t i = 0; i < p.M; ++i)
        for (int64_t k = 0; k < p.K; ++k) {
          const double a = p.A[i * p.lda + k];
          const double r = static_cast<double>(h[i * ldh + k]) +
                           static_cast<double>(l[i * ldh + k]) / 2048.0;
          CHECK(std::fabs(r - a) <= std::fabs(a) * 0x1p-21 + 0x1p-35);
        }
      (void)hipFree(hi);
      (void)hipFree(lo);
    }
    (void)hipFree(rep);
    (void)hipFree(ws_ex);
    (void)hipFree(ws);
  }
}

}  // namespace

int main(int argc, char** argv) {
  const bool gpu = argc > 1 && std::strcmp(argv[1], "gpu") == 0;
  check_validation();
  if (gpu) {
    int n = 0;
    CHECK(hipGetDeviceCount(&n) == hipSuccess && n > 0);
    if (n > 0) {
      check_gpu(nullptr);
      hipStream_t s = nullptr;
      HIP_OK(hipStreamCreate(&s));
      check_gpu(s);
      HIP_OK(hipStreamSynchronize(s));
      HIP_OK(hipStreamDestroy(s));
    }
  }
  if (failures) {
    std::fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  std::printf("abi_check %s: all checks passed\n", gpu ? "gpu" : "cpu");
  return 0;
}
