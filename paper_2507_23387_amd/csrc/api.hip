// C-ABI of libsgemmcube: argument validation, workspace, dispatch.
// The interface and its conventions are documented in include/sgemm_cube.h.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "internal.h"
#include "sgemm_cube.h"

namespace sgc {

Planes plan_planes(int64_t M, int64_t N, int64_t K, void* base, bool prescale) {
  Planes p{};
  p.Mp = round_up(M, kRowPad);
  p.Np = round_up(N, kRowPad);
  p.Kp = round_up(K, kKPad);
  const size_t a_bytes = static_cast<size_t>(round_up(p.Mp * p.Kp * 2, 256));
  const size_t b_bytes = static_cast<size_t>(round_up(p.Np * p.Kp * 2, 256));
  p.bytes = kFlagBytes + 2 * a_bytes + 2 * b_bytes;
  if (prescale) p.bytes += static_cast<size_t>(round_up((p.Mp + p.Np) * 4, 256));
  if (!base) return p;  // sizes only
  char* c = static_cast<char*>(base);
  p.range = reinterpret_cast<uint32_t*>(c);
  c += kFlagBytes;
  p.a_hi = reinterpret_cast<uint16_t*>(c);
  p.a_lo = reinterpret_cast<uint16_t*>(c + a_bytes);
  p.b_hi = reinterpret_cast<uint16_t*>(c + 2 * a_bytes);
  p.b_lo = reinterpret_cast<uint16_t*>(c + 2 * a_bytes + b_bytes);
  if (prescale) {
    // The row and column maxima follow the planes.
    p.row_max = reinterpret_cast<uint32_t*>(c + 2 * a_bytes + 2 * b_bytes);
    p.col_max = p.row_max + p.Mp;
  }
  return p;
}

namespace {

// Largest dimension the kernels index with 32-bit tile arithmetic; also keeps
// every grid dimension within its hardware limit.
constexpr int64_t kMaxDim = (int64_t{1} << 30);

bool valid_order(int order) {
  return order == SGEMM_CUBE_ELEMENTWISE || order == SGEMM_CUBE_TERMWISE ||
         order == SGEMM_CUBE_ELEMENTWISE_CROSS_FIRST;
}

// Public accumulation order -> internal kernel variant.
int variant_of(int order) {
  switch (order) {
    case SGEMM_CUBE_ELEMENTWISE: return kElementwise;
    case SGEMM_CUBE_TERMWISE: return kTermwise;
    default: return kCrossFirst;
  }
}

bool valid_scale(float s) {
  if (!std::isfinite(s) || s < 1.0f || s > 16777216.0f) return false;
  int e = 0;
  return std::frexp(s, &e) == 0.5f;  // exact power of two
}

// Bytes spanned by a rows x cols row-major matrix with leading dimension ld.
uint64_t span_bytes(int64_t rows, int64_t cols, int64_t ld, uint64_t elem) {
  if (rows <= 0 || cols <= 0) return 0;
  return (static_cast<uint64_t>(rows - 1) * static_cast<uint64_t>(ld) +
          static_cast<uint64_t>(cols)) * elem;
}

bool overlap(const void* p, uint64_t pn, const void* q, uint64_t qn) {
  if (pn == 0 || qn == 0) return false;
  const uintptr_t a = reinterpret_cast<uintptr_t>(p), b = reinterpret_cast<uintptr_t>(q);
  return a < b + qn && b < a + pn;
}

// Grid limits: GEMM workgroups (at most (Mp / 256) * (Np / 128)) must fit an
// int, and the split of B uses grid.y = Np / 128 <= 65535.
bool round_up_tiles_exceed(int64_t M, int64_t N) {
  const int64_t Mp = round_up(M, kRowPad), Np = round_up(N, kRowPad);
  return (Mp / 256) * (Np / 128) > INT32_MAX || Np / kPanel > 65535;
}

// ld * rows must not overflow int64 when forming addresses.
bool ld_ok(int64_t rows, int64_t ld) {
  return rows <= 1 || ld <= INT64_MAX / 8 / rows;
}

int validate_gemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                  int64_t ldb, const float* C, int64_t ldc, float scale, bool check_scale) {
  if (M < 0 || N < 0 || K < 0) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (lda < (K > 1 ? K : 1) || ldb < (N > 1 ? N : 1) || ldc < (N > 1 ? N : 1))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (check_scale && !valid_scale(scale)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if ((M > 0 && K > 0 && !A) || (K > 0 && N > 0 && !B) || (M > 0 && N > 0 && !C))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!ld_ok(M, lda) || !ld_ok(K, ldb) || !ld_ok(M, ldc)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const uint64_t cb = span_bytes(M, N, ldc, 4);
  if (overlap(C, cb, A, span_bytes(M, K, lda, 4)) || overlap(C, cb, B, span_bytes(K, N, ldb, 4)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M > kMaxDim || N > kMaxDim || K > kMaxDim) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (round_up_tiles_exceed(M, N)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  return SGEMM_CUBE_OK;
}

// A fresh stamp for every split of B (see launch_split_b); 0 is skipped.
std::atomic<uint32_t> g_stamp{0};
uint32_t next_stamp() {
  uint32_t s = g_stamp.fetch_add(1, std::memory_order_relaxed) + 1;
  return s ? s : g_stamp.fetch_add(1, std::memory_order_relaxed) + 1;
}

size_t ws_size(int64_t M, int64_t N, int64_t K, bool prescale = false) {
  if (M == 0 || N == 0 || K == 0) return 0;
  return plan_planes(M, N, K, nullptr, prescale).bytes;
}

// Option bits sgemm_cube_ex accepts.
constexpr unsigned kExOptions = SGEMM_CUBE_OPT_PRESCALE | SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM;

// Target exponents of the pre-scaled row (A) and column (B) maxima for
// s = 2^s_b: [2^EA, 2^(EA+1)) with EA = min(14, 26 - s_b) keeps hi finite and
// the scaled residual of every entry below 2^16 (Rule 2, Sec. 4.2); B's
// EB = 14 - s_b also keeps s B_hi finite for the scaled elementwise kernel.
RangeOpts range_opts(unsigned options, bool report, float scale) {
  RangeOpts o;
  o.prescale = (options & SGEMM_CUBE_OPT_PRESCALE) != 0;
  o.report = report;
  int e = 0;
  (void)std::frexp(scale, &e);
  const int s_b = e - 1;
  o.exp_a = std::min(14, 26 - s_b);
  o.exp_b = 14 - s_b;
  return o;
}

// The in-kernel split of A redoes the split of an A tile once per tile
// column of C, on the vector ALU between the matrix instructions, while the
// split pass costs one read of A and one write of its planes through HBM.
// Measured on MI355X: for the elementwise order (256-column tiles) the
// in-kernel split is 13 % faster at M x N x K = 16384 x 1024 x 8192, 1 %
// faster at 4096^3 and 4 % slower at 8192^3, so it is used up to N = 4096.
// For termwise (128-column tiles, so twice the repeats per column of C): 10 %
// faster at 16384 x 1024 x 8192, even at 4096^3 and 4 % slower at 4096 x 4096
// x 16384, so it is used up to N = 2048.
constexpr int64_t kFusedSplitMaxN = 4096;
constexpr int64_t kTermwiseFusedMaxN = 2048;

bool splits_a_in_gemm(int64_t N, const float* A, int64_t lda, int64_t K, float scale,
                      int variant) {
  const int64_t max_n = variant == kElementwise ? kFusedSplitMaxN
                        : variant == kTermwise  ? kTermwiseFusedMaxN
                                                : 0;
  return N <= max_n && fused_split_ok(A, lda, K, scale, variant);
}

// GEMM from FP32 A and a workspace whose B planes are prepared: the 256 x 256
// kernel splits A in registers when splits_a_in_gemm says so, else A is split
// into the workspace first and the GEMM runs on the planes.
hipError_t compute_from_a(const Planes& p, int64_t M, int64_t N, int64_t K, const float* A,
                          int64_t lda, float* C, int64_t ldc, float scale, int variant,
                          hipStream_t stream) {
  if (splits_a_in_gemm(N, A, lda, K, scale, variant))
    return launch_gemm_fused_a(p, M, N, K, A, lda, C, ldc, scale, variant, stream);
  const hipError_t e = launch_split_a(p, M, K, A, lda, scale, RangeOpts{}, next_stamp(), stream);
  if (e != hipSuccess) return e;
  return launch_gemm(p, M, N, C, ldc, scale, variant, stream);
}

// Enqueue the whole computation; arguments already validated.  `report`, if
// not null, receives the range classes (device word).
int run(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
        int64_t ldb, float* C, int64_t ldc, float scale, int variant, void* ws,
        hipStream_t stream, const RangeOpts& opt = RangeOpts{}, uint32_t* report = nullptr,
        bool split_b_in_gemm = false) {
  if (M == 0 || N == 0 || K == 0) {
    if (M > 0 && N > 0 && launch_zero(M, N, C, ldc, stream) != hipSuccess)
      return SGEMM_CUBE_ERR_HIP;
    if (report && launch_range_report(Planes{}, true, report, stream) != hipSuccess)
      return SGEMM_CUBE_ERR_HIP;
    return SGEMM_CUBE_OK;
  }
  const Planes p = plan_planes(M, N, K, ws, opt.prescale);
  if (split_b_in_gemm) {
    // Termwise with B split inside the GEMM kernel (validated by the caller);
    // A too where the library splits it there, else by its own pass.
    const bool fused_a = splits_a_in_gemm(N, A, lda, K, scale, variant);
    if (!fused_a &&
        launch_split_a(p, M, K, A, lda, scale, opt, next_stamp(), stream) != hipSuccess)
      return SGEMM_CUBE_ERR_HIP;
    return launch_gemm_fused_b(p, M, N, K, A, lda, fused_a, B, ldb, C, ldc, scale, stream) ==
                   hipSuccess
               ? SGEMM_CUBE_OK
               : SGEMM_CUBE_ERR_HIP;
  }
  if (!opt.prescale && !opt.report && splits_a_in_gemm(N, A, lda, K, scale, variant)) {
    // B is split into the workspace, A inside the GEMM kernel.
    if (launch_split_b(p, K, N, B, ldb, scale, opt, next_stamp(), stream) != hipSuccess)
      return SGEMM_CUBE_ERR_HIP;
    return compute_from_a(p, M, N, K, A, lda, C, ldc, scale, variant, stream) == hipSuccess
               ? SGEMM_CUBE_OK
               : SGEMM_CUBE_ERR_HIP;
  }
  if (opt.prescale && launch_absmax(p, M, N, K, A, lda, B, ldb, stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (launch_split_a(p, M, K, A, lda, scale, opt, next_stamp(), stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (launch_split_b(p, K, N, B, ldb, scale, opt, next_stamp(), stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (launch_gemm(p, M, N, C, ldc, scale, variant, stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (opt.prescale && launch_unscale(p, M, N, C, ldc, opt, stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (report && launch_range_report(p, false, report, stream) != hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  return SGEMM_CUBE_OK;
}

// Library-owned, per-device stream-ordered memory pool for the workspace of
// the allocating entry points.  The release threshold is raised so memory
// freed at the end of a call is reused by the next one instead of going back
// to the driver at every synchronisation.
std::mutex g_pool_mu;
constexpr int kMaxDevices = 64;
hipMemPool_t g_pools[kMaxDevices] = {};

int get_pool(hipMemPool_t* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return SGEMM_CUBE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_pool_mu);
  if (!g_pools[dev]) {
    hipMemPoolProps props;
    std::memset(&props, 0, sizeof props);
    props.allocType = hipMemAllocationTypePinned;
    props.location.type = hipMemLocationTypeDevice;
    props.location.id = dev;
    hipMemPool_t pool = nullptr;
    if (hipMemPoolCreate(&pool, &props) != hipSuccess) return SGEMM_CUBE_ERR_ALLOC;
    uint64_t threshold = UINT64_MAX;
    if (hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &threshold) != hipSuccess) {
      (void)hipMemPoolDestroy(pool);
      return SGEMM_CUBE_ERR_ALLOC;
    }
    g_pools[dev] = pool;
  }
  *out = g_pools[dev];
  return SGEMM_CUBE_OK;
}

int run_allocating(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                   int64_t ldb, float* C, int64_t ldc, float scale, int variant,
                   hipStream_t stream) {
  const size_t need = ws_size(M, N, K);
  if (need == 0) return run(M, N, K, A, lda, B, ldb, C, ldc, scale, variant, nullptr, stream);
  hipMemPool_t pool = nullptr;
  int st = get_pool(&pool);
  if (st != SGEMM_CUBE_OK) {
    (void)hipGetLastError();
    return st;
  }
  void* ws = nullptr;
  if (hipMallocFromPoolAsync(&ws, need, pool, stream) != hipSuccess || !ws) {
    // Clear the runtime's last error, so that it is not reported by the
    // launch check of a later call on this thread.
    (void)hipGetLastError();
    return SGEMM_CUBE_ERR_ALLOC;
  }
  st = run(M, N, K, A, lda, B, ldb, C, ldc, scale, variant, ws, stream);
  if (hipFreeAsync(ws, stream) != hipSuccess && st == SGEMM_CUBE_OK) st = SGEMM_CUBE_ERR_HIP;
  return st;
}

// Workspace of sgemm_cube_noalloc: a fixed device array, one copy per GPU,
// held for the life of the process.  Host code must not use the array's name
// as a device address (on the host it names a stand-in object): its device
// address is looked up once per device with hipGetSymbolAddress, with that
// device current, and only that address is passed to kernels.  The array's
// header words are stamped by every split (a fresh stamp per call), so nothing
// in it has to start at zero; the planes are fully rewritten by the splits of
// each call, padding included.
static __device__ __align__(256) unsigned char scratch[SGEMM_CUBE_NOALLOC_WORKSPACE_BYTES];
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return SGEMM_CUBE_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return SGEMM_CUBE_ERR_HIP;
    if (reinterpret_cast<uintptr_t>(p) % 256 != 0) return SGEMM_CUBE_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return SGEMM_CUBE_OK;
}

// sgemm_cube_compute, sgemm_cube_compute_stages and sgemm_cube_compute_tile;
// stages == 0 and tile_m == 0 mean the library's default kernels.
int compute(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, float scale, int accum_order,
            int stages, const void* ws, size_t ws_bytes, hipStream_t stream, int tile_m = 0,
            int tile_n = 0, int block_k = 0, int waves = 0) {
  if (!valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M < 0 || N < 0 || K < 0 || ldc < (N > 1 ? N : 1) || !valid_scale(scale))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (stages < 0 || stages > 2) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const bool tile = tile_m != 0 || tile_n != 0 || block_k != 0 || waves != 0;
  if (tile && !tile_config_ok(tile_m, tile_n, block_k, waves))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if ((stages != 0 || tile) && accum_order != SGEMM_CUBE_ELEMENTWISE)
    return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (M > kMaxDim || N > kMaxDim || K > kMaxDim) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (round_up_tiles_exceed(M, N)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (M == 0 || N == 0) return SGEMM_CUBE_OK;
  if (!C || !ld_ok(M, ldc)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (K == 0)
    return launch_zero(M, N, C, ldc, stream) == hipSuccess ? SGEMM_CUBE_OK : SGEMM_CUBE_ERR_HIP;
  const size_t need = ws_size(M, N, K);
  if (ws_bytes < need || !ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (overlap(ws, need, C, span_bytes(M, N, ldc, 4))) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const Planes p = plan_planes(M, N, K, const_cast<void*>(ws));
  const hipError_t e =
      tile ? launch_gemm_tile(p, M, N, C, ldc, scale, tile_m, tile_n, block_k, waves, stream)
      : stages == 0
          ? launch_gemm(p, M, N, C, ldc, scale, variant_of(accum_order), stream)
          : launch_gemm_stages(p, M, N, C, ldc, scale, stages, stream);
  return e == hipSuccess ? SGEMM_CUBE_OK : SGEMM_CUBE_ERR_HIP;
}

}  // namespace
}  // namespace sgc

#pragma GCC visibility push(default)
extern "C" {

int sgemm_cube(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
               int64_t ldb, float* C, int64_t ldc, float scale, int accum_order,
               hipStream_t stream) {
  if (!sgc::valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const int st = sgc::validate_gemm(M, N, K, A, lda, B, ldb, C, ldc, scale, true);
  if (st != SGEMM_CUBE_OK) return st;
  return sgc::run_allocating(M, N, K, A, lda, B, ldb, C, ldc, scale,
                             sgc::variant_of(accum_order), stream);
}

int sgemm_cube_noalloc(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                       const float* B, int64_t ldb, float* C, int64_t ldc, float scale,
                       int accum_order, hipStream_t stream) {
  if (!sgc::valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const int st = sgc::validate_gemm(M, N, K, A, lda, B, ldb, C, ldc, scale, true);
  if (st != SGEMM_CUBE_OK) return st;
  const size_t need = sgc::ws_size(M, N, K);
  if (need > SGEMM_CUBE_NOALLOC_WORKSPACE_BYTES) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  void* ws = nullptr;
  if (need > 0) {
    const int sst = sgc::scratch_address(&ws);
    if (sst != SGEMM_CUBE_OK) return sst;
  }
  return sgc::run(M, N, K, A, lda, B, ldb, C, ldc, scale, sgc::variant_of(accum_order), ws,
                  stream);
}

int sgemm_cube_ws(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                  int64_t ldb, float* C, int64_t ldc, float scale, int accum_order, void* ws,
                  size_t ws_bytes, hipStream_t stream) {
  if (!sgc::valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  int st = sgc::validate_gemm(M, N, K, A, lda, B, ldb, C, ldc, scale, true);
  if (st != SGEMM_CUBE_OK) return st;
  const size_t need = sgc::ws_size(M, N, K);
  if (ws_bytes < need || (need > 0 && (!ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (need > 0) {
    if (sgc::overlap(ws, need, A, sgc::span_bytes(M, K, lda, 4)) ||
        sgc::overlap(ws, need, B, sgc::span_bytes(K, N, ldb, 4)) ||
        sgc::overlap(ws, need, C, sgc::span_bytes(M, N, ldc, 4)))
      return SGEMM_CUBE_ERR_INVALID_VALUE;
  }
  return sgc::run(M, N, K, A, lda, B, ldb, C, ldc, scale, sgc::variant_of(accum_order), ws,
                  stream);
}

int sgemm_cube_ex(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                  int64_t ldb, float* C, int64_t ldc, float scale, int accum_order,
                  unsigned options, void* ws, size_t ws_bytes, uint32_t* range_report,
                  hipStream_t stream) {
  if (!sgc::valid_order(accum_order) || (options & ~sgc::kExOptions))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  int st = sgc::validate_gemm(M, N, K, A, lda, B, ldb, C, ldc, scale, true);
  if (st != SGEMM_CUBE_OK) return st;
  const bool prescale = (options & SGEMM_CUBE_OPT_PRESCALE) != 0;
  const bool split_b = (options & SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM) != 0;
  if (split_b && (accum_order != SGEMM_CUBE_TERMWISE || prescale || range_report ||
                  !sgc::fused_split_b_ok(B, ldb, N, K)))
    return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const size_t need = sgc::ws_size(M, N, K, prescale);
  if (ws_bytes < need || (need > 0 && (!ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  const uint64_t ab = sgc::span_bytes(M, K, lda, 4), bb = sgc::span_bytes(K, N, ldb, 4);
  const uint64_t cb = sgc::span_bytes(M, N, ldc, 4);
  if (need > 0 && (sgc::overlap(ws, need, A, ab) || sgc::overlap(ws, need, B, bb) ||
                   sgc::overlap(ws, need, C, cb)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (range_report && (reinterpret_cast<uintptr_t>(range_report) % 4 != 0 ||
                       sgc::overlap(range_report, 4, A, ab) ||
                       sgc::overlap(range_report, 4, B, bb) ||
                       sgc::overlap(range_report, 4, C, cb) ||
                       sgc::overlap(range_report, 4, ws, need)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  return sgc::run(M, N, K, A, lda, B, ldb, C, ldc, scale, sgc::variant_of(accum_order), ws,
                  stream, sgc::range_opts(options, range_report != nullptr, scale), range_report,
                  split_b);
}

size_t sgemm_cube_ex_workspace_size(int64_t M, int64_t N, int64_t K, int accum_order,
                                    unsigned options) {
  if (!sgc::valid_order(accum_order) || (options & ~sgc::kExOptions)) return 0;
  if (M < 0 || N < 0 || K < 0 || M > sgc::kMaxDim || N > sgc::kMaxDim || K > sgc::kMaxDim)
    return 0;
  return sgc::ws_size(M, N, K, (options & SGEMM_CUBE_OPT_PRESCALE) != 0);
}

int sgemm_cube_prepare(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                       const float* B, int64_t ldb, float scale, void* ws, size_t ws_bytes,
                       hipStream_t stream) {
  if (M < 0 || N < 0 || K < 0) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (lda < (K > 1 ? K : 1) || ldb < (N > 1 ? N : 1) || !sgc::valid_scale(scale))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!sgc::ld_ok(M, lda) || !sgc::ld_ok(K, ldb)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M > sgc::kMaxDim || N > sgc::kMaxDim || K > sgc::kMaxDim) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const size_t need = sgc::ws_size(M, N, K);
  if (need == 0) return SGEMM_CUBE_OK;
  if (ws_bytes < need || !ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (sgc::overlap(ws, need, A, sgc::span_bytes(M, K, lda, 4)) ||
      sgc::overlap(ws, need, B, sgc::span_bytes(K, N, ldb, 4)))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (sgc::round_up_tiles_exceed(M, N)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const sgc::Planes p = sgc::plan_planes(M, N, K, ws);
  const sgc::RangeOpts plain;
  if (A && sgc::launch_split_a(p, M, K, A, lda, scale, plain, sgc::next_stamp(), stream) !=
               hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  if (B && sgc::launch_split_b(p, K, N, B, ldb, scale, plain, sgc::next_stamp(), stream) !=
               hipSuccess)
    return SGEMM_CUBE_ERR_HIP;
  return SGEMM_CUBE_OK;
}

int sgemm_cube_compute(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, float scale,
                       int accum_order, const void* ws, size_t ws_bytes, hipStream_t stream) {
  return sgc::compute(M, N, K, C, ldc, scale, accum_order, 0, ws, ws_bytes, stream);
}

int sgemm_cube_compute_b(int64_t M, int64_t N, int64_t K, const float* B, int64_t ldb,
                         float* C, int64_t ldc, float scale, int accum_order, const void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  if (!sgc::valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M < 0 || N < 0 || K < 0 || ldb < (N > 1 ? N : 1) || ldc < (N > 1 ? N : 1) ||
      !sgc::valid_scale(scale))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if ((K > 0 && N > 0 && !B) || (M > 0 && N > 0 && !C)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!sgc::ld_ok(K, ldb) || !sgc::ld_ok(M, ldc)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M > sgc::kMaxDim || N > sgc::kMaxDim || K > sgc::kMaxDim) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (sgc::round_up_tiles_exceed(M, N)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const uint64_t bb = sgc::span_bytes(K, N, ldb, 4), cb = sgc::span_bytes(M, N, ldc, 4);
  if (sgc::overlap(C, cb, B, bb)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (accum_order != SGEMM_CUBE_TERMWISE) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (M == 0 || N == 0) return SGEMM_CUBE_OK;
  if (K == 0)
    return sgc::launch_zero(M, N, C, ldc, stream) == hipSuccess ? SGEMM_CUBE_OK
                                                                : SGEMM_CUBE_ERR_HIP;
  if (!sgc::fused_split_b_ok(B, ldb, N, K)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const size_t need = sgc::ws_size(M, N, K);
  if (ws_bytes < need || !ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (sgc::overlap(ws, need, B, bb) || sgc::overlap(ws, need, C, cb))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  const sgc::Planes p = sgc::plan_planes(M, N, K, const_cast<void*>(ws));
  return sgc::launch_gemm_fused_b(p, M, N, K, nullptr, 0, false, B, ldb, C, ldc, scale,
                                  stream) == hipSuccess
             ? SGEMM_CUBE_OK
             : SGEMM_CUBE_ERR_HIP;
}

int sgemm_cube_compute_a(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                         float* C, int64_t ldc, float scale, int accum_order, void* ws,
                         size_t ws_bytes, hipStream_t stream) {
  if (!sgc::valid_order(accum_order)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M < 0 || N < 0 || K < 0 || lda < (K > 1 ? K : 1) || ldc < (N > 1 ? N : 1) ||
      !sgc::valid_scale(scale))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if ((M > 0 && K > 0 && !A) || (M > 0 && N > 0 && !C)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!sgc::ld_ok(M, lda) || !sgc::ld_ok(M, ldc)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M > sgc::kMaxDim || N > sgc::kMaxDim || K > sgc::kMaxDim) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  if (sgc::round_up_tiles_exceed(M, N)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  const uint64_t ab = sgc::span_bytes(M, K, lda, 4), cb = sgc::span_bytes(M, N, ldc, 4);
  if (sgc::overlap(C, cb, A, ab)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (M == 0 || N == 0) return SGEMM_CUBE_OK;
  if (K == 0)
    return sgc::launch_zero(M, N, C, ldc, stream) == hipSuccess ? SGEMM_CUBE_OK
                                                                : SGEMM_CUBE_ERR_HIP;
  const size_t need = sgc::ws_size(M, N, K);
  if (ws_bytes < need || !ws || reinterpret_cast<uintptr_t>(ws) % 256 != 0)
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (sgc::overlap(ws, need, A, ab) || sgc::overlap(ws, need, C, cb))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  const sgc::Planes p = sgc::plan_planes(M, N, K, ws);
  return sgc::compute_from_a(p, M, N, K, A, lda, C, ldc, scale, sgc::variant_of(accum_order),
                             stream) == hipSuccess
             ? SGEMM_CUBE_OK
             : SGEMM_CUBE_ERR_HIP;
}

int sgemm_cube_splits_a_in_gemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                                float scale, int accum_order) {
  if (M <= 0 || N <= 0 || K <= 0 || !A || !sgc::valid_scale(scale)) return 0;
  if (lda < K || !sgc::ld_ok(M, lda) || M > sgc::kMaxDim || N > sgc::kMaxDim ||
      K > sgc::kMaxDim || sgc::round_up_tiles_exceed(M, N))
    return 0;
  if (accum_order < SGEMM_CUBE_ELEMENTWISE || accum_order > SGEMM_CUBE_ELEMENTWISE_CROSS_FIRST)
    return 0;
  return sgc::splits_a_in_gemm(N, A, lda, K, scale, sgc::variant_of(accum_order)) ? 1 : 0;
}

int sgemm_cube_compute_stages(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                              float scale, int accum_order, int stages, const void* ws,
                              size_t ws_bytes, hipStream_t stream) {
  if (stages < 1) return SGEMM_CUBE_ERR_INVALID_VALUE;
  return sgc::compute(M, N, K, C, ldc, scale, accum_order, stages, ws, ws_bytes, stream);
}

int sgemm_cube_compute_tile(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, float scale,
                            int accum_order, int tile_m, int tile_n, int block_k, int waves,
                            const void* ws, size_t ws_bytes, hipStream_t stream) {
  if (tile_m == 0 && tile_n == 0 && block_k == 0 && waves == 0)
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  return sgc::compute(M, N, K, C, ldc, scale, accum_order, 0, ws, ws_bytes, stream, tile_m,
                      tile_n, block_k, waves);
}

size_t sgemm_cube_workspace_size(int64_t M, int64_t N, int64_t K, int accum_order) {
  if (!sgc::valid_order(accum_order)) return 0;
  if (M < 0 || N < 0 || K < 0 || M > sgc::kMaxDim || N > sgc::kMaxDim || K > sgc::kMaxDim)
    return 0;
  return sgc::ws_size(M, N, K);
}

int sgemm_cube_split(int64_t rows, int64_t cols, const float* X, int64_t ldx, uint16_t* hi,
                     uint16_t* lo, int64_t ldh, float scale, hipStream_t stream) {
  if (rows < 0 || cols < 0) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (ldx < (cols > 1 ? cols : 1) || ldh < (cols > 1 ? cols : 1))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!sgc::valid_scale(scale)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (rows == 0 || cols == 0) return SGEMM_CUBE_OK;
  if (!X || !hi || !lo) return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (!sgc::ld_ok(rows, ldx) || !sgc::ld_ok(rows, ldh)) return SGEMM_CUBE_ERR_INVALID_VALUE;
  const uint64_t xb = sgc::span_bytes(rows, cols, ldx, 4);
  const uint64_t hb = sgc::span_bytes(rows, cols, ldh, 2);
  if (sgc::overlap(hi, hb, lo, hb) || sgc::overlap(hi, hb, X, xb) || sgc::overlap(lo, hb, X, xb))
    return SGEMM_CUBE_ERR_INVALID_VALUE;
  if (cols > (int64_t{1} << 40)) return SGEMM_CUBE_ERR_NOT_SUPPORTED;
  return sgc::launch_split_rows(rows, cols, X, ldx, hi, lo, ldh, scale, stream) ==
                 hipSuccess
             ? SGEMM_CUBE_OK
             : SGEMM_CUBE_ERR_HIP;
}

int sgemm_cube_hgemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                     const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream) {
  const int st = sgc::validate_gemm(M, N, K, A, lda, B, ldb, C, ldc, 1.0f, false);
  if (st != SGEMM_CUBE_OK) return st;
  // The hi-only baseline does not read the residual planes; the split still
  // fills them so the whole split pass is shared.
  return sgc::run_allocating(M, N, K, A, lda, B, ldb, C, ldc, 1.0f, sgc::kHiOnly, stream);
}

const char* sgemm_cube_status_string(int status) {
  switch (status) {
    case SGEMM_CUBE_OK: return "SGEMM_CUBE_OK";
    case SGEMM_CUBE_ERR_INVALID_VALUE: return "SGEMM_CUBE_ERR_INVALID_VALUE";
    case SGEMM_CUBE_ERR_NOT_SUPPORTED: return "SGEMM_CUBE_ERR_NOT_SUPPORTED";
    case SGEMM_CUBE_ERR_ALLOC: return "SGEMM_CUBE_ERR_ALLOC";
    case SGEMM_CUBE_ERR_HIP: return "SGEMM_CUBE_ERR_HIP";
    default: return "SGEMM_CUBE_UNKNOWN_STATUS";
  }
}

int sgemm_cube_block_k(void) { return sgc::kBlockScaled; }

}  // extern "C"
#pragma GCC visibility pop
