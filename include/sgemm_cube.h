/*
 * sgemm_cube.h -- FP32-accuracy GEMM from three FP16 MFMA products on
 * AMD Instinct MI355X (gfx950).
 *
 * Method (arXiv 2507.23387, "SGEMM-cube"):
 *   Sec. 3.3 / Eq. recover_eqn: every FP32 operand entry a is split into an
 *   FP16 high word hi = fl16(a) and an FP16 scaled residual
 *   lo = fl16((a - hi) * s), fl16 = round to nearest even with gradual
 *   underflow.  The product is rebuilt from three FP16 GEMMs accumulated in
 *   FP32,
 *       C ~= A_hi B_hi + (A_lo B_hi + A_hi B_lo) / s,
 *   and the lo*lo term is dropped (bounded by Eq. ll_bound).
 *   Sec. 4.5: the three terms are accumulated either elementwise
 *   (Eq. elementwise: one running FP32 accumulator, each k-block's three
 *   products folded into it in turn) or termwise (Eq. termwise: three
 *   separate FP32 accumulations, combined once at the end as
 *   (HH + XA/s) + XB/s).
 *
 * Conventions shared by every entry point below:
 *   - Matrices are ROW-MAJOR.  A is M x K with leading dimension lda >= K,
 *     B is K x N with ldb >= N, C is M x N with ldc >= N (all counted in
 *     elements).  Column-major callers pass the operands swapped
 *     (C^T = B^T A^T).
 *   - A, B, C (and the workspace) are DEVICE pointers owned by the caller,
 *     who keeps them alive until the enqueued work completes.
 *   - Every call is asynchronous: it validates its arguments on the host,
 *     enqueues kernels on `stream` (a hipStream_t; 0 = the null stream) and
 *     returns.  Argument errors are reported BEFORE any device work and leave
 *     C untouched.  Device faults surface at the caller's next stream
 *     synchronisation.
 *   - No range guard: inputs with |a| >= 65520 (hi overflow) or with a scaled
 *     residual >= 65520 (lo overflow, Rule 2 of Sec. 4.2 violated) produce
 *     IEEE inf/NaN in the affected outputs, deterministically (Sec. 3.1 scope).
 *     Entries below 2^-14 have a subnormal hi and lose the 22-bit guarantee of
 *     Eq. split_error (Sec. 4.2); they are still computed as defined.
 *     sgemm_cube_ex adds power-of-two pre-scaling and a range report.
 *   - Thread-safe; the library keeps no per-call state, except that calls of
 *     sgemm_cube_noalloc that overlap on one GPU share its fixed workspace.
 */
#ifndef SGEMM_CUBE_H_
#define SGEMM_CUBE_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Accumulation orders (Sec. 4.5). */
typedef enum {
  SGEMM_CUBE_ELEMENTWISE = 0,             /* Eq. elementwise */
  SGEMM_CUBE_TERMWISE = 1,                /* Eq. termwise */
  SGEMM_CUBE_ELEMENTWISE_CROSS_FIRST = 2  /* the reordering proposed at the end of
                                             Sec. 4.5: per block g,
                                             acc = acc + ((XA_g + XB_g) / s + HH_g),
                                             blocks of sgemm_cube_block_k() */
} sgemm_cube_order_t;

/* Status codes returned by every entry point. */
typedef enum {
  SGEMM_CUBE_OK = 0,
  SGEMM_CUBE_ERR_INVALID_VALUE = 1, /* bad dimension, stride, pointer, scale or order */
  SGEMM_CUBE_ERR_NOT_SUPPORTED = 2, /* shape beyond the library's indexing limits or
                                       sgemm_cube_noalloc's fixed workspace; an option
                                       or measurement hook used outside the orders and
                                       layouts it covers */
  SGEMM_CUBE_ERR_ALLOC = 3,         /* workspace could not be obtained */
  SGEMM_CUBE_ERR_HIP = 4            /* a HIP runtime call or kernel launch failed */
} sgemm_cube_status_t;

/*
 * C = SGEMM-cube(A, B): FP32 in, FP32 out, C overwritten (no alpha/beta).
 *
 *   M, N, K      >= 0.  M == 0 or N == 0: nothing is done.  K == 0: C := +0.
 *   A, lda       row-major M x K, lda >= max(1, K); non-NULL when M*K > 0.
 *   B, ldb       row-major K x N, ldb >= max(1, N); non-NULL when K*N > 0.
 *   C, ldc       row-major M x N, ldc >= max(1, N); non-NULL when M*N > 0;
 *                must not overlap A or B.
 *   scale        the residual scaling factor s = 2^{s_b} of Sec. 4.2: a finite
 *                exact power of two in [1, 2^24].  Eq. sf_bounds gives the
 *                valid range for an input's exponent window; 2^11 is the fixed
 *                choice valid over the whole normal-FP16 range.  Any other
 *                value -> SGEMM_CUBE_ERR_INVALID_VALUE.
 *   accum_order  SGEMM_CUBE_ELEMENTWISE, SGEMM_CUBE_TERMWISE or
 *                SGEMM_CUBE_ELEMENTWISE_CROSS_FIRST.
 *   stream       HIP stream the work is enqueued on.
 *
 * Needs device workspace of sgemm_cube_workspace_size(M, N, K, accum_order)
 * bytes, which this entry point takes stream-ordered from a library-owned
 * memory pool (hipMallocFromPoolAsync / hipFreeAsync on `stream`); failure ->
 * SGEMM_CUBE_ERR_ALLOC.  Use sgemm_cube_ws to pass your own workspace.
 */
int sgemm_cube(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
               int64_t ldb, float* C, int64_t ldc, float scale, int accum_order,
               hipStream_t stream);

/*
 * Same as sgemm_cube, with caller-provided device workspace `ws` of
 * `ws_bytes` bytes (>= sgemm_cube_workspace_size(...), 256-byte aligned).
 * `ws` may be NULL only when the required size is 0.  The workspace must not
 * overlap A, B or C; its contents on entry are irrelevant and on exit are
 * unspecified.  Calls that share a workspace must be ordered on one stream.
 */
int sgemm_cube_ws(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                  int64_t ldb, float* C, int64_t ldc, float scale, int accum_order, void* ws,
                  size_t ws_bytes, hipStream_t stream);

/*
 * For callers that cannot allocate device memory: code recorded under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same computation, arguments, validation and results as sgemm_cube (bit for
 * bit: the same kernels run), but the workspace is a fixed device array inside
 * the library, SGEMM_CUBE_NOALLOC_WORKSPACE_BYTES (64 MiB) on every GPU the
 * library runs on, held until the process ends.  No device memory is
 * allocated or freed by this call.
 *   Problems whose workspace (sgemm_cube_workspace_size) exceeds that size ->
 *   SGEMM_CUBE_ERR_NOT_SUPPORTED before any device work; the workspace is
 *   256 + 4 * Kp * (Mp + Np) bytes with Mp, Np = M, N rounded up to 256 and
 *   Kp = K rounded up to 64, so e.g. M = N = K = 2048 fits.
 *   All calls on one GPU share its array: calls that overlap in time on one
 *   GPU (different streams, or different host threads without ordering) race
 *   and give undefined results; calls ordered on one stream are safe.  The
 *   array's contents carry over between calls and are never read before each
 *   call rewrites them.
 * The first call on each device looks up the array's device address
 * (hipGetSymbolAddress) with that device current; a failure there ->
 * SGEMM_CUBE_ERR_HIP.
 */
#define SGEMM_CUBE_NOALLOC_WORKSPACE_BYTES ((size_t)64 << 20)
int sgemm_cube_noalloc(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                       const float* B, int64_t ldb, float* C, int64_t ldc, float scale,
                       int accum_order, hipStream_t stream);

/* Options of sgemm_cube_ex (bit mask). */
enum { SGEMM_CUBE_OPT_PRESCALE = 1, SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM = 2 };

/* Range classes reported by sgemm_cube_ex (bit mask; Sec. 3.1 and 4.2). */
enum {
  SGEMM_CUBE_RANGE_NONFINITE = 1,    /* an input entry is inf or NaN */
  SGEMM_CUBE_RANGE_HI_OVERFLOW = 2,  /* a finite entry has |a| >= 65520: fl16(a) is infinite */
  SGEMM_CUBE_RANGE_LO_OVERFLOW = 4,  /* a scaled residual overflowed FP16 (Rule 2 violated) */
  SGEMM_CUBE_RANGE_HI_SUBNORMAL = 8  /* a nonzero hi is FP16-subnormal: the 22-bit guarantee
                                        of Sec. 4.2 does not hold for that entry */
};

/*
 * sgemm_cube_ws with the range extensions that Sec. 4.2 leaves out of scope
 * and Sec. 7 and 8 name as the way to widen the method's range (explicit
 * exponent management of the high part, input-dependent scaling, an overflow
 * guard):
 *   options      0, SGEMM_CUBE_OPT_PRESCALE or SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM.
 *                With PRESCALE, row i of A is
 *                multiplied by 2^p_i and column j of B by 2^q_j before the
 *                split, powers of two that bring the row's (column's) largest
 *                finite magnitude into [2^EA, 2^(EA+1)) with
 *                EA = min(14, 26 - s_b) (columns: [2^EB, 2^(EB+1)),
 *                EB = 14 - s_b, for scale = 2^s_b); the three-product GEMM
 *                runs on the scaled operands and C_ij = 2^-(p_i + q_j) C'_ij.
 *                The scaling is exact, so entries whose hi would be subnormal
 *                or would overflow FP16 are brought into the normal range as
 *                long as they are within ~28 (A) / ~17 (B, s = 2^11) binades
 *                of their row's (column's) largest entry.  A row (column) with
 *                no nonzero finite entry is left unscaled.  Costs one extra
 *                read of A and B and one read-write of C.
 *                With SPLIT_B_IN_GEMM (the fused split of Sec. 3.3 applied to
 *                B as well as A), the termwise GEMM kernel reads B as FP32 and
 *                splits it itself, each B tile once per tile row of C, instead
 *                of a split pass writing B's planes; A is split inside the
 *                kernel too where sgemm_cube_splits_a_in_gemm says so, so then
 *                no plane reaches HBM.  The result is that of the termwise
 *                order without the option, bit for bit.  Requires
 *                accum_order = SGEMM_CUBE_TERMWISE, no PRESCALE, range_report
 *                NULL, B 16-byte aligned, ldb and N multiples of 4, K a
 *                multiple of 64 and ldb < 2^22; otherwise
 *                SGEMM_CUBE_ERR_NOT_SUPPORTED.  The workspace is that of the
 *                call without the option.
 *   range_report NULL, or a 4-byte-aligned DEVICE pointer to one uint32 that
 *                receives, in stream order, the OR of the SGEMM_CUBE_RANGE_*
 *                classes found among the (pre-scaled) entries of A and B; 0 when
 *                M, N or K is 0.  Must not overlap A, B, C or the workspace.
 *   ws, ws_bytes at least sgemm_cube_ex_workspace_size(M, N, K, accum_order,
 *                options) bytes, 256-byte aligned; otherwise as sgemm_cube_ws.
 * Other arguments and errors as sgemm_cube_ws; unknown option bits ->
 * SGEMM_CUBE_ERR_INVALID_VALUE.
 */
int sgemm_cube_ex(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda, const float* B,
                  int64_t ldb, float* C, int64_t ldc, float scale, int accum_order,
                  unsigned options, void* ws, size_t ws_bytes, uint32_t* range_report,
                  hipStream_t stream);

/* Workspace bytes sgemm_cube_ex needs (0 for degenerate shapes or invalid
 * arguments). */
size_t sgemm_cube_ex_workspace_size(int64_t M, int64_t N, int64_t K, int accum_order,
                                    unsigned options);

/*
 * Two-phase form of sgemm_cube_ws, for callers that reuse a split operand
 * (for example a constant B) or time the two passes separately:
 *   sgemm_cube_prepare  splits A and B (Sec. 3.3) into the workspace;
 *   sgemm_cube_compute  runs the three-product MFMA GEMM and the FP32
 *                       reconstruction (Eq. recover_eqn, Sec. 4.5) from it.
 * sgemm_cube_ws(...) == prepare(...) followed by compute(...) on one stream.
 * M, N, K, the operands, scale, ws and ws_bytes follow sgemm_cube_ws; compute
 * must be called with the same M, N, K and scale as the prepare whose
 * workspace it reads (the library cannot check this).  prepare with A == NULL
 * (or B == NULL) leaves that operand's planes untouched, so one operand can
 * be re-split while the other's planes are kept.
 */
int sgemm_cube_prepare(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                       const float* B, int64_t ldb, float scale, void* ws, size_t ws_bytes,
                       hipStream_t stream);
int sgemm_cube_compute(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, float scale,
                       int accum_order, const void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * The second half of sgemm_cube_ws for a workspace whose B planes are
 * prepared (sgemm_cube_prepare with A == NULL): splits A (Sec. 3.3) and runs
 * the three-product GEMM (Eq. recover_eqn, Sec. 4.5), reading A as FP32.
 * Gives the same bits as sgemm_cube_ws(...), i.e. as prepare(A = NULL, B)
 * followed by prepare(A, B = NULL) and compute.
 * Where sgemm_cube_splits_a_in_gemm(M, N, K, A, lda, scale, accum_order)
 * returns 1, the split of A happens inside the GEMM kernel (in registers, with
 * the same arithmetic as the split kernels, so the result is the same) and the
 * A planes are not written unless the scaled kernel cannot run (some
 * |fl16(B)| * scale > 65504); no pass over A goes through HBM besides the
 * GEMM's own reads.  Otherwise A is split into the workspace first.
 * sgemm_cube, sgemm_cube_ws and sgemm_cube_noalloc follow the same rule.
 * M, N, K, A, lda, C, ldc, scale, accum_order, ws, ws_bytes and the errors
 * follow sgemm_cube_ws; C must not overlap A or the workspace.  Must use the
 * same M, N, K and scale as the prepare of B (the library cannot check this).
 * Afterwards the workspace's A planes are unspecified.
 */
int sgemm_cube_compute_a(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                         float* C, int64_t ldc, float scale, int accum_order, void* ws,
                         size_t ws_bytes, hipStream_t stream);

/*
 * The mirror image for a workspace whose A planes are prepared
 * (sgemm_cube_prepare with B == NULL), termwise order only: the GEMM kernel
 * reads B as FP32 and splits it itself (Sec. 3.3: the fused split, applied to
 * B; each B tile is split once per tile row of C), so B's planes are never
 * written.  Gives the same bits as sgemm_cube_ws(...) with the termwise
 * order.  On MI355X the in-kernel split costs the GEMM more than the split
 * pass of B it replaces, so sgemm_cube_prepare(A = NULL, B) followed by
 * sgemm_cube_compute is faster on the same A planes; this call measures that
 * trade-off and keeps B's planes out of the workspace.
 * accum_order other than SGEMM_CUBE_TERMWISE, or B not 16-byte aligned, ldb
 * or N not a multiple of 4, K not a multiple of 64, or ldb >= 2^22 ->
 * SGEMM_CUBE_ERR_NOT_SUPPORTED.  M, N, K, B, ldb, C, ldc, scale, ws,
 * ws_bytes and the other errors follow sgemm_cube_ws; C must not overlap B
 * or the workspace.  Must use the same M, N, K and scale as the prepare of A
 * (the library cannot check this).
 */
int sgemm_cube_compute_b(int64_t M, int64_t N, int64_t K, const float* B, int64_t ldb,
                         float* C, int64_t ldc, float scale, int accum_order, const void* ws,
                         size_t ws_bytes, hipStream_t stream);

/*
 * 1 when sgemm_cube, sgemm_cube_ws, sgemm_cube_noalloc and
 * sgemm_cube_compute_a with these arguments split A inside the GEMM kernel
 * instead of in a pass of its own, else 0 (also for arguments those calls
 * reject).  The in-kernel split repeats the split of each A tile for every
 * tile column of C, so it is chosen only where that costs less than the
 * pass over A: A 16-byte aligned, lda a multiple of 4 and below 2^22, K a
 * multiple of 64, and the elementwise order with N <= 4096 and
 * scale <= 2^15, or the termwise order with N <= 2048 (any scale).  Enqueues nothing and reads no device
 * memory (A is only looked at as an address).  Both choices give the same
 * bits.
 */
int sgemm_cube_splits_a_in_gemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                                float scale, int accum_order);

/*
 * Measurement hook for the pipeline ablation (Sec. 5.4 measures double
 * buffering against a single buffer): sgemm_cube_compute with the elementwise
 * order on the 256 x 256 kernel, 1 <= stages <= 2.  stages = 2 (the library's
 * own choice) copies the operands of the coming k-steps into LDS while a step
 * computes; stages = 1 issues the same copies at the end of each step and
 * waits for them there, so no copy overlaps the matrix instructions.  Both
 * use the same LDS slots and compute identical results.
 * accum_order other than SGEMM_CUBE_ELEMENTWISE ->
 * SGEMM_CUBE_ERR_NOT_SUPPORTED; stages outside 1..2 ->
 * SGEMM_CUBE_ERR_INVALID_VALUE; otherwise as sgemm_cube_compute
 * (when the range flag selects the unscaled fallback kernel, that kernel
 * keeps its own pipeline).
 */
int sgemm_cube_compute_stages(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc,
                              float scale, int accum_order, int stages, const void* ws,
                              size_t ws_bytes, hipStream_t stream);

/*
 * Measurement hook for the tile-shape and k-depth sweep (Sec. 6.3 sweeps the
 * block sizes b_m, b_k, b_n of its pipeline): sgemm_cube_compute with the
 * elementwise order on a generic kernel with tile_m x tile_n tiles of C and
 * block_k of k per double-buffered LDS stage, computed by workgroups of
 * `waves` waves, one of (tile_m, tile_n, block_k, waves) =
 *   (256, 256, 32, 4), (256, 128, 32, 4), (128, 256, 32, 4), (128, 128, 32, 4)
 *   with two workgroups per compute unit, (128, 128, 64, 4), and
 *   (256, 256, 32, 8): two waves per SIMD, each wave 128 x 64 of the tile.
 * Every configuration applies the library's MFMA operations to each
 * accumulator in the same order, so all of them, and sgemm_cube_compute,
 * give identical results.  The generic kernel keeps one code shape for every
 * tile (A fragments read at the start of each 32-wide k-step, B streamed per
 * 16-column block, the next stage's copies spread over the first k-step);
 * the library's own 256 x 256 kernel is scheduled by hand and is faster.
 * accum_order other than SGEMM_CUBE_ELEMENTWISE ->
 * SGEMM_CUBE_ERR_NOT_SUPPORTED; another (tile_m, tile_n, block_k, waves) ->
 * SGEMM_CUBE_ERR_INVALID_VALUE; otherwise as sgemm_cube_compute (scales
 * above 2^15, or a range flag that the split of B set, take the unscaled
 * fallback kernel as there).
 */
int sgemm_cube_compute_tile(int64_t M, int64_t N, int64_t K, float* C, int64_t ldc, float scale,
                            int accum_order, int tile_m, int tile_n, int block_k, int waves,
                            const void* ws, size_t ws_bytes, hipStream_t stream);

/* Device workspace in bytes that sgemm_cube_ws needs for this problem
 * (0 for degenerate shapes); 0 also for invalid arguments. */
size_t sgemm_cube_workspace_size(int64_t M, int64_t N, int64_t K, int accum_order);

/*
 * The two-component split alone (Sec. 3.3, Eq. recover_eqn), exposed so the
 * split can be checked bit for bit:
 *   hi[i*ldh + j] = fl16(X[i*ldx + j])
 *   lo[i*ldh + j] = fl16((X[i*ldx + j] - hi) * scale)
 * for 0 <= i < rows, 0 <= j < cols, as IEEE binary16 bit patterns.
 *   rows, cols >= 0; ldx >= max(1, cols); ldh >= max(1, cols);
 *   X, hi, lo device pointers, non-NULL when rows*cols > 0; hi and lo must not
 *   overlap each other or X.  scale as for sgemm_cube.
 */
int sgemm_cube_split(int64_t rows, int64_t cols, const float* X, int64_t ldx, uint16_t* hi,
                     uint16_t* lo, int64_t ldh, float scale, hipStream_t stream);

/*
 * Native-FP16 baseline (the HGEMM the paper compares against in Sec. 6.2):
 *   C = sum_k fl16(A[i,k]) fl16(B[k,j]), FP16 products accumulated in FP32,
 * i.e. the high-high term of Eq. recover_eqn alone.  Arguments and workspace
 * handling as for sgemm_cube.
 */
int sgemm_cube_hgemm(int64_t M, int64_t N, int64_t K, const float* A, int64_t lda,
                     const float* B, int64_t ldb, float* C, int64_t ldc, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* sgemm_cube_status_string(int status);

/* Size in elements of the elementwise k-block g of Eq. elementwise (32). On
 * the main path a block is one MFMA k-step: the running accumulator holds
 * scale * acc and each block's three products are summed into it by the
 * matrix unit in the order HH, XA, XB, each sum rounded once together with
 * the accumulator.  When scale > 2^15 (scale is then not a finite FP16 value)
 * or some |fl16(B)| * scale exceeds 65504 (scale * B_hi would overflow FP16)
 * the elementwise order runs unscaled with blocks of the same size instead:
 * HH into the accumulator, XA_g and XB_g summed separately,
 * acc = (acc + XA_g / s) + XB_g / s.  The cross-terms-first order uses the
 * same block size. */
int sgemm_cube_block_k(void);

#ifdef __cplusplus
}
#endif

#endif /* SGEMM_CUBE_H_ */
