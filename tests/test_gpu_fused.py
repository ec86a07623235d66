"""The elementwise GEMM that splits A in registers (the 256 x 256 kernel with
its A copies taken from FP32 A) against the path through the split kernels
and the A planes (sgemm_cube_prepare + sgemm_cube_compute).

sgemm_cube, sgemm_cube_ws and sgemm_cube_compute_a take the fused path where
sgemm_cube_splits_a_in_gemm says so (the elementwise order, N <= 4096,
s <= 2^15, A 16-byte aligned, lda a multiple of 4, K a multiple of 64);
otherwise they split A into the workspace first.  Both
paths apply the same MFMA operations to every accumulator in the same order
(HH, XA, XB per block), so when the in-register split produces the same bits
as the split kernels (which the split tests pin to the oracle bit for bit)
the results are identical bit for bit; the fused result must also meet the
parity bar against the oracle.  When s * B_hi overflows FP16 the fused kernel
writes the A planes itself and the unscaled kernel runs: again bit-identical
to the planes path."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu

# K a multiple of 64 and N <= 4096 (fused), with ragged M and N; the last
# three take the planes path (K not a multiple of 64, N above 4096) and must
# agree all the same.
SHAPES = [(1, 1, 64), (17, 33, 128), (129, 700, 64), (256, 256, 256), (300, 200, 1024),
          (513, 640, 192), (200, 129, 4096), (40, 4096, 128), (17, 33, 68), (300, 200, 1000),
          (40, 4097, 128)]
FUSED = {shape: shape[2] % 64 == 0 and shape[1] <= 4096 for shape in SHAPES}


def _kb():
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


def _paths(A, B, scale=2048.0, lda=None, order="elementwise"):
    """(C through sgemm_cube_ws, C through prepare(A = NULL, B) + compute_a(A),
    C through prepare(A, B) + compute on the planes)."""
    import torch

    from paper_2507_23387_amd import binding

    M, K = A.shape
    N = B.shape[1]
    lda = K if lda is None else lda
    buf = torch.zeros((M * lda + 4,), dtype=torch.float32, device="cuda")
    dA = buf[:M * lda].view(M, lda)
    dA[:, :K].copy_(torch.from_numpy(A))
    dB = to_dev(B)
    stream = torch.cuda.current_stream().cuda_stream
    code = binding.ORDERS[order]
    ws = binding.workspace(M, N, K)
    n = ws.numel()
    C = [torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda") for _ in range(3)]
    assert binding.sgemm_cube_ws(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), N, C[0].data_ptr(),
                                 N, scale, code, ws.data_ptr(), n, stream) == 0
    assert binding.sgemm_cube_prepare(M, N, K, None, lda, dB.data_ptr(), N, scale,
                                      ws.data_ptr(), n, stream) == 0
    assert binding.sgemm_cube_compute_a(M, N, K, dA.data_ptr(), lda, C[1].data_ptr(), N, scale,
                                        code, ws.data_ptr(), n, stream) == 0
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), N, scale,
                                      ws.data_ptr(), n, stream) == 0
    assert binding.sgemm_cube_compute(M, N, K, C[2].data_ptr(), N, scale, code,
                                      ws.data_ptr(), n, stream) == 0
    torch.cuda.synchronize()
    return [c.cpu().numpy() for c in C]


def _both_paths(A, B, scale=2048.0, lda=None, order="elementwise"):
    """(fused C, planes C), after checking that sgemm_cube_ws and compute_a
    agree bit for bit."""
    Cw, Ca, Cp = _paths(A, B, scale, lda, order)
    _same_bits(Cw, Ca)
    return Cw, Cp


def _same_bits(X, Y):
    """Bitwise equal, NaNs compared by class (their payloads may differ)."""
    nx, ny = np.isnan(X), np.isnan(Y)
    assert np.array_equal(nx, ny)
    assert np.array_equal(X[~nx].view(np.uint32), Y[~ny].view(np.uint32))


def _mixed_operands(M, N, K, seed):
    """N(0,1) operands with rows and columns of A and B moved to other binades
    (FP16-subnormal hi at 2^-17, large values at 2^9), so the in-register
    split meets normal, subnormal and large hi words."""
    A, B = workloads.make_operands(M, N, K, seed, "normal")
    A[::5] *= np.float32(2.0**-17)
    A[1::7] *= np.float32(2.0**9)
    B[:, ::3] *= np.float32(2.0**-3)
    return A, B


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_fused_split_gives_the_bits_of_the_planes_path(gpu, shape):
    M, N, K = shape
    A, B = _mixed_operands(M, N, K, M + 3 * N + K)
    log(f"fused vs planes {M}x{N}x{K}")
    from paper_2507_23387_amd import binding

    dA = to_dev(A)
    assert binding.sgemm_cube_splits_a_in_gemm(M, N, K, dA.data_ptr(), K, 2048.0,
                                               binding.ELEMENTWISE) == int(FUSED[shape])
    Cf, Cp = _both_paths(A, B)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "elementwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"fused {shape}")


def test_identity_b_reconstructs_every_split_of_a(gpu):
    """With B = I (exact in FP16, B_lo = 0) each output is the rounded
    s-scaled sum s hi + lo of one entry of A, divided by s: a change in any
    bit of the in-register split of A changes C.  Compared with the same sum
    formed from the oracle's split."""
    M = K = N = 512
    rng = np.random.default_rng(41)
    mant = rng.uniform(1.0, 2.0, size=(M, K))
    expo = rng.integers(-26, 14, size=(M, K))
    A = (np.where(rng.random((M, K)) < 0.5, -1.0, 1.0) * np.ldexp(mant, expo)).astype(np.float32)
    B = np.eye(K, N, dtype=np.float32)
    log("fused identity B")
    Cf, Cp = _both_paths(A, B)
    _same_bits(Cf, Cp)
    hi, lo = oracle.split(A, 2048.0)
    hi64 = oracle.f16_to_f32(hi).astype(np.float64)
    lo64 = oracle.f16_to_f32(lo).astype(np.float64)
    # s hi + lo has at most 24 significant bits where lo's last bit is within
    # 23 bits of s hi's leading bit; there the sum is exact and so is C.
    want = (hi64 * 2048.0 + lo64).astype(np.float32).astype(np.float64) / 2048.0
    exact = np.abs(want - (hi64 + lo64 / 2048.0)) == 0
    assert exact.mean() > 0.5
    got = Cf.astype(np.float64)
    assert np.array_equal(got[exact] == 0, want[exact] == 0)
    nz = exact & (want != 0)
    assert np.array_equal(got[nz], want[nz])


@pytest.mark.parametrize("edge", ["scaled_limit", "fallback"])
def test_fused_range_switch(gpu, edge):
    """|B_hi| s at 65504 keeps the scaled kernel; one FP16 ulp above makes the
    fused kernel write the A planes and the unscaled kernel compute C."""
    M, N, K = 300, 260, 256
    A, B = workloads.make_operands(M, N, K, 22, "uniform_pm1")
    B[5, 7] = 31.984375 if edge == "scaled_limit" else 32.0
    log(f"fused range switch {edge}")
    Cf, Cp = _both_paths(A, B)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "elementwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"fused range switch {edge}")


@pytest.mark.parametrize("s_b", [0, 13, 15])
def test_fused_split_at_other_scales(gpu, s_b):
    """The in-kernel split at s = 1, 2^13 and 2^15 (the largest scale the
    scaled kernel takes; |B| < 1 keeps the range flag clear), with A values
    whose hi is FP16-subnormal and whose scaled residual is subnormal."""
    M, N, K = 257, 300, 192
    A, B = workloads.make_operands(M, N, K, 30 + s_b, "uniform_pm1")
    A[::3] *= np.float32(2.0**-16)
    B *= np.float32(0.999)
    scale = 2.0**s_b
    log(f"fused split at s = 2^{s_b}")
    Cf, Cp = _both_paths(A, B, scale)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, scale, "elementwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"fused s=2^{s_b}")


def test_fused_non_finite_inputs(gpu):
    M, N, K = 40, 50, 128
    A, B = workloads.make_operands(M, N, K, 23, "uniform_pm1")
    A[3, 5] = 70000.0      # hi overflows
    A[7, 9] = -np.inf
    A[20, 21] = 32784.0    # lo overflows with s = 2^12
    A[30, 127] = np.nan    # in the last k-step
    A[31, 64] = -0.0
    A[32, 65] = 2.0**-140  # FP32 subnormal
    log("fused non-finite")
    Cf, Cp = _both_paths(A, B, 4096.0)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 4096.0, "elementwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), "fused non-finite")


def test_compute_a_after_prepare_of_b(gpu):
    """prepare(A = NULL, B) + compute_a(A) == sgemm_cube_ws, for every order
    (the orders other than elementwise split A into the workspace first)."""
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 300, 257, 516
    A, B = workloads.make_operands(M, N, K, 24, "normal")
    dA, dB = to_dev(A), to_dev(B)
    stream = torch.cuda.current_stream().cuda_stream
    for order in ("elementwise", "termwise", "elementwise_cross_first"):
        log(f"compute_a {order}")
        code = binding.ORDERS[order]
        ws = binding.workspace(M, N, K)
        C1 = binding.matmul(dA, dB, 2048.0, order)
        C2 = torch.empty_like(C1)
        assert binding.sgemm_cube_prepare(M, N, K, None, K, dB.data_ptr(), N, 2048.0,
                                          ws.data_ptr(), ws.numel(), stream) == 0
        assert binding.sgemm_cube_compute_a(M, N, K, dA.data_ptr(), K, C2.data_ptr(), N, 2048.0,
                                            code, ws.data_ptr(), ws.numel(), stream) == 0
        torch.cuda.synchronize()
        assert torch.equal(C1, C2)


def test_padded_lda_takes_the_fused_path_bitwise(gpu):
    """lda = K + 4 (rows 16-byte aligned) on ragged M and N, and lda = K + 1
    (the planes path): both equal the planes path bit for bit."""
    M, N, K = 133, 71, 320
    A, B = _mixed_operands(M, N, K, 31)
    for lda in (K + 4, K + 1):
        log(f"fused padded lda {lda}")
        Cf, Cp = _both_paths(A, B, lda=lda)
        _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "elementwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), "padded lda")


def test_unaligned_a_splits_into_the_workspace(gpu):
    """compute_a with A misaligned by one element, or K not a multiple of 4,
    splits A into the workspace first; the result equals sgemm_cube's (which
    takes the fused path for the aligned copy at K = 256)."""
    import torch

    from paper_2507_23387_amd import binding

    for (M, N, K, off) in ((130, 140, 256, 1), (130, 140, 258, 0)):
        A, B = workloads.make_operands(M, N, K, 25, "normal")
        buf = torch.zeros(off + M * K, dtype=torch.float32, device="cuda")
        Av = buf[off:].view(M, K)
        Av.copy_(torch.from_numpy(A))
        dB = to_dev(B)
        stream = torch.cuda.current_stream().cuda_stream
        log(f"compute_a unaligned {M}x{N}x{K} off {off}")
        ws = binding.workspace(M, N, K)
        C1 = torch.empty((M, N), dtype=torch.float32, device="cuda")
        assert binding.sgemm_cube_prepare(M, N, K, None, K, dB.data_ptr(), N, 2048.0,
                                          ws.data_ptr(), ws.numel(), stream) == 0
        assert binding.sgemm_cube_compute_a(M, N, K, Av.data_ptr(), K, C1.data_ptr(), N, 2048.0,
                                            binding.ELEMENTWISE, ws.data_ptr(), ws.numel(),
                                            stream) == 0
        C2 = binding.matmul(to_dev(A), dB, 2048.0, "elementwise")
        torch.cuda.synchronize()
        assert torch.equal(C1, C2)


# --- termwise: the 256 x 128 kernel that splits A in registers ----------------

TW_SHAPES = [(1, 1, 64), (17, 33, 128), (129, 700, 64), (300, 200, 1024), (513, 1024, 192),
             (200, 129, 4096), (40, 2048, 128), (300, 200, 1000), (40, 2049, 128)]


@pytest.mark.parametrize("shape", TW_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_termwise_fused_split_gives_the_bits_of_the_planes_path(gpu, shape):
    """Termwise (Eq. termwise) with the split of A inside the 256 x 128
    kernel: the same bits as the planes path, and parity with the oracle.
    K a multiple of 64 and N <= 2048 take the fused kernel; the last two
    shapes take the planes path and must agree all the same."""
    from paper_2507_23387_amd import binding

    M, N, K = shape
    A, B = _mixed_operands(M, N, K, 7 * M + N + K)
    dA = to_dev(A)
    fused = K % 64 == 0 and N <= 2048
    assert binding.sgemm_cube_splits_a_in_gemm(M, N, K, dA.data_ptr(), K, 2048.0,
                                               binding.TERMWISE) == int(fused)
    log(f"termwise fused vs planes {M}x{N}x{K}")
    Cf, Cp = _both_paths(A, B, order="termwise")
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "termwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"termwise fused {shape}")


@pytest.mark.parametrize("s_b", [0, 13, 20, 24])
def test_termwise_fused_split_at_other_scales(gpu, s_b):
    """Termwise needs no s B_hi, so the in-kernel split runs at every scale,
    2^24 included; subnormal hi and scaled residuals on a third of the rows."""
    M, N, K = 257, 300, 192
    A, B = workloads.make_operands(M, N, K, 60 + s_b, "uniform_pm1")
    A[::3] *= np.float32(2.0**-16)
    scale = 2.0**s_b
    log(f"termwise fused split at s = 2^{s_b}")
    Cf, Cp = _both_paths(A, B, scale, order="termwise")
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, scale, "termwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"termwise fused s=2^{s_b}")


def test_termwise_fused_non_finite_and_padded_lda(gpu):
    M, N, K = 133, 71, 320
    A, B = workloads.make_operands(M, N, K, 61, "uniform_pm1")
    A[3, 5] = 70000.0      # hi overflows
    A[7, 9] = np.inf
    A[11, 300] = np.nan
    log("termwise fused: non-finite inputs, lda = K + 12")
    Cf, Cp = _both_paths(A, B, lda=K + 12, order="termwise")
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "termwise", kb=_kb())
    _same_bits(np.isfinite(Cf).astype(np.float32), np.isfinite(Co).astype(np.float32))
