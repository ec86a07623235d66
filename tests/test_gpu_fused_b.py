"""The termwise GEMM that splits B inside the kernel (sgemm_cube_ex with
SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM, and sgemm_cube_compute_b on prepared A
planes) against the same call without the option.

With the option the 256 x 128 termwise kernel copies FP32 rows of B into LDS
and the workgroup splits them into the tiled B planes of the stage itself;
A is split inside the kernel as well where the library does that for
termwise (N <= 2048, A 16-byte aligned, lda a multiple of 4, K a multiple
of 64), otherwise by the split pass.  Everything after the split is the
planes path, so the result must equal the call without the option bit for
bit (NaNs by class), and meet the parity bar against the oracle.  Shapes
cover ragged M, N a multiple of 4 but not of 128 (the last tile column
copies repeated columns past N), both routes for A, padded lda, ldb and ldc,
every scale from 2^0 to 2^24, and non-finite, FP16-overflowing and
subnormal entries of B."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, padded, to_dev
from tests.helpers import abs_ab, assert_discriminates, assert_parity, band_rows

pytestmark = pytest.mark.gpu

SHAPES = [(1, 4, 64), (17, 36, 128), (129, 700, 64), (300, 200, 1024), (513, 1024, 192),
          (200, 132, 4096), (40, 2048, 128), (256, 128, 64), (40, 2052, 128),
          (300, 2500, 320)]


def _kb():
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


def _same_bits(X, Y):
    """Bitwise equal, NaNs compared by class (their payloads may differ)."""
    nx, ny = np.isnan(X), np.isnan(Y)
    assert np.array_equal(nx, ny)
    assert np.array_equal(X[~nx].view(np.uint32), Y[~ny].view(np.uint32))


def _mixed_operands(M, N, K, seed):
    """N(0,1) operands with columns of B and rows of A moved to other binades
    (FP16-subnormal hi at 2^-17, large values at 2^9)."""
    A, B = workloads.make_operands(M, N, K, seed, "normal")
    B[:, ::5] *= np.float32(2.0**-17)
    B[:, 1::7] *= np.float32(2.0**9)
    A[::3] *= np.float32(2.0**-3)
    return A, B


def _with_and_without(A, B, scale=2048.0, pads=(0, 0, 0), a_offset=0):
    """(C with the option, C without), each written into a NaN-filled C with
    ldc = N + pads[2]; the columns past N and the rows past M stay NaN.  The
    third route, sgemm_cube_prepare(A, B = NULL) + sgemm_cube_compute_b, is
    checked against the first bit for bit here."""
    import torch

    from paper_2507_23387_amd import binding

    M, K = A.shape
    N = B.shape[1]
    lda, ldb, ldc = K + pads[0], N + pads[1], N + pads[2]
    _, dA = padded(A, lda, offset=a_offset)
    _, dB = padded(B, ldb)
    stream = torch.cuda.current_stream().cuda_stream
    opt = binding.OPT_SPLIT_B_IN_GEMM
    out = []
    for options in (opt, 0):
        nbytes = binding.sgemm_cube_ex_workspace_size(M, N, K, binding.TERMWISE, options)
        ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device="cuda")
        cbuf, dC = padded(np.full((M, N), np.nan, np.float32), ldc)
        cbuf.fill_(float("nan"))
        st = binding.sgemm_cube_ex(M, N, K, dA.data_ptr(), lda, dB.data_ptr(), ldb,
                                   dC.data_ptr(), ldc, scale, binding.TERMWISE, options,
                                   ws.data_ptr(), nbytes, None, stream)
        assert st == 0, binding.sgemm_cube_status_string(st)
        torch.cuda.synchronize()
        full = cbuf.cpu().numpy()
        assert np.isnan(full[:M * ldc].reshape(M, ldc)[:, N:]).all()
        assert np.isnan(full[M * ldc:]).all()
        out.append(full[:M * ldc].reshape(M, ldc)[:, :N].copy())
    ws = binding.workspace(M, N, K)
    cbuf, dC = padded(np.full((M, N), np.nan, np.float32), ldc)
    cbuf.fill_(float("nan"))
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), lda, None, ldb, scale,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    st = binding.sgemm_cube_compute_b(M, N, K, dB.data_ptr(), ldb, dC.data_ptr(), ldc, scale,
                                      binding.TERMWISE, ws.data_ptr(), ws.numel(), stream)
    assert st == 0, binding.sgemm_cube_status_string(st)
    torch.cuda.synchronize()
    full = cbuf.cpu().numpy()
    assert np.isnan(full[:M * ldc].reshape(M, ldc)[:, N:]).all()
    _same_bits(full[:M * ldc].reshape(M, ldc)[:, :N], out[0])
    return out[0], out[1]


def _fused_a(M, N, K, a_offset=0, lda=None):
    return N <= 2048 and K % 64 == 0 and a_offset % 4 == 0 and (lda or K) % 4 == 0


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_split_b_in_gemm_gives_the_bits_of_the_planes_path(gpu, shape):
    from paper_2507_23387_amd import binding

    M, N, K = shape
    A, B = _mixed_operands(M, N, K, 5 * M + N + 3 * K)
    log(f"split of B in the GEMM vs planes {M}x{N}x{K} "
        f"(A {'in the GEMM' if _fused_a(M, N, K) else 'split pass'})")
    import torch

    dA = torch.from_numpy(A).cuda()
    assert binding.sgemm_cube_splits_a_in_gemm(M, N, K, dA.data_ptr(), K, 2048.0,
                                               binding.TERMWISE) == int(_fused_a(M, N, K))
    Cf, Cp = _with_and_without(A, B)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "termwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"split B in GEMM {shape}")


@pytest.mark.parametrize("s_b", [0, 13, 20, 24])
def test_split_b_in_gemm_at_other_scales(gpu, s_b):
    """Termwise needs no s B_hi, so the in-kernel split of B runs at every
    scale; FP16-subnormal hi and scaled residuals in a third of B's columns."""
    M, N, K = 257, 300, 192
    A, B = workloads.make_operands(M, N, K, 80 + s_b, "uniform_pm1")
    B[:, ::3] *= np.float32(2.0**-16)
    scale = 2.0**s_b
    log(f"split of B in the GEMM at s = 2^{s_b}")
    Cf, Cp = _with_and_without(A, B, scale)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, scale, "termwise", kb=_kb())
    assert_parity(Cf, Co, K, abs_ab(A, B), f"split B in GEMM s=2^{s_b}")


@pytest.mark.parametrize("a_offset", [0, 1])
def test_split_b_in_gemm_non_finite_and_padding(gpu, a_offset):
    """Non-finite, FP16-overflowing, FP32-subnormal and signed-zero entries of
    B, padded lda, ldb and ldc; a_offset = 1 misaligns A, which then takes
    the split pass while B is still split in the GEMM."""
    M, N, K = 133, 72, 320
    A, B = workloads.make_operands(M, N, K, 62 + a_offset, "uniform_pm1")
    B[5, 3] = 70000.0      # hi overflows
    B[9, 7] = np.inf
    B[300, 11] = np.nan    # in the last k-step
    B[64, 31] = -0.0
    B[65, 32] = 2.0**-140  # FP32 subnormal
    B[2, 71] = -np.inf     # the last column
    log(f"split of B in the GEMM: non-finite B, padded strides, A offset {a_offset}")
    Cf, Cp = _with_and_without(A, B, pads=(12, 8, 5), a_offset=a_offset)
    _same_bits(Cf, Cp)
    Co = oracle.sgemm(A, B, 2048.0, "termwise", kb=_kb())
    assert not np.isfinite(Co[:, [3, 7, 11, 71]]).any()
    assert_parity(Cf, Co, K, abs_ab(A, B), "split B in GEMM, non-finite B")


def test_split_b_in_gemm_larger_problem(gpu):
    """Several rounds of tiles along M and N, both operands split in the
    GEMM, uniform data."""
    M, N, K = 2304, 1920, 1024
    A, B = workloads.make_operands(M, N, K, 90, "uniform_pm1")
    log(f"split of B in the GEMM {M}x{N}x{K}")
    Cf, Cp = _with_and_without(A, B)
    _same_bits(Cf, Cp)
    rows = np.arange(0, M, 97)
    Co = oracle.sgemm_rows(A, B, rows, 2048.0, "termwise", kb=_kb())
    assert_parity(Cf[rows], Co, K, abs_ab(A[rows], B), "split B in GEMM, sampled rows")


@pytest.mark.parametrize("name", ["c5", "c2", "c4"])
def test_split_b_in_gemm_full_size_workloads(gpu, name):
    """The termwise workloads at full size with B split in the GEMM kernel
    (16384 x 1024 x 8192: A too; 4096^3 and 4096 x 4096 x 16384: A by its
    split pass), in the launch configuration of bench.py --split-b-in-gemm.
    C is prefilled with NaN, so the all-finite check shows every entry was
    written; one row in every 256-row band is held to the oracle with the
    parity bar and the discriminator against the hi-only product."""
    import torch

    from paper_2507_23387_amd import binding

    w = workloads.get(name)
    A, B = workloads.workload_operands(name)
    scale = 2.0**11
    log(f"split of B in the GEMM, workload {w.name}")
    dA, dB = to_dev(A), to_dev(B)
    Cd = torch.full((w.M, w.N), float("nan"), dtype=torch.float32, device="cuda")
    binding.matmul_ex(dA, dB, scale, "termwise", split_b_in_gemm=True, out=Cd)
    torch.cuda.synchronize()
    C = Cd.cpu().numpy()
    del dA, dB, Cd
    assert np.isfinite(C).all()
    rows = band_rows(w.M, w.seed + 29)
    Co = oracle.sgemm_rows(A, B, rows, scale, "termwise", kb=_kb())
    Ch = oracle.sgemm_rows(A, B, rows, scale, "hi_only", kb=_kb())
    assert_parity(C[rows], Co, w.K, abs_ab(A, B, rows), f"{name} split B in GEMM")
    assert_discriminates(C[rows], Co, Ch, f"{name} split B in GEMM")
