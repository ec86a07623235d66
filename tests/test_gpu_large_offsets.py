"""Large operands: every plane of A past 4 GiB, FP32 A past 8 GiB.

M = 69632, N = 256, K = 32768: A is 9.1 GB of FP32, and each of its FP16
planes 4.56 GB, so the split kernels' stores, the GEMM's copies from the
planes and the in-kernel split's copies from FP32 A all reach offsets beyond
2^32 bytes inside one operand.  Both orders run on the library's default path
(A split inside the GEMM kernel: N <= 2048) and on the plane path
(sgemm_cube_prepare + sgemm_cube_compute), which must give the same bits;
one row in every 256-row band of C (272 rows, offsets rotating) is held to
the oracle with the parity bar and the discriminator.  C is prefilled with
NaN, so the all-finite check proves that every entry was written.

A is drawn on the GPU from a seeded torch generator (uniform in [-1, 1)); the
oracle gets the sampled rows copied back."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_discriminates, assert_parity, band_rows

pytestmark = pytest.mark.gpu

M, N, K = 69632, 256, 32768


def _kb():
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


@pytest.fixture(scope="module")
def operands():
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(71)
    dA = torch.rand((M, K), generator=g, device="cuda", dtype=torch.float32) * 2.0 - 1.0
    rng = np.random.default_rng(72)
    B = rng.uniform(-1.0, 1.0, (K, N)).astype(np.float32)
    dB = to_dev(B)
    rows = band_rows(M, 73)
    A_rows = dA[torch.from_numpy(rows).to("cuda")].cpu().numpy()
    yield dA, dB, B, rows, A_rows
    del dA, dB
    torch.cuda.empty_cache()


@pytest.mark.parametrize("order", ["elementwise", "termwise"])
def test_planes_beyond_4_gib(gpu, operands, order):
    import torch

    from paper_2507_23387_amd import binding

    dA, dB, B, rows, A_rows = operands
    code = binding.ORDERS[order]
    # Each A plane (M x K halves) is past 4 GiB; the workspace holds two of them.
    assert M * K * 2 > (1 << 32)
    assert binding.sgemm_cube_workspace_size(M, N, K, code) > 2 * M * K * 2
    assert binding.sgemm_cube_splits_a_in_gemm(M, N, K, dA.data_ptr(), K, 2048.0, code) == 1
    stream = torch.cuda.current_stream().cuda_stream
    log(f"large operands {M}x{N}x{K} {order}: default path")
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    assert binding.sgemm_cube(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                              2048.0, code, stream) == 0
    log(f"large operands {order}: plane path")
    ws = binding.workspace(M, N, K)
    Cp = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, 2048.0,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    assert binding.sgemm_cube_compute(M, N, K, Cp.data_ptr(), N, 2048.0, code, ws.data_ptr(),
                                      ws.numel(), stream) == 0
    torch.cuda.synchronize()
    del ws
    assert bool(torch.isfinite(C).all())
    assert torch.equal(C.view(torch.int32), Cp.view(torch.int32))
    got = C[torch.from_numpy(rows).to("cuda")].cpu().numpy()
    del C, Cp
    sel = np.arange(len(rows))
    Co = oracle.sgemm_rows(A_rows, B, sel, 2048.0, order, kb=_kb())
    Ch = oracle.sgemm_rows(A_rows, B, sel, 2048.0, "hi_only", kb=_kb())
    assert_parity(got, Co, K, abs_ab(A_rows, B), f"large {order}")
    assert_discriminates(got, Co, Ch, f"large {order}")
