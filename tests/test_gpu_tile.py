"""The tile-shape and k-depth sweep kernel (sgemm_cube_compute_tile) against
the library's elementwise GEMM (sgemm_cube_compute) on the same prepared
workspace.  Every configuration applies the same MFMA operations to each
accumulator in the same order as the library's 256 x 256 kernel, so the
results must be identical bit for bit: ragged shapes that leave partial
tiles in both dimensions, a K that is not a multiple of the stage depth, a
B whose s B_hi overflows FP16 (range flag: both take the unscaled kernel),
a scale above 2^15 and one larger problem.  The library's result is itself
held to the oracle by the parity tests."""
import numpy as np
import pytest

import workloads
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1, 1), (300, 200, 320), (513, 700, 256), (129, 130, 96), (256, 256, 64)]


def _configs():
    from paper_2507_23387_amd import binding

    return binding.TILE_CONFIGS


def _compare(A, B, scale, configs):
    import torch

    from paper_2507_23387_amd import binding

    M, K = A.shape
    N = B.shape[1]
    dA, dB = to_dev(A), to_dev(B)
    stream = torch.cuda.current_stream().cuda_stream
    ws = binding.workspace(M, N, K)
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, scale,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    ref = torch.full((M, N), float("nan"), device="cuda")
    assert binding.sgemm_cube_compute(M, N, K, ref.data_ptr(), N, scale, binding.ELEMENTWISE,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    for cfg in configs:
        C = torch.full((M, N), float("nan"), device="cuda")
        assert binding.sgemm_cube_compute_tile(M, N, K, C.data_ptr(), N, scale,
                                               binding.ELEMENTWISE, *cfg, ws.data_ptr(),
                                               ws.numel(), stream) == 0
        torch.cuda.synchronize()
        assert torch.isfinite(ref).all()
        eq = torch.eq(C.view(torch.int32), ref.view(torch.int32))
        assert bool(eq.all()), f"{cfg}: {int((~eq).sum())} of {M * N} differ"


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_tile_configs_give_the_library_bits(gpu, shape):
    M, N, K = shape
    A, B = workloads.make_operands(M, N, K, 40 + M, "normal")
    log(f"tile sweep kernels vs library {M}x{N}x{K}")
    _compare(A, B, 2048.0, _configs())


def test_tile_configs_range_flag_and_large_scale(gpu):
    M, N, K = 200, 300, 192
    A, B = workloads.make_operands(M, N, K, 41, "uniform_pm1")
    B[7, 11] = np.float32(100.0)            # |B_hi| s > 65504 at s = 2^11: range flag
    log("tile sweep kernels: range flag, s = 2^11")
    _compare(A, B, 2048.0, _configs())
    A, B = workloads.make_operands(M, N, K, 42, "uniform_pm1")
    log("tile sweep kernels: s = 2^16 (unscaled kernel)")
    _compare(A, B, 65536.0, _configs())


def test_tile_configs_larger_problem(gpu):
    M, N, K = 2048, 1536, 1024
    A, B = workloads.make_operands(M, N, K, 43, "uniform_pm1")
    log(f"tile sweep kernels vs library {M}x{N}x{K}")
    _compare(A, B, 2048.0, _configs())
