"""sgemm_cube_noalloc: the entry point for callers that cannot allocate device
memory.  Its workspace is a fixed 64 MiB device array inside the library; the
kernels are the ones sgemm_cube runs, so its output must equal sgemm_cube's
bit for bit, and meet the oracle's bar (|C - C_oracle| <= 2 K 2^-24 |A||B|).
Two calls in a row, the second on a smaller problem, check that nothing of
the first call's contents in the shared array leaks into the second; a
problem whose workspace exceeds the array is refused before any device work."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu

ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]
NOT_SUPPORTED = 2


def _noalloc(dA, dB, scale, order):
    import torch

    from paper_2507_23387_amd import binding

    M, K = dA.shape
    N = dB.shape[1]
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    st = binding.sgemm_cube_noalloc(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                                    scale, binding.ORDERS[order],
                                    torch.cuda.current_stream().cuda_stream)
    assert st == 0, binding.sgemm_cube_status_string(st)
    return C


@pytest.mark.parametrize("order", ORDERS)
def test_noalloc_matches_sgemm_cube_on_two_calls(gpu, order):
    import torch

    from paper_2507_23387_amd import binding

    kb = binding.sgemm_cube_block_k()
    # The first problem's planes fill most of the array (47 MiB of 64); the
    # second is smaller and ragged in every dimension.
    shapes = [(2000, 1900, 3000), (300, 200, 129)]
    for n, (M, N, K) in enumerate(shapes):
        assert binding.sgemm_cube_workspace_size(M, N, K) <= binding.NOALLOC_WORKSPACE_BYTES
        A, B = workloads.make_operands(M, N, K, 40 + n, "normal")
        dA, dB = to_dev(A), to_dev(B)
        log(f"noalloc {order} call {n} {M}x{N}x{K}")
        C = _noalloc(dA, dB, 2048.0, order)
        ref = binding.matmul(dA, dB, 2048.0, order)
        torch.cuda.synchronize()
        Cn = C.cpu().numpy()
        assert np.isfinite(Cn).all()
        assert torch.equal(C, ref), f"call {n}: differs from sgemm_cube"
        rows = np.arange(M) if M <= 300 else workloads.sample_rows(M, 24, n)
        Co = oracle.sgemm_rows(A, B, rows, 2048.0, order, kb=kb)
        assert_parity(Cn[rows], Co, K, abs_ab(A, B, rows), f"noalloc {order} call {n}")


def test_noalloc_refuses_problems_beyond_its_array(gpu):
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 4096, 4096, 2049      # 256 + 4 * 2112 * 8192 bytes > 64 MiB
    assert binding.sgemm_cube_workspace_size(M, N, K) > binding.NOALLOC_WORKSPACE_BYTES
    A = torch.zeros((M, K), device="cuda")
    B = torch.zeros((K, N), device="cuda")
    C = torch.full((M, N), 7.0, device="cuda")
    log("noalloc too large")
    st = binding.sgemm_cube_noalloc(M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N,
                                    2048.0, 0, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == NOT_SUPPORTED
    assert bool((C == 7.0).all())


def test_noalloc_degenerate_shapes(gpu):
    import torch

    from paper_2507_23387_amd import binding

    stream = torch.cuda.current_stream().cuda_stream
    C = torch.full((5, 6), float("nan"), device="cuda")
    A = torch.empty((5, 0), device="cuda")
    B = torch.empty((0, 6), device="cuda")
    log("noalloc K=0")
    assert binding.sgemm_cube_noalloc(5, 6, 0, A.data_ptr(), 1, B.data_ptr(), 6, C.data_ptr(), 6,
                                      2048.0, 1, stream) == 0
    torch.cuda.synchronize()
    assert bool((C == 0).all())
