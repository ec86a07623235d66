"""The calls that take no stream-ordered allocation -- sgemm_cube_ws with a
caller workspace, sgemm_cube_noalloc, and sgemm_cube_ex with the split of B
inside the GEMM -- captured into a HIP graph and
replayed.  The library enqueues kernels only (no memset, copy or allocation
on the stream), so a captured call must give, on every replay, the bits of
the same call made eagerly.  Each case is first called eagerly (which also
sets the kernels' LDS limits and looks up the fixed workspace's address), then
captured once and replayed three times; between the replays the output is
refilled with NaN and other eager work runs on the stream (another library
call with its own buffers), with synchronisations, and every replay is
checked against the eager result."""
import numpy as np
import pytest

import workloads
from tests.gpu_util import log, to_dev

pytestmark = pytest.mark.gpu

# (M, N, K, order): the in-kernel split of A (elementwise N <= 4096, termwise
# N <= 2048, K % 64 == 0), the plane path (N or K outside those), the range
# fallback (|B_hi| s > 65504) and cross-terms-first.
CASES = [(300, 260, 320, "elementwise"), (130, 4200, 128, "elementwise"),
         (300, 200, 256, "termwise"), (257, 300, 100, "termwise"),
         (200, 190, 192, "elementwise_range"), (150, 140, 320, "elementwise_cross_first")]


def _operands(M, N, K, order, seed):
    A, B = workloads.make_operands(M, N, K, seed, "normal")
    if order == "elementwise_range":
        B[3, 4] = np.float32(40.0)      # x 2^11 > 65504: the unscaled kernel runs
    return A, B


# The termwise call with B split inside the GEMM (sgemm_cube_ex with
# SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM): A split in the GEMM too (N <= 2048), and A
# through its split pass (N > 2048).
SPLIT_B_CASES = [(300, 204, 320, "termwise"), (130, 2100, 128, "termwise")]


PARAMS = ([(c, e) for c in CASES for e in ("ws", "noalloc")] +
          [(c, e) for c in SPLIT_B_CASES for e in ("ws", "noalloc", "ex_split_b")])


@pytest.mark.parametrize("case,entry", PARAMS,
                         ids=[f"{e}-{c[3]}-{c[0]}x{c[1]}x{c[2]}" for c, e in PARAMS])
def test_captured_call_replays_the_eager_bits(gpu, case, entry):
    import torch

    from paper_2507_23387_amd import binding

    M, N, K, order = case
    code = binding.ORDERS["elementwise" if order == "elementwise_range" else order]
    A, B = _operands(M, N, K, order, M + N + K)
    dA, dB = to_dev(A), to_dev(B)
    ws = binding.workspace(M, N, K)
    C = torch.full((M, N), float("nan"), device="cuda")

    def call(stream):
        if entry == "ws":
            return binding.sgemm_cube_ws(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                         C.data_ptr(), N, 2048.0, code, ws.data_ptr(),
                                         ws.numel(), stream)
        if entry == "ex_split_b":
            return binding.sgemm_cube_ex(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                         C.data_ptr(), N, 2048.0, code,
                                         binding.OPT_SPLIT_B_IN_GEMM, ws.data_ptr(),
                                         ws.numel(), None, stream)
        return binding.sgemm_cube_noalloc(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                          C.data_ptr(), N, 2048.0, code, stream)

    log(f"graph {entry} {order} {M}x{N}x{K}: eager")
    assert call(torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    ref = C.clone()
    assert bool(torch.isfinite(ref).all())

    # Other eager work between replays: a call with its own operands.
    A2, B2 = workloads.make_operands(64, 96, 128, 5, "uniform_pm1")
    dA2, dB2 = to_dev(A2), to_dev(B2)

    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    log(f"graph {entry} {order}: capture")
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            st = call(cap.cuda_stream)
    assert st == 0
    torch.cuda.current_stream().wait_stream(cap)
    for rep in range(3):
        C.fill_(float("nan"))
        torch.cuda.synchronize()
        log(f"graph {entry} {order}: replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int32), ref.view(torch.int32)), f"replay {rep}"
        other = binding.matmul(dA2, dB2, 2048.0, "termwise")
        torch.cuda.synchronize()
        assert bool(torch.isfinite(other).all())
    del g
