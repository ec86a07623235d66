"""The copy/compute overlap hook (sgemm_cube_compute_stages): the setting
without overlap (stages = 1) computes the same bits as the default pipeline
(stages = 2), and those bits meet the parity bar against the oracle."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu


def _kb():
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


def _run(A, B, stages_list, scale=2048.0):
    import torch

    from paper_2507_23387_amd import binding

    M, K = A.shape
    N = B.shape[1]
    dA, dB = to_dev(A), to_dev(B)
    ws = binding.workspace(M, N, K)
    stream = torch.cuda.current_stream().cuda_stream
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, scale,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    out = {}
    for st in stages_list:
        C = torch.empty((M, N), dtype=torch.float32, device="cuda")
        if st == 0:
            rc = binding.sgemm_cube_compute(M, N, K, C.data_ptr(), N, scale, 0, ws.data_ptr(),
                                            ws.numel(), stream)
        else:
            rc = binding.sgemm_cube_compute_stages(M, N, K, C.data_ptr(), N, scale, 0, st,
                                                   ws.data_ptr(), ws.numel(), stream)
        assert rc == 0
        out[st] = C
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("shape", [(1, 1, 1), (300, 257, 515), (513, 640, 2048)],
                         ids=lambda s: "x".join(map(str, s)))
def test_every_stage_count_computes_the_same_bits(gpu, shape):
    M, N, K = shape
    A, B = workloads.make_operands(M, N, K, M + 2 * N + K, "normal")
    log(f"pipeline stages {shape}")
    res = _run(A, B, [0, 1, 2])
    for st in (1, 2):
        assert np.array_equal(res[st].view(np.uint32), res[0].view(np.uint32)), st
    Co = oracle.sgemm(A, B, 2048.0, "elementwise", kb=_kb())
    assert_parity(res[1], Co, K, abs_ab(A, B), f"stages {shape}")


def test_stage_counts_on_the_4096_cube_sampled_rows(gpu):
    w = workloads.get("c2")
    A, B = workloads.workload_operands(w)
    log("pipeline stages c2")
    res = _run(A, B, [0, 1])
    assert np.array_equal(res[1].view(np.uint32), res[0].view(np.uint32))
    rows = workloads.sample_rows(w.M, 8, w.seed)
    Co = oracle.sgemm_rows(A, B, rows, 2048.0, "elementwise", kb=_kb())
    assert_parity(res[1][rows], Co, w.K, abs_ab(A, B, rows), "stages c2")
