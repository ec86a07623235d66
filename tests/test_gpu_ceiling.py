"""The diagnostic register-only MFMA loop (sgemm_cube_mfma_loop): with every
operand 0.5 each v_mfma_f32_16x16x32_f16 adds 32 * 0.25 = 8 to each of the 4
values a lane holds of an accumulator, so after `iters` iterations a thread's
64 accumulators sum to 64 * 4 * 8 * iters = 2048 * iters, exactly in FP32."""
import numpy as np
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu


def _run(torch, sgc, workgroups, iters, values):
    ops = torch.from_numpy(values.astype(np.float16).view(np.int16).copy()).cuda()
    out = torch.full((workgroups * 256,), -1.0, dtype=torch.float32, device="cuda")
    st = sgc.sgemm_cube_mfma_loop(workgroups, iters, ops.data_ptr(), ops.numel() * 2,
                                  out.data_ptr(), out.numel() * 4,
                                  torch.cuda.current_stream().cuda_stream)
    assert st == 0, st
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("workgroups,iters", [(1, 1), (8, 100), (300, 8192)])
def test_constant_operands_give_exact_sum(gpu, workgroups, iters):
    import torch

    import paper_2507_23387_amd as sgc

    log(f"mfma loop workgroups={workgroups} iters={iters}")
    out = _run(torch, sgc, workgroups, iters, np.full(32768, 0.5))
    assert np.all(out == 2048.0 * iters)


def test_zero_operands_give_zero(gpu):
    import torch

    import paper_2507_23387_amd as sgc

    log("mfma loop zero operands")
    out = _run(torch, sgc, 4, 10, np.zeros(32768))
    assert np.all(out == 0.0)
