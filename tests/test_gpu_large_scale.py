"""Residual scales above 2^15 on every entry point and order, against the oracle.

The C-ABI accepts any power of two s in [1, 2^24] (Sec. 4.2, s_f = 2^{s_b};
Rule 2 bounds the usable s_b by the input's exponent window, not by the
format).  The scaled elementwise kernels form s * B_hi in FP16, where s itself
is only finite up to 2^15, so from 2^16 on the library must take its unscaled
elementwise kernel.  These cases use |B| < 1, so |B_hi| * s never exceeds
65504 for s <= 2^15 and the range flag of the split of B stays clear: only the
host-side routing keeps the result finite.  B also holds whole zero rows and
columns and scattered zeros (0 * inf would be NaN).

Bar: |C_gpu - C_oracle|_ij <= 2 K 2^-24 (|A||B|)_ij, identical inf/NaN
patterns (here: none), C prefilled with NaN so every entry is checked to be
written."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu

SCALES = [2.0**15, 2.0**16, 2.0**20, 2.0**24]
ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]
M, N, K = 300, 260, 257


def _operands(seed):
    rng = np.random.default_rng(seed)
    A = rng.uniform(-1.0, 1.0, (M, K)).astype(np.float32)
    B = (rng.uniform(-1.0, 1.0, (K, N)) * 0.999).astype(np.float32)
    B[rng.random((K, N)) < 0.1] = 0.0
    B[::7, :] = 0.0
    B[:, ::5] = 0.0
    assert np.abs(B).max() < 1.0
    return A, B


def _kb():
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


def _nan_c():
    import torch

    return torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")


def _check(C, A, B, scale, order, what, prescale=False):
    import torch

    torch.cuda.synchronize()
    Cn = C.cpu().numpy()
    assert np.isfinite(Cn).all(), f"{what}: non-finite output"
    fn = oracle.sgemm_prescaled if prescale else oracle.sgemm
    Co = fn(A, B, scale, order, kb=_kb())
    assert np.isfinite(Co).all()
    assert_parity(Cn, Co, K, abs_ab(A, B), what)


@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("scale", SCALES, ids=lambda s: f"s2^{int(np.log2(s))}")
def test_large_scale_every_entry_point(gpu, order, scale):
    import torch

    from paper_2507_23387_amd import binding

    A, B = _operands(int(np.log2(scale)) + 3 * ORDERS.index(order))
    dA, dB = to_dev(A), to_dev(B)
    code = binding.ORDERS[order]
    stream = torch.cuda.current_stream().cuda_stream
    tag = f"{order} s=2^{int(np.log2(scale))}"

    log(f"large scale sgemm_cube {tag}")
    C = _nan_c()
    binding.matmul(dA, dB, scale, order, out=C)
    _check(C, A, B, scale, order, f"sgemm_cube {tag}")

    log(f"large scale sgemm_cube_ws {tag}")
    ws = binding.workspace(M, N, K)
    nbytes = ws.numel()
    C = _nan_c()
    binding.matmul(dA, dB, scale, order, out=C, workspace=ws)
    _check(C, A, B, scale, order, f"sgemm_cube_ws {tag}")

    log(f"large scale prepare + compute {tag}")
    C = _nan_c()
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, scale,
                                      ws.data_ptr(), nbytes, stream) == 0
    assert binding.sgemm_cube_compute(M, N, K, C.data_ptr(), N, scale, code, ws.data_ptr(),
                                      nbytes, stream) == 0
    _check(C, A, B, scale, order, f"prepare+compute {tag}")

    log(f"large scale prepare(B) + compute_a {tag}")
    C = _nan_c()
    assert binding.sgemm_cube_prepare(M, N, K, 0, K, dB.data_ptr(), N, scale, ws.data_ptr(),
                                      nbytes, stream) == 0
    assert binding.sgemm_cube_compute_a(M, N, K, dA.data_ptr(), K, C.data_ptr(), N, scale, code,
                                        ws.data_ptr(), nbytes, stream) == 0
    _check(C, A, B, scale, order, f"compute_a {tag}")

    if order == "elementwise":
        for stages in (1, 2):
            log(f"large scale compute_stages({stages}) {tag}")
            C = _nan_c()
            assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                              scale, ws.data_ptr(), nbytes, stream) == 0
            assert binding.sgemm_cube_compute_stages(M, N, K, C.data_ptr(), N, scale, code,
                                                     stages, ws.data_ptr(), nbytes,
                                                     stream) == 0
            _check(C, A, B, scale, order, f"compute_stages({stages}) {tag}")

    for prescale in (False, True):
        log(f"large scale sgemm_cube_ex prescale={prescale} {tag}")
        C = _nan_c()
        binding.matmul_ex(dA, dB, scale, order, prescale=prescale, out=C)
        _check(C, A, B, scale, order, f"sgemm_cube_ex prescale={prescale} {tag}", prescale)


def test_scale_2_15_keeps_the_scaled_kernel_bitwise_stable(gpu):
    """At s = 2^15 (the largest scale the scaled kernel takes) the three
    entry points that share the GEMM launch give the same bits."""
    import torch

    from paper_2507_23387_amd import binding

    A, B = _operands(99)
    dA, dB = to_dev(A), to_dev(B)
    log("s=2^15 entry points agree")
    C1 = binding.matmul(dA, dB, 2.0**15, "elementwise")
    C2 = binding.matmul(dA, dB, 2.0**15, "elementwise", workspace=binding.workspace(M, N, K))
    C3 = binding.matmul_ex(dA, dB, 2.0**15, "elementwise")
    torch.cuda.synchronize()
    assert torch.equal(C1, C2) and torch.equal(C1, C3)
