"""GPU range extensions (sgemm_cube_ex) against the oracle.

Pre-scaling: parity with the oracle's pre-scaled product on ragged shapes
whose rows and columns span wide exponent ranges and on the 2^-14-scaled
workload; bit-for-bit invariance on inputs whose hi and lo words stay normal;
Eq. main_bound restored for deeply subnormal hi.  Range report: equal to the
oracle's range classes of the (pre-scaled) operands.  Degenerate shapes and
the plain path.
"""
import numpy as np
import pytest

import oracle
import workloads
from oracle import bounds
from tests.gpu_util import log, to_dev
from tests.helpers import abs_ab, assert_parity, ref64
from tests.test_oracle_range import _normal_two_word_operands

pytestmark = pytest.mark.gpu

ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]


def _kb():
    """The oracle's block size matching the GPU's (one 32-wide MFMA k-step)."""
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


def _ex(A, B, scale, order, prescale, report=False):
    import torch

    from paper_2507_23387_amd import binding

    out = binding.matmul_ex(to_dev(A), to_dev(B), scale=scale, order=order, prescale=prescale,
                            report=report)
    torch.cuda.synchronize()
    if report:
        C, bits = out
        return C.cpu().numpy(), int(bits.cpu().item())
    return out.cpu().numpy()


def _wide_range_operands(M, N, K, seed):
    rng = np.random.default_rng(seed)
    A = rng.uniform(-1, 1, (M, K)) * np.ldexp(1.0, rng.integers(-30, 20, size=(M, 1)))
    B = rng.uniform(-1, 1, (K, N)) * np.ldexp(1.0, rng.integers(-30, 20, size=(1, N)))
    return A.astype(np.float32), B.astype(np.float32)


@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("shape", [(1, 1, 1), (129, 130, 65), (300, 257, 515)],
                         ids=lambda s: "x".join(map(str, s)))
def test_prescaled_parity(gpu, order, shape):
    M, N, K = shape
    A, B = _wide_range_operands(M, N, K, M + N + K)
    log(f"ex prescale {order} {shape}")
    C = _ex(A, B, 2048.0, order, True)
    Co = oracle.sgemm_prescaled(A, B, 2048.0, order, kb=_kb())
    assert_parity(C, Co, K, abs_ab(A, B), f"prescale {order} {shape}")


@pytest.mark.parametrize("order", ORDERS)
def test_prescaling_is_exact_on_normal_two_word_inputs(gpu, order):
    A, B = _normal_two_word_operands(200, 190, 320, 7)
    rng = np.random.default_rng(8)
    A = np.ldexp(A, rng.integers(-6, 7, size=(200, 1)).astype(np.int32)).astype(np.float32)
    B = np.ldexp(B, rng.integers(-3, 4, size=(1, 190)).astype(np.int32)).astype(np.float32)
    log(f"ex prescale invariance {order}")
    plain = _ex(A, B, 2048.0, order, False)
    pre = _ex(A, B, 2048.0, order, True)
    assert np.array_equal(plain.view(np.uint32), pre.view(np.uint32))


def test_prescaling_restores_main_bound_for_deep_subnormal_hi(gpu):
    """|a| ~ 2^-22: hi is FP16-subnormal with 2 significant bits (Sec. 4.2,
    after Rule 1); unscaled the termwise result breaks Eq. main_bound,
    pre-scaled it meets it (the oracle shows the same, test_oracle_range)."""
    rng = np.random.default_rng(3)
    M, N, K = 24, 20, 32
    A = np.ldexp(rng.uniform(-1, 1, (M, K)), -22).astype(np.float32)
    B = np.ldexp(rng.uniform(-1, 1, (K, N)), -22).astype(np.float32)
    ref = ref64(A, B)
    absab = abs_ab(A, B)
    coef = float(bounds.main_bound_coef(K))
    log("ex prescale deep subnormal")
    plain = _ex(A, B, 2048.0, "termwise", False)
    pre = _ex(A, B, 2048.0, "termwise", True)
    assert np.any(np.abs(plain.astype(np.float64) - ref) > coef * absab)
    assert np.all(np.abs(pre.astype(np.float64) - ref) <= coef * absab)


def test_prescaled_subnormal_hi_workload(gpu):
    """The 2^-14-scaled workload pre-scaled: parity with the oracle's
    pre-scaled product and Eq. main_bound on sampled rows."""
    w = workloads.get("c5")
    A, B = workloads.workload_operands(w)
    rows = workloads.sample_rows(w.M, 8, w.seed)
    log("ex prescale c5 termwise")
    pre = _ex(A, B, 2048.0, "termwise", True)[rows]
    coef = float(bounds.main_bound_coef(w.K))
    assert np.all(np.abs(pre.astype(np.float64) - ref64(A, B, rows)) <= coef * abs_ab(A, B, rows))
    As, Bs = _prescaled_inputs(A, B, 2048.0)
    Cs = oracle.sgemm_rows(As, Bs, rows, 2048.0, "termwise", kb=_kb())
    _assert_unscaled_parity(pre, Cs, A, B, rows, w.K)


def _prescaled_inputs(A, B, scale):
    ea, eb = oracle.prescale_targets(scale)
    p = oracle.prescale_exponents(A, 1, ea)
    q = oracle.prescale_exponents(B, 0, eb)
    As = np.ldexp(A, p[:, None].astype(np.int32)).astype(np.float32)
    Bs = np.ldexp(B, q[None, :].astype(np.int32)).astype(np.float32)
    return As, Bs


def _assert_unscaled_parity(C_rows, Cs_rows, A, B, rows, K):
    ea, eb = oracle.prescale_targets(2048.0)
    p = oracle.prescale_exponents(A, 1, ea)[rows]
    q = oracle.prescale_exponents(B, 0, eb)
    Co = np.ldexp(Cs_rows, (-(p[:, None] + q[None, :])).astype(np.int32)).astype(np.float32)
    assert_parity(C_rows, Co, K, abs_ab(A, B, rows), "prescaled rows")


def _special_operands():
    rng = np.random.default_rng(11)
    A = rng.uniform(-1, 1, (40, 70)).astype(np.float32)
    B = rng.uniform(-1, 1, (70, 50)).astype(np.float32)
    return A, B


@pytest.mark.parametrize("case", ["clean", "hi_overflow", "lo_overflow", "subnormal", "nan",
                                  "all"])
@pytest.mark.parametrize("prescale", [False, True], ids=["plain", "prescale"])
def test_range_report_matches_oracle(gpu, case, prescale):
    A, B = _special_operands()
    scale = 4096.0
    if case in ("hi_overflow", "all"):
        A[3, 5] = 70000.0
    if case in ("lo_overflow", "all"):
        B[20, 21] = 32784.0
    if case in ("subnormal", "all"):
        A[7, :] = np.ldexp(A[7, :], -20)
    if case in ("nan", "all"):
        B[11, 13] = np.nan
    log(f"ex range report {case} prescale={prescale}")
    _, bits = _ex(A, B, scale, "termwise", prescale, report=True)
    As, Bs = _prescaled_inputs(A, B, scale) if prescale else (A, B)
    want = oracle.range_classes(As, scale) | oracle.range_classes(Bs, scale)
    assert bits == want, (bits, want)
    if case == "clean":
        assert bits == 0
    if prescale and case == "subnormal":
        assert bits == 0        # the small row is scaled into the normal range


def test_plain_ex_equals_sgemm_ws_and_degenerate_shapes(gpu):
    import torch

    from paper_2507_23387_amd import binding

    A, B = workloads.make_operands(130, 70, 90, 14, "normal")
    log("ex plain == ws")
    for order in ORDERS:
        C1 = binding.matmul(to_dev(A), to_dev(B), 2048.0, order)
        C2 = binding.matmul_ex(to_dev(A), to_dev(B), 2048.0, order)
        torch.cuda.synchronize()
        assert torch.equal(C1, C2)
    log("ex K=0 / M=0")
    stream = torch.cuda.current_stream().cuda_stream
    C = torch.full((5, 6), float("nan"), device="cuda")
    Ad = torch.empty((5, 0), device="cuda")
    Bd = torch.empty((0, 6), device="cuda")
    bits = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    assert binding.sgemm_cube_ex(5, 6, 0, Ad.data_ptr(), 1, Bd.data_ptr(), 6, C.data_ptr(), 6,
                                 2048.0, 1, binding.OPT_PRESCALE, 0, 0, bits.data_ptr(),
                                 stream) == 0
    torch.cuda.synchronize()
    assert (C.cpu().numpy() == 0).all() and int(bits.item()) == 0
    bits.fill_(7)
    B4 = torch.ones((4, 6), device="cuda")
    assert binding.sgemm_cube_ex(0, 6, 4, 0, 4, B4.data_ptr(), 6, C.data_ptr(), 6, 2048.0, 1, 0,
                                 0, 0, bits.data_ptr(), stream) == 0
    torch.cuda.synchronize()
    assert int(bits.item()) == 0
