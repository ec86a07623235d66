"""How the matrix unit sums FP16 x FP16 products into FP32, probed through the
C-ABI (sgemm_cube_hgemm on FP16-exact inputs, so hi = a and the kernel is a
chain of v_mfma_f32_16x16x32_f16 starting from zero, one k-step of
sgemm_cube_block_k() = 32 products per instruction).

The parity tolerance rests on these properties (the paper assumes an RN FP32
accumulation in the matrix unit, Sec. 4.3, and names checking it as open work,
Sec. 7):
  * products are exact;
  * the products of a k-step are aligned to the largest of them with few
    guard bits and no sticky bit, so small products next to a large one are
    cut off before rounding: 1 + 2^-24 + 2^-30 as three products of one
    k-step gives 1 (the exact sum rounds to 1 + 2^-23), and a small term next
    to cancelling large ones is lost (2^20 - 2^20 + 2^-20 -> 0);
  * the accumulator is then added to that product sum with one rounding: 1 in
    the accumulator plus products 2^-24 + 2^-30 of the next k-step gives
    1 + 2^-23, where sequential round-to-nearest would give 1;
  * the error of one k-step stays within 2 u32 of the sum of the magnitudes of
    its terms, which is what the parity tolerance uses.
"""
import numpy as np
import pytest

from tests.gpu_util import hgemm, log

pytestmark = pytest.mark.gpu


def _dot(a, b):
    """One output entry C[0,0] = sum_k a_k b_k through a 1 x 1 x K hgemm."""
    A = np.asarray(a, dtype=np.float32).reshape(1, -1)
    B = np.asarray(b, dtype=np.float32).reshape(-1, 1)
    return float(hgemm(A, B)[0, 0])


def _exact(a, b):
    from fractions import Fraction

    return sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(a, b))


CASES = {
    # name: (a, b) with every entry exactly representable in FP16
    "fused_single_rounding": ([1.0, 2.0**-12, 2.0**-15], [1.0, 2.0**-12, 2.0**-15]),
    "cancellation_truncates": ([2.0**10, -(2.0**10), 2.0**-10], [2.0**10, 2.0**10, 2.0**-10]),
    "exact_products": ([2047.0, -2045.0, 3.0], [2047.0, 2043.0, 5.0]),
    "subnormal_products": ([2.0**-24, 2.0**-24, 3 * 2.0**-24], [1.0, 2.0**-14, 2.0**-14]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_one_k_step_error_is_within_two_ulps_of_the_term_sum(gpu, name):
    a, b = CASES[name]
    log(f"mfma numerics {name}")
    got = _dot(a, b)
    exact = _exact(a, b)
    mag = sum(abs(float(x) * float(y)) for x, y in zip(a, b))
    assert abs(got - float(exact)) <= 2 * 2.0**-24 * mag, (name, got, float(exact))


def test_small_products_next_to_a_large_one_are_cut_off(gpu):
    a, b = CASES["fused_single_rounding"]
    log("mfma numerics alignment within a k-step")
    # Round-to-nearest FP32 of the exact sum (exact in float64 here) would be 1 + 2^-23.
    assert np.float32(float(_exact(a, b))) == np.float32(1.0 + 2.0**-23)
    assert _dot(a, b) == 1.0


def test_accumulator_plus_products_of_the_next_k_step(gpu):
    """1 in the accumulator (first k-step), 2^-24 + 2^-30 as products of the
    second k-step: one rounding of the exact sum, 1 + 2^-23 (sequential
    round-to-nearest would give 1)."""
    from paper_2507_23387_amd import binding

    kb = binding.sgemm_cube_block_k()
    a = np.zeros(2 * kb)
    b = np.zeros(2 * kb)
    a[0] = b[0] = 1.0
    a[kb], b[kb] = 2.0**-12, 2.0**-12
    a[kb + 1], b[kb + 1] = 2.0**-15, 2.0**-15
    log("mfma numerics accumulator")
    got = _dot(a, b)
    assert got == 1.0 + 2.0**-23


def test_small_term_lost_to_alignment(gpu):
    a, b = CASES["cancellation_truncates"]
    log("mfma numerics truncation")
    assert _dot(a, b) == 0.0


def test_products_exact_and_integer_sums_exact(gpu):
    a, b = CASES["exact_products"]
    assert _dot(a, b) == float(_exact(a, b))      # 4190209 - 4177935 + 15 = 12289
    a, b = CASES["subnormal_products"]
    assert _dot(a, b) == 2.0**-24 + 2.0**-36      # FP16-subnormal operands, exact products
