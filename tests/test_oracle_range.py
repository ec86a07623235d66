"""Pins of the oracle's range extensions (pre-scaling, range classes).

The paper names explicit exponent management of the high part (Sec. 4.2),
input-dependent scaling and an overflow guard (Sec. 7, 8) as the way to widen
the method's range without fixing a rule; the oracle's reading is documented in
oracle/__init__.py.  It is pinned here by what the mathematics fixes:
power-of-two scaling is exact, so on inputs whose hi and lo words stay normal
the pre-scaled result equals the plain one bit for bit; on inputs whose hi is
FP16-subnormal (outside Rule 1's reach) pre-scaling brings Eq. main_bound back;
and the range classes of the values Sec. 3.1 and Sec. 4.2 name.
"""
import numpy as np
import pytest

import oracle
from oracle import bounds


def _normal_two_word_operands(M, N, K, seed):
    """Entries a = h + l / 2^11 with h an FP16 value in [0.5, 1) and l an FP16
    value in [1/8, 1/2): fl16(a) = h and the scaled residual is exactly l, both
    normal before and after any power-of-two scaling used below."""
    rng = np.random.default_rng(seed)

    def draw(shape):
        h = (1024 + rng.integers(0, 1024, size=shape)) * 2.0**-11      # [0.5, 1), 11 bits
        l = (1024 + rng.integers(0, 1024, size=shape)) * 2.0**-13      # [1/8, 1/4), 11 bits
        l = np.where(rng.random(shape) < 0.5, l, 2 * l - 2.0**-12)     # some in [1/4, 1/2)
        sign = rng.choice([-1.0, 1.0], size=shape)
        return (sign * (h + l * 2.0**-11)).astype(np.float32)

    return draw((M, K)), draw((K, N))


@pytest.mark.parametrize("order,kb", [("elementwise", 16), ("termwise", 16),
                                      ("elementwise_cross_first", 32), ("hi_only", 16)])
def test_prescaling_is_exact_when_hi_and_lo_stay_normal(order, kb):
    A, B = _normal_two_word_operands(37, 29, 96, 1)
    # Row scales of 2^-6 .. 2^6 and column scales of 2^-3 .. 2^3 on top.
    rng = np.random.default_rng(2)
    A = np.ldexp(A, rng.integers(-6, 7, size=(37, 1)).astype(np.int32)).astype(np.float32)
    B = np.ldexp(B, rng.integers(-3, 4, size=(1, 29)).astype(np.int32)).astype(np.float32)
    plain = oracle.sgemm(A, B, 2048.0, order, kb=kb)
    pre = oracle.sgemm_prescaled(A, B, 2048.0, order, kb=kb)
    assert np.array_equal(plain.view(np.uint32), pre.view(np.uint32))


def test_prescaling_restores_main_bound_for_subnormal_hi():
    """|a| ~ 2^-22: hi is FP16-subnormal with 2 significant bits and the
    two-word representation loses the 22-bit guarantee (Sec. 4.2, after
    Rule 1), so Eq. main_bound fails; scaled into the normal range it holds."""
    rng = np.random.default_rng(3)
    M, N, K = 24, 20, 32
    A = np.ldexp(rng.uniform(-1, 1, (M, K)), -22).astype(np.float32)
    B = np.ldexp(rng.uniform(-1, 1, (K, N)), -22).astype(np.float32)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    absab = np.abs(A).astype(np.float64) @ np.abs(B).astype(np.float64)
    coef = float(bounds.main_bound_coef(K))
    plain = np.abs(oracle.sgemm(A, B, 2048.0, "termwise").astype(np.float64) - ref)
    pre = np.abs(oracle.sgemm_prescaled(A, B, 2048.0, "termwise").astype(np.float64) - ref)
    assert np.any(plain > coef * absab)
    assert np.all(pre <= coef * absab)


def test_prescale_exponents_place_the_maximum():
    X = np.array([[3.0, -0.75, 1e-3], [0, 0, 0], [np.inf, 5e-9, -np.nan],
                  [-65504.0, 1, 2]], dtype=np.float32)
    p = oracle.prescale_exponents(X, 1, 14)
    assert p[1] == 0                                       # all-zero row: unscaled
    for i in (0, 2, 3):
        m = np.max(np.abs(np.where(np.isfinite(X[i]), X[i], 0)))
        scaled = np.ldexp(np.float64(m), int(p[i]))
        assert 2.0**14 <= scaled < 2.0**15
    q = oracle.prescale_exponents(X, 0, 3)
    for j in range(3):
        col = X[:, j]
        m = np.max(np.abs(np.where(np.isfinite(col), col, 0)))
        assert 8.0 <= np.ldexp(np.float64(m), int(q[j])) < 16.0
    assert oracle.prescale_targets(2.0**11) == (14, 3)
    assert oracle.prescale_targets(2.0**13) == (13, 1)
    assert oracle.prescale_targets(1.0) == (14, 14)


@pytest.mark.parametrize("value,scale,bits", [
    (1.0, 2048.0, 0),
    (65504.0, 2048.0, 0),              # largest finite FP16
    (65519.0, 2048.0, 0),              # still rounds down to 65504
    (65520.0, 2048.0, oracle.RANGE_HI_OVERFLOW),   # Sec. 3.1: |a| >= 65520 overflows
    (-1e6, 2048.0, oracle.RANGE_HI_OVERFLOW),
    (32784.0, 4096.0, oracle.RANGE_LO_OVERFLOW),   # Sec. 4.2: residual 16, times 2^12
    (32784.0, 2048.0, 0),
    (2.0**-20, 2048.0, oracle.RANGE_HI_SUBNORMAL),  # below 2^-14
    (2.0**-14, 2048.0, 0),             # smallest normal FP16
    (2.0**-30, 2048.0, 0),             # hi rounds to zero: no subnormal hi
    (np.inf, 2048.0, oracle.RANGE_NONFINITE),
    (np.nan, 2048.0, oracle.RANGE_NONFINITE),
])
def test_range_classes_of_named_values(value, scale, bits):
    assert oracle.range_classes(np.array([[value, 0.5]], np.float32), scale) == bits
