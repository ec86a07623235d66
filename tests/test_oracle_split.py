"""Pins for the oracle's two-component split (Sec. 3.3; Eq. recover_eqn):
hi = fl16(a), r = a - hi, lo = fl16(r * s_f).

Checked against what the paper fixes, mostly exhaustively over whole binades
(all 2^23 mantissas of an FP32 exponent):
  * the worked overflow example of Sec. 4.2 (golden file);
  * Eq. split_error together with the scaling bounds Eq. sf_bounds (Rules 1-2);
  * the sign flip of the residual when hi rounds away from zero (Sec. 3.3);
  * the residual-class counts of the probability model of Sec. 4.1, exactly;
  * the 12-exponent shift of the retained-precision curve under s_b = 12
    (Sec. 4.2).
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from oracle import bounds
from tests.helpers import claims, read_table


def binade(e_off: int) -> np.ndarray:
    """All 2^23 positive FP32 values with unbiased exponent e_off."""
    m = np.arange(1 << 23, dtype=np.uint32)
    return (np.uint32(e_off + 127) << np.uint32(23) | m).view(np.float32)


def split64(x: np.ndarray, s_b: int):
    hi, lo = oracle.split(x.reshape(1, -1), 2.0**s_b)
    h = oracle.f16_to_f32(hi[0]).astype(np.float64)
    l = oracle.f16_to_f32(lo[0]).astype(np.float64)
    return h, l


_BUF = {}


def _buf(name, n):
    b = _BUF.get(name)
    if b is None or b.size < n:
        b = _BUF[name] = np.empty(n, dtype=np.float64)
    return b[:n]


def rel_repr_error(x: np.ndarray, s_b: int) -> np.ndarray:
    """|a - hi - lo/s_f| / |a| in FP64 (exact up to the final division).
    Works in reused buffers: fresh large allocations are slow to fault in."""
    hi, lo = oracle.split(x.reshape(1, -1), 2.0**s_b)
    n = x.size
    a, h, l = _buf("a", n), _buf("h", n), _buf("l", n)
    a[:] = x
    h[:] = oracle.f16_to_f32(hi[0])
    l[:] = oracle.f16_to_f32(lo[0])
    np.multiply(l, 2.0**-s_b, out=l)
    np.subtract(a, h, out=h)
    np.subtract(h, l, out=h)
    np.abs(h, out=h)
    np.abs(a, out=a)
    np.divide(h, a, out=h)
    return h


def test_worked_example_sec_4_2():
    for V, s_b, e_hi, e_res, e_lo in read_table("split_worked_example.txt"):
        V, s_b = float(V), int(s_b)
        hi, lo = oracle.split(np.array([[V]], dtype=np.float32), 2.0**s_b)
        h = float(oracle.f16_to_f32(hi)[0, 0])
        l = float(oracle.f16_to_f32(lo)[0, 0])
        assert h == float(e_hi)
        assert V - h == float(e_res)
        assert l == float(e_lo), (V, s_b, l)


def test_unique_fixed_scale_over_full_fp16_range():
    """Eq. sf_bounds: -3 - e_min <= s_b <= 26 - e_max; with e_min = -14 and
    e_max = 15 the only choice is s_b = 11 (Sec. 4.2)."""
    lo, hi = -3 - (-14), 26 - 15
    assert lo == hi == int(claims()["unique_fixed_sb"])


def _window(s_b: int):
    """Exponents where Eq. sf_bounds holds for a single binade and hi is a
    normal FP16: e >= -3 - s_b, e >= -14, e <= 26 - s_b, e <= 15."""
    return range(max(-3 - s_b, -14), min(26 - s_b, 15) + 1)


@pytest.mark.parametrize("s_b", [0, 11, 12])
def test_split_error_bound_inside_scaling_window(s_b):
    """Eq. split_error: |V - (V_high + V_low / s_f)| <= 2^-22 |V| whenever
    Rules 1-2 (Eq. sf_bounds) hold, for every value of every such binade."""
    bound = 2.0 ** claims()["split_error_log2"]
    for e in _window(s_b):
        x = binade(e)
        if e == 15:
            x = x[x < 65520.0]  # beyond that hi itself overflows (Sec. 3.1)
        err = rel_repr_error(x, s_b)
        assert np.all(err <= bound), (s_b, e, err.max())


@pytest.mark.parametrize("s_b", [0, 6])
def test_split_error_bound_fails_below_rule_1(s_b):
    """One exponent below the Rule-1 limit the 22-bit guarantee is lost: some
    value of the binade has representation error above 2^-22 (Sec. 4.2)."""
    e = -3 - s_b - 1
    err = rel_repr_error(binade(e), s_b)
    assert err.max() > 2.0**-22


def test_lo_overflow_beyond_rule_2():
    """Rule 2: s_b = 12 is safe only for e_max <= 14; in the binade of 2^15
    some scaled residuals overflow (the worked example is one of them)."""
    x = binade(15)
    x = x[x < 65520.0]
    _, lo = oracle.split(x.reshape(1, -1), 2.0**12)
    assert np.isinf(oracle.f16_to_f32(lo)).any()
    _, lo = oracle.split(binade(14).reshape(1, -1), 2.0**12)
    assert np.isfinite(oracle.f16_to_f32(lo)).all()


@pytest.mark.parametrize("e", [-14, -5, 0, 3, 14])
def test_sign_flip_iff_rounded_away(e):
    """Sec. 3.3: the residual's sign differs from V's exactly when RN rounded
    the high part away from zero (carry c = 1)."""
    x = binade(e)
    h, l = split64(x, 11)
    rounded_up = h > x.astype(np.float64)
    nz = l != 0
    assert np.array_equal((l < 0)[nz], rounded_up[nz])
    # Without residual underflow (every nonzero |r| * s_f >= 2^-24, i.e. the
    # smallest residual ulp32(V) = 2^(e-23) scaled by 2^11 stays >= 2^-24),
    # lo is zero only where hi already equals the input.
    if e - 23 + 11 >= -24:
        assert np.array_equal(l == 0, h == x.astype(np.float64))


@pytest.mark.parametrize("e", [-14, -11, -3, 0, 7, 14])
def test_residual_class_counts_match_probability_model(e):
    """Sec. 4.1: over a binade with uniformly distributed low mantissa bits,
    the joint frequency of (X, N) equals P(X, N = n) exactly, where X says
    whether hi was truncated (T) or rounded up (R), and N counts the leading
    zeros of the residual below the split (-1 = the midpoint tie)."""
    x = binade(e)
    h, _ = split64(x, 11)
    a = x.astype(np.float64)
    r = a - h  # exact
    X_R = np.abs(h) > np.abs(a)
    N = np.full(a.shape, 12, dtype=np.int64)
    nz = r != 0
    _, ex = np.frexp(np.abs(r[nz]))
    N[nz] = (e - 12) - (ex - 1)
    total = 1 << 23
    for n in range(-1, 13):
        for xcls, mask in (("T", ~X_R), ("R", X_R)):
            got = int(np.count_nonzero(mask & (N == n)))
            want = bounds.p_class(xcls, n) * total
            assert want.denominator == 1
            assert got == want.numerator, (e, xcls, n, got, want)
    assert not np.any(X_R & (N == 12))


def test_probability_claims_sec_4_1():
    c = claims()
    total = sum(bounds.p_class(x, n) for x in "TR" for n in range(-2, 14))
    assert total == c["p_class_total"]
    p0 = bounds.p_gradual_or_underflow(0)
    assert p0 > c["p_ugu_at_0_exceeds"]
    assert p0 == Fraction(1, 8) - Fraction(1, 2**13)
    lim = int(c["p_u_significant_below"])
    assert bounds.p_underflow(lim + 2) < Fraction(1, 10)
    near = int(c["p_u_near_one_below"])
    assert bounds.p_underflow(near - 1) > Fraction(999, 1000)
    # monotone in the exponent
    vals = [bounds.p_underflow(e) for e in range(-30, 5)]
    assert all(a >= b for a, b in zip(vals, vals[1:]))


@pytest.mark.parametrize("e", [-12, -3, 0])
def test_range_event_frequency_matches_model(e):
    """Sec. 4.1 range events, measured on the oracle's hi: the fraction of a
    binade whose exact nonzero residual lies below 2^-14 (gradual underflow or
    underflow) equals the model's sum over the classes that trigger it."""
    x = binade(e)
    h, _ = split64(x, 11)
    r = np.abs(x.astype(np.float64) - h)
    got = int(np.count_nonzero((r != 0) & (r < 2.0**-14)))
    lo = e - bounds.L_M_HIGH + bounds.B_LOW - 2
    want = sum(bounds.p_class("T", n) + bounds.p_class("R", n)
               for n in range(max(lo, -1), 12)) * (1 << 23)
    assert got == want


def test_scaling_shifts_precision_curve_by_s_b():
    """Sec. 4.2: s_b = 12 shifts the retained-precision curve left by 12
    exponents.  Elementwise: the representation error of m * 2^e with s_b = 12
    equals that of m * 2^(e+12) with s_b = 0, while hi stays a normal FP16."""
    shift = int(claims()["shift_exponents_sb12"])
    for e in (-14, -12, -8, -4, 0, 2):  # e + 12 <= 14 keeps hi finite
        a = rel_repr_error(binade(e), shift).copy()
        b = rel_repr_error(binade(e + shift), 0)
        assert np.array_equal(a, b), e


def test_unscaled_range_boundaries():
    """Sec. 4.2: without scaling the exact residual sits about 12 exponents
    below the input, so it enters the FP16 subnormal range once E_offset < -2
    and falls below 2^-24 once E_offset < -12 (here: for the typical N = 0
    class, i.e. the largest non-tie residuals of the binade)."""
    c = claims()
    g, u = int(c["gradual_boundary_unscaled"]), int(c["underflow_boundary_unscaled"])
    for e, limit in ((g, 2.0**-14), (u, 2.0**-24)):
        for ee, inside in ((e, True), (e - 1, False)):
            x = binade(ee)
            h, _ = split64(x, 0)
            r = np.abs(x.astype(np.float64) - h)
            r_max_nontie = r[r < 2.0 ** (ee - 11)].max()
            assert (r_max_nontie >= limit) == inside, (e, ee, r_max_nontie)
