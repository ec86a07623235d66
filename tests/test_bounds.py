"""Pins for the exact-rational bound calculators against the statements the
paper prints about them (Sec. 4.3 and Sec. 4.4)."""
from fractions import Fraction

from oracle import bounds
from tests.helpers import claims


def test_ll_coefficient_between_gamma4_and_gamma5():
    """Eq. ll_bound: u16^2 (1+u16)^2 is slightly larger than gamma_4 and
    smaller than gamma_5 (Sec. 4.3)."""
    k = int(claims()["ll_coef_between_gamma"])
    assert bounds.gamma(k) < bounds.LL_COEF < bounds.gamma(k + 1)
    assert bounds.LL_COEF == Fraction(2049**2, 2**44)


def test_ratio_to_gamma_k_first_below_two_at_15():
    """Sec. 4.4: the exact main-bound coefficient's ratio to the classical
    gamma_k falls below 2 at k = 15 (and not before)."""
    k15 = int(claims()["ratio_below_two_at_k"])
    for k in range(1, k15):
        assert bounds.main_bound_coef(k) / bounds.gamma(k) >= 2, k
    assert bounds.main_bound_coef(k15) / bounds.gamma(k15) < 2
    # and tends to 1 as k grows
    r = [bounds.main_bound_coef(k) / bounds.gamma(k) for k in (100, 10_000, 1_000_000)]
    assert r[0] > r[1] > r[2] > 1 and r[2] < Fraction(1001, 1000) * (1 + 4 * bounds.U16)


def test_first_order_form():
    """Eq. main_bound_first_order: coefficient = gamma_k + 14 u32 + O(u16^3 +
    gamma_k u16), i.e. the scheme-specific additive constant is 14 u32."""
    extra = int(claims()["first_order_extra_u32"])
    u16, u32 = bounds.U16, bounds.U32
    for k in (1, 10, 100, 1000, 16384):
        g = bounds.gamma(k)
        diff = bounds.main_bound_coef(k) - bounds.first_order_coef(k)
        assert abs(diff) <= 8 * (u16**3 + g * u16), k
        assert bounds.first_order_coef(k) == g + extra * u32


def test_tau_is_about_12_u32():
    """tau = u16^2 (3 + 2u16 + 2u16^2) = 12 u32 (1 + O(u16)); u16^2 = 4 u32."""
    assert bounds.U16**2 == 4 * bounds.U32
    t = bounds.TAU / bounds.U32
    assert 12 < t < Fraction(12004, 1000)


def test_gamma_definition():
    assert bounds.gamma(1) == Fraction(1, 2**24 - 1)
    assert bounds.gamma(2) == Fraction(2, 2**24 - 2)


def test_depth_counts():
    # one block: kb - 1 inner additions + 3 merges (elementwise), +2 (termwise)
    assert bounds.elementwise_depth(64, 64) == 63 + 3
    assert bounds.termwise_depth(64, 64) == 63 + 2
    assert bounds.elementwise_depth(128, 64) == 63 + 6
    assert bounds.termwise_depth(128, 64) == 63 + 1 + 2
    # never deeper than the plain sequential K-term chain for termwise blocks
    for K in (1, 2, 63, 64, 65, 1000, 8192):
        assert bounds.termwise_depth(K, 64) <= K + 2
