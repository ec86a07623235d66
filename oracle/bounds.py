"""Exact-rational calculators for the constants of the SGEMM-cube analysis.

TEST INFRASTRUCTURE (part of the oracle).  Everything is a
``fractions.Fraction`` so the statements the paper prints about the constants
can be checked exactly.

* Sec. 3.2 notation table: u16 = 2^-11, u32 = 2^-24,
  gamma_k = k u32 / (1 - k u32), a = 1 + u16,
  tau = u16^2 (3 + 2 u16 + 2 u16^2).
* Eq. ll_bound (Sec. 4.3): the dropped lo*lo term is bounded by
  u16^2 (1 + u16)^2 |A||B|.
* Eq. truncation / Eq. main_bound / Eq. main_bound_first_order (Sec. 4.4).
* The residual-class probability model P(X, N = n) and the sums P_{u+gu},
  P_u of Sec. 4.1.
"""
from __future__ import annotations

from fractions import Fraction as Fr

U16 = Fr(1, 2**11)
U32 = Fr(1, 2**24)
L_M = 23        # stored mantissa bits of FP32
L_M_HIGH = 10   # stored mantissa bits of FP16
B_LOW = 15      # FP16 exponent bias


def gamma(k: int) -> Fr:
    """gamma_k = k u32 / (1 - k u32) (Sec. 3.2 notation table)."""
    if k * U32 >= 1:
        raise ValueError("gamma_k undefined for k u32 >= 1")
    return k * U32 / (1 - k * U32)


A_COEF = 1 + U16                                  # a = 1 + u16
TAU = U16**2 * (3 + 2 * U16 + 2 * U16**2)          # Eq. truncation
LL_COEF = U16**2 * (1 + U16) ** 2                  # Eq. ll_bound


def main_bound_coef(k: int) -> Fr:
    """Coefficient of |A||B| in Eq. main_bound (termwise, RN throughout):
    tau + gamma_k a^2 (1+2u16) + gamma_2 (1+gamma_k) a^2 (1+2u16)."""
    g = gamma(k)
    s = A_COEF**2 * (1 + 2 * U16)
    return TAU + g * s + gamma(2) * (1 + g) * s


def first_order_coef(k: int) -> Fr:
    """Eq. main_bound_first_order: gamma_k + 14 u32."""
    return gamma(k) + 14 * U32


def elementwise_depth(K: int, kb: int) -> int:
    """Largest number of FP32 roundings any single exact term passes through in
    the blocked elementwise order (Eq. elementwise with blocks of kb): up to
    kb-1 inside its block sum, then three merges per block from its own block
    to the last.  The paper prints no elementwise bound (Sec. 4.5); this depth
    feeds the standard summation bound |C - S| <= gamma_depth * sum|terms|."""
    if K == 0:
        return 0
    nblocks = -(-K // kb)
    return (min(kb, K) - 1) + 3 * nblocks


def cross_first_depth(K: int, kb: int) -> int:
    """Same count for the cross-terms-first order (end of Sec. 4.5): up to
    kb-1 inside a block sum, then X_g = XA_g + XB_g, then X_g / s + HH_g (the
    division by the power of two s is exact), then the addition to the
    running sum in the term's own block and one more in each later block."""
    if K == 0:
        return 0
    nblocks = -(-K // kb)
    return (min(kb, K) - 1) + 2 + nblocks


def termwise_depth(K: int, kb: int) -> int:
    """Same count for the blocked termwise order: up to kb-1 inside the block,
    up to G more in the stream sum over blocks, then the two final additions."""
    if K == 0:
        return 0
    nblocks = -(-K // kb)
    return (min(kb, K) - 1) + (nblocks - 1) + 2


# --- Sec. 4.1: residual-class probability model ------------------------------

def p_class(x: str, n: int) -> Fr:
    """P(X, N = n): probability that the high-part conversion is of type X
    ('T' truncated, c = 0; 'R' rounded up, c = 1) and the residual has n
    leading zeros below the split (n = -1 is the midpoint tie)."""
    top = L_M - L_M_HIGH - 1  # = 12
    if x not in ("T", "R"):
        raise ValueError(x)
    if n < -1:
        return Fr(0)
    if n == -1:
        return Fr(1, 2 ** (L_M - L_M_HIGH + 1))
    if 0 <= n < top:
        return Fr(1, 2 ** (n + 2))
    if n == top:
        return Fr(1, 2 ** (L_M - L_M_HIGH)) if x == "T" else Fr(0)
    return Fr(0)


def p_gradual_or_underflow(e_off: int) -> Fr:
    """P_{u+gu}(E_offset): the exact residual lies in or below the FP16
    subnormal range (N > E_offset - l_Mhigh + b_low - 3)."""
    lo = e_off - L_M_HIGH + B_LOW - 2
    top = L_M - L_M_HIGH - 1
    return sum((p_class("T", n) + p_class("R", n) for n in range(max(lo, -1), top + 1)),
               Fr(0))


def p_underflow(e_off: int) -> Fr:
    """P_u(E_offset): the exact residual lies below 2^-24
    (N > E_offset + b_low - 3)."""
    lo = e_off + B_LOW - 2
    top = L_M - L_M_HIGH - 1
    return sum((p_class("T", n) + p_class("R", n) for n in range(max(lo, -1), top + 1)),
               Fr(0))
