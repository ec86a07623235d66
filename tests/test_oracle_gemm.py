"""Pins for the oracle's three-product GEMM (Eq. recover_eqn, Sec. 4.3) and its
accumulation orders (Eq. elementwise, Eq. termwise, Sec. 4.5).

What fixes the answer independently of the oracle:
  * exact recovery: inputs built so that a = hi + lo/s_f exactly, B exactly
    FP16, and every partial sum exact in FP32 -> C equals A*B exactly;
  * the dropped lo*lo term: with single products the deficit A*B - C is
    exactly r_A r_B (the term Eq. recover_eqn drops), r = a - fl16(a) taken
    from numpy's own float16 conversion;
  * Eq. ll_bound, Eq. truncation and Eq. main_bound, checked by brute force in
    exact rational arithmetic on small inputs, and Eq. main_bound at the
    256^3 workload against an FP64 GEMM;
  * textbook reductions: FP16-exact inputs make every order a plain FP32 GEMM;
    one block (kb >= K) makes the elementwise and termwise orders identical.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from oracle import bounds
from tests.helpers import abs_ab, claims, ref64

ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]


def _fp16_exact(rng, shape, lo=-4, hi=4):
    return rng.integers(lo, hi + 1, size=shape).astype(np.float32)


@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("kb", [1, 7, 64, 1000])
def test_exact_recovery_when_inputs_fit_hi_plus_lo(order, kb):
    """A = n * 2^-7 with |n| < 2^15 (so hi keeps 11 bits and the residual,
    a multiple of 2^-7 below 2^-3, is exact in FP16 after scaling by 2^11);
    B small integers (exact FP16, lo_B = 0).  Every block sum and merge is an
    integer multiple of 2^-7 below 2^16, exact in FP32, so C == A B."""
    rng = np.random.default_rng(11)
    M, N, K = 9, 13, 64
    A = (rng.integers(-(2**15) + 1, 2**15, size=(M, K)) * 2.0**-7).astype(np.float32)
    B = _fp16_exact(rng, (K, N))
    # the construction really does exercise the residual
    hi, lo = oracle.split(A, 2.0**11)
    assert np.count_nonzero(lo) > A.size // 2
    C = oracle.sgemm(A, B, 2.0**11, order, kb=kb)
    assert np.array_equal(C.astype(np.float64), ref64(A, B))


@pytest.mark.parametrize("order", ORDERS)
def test_dropped_low_low_term_is_exactly_the_deficit(order):
    """K = 1 and a, b in [2^11, 1.5 * 2^11) scaled by signs: hh + xa/s + xb/s is
    an integer below 2^24 (exact), so A B - C = r_A r_B, the product of the
    two residuals that Eq. recover_eqn drops."""
    rng = np.random.default_rng(5)
    M, N = 40, 50
    A = (rng.integers(2**11, 3 * 2**10, size=(M, 1)) * rng.choice([-1, 1], (M, 1))).astype(
        np.float32)
    B = (rng.integers(2**11, 3 * 2**10, size=(1, N)) * rng.choice([-1, 1], (1, N))).astype(
        np.float32)
    C = oracle.sgemm(A, B, 2.0**11, order).astype(np.float64)
    rA = A.astype(np.float64) - A.astype(np.float16).astype(np.float64)
    rB = B.astype(np.float64) - B.astype(np.float16).astype(np.float64)
    deficit = ref64(A, B) - C
    assert np.array_equal(deficit, rA @ rB)
    assert np.count_nonzero(rA @ rB) > 0


def _window_operands(rng, M, N, K, s_b=11):
    """Entries sign * u * 2^e with e in [-12, 12]: hi normal, Rules 1-2 hold
    for s_b = 11 (the long-K workload's distribution)."""
    sign = rng.choice([-1.0, 1.0], size=(M + N, K))
    u = rng.uniform(1.0, 2.0, size=(M + N, K))
    e = rng.integers(-12, 13, size=(M + N, K))
    X = np.ldexp(sign * u, e).astype(np.float32)
    return X[:M], X[M:].T.copy()


def _exact(X):
    return [[Fraction(float(v)) for v in row] for row in X]


def _exact_matmul(A, B):
    M, K, N = len(A), len(B), len(B[0])
    return [[sum((A[i][k] * B[k][j] for k in range(K)), Fraction(0)) for j in range(N)]
            for i in range(M)]


def _adversarial(rng, M, N, K):
    """Heavy cancellation in row 0 of C: its last A entry is 2^12 and the last
    row of B cancels the rest of the inner product (entries kept inside the
    Rule 1-2 window, |x| in [2^-12, 2^13))."""
    sign = rng.choice([-1.0, 1.0], size=(M + N, K))
    u = rng.uniform(1.0, 2.0, size=(M + N, K))
    e = rng.integers(-6, 4, size=(M + N, K))
    X = np.ldexp(sign * u, e).astype(np.float32)
    A, B = X[:M].copy(), X[M:].T.copy()
    A[0, -1] = 2.0**12
    last = -(A[0, :-1].astype(np.float64) @ B[:-1, :].astype(np.float64)) / 2.0**12
    last = np.where(np.abs(last) < 2.0**-12, np.copysign(2.0**-12, last), last)
    B[-1, :] = last.astype(np.float32)
    return A, B


@pytest.mark.parametrize("case", range(6))
def test_truncation_and_main_bound_brute_force(case):
    """Exact rationals on small inputs:
      Eq. truncation: T = AB - S satisfies |T| <= tau |A||B|, S the exact sum
        of the three computed terms built from the oracle's split;
      Eq. ll_bound: |R_A R_B| / s^2 <= u16^2 (1+u16)^2 |A||B|;
      Eq. main_bound: the termwise result satisfies |AB - C| <= coef(k) |A||B|;
      the elementwise and the cross-terms-first results satisfy
        |S - C| <= gamma_d sum|terms| with d the order's longest rounding
        chain (the paper prints no bound for either)."""
    rng = np.random.default_rng(100 + case)
    M, N, K = 4, 5, [1, 3, 8, 8, 16, 5][case]
    kb = [1, 2, 3, 8, 4, 64][case]
    if case % 2:
        A, B = _adversarial(rng, M, N, K)
    else:
        A, B = _window_operands(rng, M, N, K)
    s = 2.0**11
    Ahi, Alo = oracle.split(A, s)
    Bhi, Blo = oracle.split(B, s)
    ah, al = _exact(oracle.f16_to_f32(Ahi)), _exact(oracle.f16_to_f32(Alo))
    bh, bl = _exact(oracle.f16_to_f32(Bhi)), _exact(oracle.f16_to_f32(Blo))
    Ae, Be = _exact(A), _exact(B)
    AB = _exact_matmul(Ae, Be)
    absA = [[abs(v) for v in r] for r in Ae]
    absB = [[abs(v) for v in r] for r in Be]
    absAB = _exact_matmul(absA, absB)
    sf = Fraction(int(s))
    S = [[sum((ah[i][k] * bh[k][j] + (al[i][k] * bh[k][j] + ah[i][k] * bl[k][j]) / sf
               for k in range(K)), Fraction(0)) for j in range(N)] for i in range(M)]
    LL = [[sum((al[i][k] * bl[k][j] for k in range(K)), Fraction(0)) / sf**2 for j in range(N)]
          for i in range(M)]
    terms = [[sum((abs(ah[i][k] * bh[k][j]) + abs(al[i][k] * bh[k][j]) / sf
                   + abs(ah[i][k] * bl[k][j]) / sf for k in range(K)), Fraction(0))
              for j in range(N)] for i in range(M)]
    Ct = oracle.sgemm(A, B, s, "termwise", kb=kb)
    Ce = oracle.sgemm(A, B, s, "elementwise", kb=kb)
    Cc = oracle.sgemm(A, B, s, "elementwise_cross_first", kb=kb)
    coef = bounds.main_bound_coef(K)
    d = bounds.elementwise_depth(K, kb)
    ge = bounds.gamma(d)
    gc = bounds.gamma(bounds.cross_first_depth(K, kb))
    for i in range(M):
        for j in range(N):
            T = AB[i][j] - S[i][j]
            assert abs(T) <= bounds.TAU * absAB[i][j]
            assert abs(LL[i][j]) <= bounds.LL_COEF * absAB[i][j]
            assert abs(AB[i][j] - Fraction(float(Ct[i, j]))) <= coef * absAB[i][j]
            assert abs(S[i][j] - Fraction(float(Ce[i, j]))) <= ge * terms[i][j]
            assert abs(S[i][j] - Fraction(float(Cc[i, j]))) <= gc * terms[i][j]


def test_main_bound_at_256_cubed_against_fp64():
    """Eq. main_bound for the termwise order on the 256^3 U[-1,1] workload,
    with the FP64 GEMM as the exact product (its own error, about 1e-16
    relative to |A||B|, is far below the bound's slack).  The few entries
    below 2^-14 (subnormal hi) lie outside the bound's assumptions but do not
    break it at this size."""
    A, B = workloads.workload_operands("c1")
    K = A.shape[1]
    C = oracle.sgemm(A, B, 2.0**11, "termwise").astype(np.float64)
    coef = float(bounds.main_bound_coef(K))
    err = np.abs(ref64(A, B) - C)
    assert np.all(err <= coef * abs_ab(A, B))
    # and it is far more accurate than FP16 (Sec. 6.2: HGEMM error ~1e-4)
    Ch = oracle.sgemm(A, B, 2.0**11, "hi_only").astype(np.float64)
    fro = lambda X: np.linalg.norm(X)
    ref = ref64(A, B)
    assert fro(ref - C) / fro(ref) < 1e-6 < fro(ref - Ch) / fro(ref)


@pytest.mark.parametrize("kb", [1, 5, 64])
def test_fp16_exact_inputs_reduce_to_plain_fp32_gemm(kb):
    """With A and B exactly FP16 both residuals vanish (XA = XB = 0); every
    order then computes the blocked FP32 sum of hi*hi, and with one block it
    is the plain sequential FP32 GEMM computed here with numpy float32."""
    rng = np.random.default_rng(3)
    M, N, K = 17, 19, 40
    A = rng.standard_normal((M, K)).astype(np.float16).astype(np.float32)
    B = rng.standard_normal((K, N)).astype(np.float16).astype(np.float32)
    outs = [oracle.sgemm(A, B, 2.0**11, o, kb=kb) for o in ORDERS + ["hi_only"]]
    for C in outs[1:]:
        assert np.array_equal(C, outs[0])
    plain = np.zeros((M, N), dtype=np.float32)
    for k in range(K):
        plain = plain + np.outer(A[:, k], B[k, :]).astype(np.float32)
    one_block = oracle.sgemm(A, B, 2.0**11, "termwise", kb=K)
    assert np.array_equal(one_block, plain)


def test_one_block_makes_elementwise_equal_termwise():
    """kb >= K: G = 0, and Eq. elementwise ((0 + hh) + xa/s) + xb/s is the
    same expression as Eq. termwise (HH + XA/s) + XB/s."""
    A, B = workloads.make_operands(23, 31, 50, 9, "normal")
    Ce = oracle.sgemm(A, B, 2.0**11, "elementwise", kb=64)
    Ct = oracle.sgemm(A, B, 2.0**11, "termwise", kb=64)
    assert np.array_equal(Ce, Ct)
    Ce2 = oracle.sgemm(A, B, 2.0**11, "elementwise", kb=8)
    assert not np.array_equal(Ce2, Ct)  # blocks do change the rounding


def test_degenerate_shapes():
    A = np.zeros((3, 0), np.float32)
    B = np.zeros((0, 4), np.float32)
    for o in ORDERS + ["hi_only"]:
        C = oracle.sgemm(A, B, 2.0**11, o)
        assert C.shape == (3, 4) and np.all(C == 0)
    assert oracle.sgemm(np.zeros((0, 5), np.float32), np.ones((5, 2), np.float32),
                        2.0**11).shape == (0, 2)


def test_rows_sampling_matches_full():
    A, B = workloads.make_operands(64, 48, 130, 4, "uniform_pm1")
    full = oracle.sgemm(A, B, 2.0**11, "termwise")
    rows = workloads.sample_rows(64, 10, 1)
    assert np.array_equal(oracle.sgemm_rows(A, B, rows, 2.0**11, "termwise"), full[rows])


def test_threads_do_not_change_results():
    A, B = workloads.make_operands(33, 65, 200, 8, "normal")
    C1 = oracle.sgemm(A, B, 2.0**11, "elementwise", threads=1)
    C8 = oracle.sgemm(A, B, 2.0**11, "elementwise", threads=8)
    assert np.array_equal(C1, C8)


def test_termwise_more_accurate_than_elementwise_on_long_k():
    """Sec. 6.2: termwise accumulation is the more accurate order as k grows.
    At K = 4096 with U[0, 1] inputs (no cancellation) termwise's error must be
    below elementwise's."""
    A, B = workloads.offset_exponent_operands(8, 64, 4096, 21, 0, symmetric=False)
    ref = ref64(A, B)
    fro = lambda X: np.linalg.norm(X)
    e_el = fro(ref - oracle.sgemm(A, B, 2.0**12, "elementwise")) / fro(ref)
    e_tw = fro(ref - oracle.sgemm(A, B, 2.0**12, "termwise")) / fro(ref)
    assert e_tw < e_el


def test_scale_claims_constants():
    c = claims()
    assert bounds.U16 == Fraction(2) ** int(c["u16_log2"])
    assert bounds.U32 == Fraction(2) ** int(c["u32_log2"])
