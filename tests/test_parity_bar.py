"""The full-size GPU parity checks, exercised on the CPU with results whose
correctness is known.

At long K the componentwise bar 2K u32 (|A||B|)_ij is wider than the
correction terms A_lo B_hi / s and A_hi B_lo / s themselves, so on its own it
would accept a kernel that dropped one of them.  The GPU tests therefore also
require max|C_gpu - C_oracle| <= 0.1 max|C_oracle - C_hi_only| (and the same
for Frobenius norms).  Here a result that drops XB (or mis-scales the cross
terms) must fail that check while passing the componentwise bar, and a result
that sums the same three terms exactly (a correct kernel with a better
summation than FP32) must pass both.  The sampled rows cover every 256-row
band of C."""
import numpy as np
import pytest

import oracle
import workloads
from tests.helpers import abs_ab, assert_discriminates, assert_parity, band_rows


@pytest.mark.parametrize("M", [256, 4096, 8192, 16384])
def test_band_rows_cover_every_tile_band(M):
    rows = band_rows(M, 3)
    assert rows[0] == 0 and rows[-1] == M - 1
    assert set(rows // 256) == set(range(M // 256))
    offsets = {int(r % 256) for r in rows}
    assert len(offsets) >= min(M // 256, 8)


@pytest.fixture(scope="module")
def c2_rows():
    w = workloads.get("c2")
    A, B = workloads.workload_operands(w)
    rows = band_rows(w.M, 5)
    s = 2.0**11
    ha, la = oracle.split(A[rows], s)
    hb, lb = oracle.split(B, s)
    wid = lambda h: oracle.f16_to_f32(h).astype(np.float64)
    HH = wid(ha) @ wid(hb)
    XA = wid(la) @ wid(hb)
    XB = wid(ha) @ wid(lb)
    return w, A, B, rows, s, HH, XA, XB


def test_dropped_cross_term_passes_the_bar_but_not_the_discriminator(c2_rows):
    w, A, B, rows, s, HH, XA, XB = c2_rows
    Co = oracle.sgemm_rows(A, B, rows, s, "termwise", kb=32)
    Ch = oracle.sgemm_rows(A, B, rows, s, "hi_only", kb=32)
    absab = abs_ab(A, B, rows)
    exact3 = (HH + (XA + XB) / s).astype(np.float32)
    no_xb = (HH + XA / s).astype(np.float32)
    twice = (HH + 2.0 * (XA + XB) / s).astype(np.float32)
    # A correct result passes both checks.
    assert_parity(exact3, Co, w.K, absab, "exact three-term sum")
    assert_discriminates(exact3, Co, Ch, "exact three-term sum")
    # Dropping XB stays inside the componentwise bar at K = 4096 ...
    assert_parity(no_xb, Co, w.K, absab, "XB dropped")
    # ... and is caught by the discriminator, as is a factor 2 on the cross terms.
    with pytest.raises(AssertionError):
        assert_discriminates(no_xb, Co, Ch, "XB dropped")
    with pytest.raises(AssertionError):
        assert_discriminates(twice, Co, Ch, "cross terms doubled")


def test_other_correct_orders_pass_the_discriminator(c2_rows):
    """The oracle's other orders and block sizes differ from the termwise
    result only by FP32 summation order; all pass."""
    w, A, B, rows, s, *_ = c2_rows
    Co = oracle.sgemm_rows(A, B, rows, s, "termwise", kb=32)
    Ch = oracle.sgemm_rows(A, B, rows, s, "hi_only", kb=32)
    for order, kb in (("elementwise", 32), ("elementwise", 64), ("elementwise_cross_first", 32),
                      ("termwise", 128)):
        C = oracle.sgemm_rows(A, B, rows, s, order, kb=kb)
        assert_discriminates(C, Co, Ch, f"{order} kb={kb}")
