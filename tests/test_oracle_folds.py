"""Exact pins of the multi-block folds (Sec. 4.5) on hand-worked cases.

tests/golden/fold_orders.txt lists, for two small dot products with three
blocks, every rounding step of Eq. elementwise, Eq. termwise and the
cross-terms-first order of the end of Sec. 4.5.  This test re-derives each
step here with explicit binary32 round-to-nearest operations (numpy float32,
one operation per step, no fused multiply-add), checks the listed values, and
then requires the oracle to produce exactly the listed results.  Each case
also lists the result of a plausible misreading of the fold (the cross terms
added after HH_g went into the accumulator; a block folded on its own before
joining the accumulator; the termwise cross sums added together first): those
must differ, so an oracle that made one of these mistakes fails here."""
import numpy as np
import pytest

import oracle
from tests.helpers import GOLDEN

f32 = np.float32


def _cases():
    cases, cur = [], None
    with open(f"{GOLDEN}/fold_orders.txt") as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            key, *rest = line.split()
            if key == "case":
                cur = {"name": rest[0], "block": [], "elementwise": [], "cross_first": [],
                       "result": {}, "mutant": {}}
                cases.append(cur)
            elif key in ("s", "kb"):
                cur[key] = float.fromhex(rest[0]) if key == "s" else int(rest[0])
            elif key in ("a", "b", "a_hi", "a_lo", "b_hi", "b_lo", "termwise"):
                cur[key] = [float.fromhex(v) for v in rest]
            elif key in ("block", "elementwise", "cross_first"):
                cur[key].append([float.fromhex(v) for v in rest[1:]])
            elif key in ("result", "mutant"):
                cur[key][rest[0]] = float.fromhex(rest[1])
    return cases


CASES = _cases()


def _fl16(x):
    return f32(np.float16(f32(x)))


def _derive(c):
    """Every step of the three folds, one RN binary32 operation at a time."""
    s = f32(c["s"])
    inv = f32(1.0 / c["s"])
    a = [f32(v) for v in c["a"]]
    b = [f32(v) for v in c["b"]]
    a_hi = [_fl16(v) for v in a]
    a_lo = [_fl16(f32(v - h) * s) for v, h in zip(a, a_hi)]
    b_hi = [_fl16(v) for v in b]
    b_lo = [_fl16(f32(v - h) * s) for v, h in zip(b, b_hi)]
    K, kb = len(a), c["kb"]
    blocks = []
    for k0 in range(0, K, kb):
        hh = xa = xb = f32(0.0)
        for k in range(k0, min(K, k0 + kb)):
            hh = f32(hh + f32(a_hi[k] * b_hi[k]))
            xa = f32(xa + f32(a_lo[k] * b_hi[k]))
            xb = f32(xb + f32(a_hi[k] * b_lo[k]))
        blocks.append([hh, xa, xb])
    el, acc = [], f32(0.0)
    for hh, xa, xb in blocks:
        t1 = f32(acc + hh)
        t2 = f32(t1 + f32(xa * inv))
        acc = f32(t2 + f32(xb * inv))
        el.append([t1, t2, acc])
    HH = XA = XB = f32(0.0)
    for hh, xa, xb in blocks:
        HH, XA, XB = f32(HH + hh), f32(XA + xa), f32(XB + xb)
    t = f32(HH + f32(XA * inv))
    tw = [HH, XA, XB, t, f32(t + f32(XB * inv))]
    cf, acc = [], f32(0.0)
    for hh, xa, xb in blocks:
        x = f32(xa + xb)
        blk = f32(f32(x * inv) + hh)
        acc = f32(acc + blk)
        cf.append([x, blk, acc])
    m1 = f32(0.0)
    for hh, xa, xb in blocks:
        m1 = f32(f32(m1 + hh) + f32(f32(xa + xb) * inv))
    m2 = f32(0.0)
    for hh, xa, xb in blocks:
        m2 = f32(m2 + f32(f32(hh + f32(xa * inv)) + f32(xb * inv)))
    m3 = f32(HH + f32(f32(XA * inv) + f32(XB * inv)))
    return {
        "a_hi": a_hi, "a_lo": a_lo, "b_hi": b_hi, "b_lo": b_lo, "block": blocks,
        "elementwise": el, "termwise": tw, "cross_first": cf,
        "result": {"elementwise": el[-1][2], "termwise": tw[4],
                   "elementwise_cross_first": cf[-1][2]},
        "mutant": {"cross_first_hh_into_acc_first": m1, "elementwise_block_folded_first": m2,
                   "termwise_cross_sums_added_first": m3},
    }


def _same_bits(x, y):
    return np.float32(x).view(np.uint32) == np.float32(y).view(np.uint32)


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_listed_steps_follow_from_the_equations(c):
    d = _derive(c)
    for key in ("a_hi", "a_lo", "b_hi", "b_lo", "termwise"):
        assert all(_same_bits(x, y) for x, y in zip(d[key], c[key])), key
    for key in ("block", "elementwise", "cross_first"):
        assert len(d[key]) == len(c[key]) >= 3, key
        for g, (row_d, row_c) in enumerate(zip(d[key], c[key])):
            assert all(_same_bits(x, y) for x, y in zip(row_d, row_c)), (key, g)
    for kind in ("result", "mutant"):
        for name, v in c[kind].items():
            assert _same_bits(d[kind][name], v), (kind, name)


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_the_case_separates_every_order_and_misreading(c):
    r, m = c["result"], c["mutant"]
    vals = [np.float32(r[o]).view(np.uint32) for o in
            ("elementwise", "termwise", "elementwise_cross_first")]
    assert len(set(int(v) for v in vals)) == 3
    assert not _same_bits(m["cross_first_hh_into_acc_first"], r["elementwise_cross_first"])
    assert not _same_bits(m["elementwise_block_folded_first"], r["elementwise"])
    assert not _same_bits(m["termwise_cross_sums_added_first"], r["termwise"])


@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_oracle_split_matches_the_listed_words(c):
    for x, hi_key, lo_key in (("a", "a_hi", "a_lo"), ("b", "b_hi", "b_lo")):
        hi, lo = oracle.split(np.array(c[x], dtype=np.float32), c["s"])
        assert np.array_equal(oracle.f16_to_f32(hi).ravel(), np.array(c[hi_key], np.float32))
        assert np.array_equal(oracle.f16_to_f32(lo).ravel(), np.array(c[lo_key], np.float32))


@pytest.mark.parametrize("order", ["elementwise", "termwise", "elementwise_cross_first"])
@pytest.mark.parametrize("c", CASES, ids=[c["name"] for c in CASES])
def test_oracle_folds_give_the_listed_bits(c, order):
    A = np.array(c["a"], dtype=np.float32).reshape(1, -1)
    B = np.array(c["b"], dtype=np.float32).reshape(-1, 1)
    got = oracle.sgemm(A, B, c["s"], order, kb=c["kb"])[0, 0]
    assert _same_bits(got, c["result"][order]), (order, float(got).hex())
    # The same entry inside a larger product (other rows and columns of
    # different data) is computed the same way.
    rng = np.random.default_rng(5)
    A2 = rng.uniform(-1, 1, (3, A.shape[1])).astype(np.float32)
    B2 = rng.uniform(-1, 1, (B.shape[0], 4)).astype(np.float32)
    A2[1] = A[0]
    B2[:, 2] = B[:, 0]
    got2 = oracle.sgemm(A2, B2, c["s"], order, kb=c["kb"])[1, 2]
    assert _same_bits(got2, c["result"][order])
