"""Pins for the oracle's FP32 -> FP16 conversion (Sec. 3.2: fl16 is RN-even;
Sec. 4.1: gradual underflow, 2^-25 rounds to zero).

The oracle converts by integer bit manipulation.  It is compared, for every
one of the 2^32 FP32 bit patterns, with two independent library conversions
(numpy's float32 -> float16 and torch's CPU float32 -> float16), both RN-even
with subnormal support.  NaNs are compared by class only."""
import numpy as np
import pytest
import torch

import oracle
from tests.helpers import claims

CHUNK = 1 << 24


def _is_nan16(h):
    return ((h & 0x7C00) == 0x7C00) & ((h & 0x03FF) != 0)


@pytest.mark.slow
def test_exhaustive_2_32_against_torch_and_numpy():
    """Every FP32 bit pattern against torch's CPU conversion, and every 7th
    pattern against numpy's (numpy takes a slow path for chunks that hold
    subnormal or overflowing results; the binades where those behaviours
    begin are compared exhaustively against numpy in the next test)."""
    # Every buffer is allocated once: fresh large allocations are slow to
    # fault in, and the sweep runs 256 chunks of 2^24 patterns.
    base = np.arange(CHUNK, dtype=np.uint32)
    bits = np.empty(CHUNK, dtype=np.uint32)
    ours = np.empty(CHUNK, dtype=np.uint16)
    ref_t = torch.empty(CHUNK, dtype=torch.float16)
    ref_np = np.empty((CHUNK + 6) // 7, dtype=np.float16)
    eq = np.empty(CHUNK, dtype=bool)
    x_t = torch.from_numpy(bits.view(np.float32))
    lib = oracle._load()
    for start in range(0, 1 << 32, CHUNK):
        np.add(base, np.uint32(start), out=bits)
        x = bits.view(np.float32)
        lib.oracle_convert_range(start, CHUNK, ours.ctypes.data)
        ref_t.copy_(x_t)
        r_t = ref_t.view(torch.int16).numpy().view(np.uint16)
        with np.errstate(all="ignore"):
            np.copyto(ref_np, x[::7], casting="unsafe")
        r_np = ref_np.view(np.uint16)
        sub = ours[::7]
        if (start & 0x7F800000) == 0x7F000000:
            # this chunk holds the FP32 NaNs (exponent field all ones): NaNs
            # are compared by class, everything else bit for bit
            nan = _is_nan16(r_t)
            assert np.array_equal(nan, _is_nan16(ours)), hex(start)
            assert np.array_equal(ours[~nan], r_t[~nan]), hex(start)
            nan7 = _is_nan16(r_np)
            assert np.array_equal(sub[~nan7], r_np[~nan7]), hex(start)
        else:
            np.equal(ours, r_t, out=eq)
            assert eq.all(), hex(start)
            assert np.array_equal(sub, r_np), hex(start)


@pytest.mark.parametrize("biased_exp", [101, 102, 103, 111, 112, 113, 141, 142])
def test_boundary_binades_exhaustive_against_numpy(biased_exp):
    """Whole binades (both signs) where RN-even meets the subnormal boundary
    (2^-25 halfway to zero, 2^-14 smallest normal) and the overflow threshold
    (65504 .. 65520 .. 2^16), against numpy."""
    m = np.arange(1 << 23, dtype=np.uint32)
    for sign in (0, 1):
        bits = (np.uint32(sign << 31) | (np.uint32(biased_exp) << np.uint32(23)) | m)
        x = bits.view(np.float32)
        with np.errstate(all="ignore"):
            ref = x.astype(np.float16).view(np.uint16)
        assert np.array_equal(oracle.f32_to_f16(x), ref), (biased_exp, sign)


def test_sampled_against_numpy():
    """A quick version of the exhaustive check (every binade, random mantissas)."""
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 1 << 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    ours = oracle.f32_to_f16(x)
    ref = x.astype(np.float16).view(np.uint16)
    nan = _is_nan16(ref)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(_is_nan16(ours), nan)


def test_widening_exhaustive_2_16():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ours = oracle.f16_to_f32(h)
    ref = h.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan].view(np.uint32), ref[~nan].view(np.uint32))


def test_round_trip_is_identity_on_fp16_values():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    back = oracle.f32_to_f16(oracle.f16_to_f32(h))
    nan = _is_nan16(h)
    assert np.array_equal(back[~nan], h[~nan])


def test_halfway_to_zero_and_smallest_subnormal():
    """Sec. 4.1: values below 2^-25 round to zero, 2^-25 itself is a tie that
    goes to even (zero), values just above round to 2^-24."""
    c = claims()
    half = np.float32(2.0 ** c["halfway_to_zero_log2"])
    above = np.nextafter(half, np.float32(1))
    below = np.nextafter(half, np.float32(0))
    got = oracle.f16_to_f32(oracle.f32_to_f16(np.array([below, half, above, -half, -above],
                                                        dtype=np.float32)))
    assert got[0] == 0 and got[1] == 0 and got[3] == 0
    assert got[2] == 2.0**-24 and got[4] == -(2.0**-24)
    assert np.signbit(got[3])  # sign kept on the zero


def test_overflow_threshold():
    """Largest finite FP16 is 65504; 65520 is the halfway point to 2^16."""
    x = np.array([65504, 65519.996, 65520, 1e30, np.inf, -65520], dtype=np.float32)
    got = oracle.f16_to_f32(oracle.f32_to_f16(x))
    assert got[0] == 65504 and got[1] == 65504
    assert got[2] == np.inf and got[3] == np.inf and got[4] == np.inf and got[5] == -np.inf
