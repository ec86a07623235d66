"""GPU split (sgemm_cube_split) against the oracle: bitwise equality of the
FP16 hi and lo planes (Sec. 3.3, Eq. recover_eqn); NaNs compared by class.

Covers every FP32 bit pattern (exhaustive 2^32 sweep in 16 chunks), the five
workload distributions, special values, odd shapes, padded leading
dimensions and misaligned bases (the kernel's scalar path)."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, padded, split

pytestmark = pytest.mark.gpu


def _nan16(h):
    return ((h & 0x7C00) == 0x7C00) & ((h & 0x03FF) != 0)


def assert_same_planes(got, want, what):
    nan = _nan16(want)
    assert np.array_equal(_nan16(got), nan), f"{what}: NaN pattern"
    assert np.array_equal(got[~nan], want[~nan]), (
        f"{what}: {int(np.count_nonzero(got[~nan] != want[~nan]))} mismatches")


SPECIAL = np.array([
    0.0, -0.0, 1.0, -1.0, 65504.0, 65519.996, 65520.0, -65520.0, 1e30, -1e30,
    np.inf, -np.inf, np.nan, 2.0**-14, 2.0**-15, 2.0**-24, 2.0**-25, 3 * 2.0**-26,
    2.0**-26, 1e-40, -1e-40, 1.4e-45, 32784.0, 2049.0, 2051.0, 1 + 2.0**-11,
    1 + 3 * 2.0**-12, 0.1, -0.3, 3.4028235e38,
], dtype=np.float32)


@pytest.mark.parametrize("s_b", [0, 6, 11, 12, 13, 24])
def test_special_values(gpu, s_b):
    log(f"split special values s_b={s_b}")
    X = np.tile(SPECIAL, (3, 1))
    hi, lo = split(X, 2.0**s_b)
    ohi, olo = oracle.split(X, 2.0**s_b)
    assert_same_planes(hi, ohi, "hi")
    assert_same_planes(lo, olo, "lo")


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_distributions(gpu, name):
    w = workloads.get(name)
    A, B = workloads.make_operands(min(w.M, 512), min(w.N, 384), min(w.K, 1000), w.seed, w.dist)
    for X in (A, B):
        for s in w.scales:
            log(f"split {name} {X.shape} s={s}")
            hi, lo = split(X, s)
            ohi, olo = oracle.split(X, s)
            assert_same_planes(hi, ohi, f"{name} hi")
            assert_same_planes(lo, olo, f"{name} lo")


@pytest.mark.parametrize("rows,cols,ldx,offset", [
    (1, 1, 1, 0), (1, 3, 5, 1), (7, 13, 13, 0), (7, 13, 16, 3), (33, 1027, 1030, 2),
    (128, 64, 64, 0), (5, 4096, 4100, 1),
])
def test_shapes_strides_alignment(gpu, rows, cols, ldx, offset):
    import torch

    from paper_2507_23387_amd import binding

    log(f"split shape {rows}x{cols} ldx={ldx} offset={offset}")
    rng = np.random.default_rng(rows * 1000 + cols)
    X = (rng.standard_normal((rows, cols)) * np.exp2(rng.integers(-20, 16, (rows, cols)))
         ).astype(np.float32)
    _, view = padded(X, ldx, offset=offset)
    ldh = cols + 3
    hi = torch.full((rows * ldh,), -1, dtype=torch.int16, device="cuda")
    lo = torch.full((rows * ldh,), -1, dtype=torch.int16, device="cuda")
    st = binding.sgemm_cube_split(rows, cols, view.data_ptr(), ldx, hi.data_ptr(), lo.data_ptr(),
                                  ldh, 2048.0, torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    h = hi.cpu().numpy().view(np.uint16).reshape(rows, ldh)
    l = lo.cpu().numpy().view(np.uint16).reshape(rows, ldh)
    ohi, olo = oracle.split(X, 2048.0)
    assert_same_planes(h[:, :cols], ohi, "hi")
    assert_same_planes(l[:, :cols], olo, "lo")
    assert np.all(h[:, cols:] == 0xFFFF) and np.all(l[:, cols:] == 0xFFFF)  # padding untouched


@pytest.mark.parametrize("chunk", range(16))
def test_exhaustive_2_32(gpu, chunk):
    """All 2^32 FP32 bit patterns, 2^28 per test, with s = 2^11."""
    import torch

    from paper_2507_23387_amd import binding

    n = 1 << 28
    start = chunk * n
    log(f"split exhaustive chunk {chunk}")
    bits = torch.arange(start, start + n, dtype=torch.int64, device="cuda").to(torch.int32)
    X = bits.view(torch.float32)
    rows, cols = 1 << 14, 1 << 14
    hi = torch.empty(n, dtype=torch.int16, device="cuda")
    lo = torch.empty(n, dtype=torch.int16, device="cuda")
    st = binding.sgemm_cube_split(rows, cols, X.data_ptr(), cols, hi.data_ptr(), lo.data_ptr(),
                                  cols, 2048.0, torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    del bits, X
    h = hi.cpu().numpy().view(np.uint16)
    l = lo.cpu().numpy().view(np.uint16)
    x = (np.arange(n, dtype=np.uint32) + np.uint32(start)).view(np.float32).reshape(rows, cols)
    ohi, olo = oracle.split(x, 2048.0)
    assert_same_planes(h, ohi.reshape(-1), f"hi chunk {chunk}")
    assert_same_planes(l, olo.reshape(-1), f"lo chunk {chunk}")
