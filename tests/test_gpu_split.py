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


# --- the tiled planes the GEMM reads (sgemm_cube_prepare / sgemm_cube_ex) -----

def _untile(buf, rows_p, Kp):
    """Decode a plane stored as 128-row x 16-k tiles (row r's two 8-value
    chunks swapped when bit 4 of r is set) into a rows_p x Kp array."""
    r = np.arange(rows_p)[:, None]
    k = np.arange(Kp)[None, :]
    tile = (r // 128) * (Kp // 16) + k // 16
    rr, kk = r % 128, k % 16
    return buf[tile * 2048 + rr * 16 + (((kk >> 3) ^ ((rr >> 4) & 1)) << 3) + (kk & 7)]


def _prepared_planes(A, B, scale, lda_pad=0, offset=0):
    """Run sgemm_cube_prepare on (optionally padded, misaligned) copies of A and
    B and decode the four tiled planes (A_hi, A_lo, B^T_hi, B^T_lo)."""
    import torch

    from paper_2507_23387_amd import binding

    M, K = A.shape
    N = B.shape[1]
    _, Av = padded(A, K + lda_pad, offset=offset)
    _, Bv = padded(B, N + lda_pad, offset=offset)
    ws = binding.workspace(M, N, K)
    stream = torch.cuda.current_stream().cuda_stream
    assert binding.sgemm_cube_prepare(M, N, K, Av.data_ptr(), K + lda_pad, Bv.data_ptr(),
                                      N + lda_pad, scale, ws.data_ptr(), ws.numel(), stream) == 0
    torch.cuda.synchronize()
    raw = ws.cpu().numpy()
    Mp, Np, Kp = -(-M // 256) * 256, -(-N // 256) * 256, -(-K // 64) * 64
    sizes = (Mp * Kp * 2, Mp * Kp * 2, Np * Kp * 2, Np * Kp * 2)
    planes, off = [], 256
    for n in sizes:
        planes.append(raw[off:off + n].view(np.uint16))
        off += -(-n // 256) * 256
    return (_untile(planes[0], Mp, Kp), _untile(planes[1], Mp, Kp),
            _untile(planes[2], Np, Kp), _untile(planes[3], Np, Kp))


@pytest.mark.parametrize("s_b", [0, 11, 12, 24])
@pytest.mark.parametrize("lda_pad,offset", [(0, 0), (3, 1)], ids=["aligned", "misaligned"])
def test_tiled_planes_special_values_bitwise(gpu, s_b, lda_pad, offset):
    """Every special value in both operands, in the aligned (vector) and the
    padded, misaligned (scalar) path of the tiled split kernels, against the
    oracle's split bit for bit; the padding holds zeros."""
    rng = np.random.default_rng(s_b + 10 * lda_pad)
    M, K, N = 150, 70, 130
    A = rng.choice(SPECIAL, size=(M, K)).astype(np.float32)
    B = rng.choice(SPECIAL, size=(K, N)).astype(np.float32)
    log(f"tiled planes special s_b={s_b} pad={lda_pad} off={offset}")
    ah, al, bh, bl = _prepared_planes(A, B, 2.0**s_b, lda_pad, offset)
    oah, oal = oracle.split(A, 2.0**s_b)
    obh, obl = oracle.split(B, 2.0**s_b)
    assert_same_planes(ah[:M, :K], oah, "A hi")
    assert_same_planes(al[:M, :K], oal, "A lo")
    assert_same_planes(bh[:N, :K], obh.T, "B hi")
    assert_same_planes(bl[:N, :K], obl.T, "B lo")
    for p in (ah, al):
        assert not p[M:].any() and not p[:, K:].any()
    for p in (bh, bl):
        assert not p[N:].any() and not p[:, K:].any()


def test_tiled_planes_prescaled_bitwise(gpu):
    """With pre-scaling the planes hold the split of the power-of-two-scaled
    operands (the oracle's prescale_exponents applied to A's rows and B's
    columns), bit for bit."""
    import torch

    from paper_2507_23387_amd import binding

    rng = np.random.default_rng(5)
    M, K, N = 260, 100, 140
    A = (rng.uniform(-1, 1, (M, K)) * np.ldexp(1.0, rng.integers(-40, 30, (M, 1)))).astype(np.float32)
    B = (rng.uniform(-1, 1, (K, N)) * np.ldexp(1.0, rng.integers(-40, 30, (1, N)))).astype(np.float32)
    A[3, :] = 0.0
    A[5, 7] = np.nan
    scale = 2048.0
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    n = binding.sgemm_cube_ex_workspace_size(M, N, K, 1, binding.OPT_PRESCALE)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    log("tiled planes prescaled")
    assert binding.sgemm_cube_ex(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(), N,
                                 scale, 1, binding.OPT_PRESCALE, ws.data_ptr(), n, None,
                                 torch.cuda.current_stream().cuda_stream) == 0
    torch.cuda.synchronize()
    raw = ws.cpu().numpy()
    Mp, Np, Kp = 512, 256, 128
    off, planes = 256, []
    for size in (Mp * Kp * 2, Mp * Kp * 2, Np * Kp * 2, Np * Kp * 2):
        planes.append(raw[off:off + size].view(np.uint16))
        off += size
    ea, eb = oracle.prescale_targets(scale)
    As = np.ldexp(A, oracle.prescale_exponents(A, 1, ea)[:, None].astype(np.int32)).astype(np.float32)
    Bs = np.ldexp(B, oracle.prescale_exponents(B, 0, eb)[None, :].astype(np.int32)).astype(np.float32)
    oah, oal = oracle.split(As, scale)
    obh, obl = oracle.split(Bs, scale)
    assert_same_planes(_untile(planes[0], Mp, Kp)[:M, :K], oah, "A hi")
    assert_same_planes(_untile(planes[1], Mp, Kp)[:M, :K], oal, "A lo")
    assert_same_planes(_untile(planes[2], Np, Kp)[:N, :K], obh.T, "B hi")
    assert_same_planes(_untile(planes[3], Np, Kp)[:N, :K], obl.T, "B lo")
