"""GPU GEMM (sgemm_cube, sgemm_cube_hgemm) against the oracle.

Bar: |C_gpu - C_oracle|_ij <= 2 K 2^-24 (|A||B|)_ij for every compared entry,
equality where (|A||B|)_ij = 0, identical inf/NaN patterns.  The oracle runs
with the GPU's elementwise block size (sgemm_cube_block_k() = 32), so both
sides fold the same blocks g of Eq. elementwise; the summation inside a block
differs (MFMA versus sequential, and on the scaled path each block term is
rounded together with the accumulator), which the bar covers.

Small and ragged shapes are compared in full; the five workloads at their full
size are compared on sampled rows (each output row needs only its row of A
and all of B, so the oracle computes exactly those rows)."""
import numpy as np
import pytest

import oracle
import workloads
from oracle import bounds
from tests.gpu_util import gemm, hgemm, log, padded, split, to_dev
from tests.helpers import abs_ab, assert_discriminates, assert_parity, band_rows, ref64

pytestmark = pytest.mark.gpu

ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]
SHAPES = [
    (1, 1, 1), (1, 7, 3), (5, 3, 1), (17, 33, 65), (64, 64, 64), (128, 128, 64),
    (129, 130, 65), (300, 200, 1000), (256, 256, 256), (200, 129, 4103), (513, 640, 192),
]


def _kb(order="elementwise"):
    """The oracle's block size matching the GPU's: one 32-wide k-step of
    v_mfma_f32_16x16x32_f16, the same in every order and kernel."""
    from paper_2507_23387_amd import binding

    return binding.sgemm_cube_block_k()


@pytest.mark.parametrize("order", ORDERS)
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_shapes_full_parity(gpu, order, shape):
    M, N, K = shape
    log(f"gemm {order} {M}x{N}x{K}")
    A, B = workloads.make_operands(M, N, K, M + N + K, "normal")
    C = gemm(A, B, 2048.0, order)
    Co = oracle.sgemm(A, B, 2048.0, order, kb=_kb(order))
    assert_parity(C, Co, K, abs_ab(A, B), f"{order} {shape}")


@pytest.mark.parametrize("shape", [(1, 1, 1), (129, 130, 65), (256, 256, 256), (300, 200, 1000)],
                         ids=lambda s: "x".join(map(str, s)))
def test_hgemm_parity(gpu, shape):
    M, N, K = shape
    log(f"hgemm {M}x{N}x{K}")
    A, B = workloads.make_operands(M, N, K, 77, "uniform_pm1")
    C = hgemm(A, B)
    Co = oracle.sgemm(A, B, 2048.0, "hi_only", kb=_kb())
    assert_parity(C, Co, K, abs_ab(A, B), "hgemm")


@pytest.mark.parametrize("order", ORDERS)
def test_padded_leading_dimensions_and_misaligned_bases(gpu, order):
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 133, 71, 300
    lda, ldb, ldc = K + 3, N + 5, N + 7
    log(f"gemm padded ld {order}")
    A, B = workloads.make_operands(M, N, K, 5, "uniform_pm1")
    _, Av = padded(A, lda, offset=1)
    _, Bv = padded(B, ldb, offset=3)
    Cbuf = torch.full((2 + M * ldc,), float("nan"), dtype=torch.float32, device="cuda")
    Cv = Cbuf[2:].view(M, ldc)
    st = binding.sgemm_cube(M, N, K, Av.data_ptr(), lda, Bv.data_ptr(), ldb, Cv.data_ptr(), ldc,
                            2048.0, binding.ORDERS[order], torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    Cn = Cv.cpu().numpy()
    assert np.isnan(Cn[:, N:]).all(), "wrote outside the M x N block"
    assert np.isnan(Cbuf[:2].cpu().numpy()).all()
    Co = oracle.sgemm(A, B, 2048.0, order, kb=_kb(order))
    assert_parity(Cn[:, :N], Co, K, abs_ab(A, B), "padded")


def test_k_zero_writes_zero_and_empty_is_noop(gpu):
    import torch

    from paper_2507_23387_amd import binding

    log("gemm K=0 / M=0")
    C = torch.full((5, 6), float("nan"), device="cuda")
    A = torch.empty((5, 0), device="cuda")
    B = torch.empty((0, 6), device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    assert binding.sgemm_cube(5, 6, 0, A.data_ptr(), 1, B.data_ptr(), 6, C.data_ptr(), 6, 2048.0,
                              0, stream) == 0
    torch.cuda.synchronize()
    assert (C.cpu().numpy() == 0).all()
    C.fill_(float("nan"))
    B4 = torch.ones((4, 6), device="cuda")
    assert binding.sgemm_cube(0, 6, 4, 0, 4, B4.data_ptr(), 6, C.data_ptr(), 6, 2048.0, 1,
                              stream) == 0
    torch.cuda.synchronize()
    assert np.isnan(C.cpu().numpy()).all()


@pytest.mark.parametrize("order", ORDERS)
def test_non_finite_inputs_propagate_like_the_oracle(gpu, order):
    """No range guard (Sec. 3.1): |a| >= 65520, lo overflow, inf and NaN
    inputs give the same inf/NaN pattern as the oracle."""
    M, N, K = 40, 50, 70
    A, B = workloads.make_operands(M, N, K, 9, "uniform_pm1")
    A[3, 5] = 70000.0      # hi overflows
    A[7, 9] = np.inf
    B[11, 13] = np.nan
    B[20, 21] = 32784.0    # lo overflows with s = 2^12 (Sec. 4.2 example)
    log(f"gemm non-finite {order}")
    C = gemm(A, B, 4096.0, order)
    Co = oracle.sgemm(A, B, 4096.0, order, kb=_kb(order))
    assert_parity(C, Co, K, abs_ab(A, B), "non-finite")
    assert np.isnan(Co).any()


def test_non_finite_inputs_on_the_scaled_elementwise_path(gpu):
    """The same special values with B kept inside the scaled kernel's range
    (|B_hi| s <= 65504), A carrying the hi and lo overflows instead."""
    M, N, K = 40, 50, 70
    A, B = workloads.make_operands(M, N, K, 19, "uniform_pm1")
    A[3, 5] = 70000.0      # hi overflows
    A[7, 9] = -np.inf
    A[20, 21] = 32784.0    # lo overflows with s = 2^12
    B[11, 13] = np.nan
    log("gemm non-finite, scaled elementwise path")
    C = gemm(A, B, 4096.0, "elementwise")
    Co = oracle.sgemm(A, B, 4096.0, "elementwise", kb=_kb())
    assert_parity(C, Co, K, abs_ab(A, B), "non-finite scaled")
    assert np.isnan(Co).any() and np.isinf(Co).any()


@pytest.mark.parametrize("order", ["elementwise", "elementwise_cross_first"])
@pytest.mark.parametrize("edge", ["scaled_limit", "fallback"])
def test_elementwise_range_switch(gpu, edge, order):
    """The scaled kernels of the elementwise and cross-terms-first orders need
    s * B_hi to stay finite in FP16.  B's largest hi exactly at 65504 / s
    keeps them; one FP16 ulp above switches to the unscaled fallback of the
    order.  Both meet the bar and discriminate against the FP16 product, on
    ragged shapes."""
    M, N, K = 300, 260, 257
    A, B = workloads.make_operands(M, N, K, 21, "uniform_pm1")
    B[5, 7] = 31.984375 if edge == "scaled_limit" else 32.0   # x 2^11 = 65504 or 65536
    log(f"gemm {order} range switch {edge}")
    C = gemm(A, B, 2048.0, order)
    Co = oracle.sgemm(A, B, 2048.0, order, kb=_kb())
    assert_parity(C, Co, K, abs_ab(A, B), f"range switch {edge}")
    Ch = oracle.sgemm(A, B, 2048.0, "hi_only", kb=_kb())
    assert_discriminates(C, Co, Ch, f"range switch {edge} {order}")


def _range_flag(ws):
    """The workspace header starts with two stamp words; they are equal after a
    split of B that found |B_hi| s > 65504."""
    import torch

    w = ws[:8].view(torch.int32).cpu()
    return int(w[0] == w[1])


def test_range_flag_follows_the_last_split_of_b(gpu):
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 70, 90, 33
    A, B = workloads.make_operands(M, N, K, 23, "uniform_pm1")
    Bbig = B.copy()
    Bbig[0, 0] = 40.0
    dA, dB, dBbig = to_dev(A), to_dev(B), to_dev(Bbig)
    ws = binding.workspace(M, N, K)
    nbytes = ws.numel()
    stream = torch.cuda.current_stream().cuda_stream

    def prep(a, b):
        assert binding.sgemm_cube_prepare(M, N, K, a.data_ptr() if a is not None else 0, K,
                                          b.data_ptr() if b is not None else 0, N, 2048.0,
                                          ws.data_ptr(), nbytes, stream) == 0
        torch.cuda.synchronize()

    log("range flag")
    prep(dA, dBbig)
    assert _range_flag(ws) == 1
    prep(dA, dB)
    assert _range_flag(ws) == 0
    prep(None, dBbig)
    assert _range_flag(ws) == 1
    prep(dA, None)            # re-splitting A alone keeps the flag of the B planes
    assert _range_flag(ws) == 1


def _untile(buf: np.ndarray, rows_p: int, Kp: int) -> np.ndarray:
    """Decode a plane stored as 128-row x 16-k tiles (row r's two 8-value
    chunks swapped when bit 4 of r is set) into a rows_p x Kp array."""
    r = np.arange(rows_p)[:, None]
    k = np.arange(Kp)[None, :]
    tile = (r // 128) * (Kp // 16) + k // 16
    rr, kk = r % 128, k % 16
    idx = tile * 2048 + rr * 16 + (((kk >> 3) ^ ((rr >> 4) & 1)) << 3) + (kk & 7)
    return buf[idx]


def test_prepared_planes_match_the_split_bit_for_bit(gpu):
    """The tiled planes written by sgemm_cube_prepare hold exactly the bits of
    the row-major split (A) and of the split of B, transposed, with zeros in
    the padding."""
    import torch

    from paper_2507_23387_amd import binding

    M, N, K, s = 300, 200, 100, 1024.0
    A, B = workloads.make_operands(M, N, K, 29, "normal")
    dA, dB = to_dev(A), to_dev(B)
    ws = binding.workspace(M, N, K)
    stream = torch.cuda.current_stream().cuda_stream
    log("tiled planes vs split")
    assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, s,
                                      ws.data_ptr(), ws.numel(), stream) == 0
    torch.cuda.synchronize()
    raw = ws.cpu().numpy()
    Mp, Np, Kp = 512, 256, 128
    a_bytes, b_bytes = Mp * Kp * 2, Np * Kp * 2
    planes = []
    off = 256
    for nbytes in (a_bytes, a_bytes, b_bytes, b_bytes):
        planes.append(raw[off:off + nbytes].view(np.uint16))
        off += nbytes
    a_hi, a_lo = (_untile(p, Mp, Kp) for p in planes[:2])
    b_hi, b_lo = (_untile(p, Np, Kp) for p in planes[2:])
    ah, al = split(A, s)
    bh, bl = split(B, s)
    for got, want, rows, cols in ((a_hi, ah, M, K), (a_lo, al, M, K),
                                  (b_hi, bh.T, N, K), (b_lo, bl.T, N, K)):
        assert np.array_equal(got[:rows, :cols], want)
        assert not got[rows:].any() and not got[:, cols:].any()


def test_subnormal_fp16_products_exact(gpu):
    """FP16-subnormal operands (the 2^-14-scaled workload's regime): with
    exactly representable FP16 inputs whose products and sums are exact in
    FP32, the hi-only GEMM must be exact -- the MFMA must neither flush FP16
    denormal inputs nor lose bits of the exact products."""
    rng = np.random.default_rng(4)
    M, N, K = 64, 48, 96
    A = (rng.integers(-1023, 1024, size=(M, K)) * 2.0**-24).astype(np.float32)   # subnormal
    B = rng.integers(-8, 9, size=(K, N)).astype(np.float32)
    log("hgemm subnormal exact")
    C = hgemm(A, B)
    assert np.array_equal(C.astype(np.float64), ref64(A, B))
    for order in ORDERS:
        log(f"sgemm subnormal exact {order}")
        C2 = gemm(A, B, 2048.0, order)
        assert np.array_equal(C2.astype(np.float64), ref64(A, B))


def test_deterministic_and_entry_points_agree(gpu):
    """Repeated calls are bitwise identical, and sgemm_cube (pool workspace),
    sgemm_cube_ws and prepare + compute compute the same bits."""
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 300, 257, 515
    A, B = workloads.make_operands(M, N, K, 12, "normal")
    dA, dB = to_dev(A), to_dev(B)
    stream = torch.cuda.current_stream().cuda_stream
    for order in ORDERS:
        log(f"entry points agree {order}")
        C1 = binding.matmul(dA, dB, 2048.0, order)
        C2 = binding.matmul(dA, dB, 2048.0, order)
        ws = binding.workspace(M, N, K)
        C3 = binding.matmul(dA, dB, 2048.0, order, workspace=ws)
        C4 = torch.empty_like(C1)
        nbytes = ws.numel()
        assert binding.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, 2048.0,
                                          ws.data_ptr(), nbytes, stream) == 0
        assert binding.sgemm_cube_compute(M, N, K, C4.data_ptr(), N, 2048.0,
                                          binding.ORDERS[order], ws.data_ptr(), nbytes,
                                          stream) == 0
        torch.cuda.synchronize()
        for X in (C2, C3, C4):
            assert torch.equal(C1, X)


def test_side_stream(gpu):
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 257, 300, 129
    A, B = workloads.make_operands(M, N, K, 13, "uniform_pm1")
    dA, dB = to_dev(A), to_dev(B)
    log("gemm on a side stream")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        C = binding.matmul(dA, dB, 2048.0, "termwise")
    s.synchronize()
    Co = oracle.sgemm(A, B, 2048.0, "termwise", kb=_kb())
    assert_parity(C.cpu().numpy(), Co, K, abs_ab(A, B), "side stream")


# --- the five workloads at full size, sampled rows ----------------------------

CASES = [
    ("c1", "elementwise", 2.0**11), ("c1", "termwise", 2.0**11),
    ("c2", "elementwise", 2.0**11), ("c2", "termwise", 2.0**11),
    ("c3", "elementwise", 2.0**11),
    ("c4", "elementwise", 2.0**11), ("c4", "termwise", 2.0**11),
    ("c5", "termwise", 2.0**11), ("c5", "termwise", 2.0**13),
    ("c5", "elementwise", 2.0**11), ("c5", "elementwise", 2.0**13),
    ("c2", "elementwise_cross_first", 2.0**11), ("c4", "elementwise_cross_first", 2.0**11),
    ("c5", "elementwise_cross_first", 2.0**13),
]
_CACHE = {}


def _operands(name):
    if name not in _CACHE:
        _CACHE.clear()
        _CACHE[name] = workloads.workload_operands(name)
    return _CACHE[name]


@pytest.mark.parametrize("name,order,scale", CASES,
                         ids=[f"{n}-{o}-{int(np.log2(s))}" for n, o, s in CASES])
def test_workload_parity_sampled_rows(gpu, name, order, scale):
    """Full-size workloads in the bench's launch configuration.  C is filled
    with NaN before the call, so the all-finite check proves that every entry
    was written.  The oracle computes one row in every 256-row band of C (at
    an offset that rotates from band to band), and on those rows the GPU
    must meet the 2K u32 |A||B| bar and sit within a tenth of the distance
    between the oracle and its hi-only product (a kernel that drops a
    correction term fails that, where the componentwise bar alone is loose at
    long K)."""
    import torch

    from paper_2507_23387_amd import binding

    w = workloads.get(name)
    A, B = _operands(name)
    log(f"workload {w.name} {order} s=2^{int(np.log2(scale))}")
    dA, dB = to_dev(A), to_dev(B)
    Cd = torch.full((w.M, w.N), float("nan"), dtype=torch.float32, device="cuda")
    binding.matmul(dA, dB, scale, order, out=Cd)
    torch.cuda.synchronize()
    C = Cd.cpu().numpy()
    del dA, dB, Cd
    assert C.shape == (w.M, w.N)
    # The whole output is written and finite (every workload stays in range).
    assert np.isfinite(C).all()
    rows = np.arange(w.M) if w.M <= 256 else band_rows(w.M, w.seed + 11 * len(order))
    Co = oracle.sgemm_rows(A, B, rows, scale, order, kb=_kb(order))
    Ch = oracle.sgemm_rows(A, B, rows, scale, "hi_only", kb=_kb(order))
    absab = abs_ab(A, B, rows)
    assert_parity(C[rows], Co, w.K, absab, f"{name} {order}")
    assert_discriminates(C[rows], Co, Ch, f"{name} {order}")
    # Termwise inside the exponent window of Rules 1-2 (all of the 4096^3
    # normal and long-K workloads): Eq. main_bound against an FP64 GEMM.
    if order == "termwise" and name in ("c2", "c4"):
        coef = float(bounds.main_bound_coef(w.K))
        err = np.abs(C[rows].astype(np.float64) - ref64(A, B, rows))
        assert np.all(err <= coef * absab)


def test_workspace_at_high_addresses(gpu):
    """A caller workspace placed so that the FP16 planes sit at addresses whose
    low 32 bits are >= 2^31 and one plane straddles a 4 GiB boundary: the GEMM
    kernels build each copy's 64-bit source address from two 32-bit halves,
    and every order must give the same bits as with a pool workspace."""
    import torch

    from paper_2507_23387_amd import binding

    M, N, K = 520, 300, 1056
    A, B = workloads.make_operands(M, N, K, 14, "uniform_pm1")
    dA, dB = to_dev(A), to_dev(B)
    stream = torch.cuda.current_stream().cuda_stream
    wsb = max(binding.sgemm_cube_workspace_size(M, N, K, binding.ORDERS[o]) for o in ORDERS)
    plane = binding.sgemm_cube_workspace_size(M, N, K) // 4
    buf = torch.empty((1 << 32) + wsb + 4096, dtype=torch.uint8, device="cuda")
    base = buf.data_ptr()
    # The workspace starts 1.5 planes below a 4 GiB boundary (256-byte aligned).
    target = ((1 << 32) - (3 * plane) // 2) & ~255
    off = (target - (base & 0xFFFFFFFF)) % (1 << 32)
    ws_ptr = base + off
    assert off + wsb <= buf.numel() and ws_ptr % 256 == 0
    assert ws_ptr & 0xFFFFFFFF >= 1 << 31
    assert (ws_ptr >> 32) != ((ws_ptr + wsb - 1) >> 32)
    for order in ORDERS:
        log(f"high-address workspace {order}")
        ref = binding.matmul(dA, dB, 2048.0, order)
        C = torch.empty_like(ref)
        assert binding.sgemm_cube_ws(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, C.data_ptr(),
                                     N, 2048.0, binding.ORDERS[order], ws_ptr, wsb, stream) == 0
        torch.cuda.synchronize()
        assert torch.equal(C, ref), order
    del buf
