"""Seeded random cases across the whole C-ABI surface, against the oracle.

Each case draws a shape (ragged M and N from 1 up to a few tiles, K from 40),
leading-dimension padding, a base offset of A (aligned or not, so both the in-kernel split and
the split pass run), a power-of-two scale from 2^0 to 2^24, an order, an entry
point and a value distribution (uniform, normal, rows and columns moved to
other binades, a B whose s B_hi overflows FP16; for sgemm_cube_ex with
power-of-two pre-scaling, rows of A and columns of B from 2^-30 to 2^20,
against the oracle's pre-scaled product).  The entry points that split
B inside the GEMM (sgemm_cube_ex with SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM,
sgemm_cube_compute_b) take the termwise order and the layouts they need: N,
ldb multiples of 4 and K of 64.  The GPU result, written into
a NaN-filled C with padded ldc, must meet the parity bar against the oracle
entry by entry, and the bytes of C outside the M x N block must be untouched.
A second family draws M and N from 1500 to 5000 (grids of up to 20 x 40
tiles, over several dispatch rounds and not made of whole 16 x 16 blocks, so
the general tile map runs): every entry of C must be written, and one row in
every 256-row band is held to the oracle.
The cases are fixed by the seed, so a failure names a reproducible case."""
import numpy as np
import pytest

import oracle
import workloads
from tests.gpu_util import log, padded
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu

ORDERS = ["elementwise", "termwise", "elementwise_cross_first"]
ENTRIES = ["sgemm_cube", "ws", "noalloc", "prepare_compute", "compute_a", "split_b_ex",
           "compute_b", "prescale_ex"]
N_CASES = 264
N_LARGE = 12
# The bar 2 K u32 |A||B| covers the two sides' rounding when each side's
# rounding depth is at most K.  The elementwise order's depth is kb - 1 + 3 per
# block (bounds.elementwise_depth; 34 for K <= 32 with the GPU's kb = 32), and
# the GPU's merges of a block term into the running sum each err by up to two
# units instead of one (the matrix unit's alignment), so below K ~ 40 two
# correct summations can differ by more than the bar: a 263 x 206 x 4 case with
# FP16-subnormal high words did (11 u32 |A||B| against a bar of 8).  Those K
# are left to the small-K tests on exact data; here K >= 40.
K_MIN = 40


def _case(i):
    rng = np.random.default_rng(1000 + i)
    M = int(rng.integers(1, 700))
    N = int(rng.integers(1, 700))
    K = int(rng.choice([int(rng.integers(K_MIN, 1100)), 64 * int(rng.integers(1, 17))]))
    pads = [int(rng.integers(0, 6)) for _ in range(3)]
    offset = int(rng.choice([0, 0, 1, 3]))
    s_b = int(rng.choice([0, 6, 11, 11, 12, 13, 15, 16, 20, 24]))
    order = ORDERS[i % 3]
    entry = ENTRIES[(i // 3) % len(ENTRIES)]
    if entry in ("split_b_ex", "compute_b"):
        order = "termwise"
        N = max(4, N - N % 4)
        K = 64 * max(1, K // 64)
        pads[1] -= pads[1] % 4
    dist = ["uniform", "normal", "binades", "overflow"][int(rng.integers(0, 4))]
    if entry == "prescale_ex" and dist != "overflow":
        dist = "wide"
    A, B = _values(rng, M, N, K, dist, s_b)
    return dict(M=M, N=N, K=K, pads=pads, offset=offset, s=2.0**s_b, order=order, entry=entry,
                dist=dist, A=A, B=B)


def _values(rng, M, N, K, dist, s_b):
    A = rng.uniform(-1, 1, (M, K)).astype(np.float32)
    B = rng.uniform(-1, 1, (K, N)).astype(np.float32)
    if dist == "normal":
        A = rng.standard_normal((M, K)).astype(np.float32)
        B = rng.standard_normal((K, N)).astype(np.float32)
    elif dist == "binades":
        A[::3] *= np.float32(2.0**-15)
        A[1::5] *= np.float32(2.0**10)
        B[:, ::4] *= np.float32(2.0**-8)
    elif dist == "overflow":
        B[rng.integers(0, K), rng.integers(0, N)] = np.float32(2.0**14)
    elif dist == "wide":  # rows of A and columns of B from 2^-30 to 2^20 (pre-scaling)
        A = A * np.ldexp(np.float32(1), rng.integers(-30, 21, size=(M, 1)).astype(np.int32))
        B = B * np.ldexp(np.float32(1), rng.integers(-30, 21, size=(1, N)).astype(np.int32))
        return A.astype(np.float32), B.astype(np.float32)
    # Keep Rule 2 (no lo overflow) and hi finite: the bar is for finite results.
    if s_b > 11:
        A *= np.float32(2.0**(11 - s_b))
        B *= np.float32(2.0**(11 - s_b))
    return A, B


def _large_case(i):
    rng = np.random.default_rng(5000 + i)
    M = int(rng.integers(1500, 5001))
    N = int(rng.integers(1500, 5001))
    K = int(rng.choice([int(rng.integers(K_MIN, 600)), 64 * int(rng.integers(1, 9))]))
    pads = [int(rng.integers(0, 6)) for _ in range(3)]
    offset = int(rng.choice([0, 1]))
    s_b = int(rng.choice([11, 11, 13, 16, 20]))
    order = ORDERS[i % 3]
    entry = ["sgemm_cube", "ws", "prepare_compute", "compute_a", "split_b_ex",
             "compute_b"][(i // 2) % 6]
    if entry in ("split_b_ex", "compute_b"):
        order = "termwise"
        N -= N % 4
        K = 64 * max(1, K // 64)
        pads[1] -= pads[1] % 4
    dist = ["uniform", "normal", "overflow"][int(rng.integers(0, 3))]
    A, B = _values(rng, M, N, K, dist, s_b)
    return dict(M=M, N=N, K=K, pads=pads, offset=offset, s=2.0**s_b, order=order, entry=entry,
                dist=dist, A=A, B=B)


def _run(c, what):
    """Call the case's entry point on a NaN-filled C with ldc = N + pads[2];
    returns the M x N block after checking that nothing else of C changed."""
    import torch

    from paper_2507_23387_amd import binding

    M, N, K, s = c["M"], c["N"], c["K"], c["s"]
    lda, ldb, ldc = K + c["pads"][0], N + c["pads"][1], N + c["pads"][2]
    code = binding.ORDERS[c["order"]]
    log(f"{what}: {M}x{N}x{K} lda+{c['pads'][0]} off {c['offset']} s=2^"
        f"{int(np.log2(s))} {c['order']} {c['entry']} {c['dist']}")
    _, dA = padded(c["A"], lda, offset=c["offset"])
    _, dB = padded(c["B"], ldb)
    cbuf, dC = padded(np.full((M, N), np.nan, np.float32), ldc)
    cbuf.fill_(float("nan"))
    stream = torch.cuda.current_stream().cuda_stream
    a, b, cc = dA.data_ptr(), dB.data_ptr(), dC.data_ptr()
    entry = c["entry"]
    if entry == "sgemm_cube":
        st = binding.sgemm_cube(M, N, K, a, lda, b, ldb, cc, ldc, s, code, stream)
    elif entry == "noalloc":
        st = binding.sgemm_cube_noalloc(M, N, K, a, lda, b, ldb, cc, ldc, s, code, stream)
        if st == 2:  # beyond the fixed workspace: take the allocating call instead
            st = binding.sgemm_cube(M, N, K, a, lda, b, ldb, cc, ldc, s, code, stream)
    else:
        ws = binding.workspace(M, N, K)
        n = ws.numel()
        if entry == "ws":
            st = binding.sgemm_cube_ws(M, N, K, a, lda, b, ldb, cc, ldc, s, code, ws.data_ptr(),
                                       n, stream)
        elif entry == "prepare_compute":
            st = binding.sgemm_cube_prepare(M, N, K, a, lda, b, ldb, s, ws.data_ptr(), n, stream)
            assert st == 0
            st = binding.sgemm_cube_compute(M, N, K, cc, ldc, s, code, ws.data_ptr(), n, stream)
        elif entry == "split_b_ex":
            st = binding.sgemm_cube_ex(M, N, K, a, lda, b, ldb, cc, ldc, s, code,
                                       binding.OPT_SPLIT_B_IN_GEMM, ws.data_ptr(), n, None,
                                       stream)
        elif entry == "prescale_ex":
            nb = binding.sgemm_cube_ex_workspace_size(M, N, K, code, binding.OPT_PRESCALE)
            ws = torch.empty((max(nb, 1),), dtype=torch.uint8, device="cuda")
            st = binding.sgemm_cube_ex(M, N, K, a, lda, b, ldb, cc, ldc, s, code,
                                       binding.OPT_PRESCALE, ws.data_ptr(), nb, None, stream)
        elif entry == "compute_b":
            st = binding.sgemm_cube_prepare(M, N, K, a, lda, None, ldb, s, ws.data_ptr(), n,
                                            stream)
            assert st == 0
            st = binding.sgemm_cube_compute_b(M, N, K, b, ldb, cc, ldc, s, code, ws.data_ptr(),
                                              n, stream)
        else:
            st = binding.sgemm_cube_prepare(M, N, K, None, lda, b, ldb, s, ws.data_ptr(), n,
                                            stream)
            assert st == 0
            st = binding.sgemm_cube_compute_a(M, N, K, a, lda, cc, ldc, s, code, ws.data_ptr(),
                                              n, stream)
    assert st == 0, binding.sgemm_cube_status_string(st)
    torch.cuda.synchronize()
    full = cbuf.cpu().numpy()
    # Padding columns of C and anything past the last row stay NaN.
    assert np.isnan(full[:M * ldc].reshape(M, ldc)[:, N:]).all()
    assert np.isnan(full[M * ldc:]).all()
    return full[:M * ldc].reshape(M, ldc)[:, :N]


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_case_against_the_oracle(gpu, i):
    from paper_2507_23387_amd import binding

    c = _case(i)
    got = _run(c, f"random case {i}")
    ref = oracle.sgemm_prescaled if c["entry"] == "prescale_ex" else oracle.sgemm
    want = ref(c["A"], c["B"], c["s"], c["order"], kb=binding.sgemm_cube_block_k())
    assert_parity(got, want, c["K"], abs_ab(c["A"], c["B"]), f"random case {i}")


@pytest.mark.parametrize("i", range(N_LARGE))
def test_large_random_case_against_the_oracle(gpu, i):
    from paper_2507_23387_amd import binding

    c = _large_case(i)
    got = _run(c, f"large random case {i}")
    assert np.isfinite(got).all()  # every entry written (C was NaN)
    rows = workloads.band_rows(c["M"], 7 + i)
    want = oracle.sgemm_rows(c["A"], c["B"], rows, c["s"], c["order"],
                             kb=binding.sgemm_cube_block_k())
    assert_parity(got[rows], want, c["K"], abs_ab(c["A"], c["B"], rows),
                  f"large random case {i}")
