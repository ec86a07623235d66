"""Host-side checks of the C-ABI (no GPU needed): the library loads, exports
every entry point include/sgemm_cube.h declares, and rejects invalid arguments
before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sgemm_cube.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2507_23387_amd import binding

    return binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sgemm_cube\w*)\s*\(", text)))


def test_header_declares_expected_entry_points(lib):
    assert declared_functions() == sorted(lib.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    raw = ctypes.CDLL(lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(raw, name), name


def test_internal_symbols_hidden(lib):
    raw = ctypes.CDLL(lib.LIB_PATH)
    assert not hasattr(raw, "_ZN3sgc11plan_planesElllPv")


def test_status_strings(lib):
    for code, name in lib.STATUS_NAMES.items():
        assert lib.sgemm_cube_status_string(code) == name
    assert lib.sgemm_cube_status_string(99) == "SGEMM_CUBE_UNKNOWN_STATUS"


def test_block_k(lib):
    assert lib.sgemm_cube_block_k() == 32


def test_workspace_size(lib):
    # 256-byte header (range flag), then four FP16 planes padded to 256 rows x 64 k.
    assert lib.sgemm_cube_workspace_size(8192, 8192, 8192) == 256 + 4 * 8192 * 8192 * 2
    assert lib.sgemm_cube_workspace_size(1, 1, 1) == 256 + 4 * (256 * 64 * 2)
    assert lib.sgemm_cube_workspace_size(300, 1, 65) == 256 + 2 * (512 * 128 * 2) + 2 * (256 * 128 * 2)
    assert lib.sgemm_cube_workspace_size(0, 5, 5) == 0
    assert lib.sgemm_cube_workspace_size(5, 5, 0) == 0
    assert lib.sgemm_cube_workspace_size(-1, 5, 5) == 0
    assert lib.sgemm_cube_workspace_size(5, 5, 5, 7) == 0


FAKE = 1 << 40  # a non-null address that is never dereferenced
INVALID = 1
NOT_SUPPORTED = 2


def call(lib, M=4, N=4, K=4, A=FAKE, lda=None, B=FAKE + (1 << 30), ldb=None,
         C=FAKE + (2 << 30), ldc=None, scale=2048.0, order=0):
    lda = K if lda is None else lda
    ldb = N if ldb is None else ldb
    ldc = N if ldc is None else ldc
    return lib.sgemm_cube(M, N, K, A, lda, B, ldb, C, ldc, scale, order, 0)


@pytest.mark.parametrize("kw", [
    dict(M=-1), dict(N=-1), dict(K=-1),
    dict(lda=3), dict(ldb=3), dict(ldc=3),
    dict(A=0), dict(B=0), dict(C=0),
    dict(scale=3.0), dict(scale=0.5), dict(scale=2.0**25), dict(scale=float("inf")),
    dict(scale=float("nan")), dict(scale=-2048.0), dict(scale=0.0),
    dict(order=3), dict(order=-1),
    dict(C=FAKE + 8),                        # C overlaps A
    dict(C=FAKE + (1 << 30) + 4),            # C overlaps B
])
def test_invalid_arguments_rejected_before_device_work(lib, kw):
    assert call(lib, **kw) == INVALID


def test_too_large_is_not_supported(lib):
    assert call(lib, M=(1 << 30) + 1, K=4, B=1 << 44, C=1 << 45) == NOT_SUPPORTED


def test_valid_scales_accepted_by_validation(lib):
    # Only validation is exercised here: M = 0 makes the call a no-op that
    # returns before any device work.
    for s_b in (0, 1, 11, 12, 13, 24):
        assert call(lib, M=0, scale=2.0**s_b) == 0


def test_all_orders_accepted_by_validation(lib):
    for order in (0, 1, 2):
        assert call(lib, M=0, order=order) == 0
        assert lib.sgemm_cube_workspace_size(5, 5, 5, order) > 0


def test_degenerate_shapes_are_noops(lib):
    assert call(lib, M=0) == 0
    assert call(lib, N=0, ldb=1, ldc=1) == 0
    assert call(lib, M=0, A=0, C=0) == 0        # null allowed when the extent is empty


def test_ws_requires_workspace(lib):
    need = lib.sgemm_cube_workspace_size(4, 4, 4)
    ws = FAKE + (3 << 30)
    args = (4, 4, 4, FAKE, 4, FAKE + (1 << 30), 4, FAKE + (2 << 30), 4, 2048.0, 0)
    assert lib.sgemm_cube_ws(*args, 0, need, 0) == INVALID           # null ws
    assert lib.sgemm_cube_ws(*args, ws, need - 1, 0) == INVALID      # too small
    assert lib.sgemm_cube_ws(*args, ws + 16, need, 0) == INVALID     # misaligned
    assert lib.sgemm_cube_ws(*args, FAKE, need, 0) == INVALID        # overlaps A


def test_split_validation(lib):
    X, H, L = FAKE, FAKE + (1 << 30), FAKE + (2 << 30)
    assert lib.sgemm_cube_split(-1, 4, X, 4, H, L, 4, 2048.0, 0) == INVALID
    assert lib.sgemm_cube_split(4, 4, X, 3, H, L, 4, 2048.0, 0) == INVALID
    assert lib.sgemm_cube_split(4, 4, X, 4, H, L, 3, 2048.0, 0) == INVALID
    assert lib.sgemm_cube_split(4, 4, X, 4, H, H + 4, 4, 2048.0, 0) == INVALID
    assert lib.sgemm_cube_split(4, 4, X, 4, H, L, 4, 6.0, 0) == INVALID
    assert lib.sgemm_cube_split(4, 4, 0, 4, H, L, 4, 2048.0, 0) == INVALID
    assert lib.sgemm_cube_split(0, 4, 0, 4, 0, 0, 4, 2048.0, 0) == 0


def test_prepare_compute_validation(lib):
    need = lib.sgemm_cube_workspace_size(4, 4, 4)
    ws = FAKE + (3 << 30)
    assert lib.sgemm_cube_prepare(4, 4, 4, FAKE, 4, FAKE + (1 << 30), 4, 3.0, ws, need, 0) == INVALID
    assert lib.sgemm_cube_prepare(4, 4, 4, FAKE, 4, FAKE + (1 << 30), 4, 2048.0, ws, need - 1,
                                  0) == INVALID
    assert lib.sgemm_cube_compute(4, 4, 4, FAKE, 4, 2048.0, 5, ws, need, 0) == INVALID
    assert lib.sgemm_cube_compute(4, 4, 4, FAKE, 4, 2048.0, 0, 0, need, 0) == INVALID
    assert lib.sgemm_cube_compute(4, 4, 4, ws + 64, 4, 2048.0, 0, ws, need, 0) == INVALID
    assert lib.sgemm_cube_compute(0, 4, 4, 0, 4, 2048.0, 0, 0, 0, 0) == 0


def test_hgemm_validation(lib):
    assert lib.sgemm_cube_hgemm(4, 4, 4, FAKE, 3, FAKE + (1 << 30), 4, FAKE + (2 << 30), 4,
                                0) == INVALID
    assert lib.sgemm_cube_hgemm(0, 4, 4, FAKE, 4, FAKE + (1 << 30), 4, FAKE + (2 << 30), 4,
                                0) == 0


def call_ex(lib, M=4, N=4, K=4, options=0, ws=FAKE + (3 << 30), ws_bytes=1 << 20,
            report=0, order=0, B=FAKE + (1 << 30), ldb=None):
    return lib.sgemm_cube_ex(M, N, K, FAKE, K, B, N if ldb is None else ldb, FAKE + (2 << 30),
                             N, 2048.0, order, options, ws, ws_bytes, report, 0)


def test_ex_validation(lib):
    assert call_ex(lib, options=4) == INVALID                     # unknown option bit
    assert call_ex(lib, options=8 | 2, order=1) == INVALID
    assert call_ex(lib, order=3) == INVALID
    assert call_ex(lib, ws_bytes=16) == INVALID                   # workspace too small
    assert call_ex(lib, ws=FAKE + (3 << 30) + 8) == INVALID       # not 256-byte aligned
    assert call_ex(lib, report=FAKE + (3 << 30) + 2) == INVALID   # report not 4-byte aligned
    assert call_ex(lib, report=FAKE + 4) == INVALID               # report overlaps A
    assert call_ex(lib, report=FAKE + (3 << 30) + 64) == INVALID  # report inside the workspace
    # Only validation runs: M = 0 returns before device work when no report is asked for.
    assert call_ex(lib, M=0, options=1) == 0


def test_ex_split_b_in_gemm_validation(lib):
    """SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM: termwise only, without pre-scaling or a
    range report, on B 16-byte aligned with ldb and N multiples of 4 and K a
    multiple of 64; anything else is NOT_SUPPORTED.  M = 0 keeps the valid
    calls free of device work."""
    split_b = lib.OPT_SPLIT_B_IN_GEMM
    ok = dict(M=0, N=64, K=64, options=split_b, order=1)
    assert call_ex(lib, **ok) == 0
    assert call_ex(lib, **{**ok, "ldb": 68}) == 0
    assert call_ex(lib, **{**ok, "order": 0}) == NOT_SUPPORTED     # elementwise
    assert call_ex(lib, **{**ok, "order": 2}) == NOT_SUPPORTED     # cross-terms-first
    assert call_ex(lib, **{**ok, "options": split_b | 1}) == NOT_SUPPORTED
    assert call_ex(lib, **{**ok, "report": FAKE + (3 << 30) - 64}) == NOT_SUPPORTED
    assert call_ex(lib, **{**ok, "N": 66}) == NOT_SUPPORTED        # N not a multiple of 4
    assert call_ex(lib, **{**ok, "ldb": 66}) == NOT_SUPPORTED      # ldb not a multiple of 4
    assert call_ex(lib, **{**ok, "K": 96}) == NOT_SUPPORTED        # K not a multiple of 64
    assert call_ex(lib, **{**ok, "B": FAKE + (1 << 30) + 4}) == NOT_SUPPORTED
    assert call_ex(lib, **{**ok, "ldb": 1 << 22}) == NOT_SUPPORTED
    # The other argument errors come first.
    assert call_ex(lib, **{**ok, "ldb": 60}) == INVALID            # ldb < N


def test_ex_workspace_size(lib):
    base = lib.sgemm_cube_workspace_size(300, 200, 100)
    assert lib.sgemm_cube_ex_workspace_size(300, 200, 100, 0, 0) == base
    # Pre-scaling adds the row and column maxima (Mp + Np words, 256-byte rounded).
    assert lib.sgemm_cube_ex_workspace_size(300, 200, 100, 0, 1) == base + (512 + 256) * 4
    assert lib.sgemm_cube_ex_workspace_size(300, 200, 100, 0, 4) == 0
    assert lib.sgemm_cube_ex_workspace_size(300, 200, 0, 2, 1) == 0
    # Splitting B in the GEMM keeps the workspace of the call without it.
    assert lib.sgemm_cube_ex_workspace_size(300, 200, 128, 1, 2) == \
        lib.sgemm_cube_ex_workspace_size(300, 200, 128, 1, 0)


def test_compute_stages_validation(lib):
    ws = FAKE + (3 << 30)
    call = lambda order=0, stages=2, M=4: lib.sgemm_cube_compute_stages(
        M, 4, 4, FAKE, 4, 2048.0, order, stages, ws, 1 << 20, 0)
    assert call(stages=0) == INVALID
    assert call(stages=3) == INVALID
    assert call(order=1) == NOT_SUPPORTED
    assert call(order=2) == NOT_SUPPORTED
    assert call(M=0, stages=1) == 0          # validation only: M = 0 is a no-op



def test_compute_tile_validation(lib):
    ws = FAKE + (3 << 30)
    call = lambda order=0, tm=256, tn=256, bk=32, w=4, M=4: lib.sgemm_cube_compute_tile(
        M, 4, 4, FAKE, 4, 2048.0, order, tm, tn, bk, w, ws, 1 << 20, 0)
    assert call(tm=0, tn=0, bk=0, w=0) == INVALID
    for cfg in ((64, 64, 32, 4), (256, 256, 64, 4), (256, 128, 64, 4), (128, 128, 16, 4),
                (384, 128, 32, 4), (256, 256, 32, 0), (256, 256, 32, 2), (256, 256, 32, 16),
                (256, 128, 32, 8), (128, 128, 32, 8), (0, 0, 0, 8)):
        assert call(tm=cfg[0], tn=cfg[1], bk=cfg[2], w=cfg[3]) == INVALID, cfg
    assert call(order=1) == NOT_SUPPORTED
    assert call(order=3) == INVALID
    for cfg in lib.TILE_CONFIGS:
        assert call(M=0, tm=cfg[0], tn=cfg[1], bk=cfg[2], w=cfg[3]) == 0   # validation only


def test_compute_b_validation(lib):
    """sgemm_cube_compute_b: the GEMM from prepared A planes and FP32 B,
    termwise only, on the layouts the in-kernel split of B reads."""
    B, C, ws = FAKE, FAKE + (2 << 30), FAKE + (3 << 30)
    call = lambda M=4, N=64, K=64, B=B, ldb=None, C=C, ldc=None, scale=2048.0, order=1, ws=ws, \
        ws_bytes=1 << 20: lib.sgemm_cube_compute_b(M, N, K, B, N if ldb is None else ldb, C,
                                                   N if ldc is None else ldc, scale, order, ws,
                                                   ws_bytes, 0)
    assert call(order=3) == INVALID
    assert call(ldb=63) == INVALID                 # ldb < N
    assert call(ldc=63) == INVALID                 # ldc < N
    assert call(scale=3.0) == INVALID              # not a power of two
    assert call(B=0) == INVALID
    assert call(C=0) == INVALID
    assert call(C=B + 64) == INVALID               # C overlaps B
    assert call(order=0) == NOT_SUPPORTED          # elementwise
    assert call(order=2) == NOT_SUPPORTED          # cross-terms-first
    assert call(N=66) == NOT_SUPPORTED             # N not a multiple of 4
    assert call(ldb=66) == NOT_SUPPORTED           # ldb not a multiple of 4
    assert call(K=96) == NOT_SUPPORTED             # K not a multiple of 64
    assert call(B=B + 4) == NOT_SUPPORTED          # B not 16-byte aligned
    assert call(ws_bytes=16) == INVALID            # workspace too small
    assert call(ws=ws + 8) == INVALID              # not 256-byte aligned
    assert call(M=0) == 0                          # validation only
    assert call(N=0, B=0, ldb=1, ldc=1) == 0


def test_compute_a_validation(lib):
    A, C, ws = FAKE, FAKE + (2 << 30), FAKE + (3 << 30)
    call = lambda M=4, N=4, K=4, A=A, lda=4, C=C, ldc=4, scale=2048.0, order=0, ws=ws, \
        ws_bytes=1 << 20: lib.sgemm_cube_compute_a(M, N, K, A, lda, C, ldc, scale, order, ws,
                                                   ws_bytes, 0)
    assert call(order=3) == INVALID
    assert call(lda=3) == INVALID                  # lda < K
    assert call(ldc=3) == INVALID                  # ldc < N
    assert call(scale=3.0) == INVALID              # not a power of two
    assert call(A=0) == INVALID
    assert call(C=0) == INVALID
    assert call(C=A + 8) == INVALID                # C overlaps A
    assert call(ws_bytes=16) == INVALID            # workspace too small
    assert call(ws=ws + 8) == INVALID              # not 256-byte aligned
    assert call(ws=A) == INVALID                   # workspace overlaps A
    assert call(M=-1) == INVALID
    assert call(M=1 << 31) == NOT_SUPPORTED
    assert call(M=0) == 0                          # validation only: a no-op


def test_splits_a_in_gemm_rule(lib):
    """The in-kernel split of A is chosen for the elementwise order with
    N <= 4096, scale <= 2^15, 16-byte aligned A, lda % 4 == 0 and below 2^22,
    and K % 64 == 0, and for termwise with the same layout and N <= 2048 at any
    valid scale; everything else, and invalid arguments, gets 0.  The query only
    looks at A's address."""
    q = lambda M=512, N=4096, K=1024, A=FAKE, lda=1024, scale=2048.0, order=0: \
        lib.sgemm_cube_splits_a_in_gemm(M, N, K, A, lda, scale, order)
    assert q() == 1
    assert q(N=1) == 1 and q(M=1) == 1 and q(K=64) == 1
    assert q(scale=32768.0) == 1 and q(scale=1.0) == 1
    assert q(lda=1028) == 1
    assert q(N=4097) == 0                      # many tile columns: split pass
    assert q(order=2) == 0                      # cross-terms-first: never
    assert q(order=1) == 0                      # termwise: N <= 2048 only
    assert q(order=1, N=2048) == 1              # the 256 x 128 kernel
    assert q(order=1, N=2048, scale=2.0**24) == 1   # termwise keeps no s B_hi
    assert q(order=1, N=2049) == 0 and q(order=1, N=2048, K=1000, lda=1000) == 0
    assert q(order=3) == 0 and q(order=-1) == 0
    assert q(scale=65536.0) == 0                # unscaled kernel
    assert q(scale=3.0) == 0 and q(scale=0.5) == 0
    assert q(A=FAKE + 4) == 0                   # A not 16-byte aligned
    assert q(lda=1026) == 0                     # lda not a multiple of 4
    assert q(K=1000, lda=1000) == 0             # K not a multiple of 64
    assert q(lda=1 << 22) == 0
    assert q(lda=512) == 0                      # lda < K: the calls reject it
    assert q(M=(1 << 30) + 1) == 0              # beyond the indexing limits
    assert q(M=0) == 0 and q(N=0) == 0 and q(K=0) == 0 and q(A=0) == 0


def test_noalloc_validates_before_device_work(lib):
    """sgemm_cube_noalloc validates like sgemm_cube and refuses problems whose
    workspace exceeds its fixed 64 MiB array, all before any device call."""
    def na(M=4, N=4, K=4, A=FAKE, B=FAKE + (1 << 30), C=FAKE + (2 << 30), scale=2048.0, order=0):
        return lib.sgemm_cube_noalloc(M, N, K, A, max(K, 1), B, max(N, 1), C, max(N, 1), scale,
                                      order, 0)

    assert lib.NOALLOC_WORKSPACE_BYTES == 64 << 20
    assert na(M=-1) == INVALID
    assert na(scale=3.0) == INVALID
    assert na(order=5) == INVALID
    assert na(C=FAKE + 8) == INVALID
    assert na(M=0) == 0 and na(N=0) == 0
    assert lib.sgemm_cube_workspace_size(4096, 4096, 2049) > lib.NOALLOC_WORKSPACE_BYTES
    assert na(M=4096, N=4096, K=2049, B=1 << 44, C=1 << 45) == NOT_SUPPORTED
