"""Thin Python binding of libsgemmcube (include/sgemm_cube.h).

The functions named like the C entry points take plain integers (device
pointers as ints, the HIP stream as an int handle) and return the C status
code.  The torch helpers below them only marshal arguments: they pass
``data_ptr()`` / ``stride(0)`` and the current torch stream and raise on a
non-zero status.  Every step of the computation runs in the HIP kernels of the
shared library; there is no Python or CPU fallback -- if the library is not
built, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsgemmcube.so")

ELEMENTWISE = 0
TERMWISE = 1
ELEMENTWISE_CROSS_FIRST = 2
ORDERS = {"elementwise": ELEMENTWISE, "termwise": TERMWISE,
          "elementwise_cross_first": ELEMENTWISE_CROSS_FIRST}

OPT_PRESCALE = 1
OPT_SPLIT_B_IN_GEMM = 2
RANGE_NONFINITE = 1
RANGE_HI_OVERFLOW = 2
RANGE_LO_OVERFLOW = 4
RANGE_HI_SUBNORMAL = 8

STATUS_OK = 0
STATUS_NAMES = {
    0: "SGEMM_CUBE_OK",
    1: "SGEMM_CUBE_ERR_INVALID_VALUE",
    2: "SGEMM_CUBE_ERR_NOT_SUPPORTED",
    3: "SGEMM_CUBE_ERR_ALLOC",
    4: "SGEMM_CUBE_ERR_HIP",
}

# Every symbol include/sgemm_cube.h declares.
EXPORTS = (
    "sgemm_cube", "sgemm_cube_ws", "sgemm_cube_noalloc", "sgemm_cube_ex", "sgemm_cube_ex_workspace_size",
    "sgemm_cube_prepare", "sgemm_cube_compute", "sgemm_cube_compute_a", "sgemm_cube_compute_b",
    "sgemm_cube_splits_a_in_gemm", "sgemm_cube_compute_stages", "sgemm_cube_compute_tile",
    "sgemm_cube_workspace_size", "sgemm_cube_split",
    "sgemm_cube_hgemm", "sgemm_cube_status_string",
    "sgemm_cube_block_k",
)


class SgemmCubeError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {STATUS_NAMES.get(status, status)}")


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is not built; run `python -m paper_2507_23387_amd.build` or `__graft_entry__.build()` "
            "(the HIP library is required, there is no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i64, ptr, f32, i32, sz, u32 = (ctypes.c_int64, ctypes.c_void_p, ctypes.c_float,
                                   ctypes.c_int, ctypes.c_size_t, ctypes.c_uint)
    sig = {
        "sgemm_cube": (i32, [i64, i64, i64, ptr, i64, ptr, i64, ptr, i64, f32, i32, ptr]),
        "sgemm_cube_ws": (i32, [i64, i64, i64, ptr, i64, ptr, i64, ptr, i64, f32, i32, ptr, sz,
                                ptr]),
        "sgemm_cube_noalloc": (i32, [i64, i64, i64, ptr, i64, ptr, i64, ptr, i64, f32, i32,
                                     ptr]),
        "sgemm_cube_ex": (i32, [i64, i64, i64, ptr, i64, ptr, i64, ptr, i64, f32, i32, u32, ptr,
                                sz, ptr, ptr]),
        "sgemm_cube_ex_workspace_size": (sz, [i64, i64, i64, i32, u32]),
        "sgemm_cube_prepare": (i32, [i64, i64, i64, ptr, i64, ptr, i64, f32, ptr, sz, ptr]),
        "sgemm_cube_compute": (i32, [i64, i64, i64, ptr, i64, f32, i32, ptr, sz, ptr]),
        "sgemm_cube_compute_a": (i32, [i64, i64, i64, ptr, i64, ptr, i64, f32, i32, ptr, sz,
                                       ptr]),
        "sgemm_cube_compute_b": (i32, [i64, i64, i64, ptr, i64, ptr, i64, f32, i32, ptr, sz,
                                       ptr]),
        "sgemm_cube_splits_a_in_gemm": (i32, [i64, i64, i64, ptr, i64, f32, i32]),
        "sgemm_cube_compute_stages": (i32, [i64, i64, i64, ptr, i64, f32, i32, i32, ptr, sz,
                                            ptr]),
        "sgemm_cube_compute_tile": (i32, [i64, i64, i64, ptr, i64, f32, i32, i32, i32, i32, i32,
                                          ptr, sz, ptr]),
        "sgemm_cube_workspace_size": (sz, [i64, i64, i64, i32]),
        "sgemm_cube_split": (i32, [i64, i64, ptr, i64, ptr, ptr, i64, f32, ptr]),
        "sgemm_cube_hgemm": (i32, [i64, i64, i64, ptr, i64, ptr, i64, ptr, i64, ptr]),
        "sgemm_cube_status_string": (ctypes.c_char_p, [i32]),
        "sgemm_cube_block_k": (i32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


# --- C-level names ----------------------------------------------------------

def sgemm_cube(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, stream) -> int:
    return _lib.sgemm_cube(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, stream)


def sgemm_cube_ws(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, ws, ws_bytes,
                  stream) -> int:
    return _lib.sgemm_cube_ws(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, ws,
                              ws_bytes, stream)


def sgemm_cube_noalloc(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, stream) -> int:
    return _lib.sgemm_cube_noalloc(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, stream)


NOALLOC_WORKSPACE_BYTES = 64 << 20  # SGEMM_CUBE_NOALLOC_WORKSPACE_BYTES


def sgemm_cube_ex(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, options, ws, ws_bytes,
                  range_report, stream) -> int:
    return _lib.sgemm_cube_ex(M, N, K, A, lda, B, ldb, C, ldc, scale, accum_order, options, ws,
                              ws_bytes, range_report, stream)


def sgemm_cube_ex_workspace_size(M, N, K, accum_order=ELEMENTWISE, options=0) -> int:
    return int(_lib.sgemm_cube_ex_workspace_size(M, N, K, accum_order, options))


def sgemm_cube_prepare(M, N, K, A, lda, B, ldb, scale, ws, ws_bytes, stream) -> int:
    return _lib.sgemm_cube_prepare(M, N, K, A, lda, B, ldb, scale, ws, ws_bytes, stream)


def sgemm_cube_compute(M, N, K, C, ldc, scale, accum_order, ws, ws_bytes, stream) -> int:
    return _lib.sgemm_cube_compute(M, N, K, C, ldc, scale, accum_order, ws, ws_bytes, stream)


def sgemm_cube_compute_a(M, N, K, A, lda, C, ldc, scale, accum_order, ws, ws_bytes,
                         stream) -> int:
    return _lib.sgemm_cube_compute_a(M, N, K, A, lda, C, ldc, scale, accum_order, ws, ws_bytes,
                                     stream)


def sgemm_cube_compute_b(M, N, K, B, ldb, C, ldc, scale, accum_order, ws, ws_bytes,
                         stream) -> int:
    return _lib.sgemm_cube_compute_b(M, N, K, B, ldb, C, ldc, scale, accum_order, ws, ws_bytes,
                                     stream)


def sgemm_cube_splits_a_in_gemm(M, N, K, A, lda, scale, accum_order) -> int:
    return _lib.sgemm_cube_splits_a_in_gemm(M, N, K, A, lda, scale, accum_order)


def sgemm_cube_compute_stages(M, N, K, C, ldc, scale, accum_order, stages, ws, ws_bytes,
                              stream) -> int:
    return _lib.sgemm_cube_compute_stages(M, N, K, C, ldc, scale, accum_order, stages, ws,
                                          ws_bytes, stream)


def sgemm_cube_compute_tile(M, N, K, C, ldc, scale, accum_order, tile_m, tile_n, block_k, waves,
                            ws, ws_bytes, stream) -> int:
    return _lib.sgemm_cube_compute_tile(M, N, K, C, ldc, scale, accum_order, tile_m, tile_n,
                                        block_k, waves, ws, ws_bytes, stream)


# (tile_m, tile_n, block_k, waves) configurations of sgemm_cube_compute_tile.
TILE_CONFIGS = ((256, 256, 32, 4), (256, 128, 32, 4), (128, 256, 32, 4), (128, 128, 32, 4),
                (128, 128, 64, 4), (256, 256, 32, 8))


def sgemm_cube_workspace_size(M, N, K, accum_order=ELEMENTWISE) -> int:
    return int(_lib.sgemm_cube_workspace_size(M, N, K, accum_order))


def sgemm_cube_split(rows, cols, X, ldx, hi, lo, ldh, scale, stream) -> int:
    return _lib.sgemm_cube_split(rows, cols, X, ldx, hi, lo, ldh, scale, stream)


def sgemm_cube_hgemm(M, N, K, A, lda, B, ldb, C, ldc, stream) -> int:
    return _lib.sgemm_cube_hgemm(M, N, K, A, lda, B, ldb, C, ldc, stream)


def sgemm_cube_status_string(status: int) -> str:
    return _lib.sgemm_cube_status_string(status).decode()


def sgemm_cube_block_k() -> int:
    return int(_lib.sgemm_cube_block_k())


# --- torch marshalling --------------------------------------------------------

def _check(status: int, what: str):
    if status != STATUS_OK:
        raise SgemmCubeError(status, what)


def _order(order) -> int:
    return ORDERS[order] if isinstance(order, str) else int(order)


def _mat(t, name):
    import torch

    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or not t.is_cuda:
        raise TypeError(f"{name} must be a float32 CUDA/HIP tensor")
    if t.dim() != 2 or (t.size(1) > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be 2-D with unit column stride (row-major)")
    return t.data_ptr(), max(t.stride(0), t.size(1), 1)


def _stream():
    import torch

    return torch.cuda.current_stream().cuda_stream


def matmul(A, B, scale: float = 2.0**11, order="elementwise", out=None, workspace=None):
    """C = SGEMM-cube(A, B) on the current torch stream."""
    import torch

    pa, lda = _mat(A, "A")
    pb, ldb = _mat(B, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError(f"shape mismatch {tuple(A.shape)} x {tuple(B.shape)}")
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    pc, ldc = _mat(C, "C")
    if workspace is None:
        st = sgemm_cube(M, N, K, pa, lda, pb, ldb, pc, ldc, scale, _order(order), _stream())
    else:
        st = sgemm_cube_ws(M, N, K, pa, lda, pb, ldb, pc, ldc, scale, _order(order),
                           workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                           _stream())
    _check(st, "sgemm_cube")
    return C


def matmul_ex(A, B, scale: float = 2.0**11, order="elementwise", prescale: bool = False,
              report: bool = False, out=None, split_b_in_gemm: bool = False):
    """sgemm_cube_ex on the current torch stream: optional power-of-two
    pre-scaling of A's rows and B's columns; with report=True returns (C, bits)
    where bits is a one-element int32 device tensor holding the range classes
    (RANGE_*); split_b_in_gemm=True (termwise) sets
    SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM."""
    import torch

    pa, lda = _mat(A, "A")
    pb, ldb = _mat(B, "B")
    M, K = A.shape
    K2, N = B.shape
    if K != K2:
        raise ValueError(f"shape mismatch {tuple(A.shape)} x {tuple(B.shape)}")
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    pc, ldc = _mat(C, "C")
    options = (OPT_PRESCALE if prescale else 0) | (OPT_SPLIT_B_IN_GEMM if split_b_in_gemm else 0)
    n = sgemm_cube_ex_workspace_size(M, N, K, _order(order), options)
    ws = torch.empty(max(n, 256), dtype=torch.uint8, device=A.device)
    bits = torch.zeros(1, dtype=torch.int32, device=A.device) if report else None
    st = sgemm_cube_ex(M, N, K, pa, lda, pb, ldb, pc, ldc, scale, _order(order), options,
                       ws.data_ptr(), ws.numel(), bits.data_ptr() if report else None, _stream())
    _check(st, "sgemm_cube_ex")
    return (C, bits) if report else C


def hgemm(A, B, out=None):
    """Native-FP16 baseline: C = fl16(A) fl16(B), FP32 accumulation."""
    import torch

    pa, lda = _mat(A, "A")
    pb, ldb = _mat(B, "B")
    M, K = A.shape
    N = B.shape[1]
    C = out if out is not None else torch.empty((M, N), dtype=torch.float32, device=A.device)
    pc, ldc = _mat(C, "C")
    _check(sgemm_cube_hgemm(M, N, K, pa, lda, pb, ldb, pc, ldc, _stream()), "sgemm_cube_hgemm")
    return C


def split(X, scale: float = 2.0**11):
    """(hi, lo) FP16 bit patterns of X as int16 tensors (reinterpret as uint16)."""
    import torch

    px, ldx = _mat(X, "X")
    rows, cols = X.shape
    hi = torch.empty((rows, cols), dtype=torch.int16, device=X.device)
    lo = torch.empty((rows, cols), dtype=torch.int16, device=X.device)
    _check(sgemm_cube_split(rows, cols, px, ldx, hi.data_ptr(), lo.data_ptr(), max(cols, 1),
                            scale, _stream()), "sgemm_cube_split")
    return hi, lo


def workspace(M: int, N: int, K: int, device="cuda"):
    """A torch byte tensor large enough for sgemm_cube_ws on this shape."""
    import torch

    n = sgemm_cube_workspace_size(M, N, K)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)
