"""CPU oracle for the SGEMM-cube FP32-accuracy GEMM -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path
(``paper_2507_23387_amd``) never imports it and shares no code with it.

Functions and what pins them (see tests/test_oracle_*.py):

* ``f32_to_f16`` / ``f16_to_f32``: RN-even FP32->FP16 conversion and exact
  widening (Sec. 3.2 notation table, Sec. 4.1).  Pinned by an exhaustive 2^32
  comparison with two independent library conversions (numpy, torch CPU).
* ``split``: the two-component split of Sec. 3.3 / Eq. recover_eqn.  Pinned by
  the worked example of Sec. 4.2, the exhaustive residual-class counts of
  Sec. 4.1, Eq. split_error over whole binades, the sign-flip property of
  Sec. 3.3 and the 12-exponent shift of Sec. 4.2.
* ``sgemm`` (ELEMENTWISE, TERMWISE, HI_ONLY, ELEMENTWISE_CROSS_FIRST): the
  three-product reconstruction with FP32 accumulation in the orders of
  Sec. 4.5.  Pinned by exact recovery on constructed inputs, the exact value of
  the dropped lo*lo term (Eq. recover_eqn), Eq. ll_bound, Eq. truncation and
  Eq. main_bound by brute force in exact rationals, and textbook reductions
  (FP16-exact inputs, one block).  ELEMENTWISE and ELEMENTWISE_CROSS_FIRST
  have no printed bound: each is also pinned, by brute force in exact
  rationals, to the standard summation bound gamma_d * sum|terms| around the
  exact three-term sum, d the order's longest rounding chain
  (bounds.elementwise_depth, bounds.cross_first_depth).  The multi-block
  folds of all three orders are pinned exactly by tests/golden/fold_orders.txt:
  hand-worked dot products of three blocks whose every rounding step the test
  re-derives with single binary32 operations, chosen so that the three orders
  and a plausible misreading of each give different bits.
* ``prescale_exponents`` / ``sgemm_prescaled`` / ``range_classes``: the
  range extensions the paper names without fixing a rule (exponent
  management of the high part, Sec. 4.2; input-dependent scaling and an
  overflow guard, Sec. 7 and 8), in this reading: each row of A (column of B)
  is multiplied by the power of two that brings its largest finite magnitude
  to [2^EA, 2^(EA+1)), EA = min(14, 26 - s_b) (B: EB = 14 - s_b), the method
  runs on the scaled operands, and C_ij is scaled back by 2^-(p_i + q_j).
  Pinned by exact invariance (inputs whose hi and lo stay normal give the
  unscaled result bit for bit), by Eq. main_bound holding after pre-scaling
  on inputs whose hi is FP16-subnormal, and by the range classes of the
  values Sec. 3.1 and Sec. 4.2 name (|a| >= 65520, the 32784 residual
  overflow at s_b = 12, subnormal hi).
* ``bounds``: exact-rational bound calculators (Eq. ll_bound,
  Eq. truncation, Eq. main_bound) and the residual-class probability model of
  Sec. 4.1, pinned by the statements the paper prints about them.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

ELEMENTWISE = 0
TERMWISE = 1
HI_ONLY = 2
ELEMENTWISE_CROSS_FIRST = 3

ORDERS = {
    "elementwise": ELEMENTWISE,
    "termwise": TERMWISE,
    "hi_only": HI_ONLY,
    "elementwise_cross_first": ELEMENTWISE_CROSS_FIRST,
}

DEFAULT_KB = 64  # b_k of the best block reported in Sec. 6.3

_HERE = os.path.dirname(os.path.abspath(__file__))
# SGEMM_CUBE_ORACLE_LIB names another build of oracle.c to load instead: the
# planted-mistake check of the oracle's pins (tests/oracle_mutants.py) runs the
# oracle's tests against copies with one mistake each.
_LIB_PATH = os.environ.get("SGEMM_CUBE_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build

        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, f32p, u16p = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p
    lib.oracle_f32_to_f16_bits.restype = ctypes.c_uint16
    lib.oracle_f32_to_f16_bits.argtypes = [ctypes.c_uint32]
    lib.oracle_f16_to_f32_bits.restype = ctypes.c_uint32
    lib.oracle_f16_to_f32_bits.argtypes = [ctypes.c_uint16]
    lib.oracle_convert_range.restype = None
    lib.oracle_convert_range.argtypes = [ctypes.c_uint64, ctypes.c_uint64, u16p]
    lib.oracle_convert_array.restype = None
    lib.oracle_convert_array.argtypes = [i64, f32p, u16p]
    lib.oracle_widen_array.restype = None
    lib.oracle_widen_array.argtypes = [i64, u16p, f32p]
    lib.oracle_split.restype = ctypes.c_int
    lib.oracle_split.argtypes = [i64, i64, f32p, i64, u16p, u16p, i64, ctypes.c_float]
    lib.oracle_sgemm.restype = ctypes.c_int
    lib.oracle_sgemm.argtypes = [
        i64, i64, i64, f32p, i64, f32p, i64, f32p, i64,
        ctypes.c_float, ctypes.c_int, i64, ctypes.c_int,
    ]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def f32_to_f16(x) -> np.ndarray:
    """RN-even FP32 -> FP16; returns the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().oracle_convert_array(x.size, _ptr(x), _ptr(out))
    return out


def f32_bits_to_f16(start: int, count: int) -> np.ndarray:
    """Convert the FP32 bit patterns start .. start+count-1 (exhaustive sweeps)."""
    out = np.empty(count, dtype=np.uint16)
    _load().oracle_convert_range(start, count, _ptr(out))
    return out


def f16_to_f32(h) -> np.ndarray:
    """Exact FP16 -> FP32 widening of uint16 bit patterns."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, dtype=np.float32)
    _load().oracle_widen_array(h.size, _ptr(h), _ptr(out))
    return out


def split(X, scale: float):
    """Two-component split of a 2-D FP32 array: returns (hi, lo) uint16 planes."""
    X = np.asarray(X, dtype=np.float32)
    if X.ndim == 1:
        X = X.reshape(1, -1)
    X = np.ascontiguousarray(X)
    rows, cols = X.shape
    hi = np.empty((rows, cols), dtype=np.uint16)
    lo = np.empty((rows, cols), dtype=np.uint16)
    rc = _load().oracle_split(rows, cols, _ptr(X), max(cols, 1), _ptr(hi), _ptr(lo),
                              max(cols, 1), float(scale))
    if rc != 0:
        raise RuntimeError(f"oracle_split failed ({rc})")
    return hi, lo


def sgemm(A, B, scale: float, order="elementwise", kb: int = DEFAULT_KB,
          threads: int | None = None) -> np.ndarray:
    """C = SGEMM-cube(A, B) in the given accumulation order (FP32 result)."""
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    if A.ndim != 2 or B.ndim != 2 or A.shape[1] != B.shape[0]:
        raise ValueError(f"shape mismatch {A.shape} x {B.shape}")
    M, K = A.shape
    N = B.shape[1]
    order_code = ORDERS[order] if isinstance(order, str) else int(order)
    C = np.empty((M, N), dtype=np.float32)
    rc = _load().oracle_sgemm(M, N, K, _ptr(A), max(K, 1), _ptr(B), max(N, 1), _ptr(C),
                              max(N, 1), float(scale), order_code, int(kb),
                              int(threads or 0))
    if rc != 0:
        raise RuntimeError(f"oracle_sgemm failed ({rc})")
    return C


def sgemm_rows(A, B, rows, scale: float, order="elementwise", kb: int = DEFAULT_KB,
               threads: int | None = None) -> np.ndarray:
    """Rows ``rows`` of SGEMM-cube(A, B): each output row depends only on its
    own row of A and all of B, so this is the full-size result sampled."""
    rows = np.asarray(rows, dtype=np.int64)
    return sgemm(np.asarray(A)[rows], B, scale, order, kb, threads)


def prescale_exponents(X, axis: int, target: int) -> np.ndarray:
    """Power-of-two exponents that bring the largest finite |X| of every row
    (axis=1) or column (axis=0) into [2^target, 2^(target+1)); 0 where the
    line has no nonzero finite entry."""
    X = np.abs(np.asarray(X, dtype=np.float64))
    X = np.where(np.isfinite(X), X, 0.0)
    m = X.max(axis=axis) if X.size else np.zeros(X.shape[1 - axis])
    _, e = np.frexp(m)          # m = f 2^e with f in [0.5, 1): floor(log2 m) = e - 1
    return np.where(m > 0, target - (e - 1), 0).astype(np.int64)


def prescale_targets(scale: float) -> tuple[int, int]:
    """(EA, EB) for s = 2^s_b: EA = min(14, 26 - s_b) keeps every hi finite
    and every scaled residual below 2^16 (Rule 2, Sec. 4.2); EB = 14 - s_b also
    keeps s * B_hi finite."""
    s_b = int(np.frexp(np.float64(scale))[1]) - 1
    return min(14, 26 - s_b), 14 - s_b


def sgemm_prescaled(A, B, scale: float, order="elementwise", kb: int = DEFAULT_KB,
                    threads: int | None = None) -> np.ndarray:
    """SGEMM-cube on A' = diag(2^p) A and B' = B diag(2^q), then
    C_ij = 2^-(p_i + q_j) C'_ij (each step exact unless it under/overflows)."""
    A = np.ascontiguousarray(A, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.float32)
    ea, eb = prescale_targets(scale)
    p = prescale_exponents(A, 1, ea)
    q = prescale_exponents(B, 0, eb)
    As = np.ldexp(A, p[:, None].astype(np.int32)).astype(np.float32)
    Bs = np.ldexp(B, q[None, :].astype(np.int32)).astype(np.float32)
    Cs = sgemm(As, Bs, scale, order, kb, threads)
    return np.ldexp(Cs, (-(p[:, None] + q[None, :])).astype(np.int32)).astype(np.float32)


RANGE_NONFINITE, RANGE_HI_OVERFLOW, RANGE_LO_OVERFLOW, RANGE_HI_SUBNORMAL = 1, 2, 4, 8


def range_classes(X, scale: float) -> int:
    """OR of the range classes of the entries of X under the split:
    1 non-finite entry; 2 finite entry whose fl16 is infinite (|a| >= 65520);
    4 finite hi whose scaled residual overflows FP16; 8 nonzero FP16-subnormal
    hi."""
    X = np.asarray(X, dtype=np.float32)
    if X.size == 0:
        return 0
    hi, lo = split(X.reshape(1, -1), scale)
    hi, lo = hi.ravel(), lo.ravel()
    fin = np.isfinite(X.ravel())
    hi_fin = (hi & 0x7C00) != 0x7C00
    bits = 0
    if (~fin).any():
        bits |= RANGE_NONFINITE
    if (fin & ~hi_fin).any():
        bits |= RANGE_HI_OVERFLOW
    if (hi_fin & ((lo & 0x7FFF) == 0x7C00)).any():
        bits |= RANGE_LO_OVERFLOW
    if (((hi & 0x7C00) == 0) & ((hi & 0x03FF) != 0)).any():
        bits |= RANGE_HI_SUBNORMAL
    return bits

