"""Seeded synthetic inputs for the SGEMM-cube GEMM.

This module is shared by the tests, the benchmark and the smoke check.  It
holds input generation only -- none of the method's arithmetic -- so the
oracle and the HIP path can be fed identical operands without sharing code.

The paper's workloads are synthetic random matrices (Sec. 6.1: entries drawn
i.i.d. from U[-2^e, 2^e] or U[0, 2^e]); there is no dataset.  The five named
workloads below use numpy's PCG64 (``default_rng(seed)``), drawing A first and
then B, C-contiguous, so lda = K and ldb = ldc = N.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    seed: int
    dist: str          # generator key, see make_operands
    scales: tuple      # residual scales s_f used with this workload
    orders: tuple      # accumulation orders used with this workload
    note: str

    @property
    def flops(self) -> int:
        """FP32-equivalent work 2MNK (Sec. 6.1)."""
        return 2 * self.M * self.N * self.K


WORKLOADS = {
    "square256_uniform": Workload(
        "square256_uniform", 256, 256, 256, 1, "uniform_pm1", (2.0**11,), ("elementwise",),
        "M=N=K=256, A,B ~ U[-1,1], s=2^11, elementwise"),
    "square4096_normal": Workload(
        "square4096_normal", 4096, 4096, 4096, 2, "normal", (2.0**11,),
        ("elementwise", "termwise"),
        "M=N=K=4096, A,B ~ N(0,1), s=2^11, elementwise and termwise"),
    "square8192_uniform": Workload(
        "square8192_uniform", 8192, 8192, 8192, 3, "uniform_pm1", (2.0**11,),
        ("elementwise",),
        "M=N=K=8192, A,B ~ U[-1,1], s=2^11, elementwise (peak-throughput case)"),
    "longk_wide_exponent": Workload(
        "longk_wide_exponent", 4096, 4096, 16384, 4, "wide_exponent", (2.0**11,),
        ("elementwise", "termwise"),
        "M=N=4096, K=16384, entries sign*u*2^e, u~U[1,2), e~U{-12..12}, s=2^11"),
    "rect_subnormal_hi": Workload(
        "rect_subnormal_hi", 16384, 1024, 8192, 5, "uniform_pm1_2m14", (2.0**11, 2.0**13),
        ("termwise", "elementwise"),
        "M=16384, N=1024, K=8192, entries U[-1,1]*2^-14 (FP16-subnormal hi), s=2^11 vs 2^13"),
}

# Short aliases: c1..c5 in the order above.
ALIASES = {f"c{i + 1}": k for i, k in enumerate(WORKLOADS)}


def get(name: str) -> Workload:
    return WORKLOADS[ALIASES.get(name, name)]


def _draw(rng: np.random.Generator, dist: str, shape) -> np.ndarray:
    if dist == "uniform_pm1":
        return rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
    if dist == "normal":
        return rng.standard_normal(size=shape, dtype=np.float32)
    if dist == "wide_exponent":
        sign = np.where(rng.integers(0, 2, size=shape, dtype=np.int8) == 0, -1.0, 1.0)
        u = rng.uniform(1.0, 2.0, size=shape).astype(np.float32)
        e = rng.integers(-12, 13, size=shape, dtype=np.int32)
        return np.ldexp(u * sign.astype(np.float32), e).astype(np.float32)
    if dist == "uniform_pm1_2m14":
        u = rng.uniform(-1.0, 1.0, size=shape).astype(np.float32)
        return np.ldexp(u, -14).astype(np.float32)
    raise KeyError(dist)


def make_operands(M: int, N: int, K: int, seed: int, dist: str = "uniform_pm1"):
    """A (M x K) then B (K x N), FP32, C-contiguous, from default_rng(seed)."""
    rng = np.random.default_rng(seed)
    A = _draw(rng, dist, (M, K))
    B = _draw(rng, dist, (K, N))
    return A, B


def workload_operands(w: Workload | str):
    if isinstance(w, str):
        w = get(w)
    return make_operands(w.M, w.N, w.K, w.seed, w.dist)


def offset_exponent_operands(M: int, N: int, K: int, seed: int, e: int,
                             symmetric: bool = True):
    """Sec. 6.1 accuracy inputs: U[-2^e, 2^e] (symmetric) or U[0, 2^e]."""
    rng = np.random.default_rng(seed)
    lo = -(2.0**e) if symmetric else 0.0
    A = rng.uniform(lo, 2.0**e, size=(M, K)).astype(np.float32)
    B = rng.uniform(lo, 2.0**e, size=(K, N)).astype(np.float32)
    return A, B


def sample_rows(M: int, count: int, seed: int) -> np.ndarray:
    """Sorted distinct row indices, always including the first and last rows."""
    rng = np.random.default_rng(seed + 7919)
    count = min(count, M)
    rows = set([0, M - 1])
    if count > len(rows):
        extra = rng.choice(M, size=count, replace=False)
        for r in extra:
            if len(rows) >= count:
                break
            rows.add(int(r))
    return np.array(sorted(rows), dtype=np.int64)


def band_rows(M: int, seed: int, band: int = 256) -> np.ndarray:
    """One row index in every band of `band` rows (the GEMM's tile height), at
    an in-band offset that rotates from band to band, plus the first and last
    rows: a sample that touches every row of tiles of an M-row output."""
    rng = np.random.default_rng(seed + 104729)
    start = int(rng.integers(0, band))
    rows = {0, M - 1}
    for b in range((M + band - 1) // band):
        rows.add(min(b * band + (start + 37 * b) % band, M - 1))
    return np.array(sorted(rows), dtype=np.int64)
