"""Shared test utilities: golden-file readers and the parity tolerance."""
from __future__ import annotations

import os

import numpy as np

from workloads import band_rows  # noqa: F401  (re-exported for the tests)

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_table(name: str):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def claims() -> dict:
    return {r[0]: float(r[1]) for r in read_table("paper_claims.txt")}


def abs_ab(A: np.ndarray, B: np.ndarray, rows=None) -> np.ndarray:
    """(|A||B|) in FP64 (the quantity the componentwise bounds scale with)."""
    A64 = np.abs(np.asarray(A, dtype=np.float64))
    if rows is not None:
        A64 = A64[rows]
    return A64 @ np.abs(np.asarray(B, dtype=np.float64))


def ref64(A: np.ndarray, B: np.ndarray, rows=None) -> np.ndarray:
    A64 = np.asarray(A, dtype=np.float64)
    if rows is not None:
        A64 = A64[rows]
    return A64 @ np.asarray(B, dtype=np.float64)


def parity_tolerance(K: int, absab: np.ndarray) -> np.ndarray:
    """|C_gpu - C_oracle|_ij <= 2 K 2^-24 (|A||B|)_ij.

    Both sides sum the same exact FP16 x FP16 products (the split is bitwise
    identical); each side's FP32 summation error is at most about
    depth * u32 * (|A||B|)_ij with depth <= K, so the sum of the two is covered
    by 2K u32.  Where (|A||B|)_ij = 0 the tolerance is 0 (equality)."""
    return 2.0 * K * 2.0**-24 * absab


def assert_parity(C_gpu: np.ndarray, C_ref: np.ndarray, K: int, absab: np.ndarray,
                  what: str = ""):
    C_gpu = np.asarray(C_gpu, dtype=np.float64)
    C_ref = np.asarray(C_ref, dtype=np.float64)
    assert C_gpu.shape == C_ref.shape, (C_gpu.shape, C_ref.shape)
    fin = np.isfinite(C_ref)
    # non-finite results must agree in class (inf sign, NaN)
    assert np.array_equal(np.isnan(C_gpu), np.isnan(C_ref)), f"{what}: NaN pattern differs"
    inf_ref = np.isinf(C_ref)
    assert np.array_equal(np.isinf(C_gpu), inf_ref), f"{what}: inf pattern differs"
    assert np.array_equal(np.sign(C_gpu[inf_ref]), np.sign(C_ref[inf_ref])), f"{what}: inf sign"
    err = np.abs(C_gpu[fin] - C_ref[fin])
    tol = parity_tolerance(K, absab[fin])
    bad = err > tol
    if bad.any():
        idx = np.argmax(np.where(bad, err / np.maximum(tol, 1e-300), 0))
        raise AssertionError(
            f"{what}: {int(bad.sum())} entries exceed 2K u32 |A||B|; worst err={err[idx]:.3e} "
            f"tol={tol[idx]:.3e}")


def assert_discriminates(C_gpu: np.ndarray, C_ref: np.ndarray, C_hi: np.ndarray, what: str = "",
                         frac: float = 0.1):
    """The GPU result must sit much closer to the oracle than the oracle's
    hi-only product (the native FP16 GEMM, both correction terms dropped)
    does: max|C_gpu - C_oracle| <= frac * max|C_oracle - C_hi| and the same
    for the Frobenius norms.  At long K the componentwise bar 2K u32 |A||B| is
    looser than the correction terms themselves, so this is what fails when a
    kernel drops or mis-scales a cross term."""
    g = np.asarray(C_gpu, dtype=np.float64)
    r = np.asarray(C_ref, dtype=np.float64)
    h = np.asarray(C_hi, dtype=np.float64)
    d, D = np.abs(g - r), np.abs(r - h)
    assert D.max() > 0, f"{what}: hi-only equals the full result; nothing to discriminate"
    assert d.max() <= frac * D.max(), (
        f"{what}: max|gpu - oracle| = {d.max():.3e} > {frac} * max|oracle - hi_only| "
        f"= {frac * D.max():.3e}")
    assert np.linalg.norm(d) <= frac * np.linalg.norm(D), (
        f"{what}: ||gpu - oracle||_F = {np.linalg.norm(d):.3e} > {frac} * "
        f"||oracle - hi_only||_F = {frac * np.linalg.norm(D):.3e}")
