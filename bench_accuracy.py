"""Accuracy sweeps of the GPU path against an FP64 reference (Sec. 6.2).

Runs the experiments of Sec. 6.1-6.2 on this GPU with synthetic inputs:

  offset   relative Frobenius error (Eq. err) vs the FP32 offset exponent e,
           entries U[-2^e, 2^e] (symmetric) and U[0, 2^e] (non-negative),
           s = 2^s_b for s_b in {0, 6, 11, 12}, averaged over seeds, m = n = k;
  mn       error vs m = n at k = 64 x 44 = 2816, e = 0, symmetric;
  k        error vs k at m = n = 1024;
  mkn      error vs m = n = k;
  maxnorm  componentwise errors on adversarial inputs (the max-norm study the
           paper leaves open): max |C - C64| / (|A||B|) and the largest
           relative error over nonzero entries;
  prescale the offset sweep's low and high exponents again with the
           power-of-two pre-scaling of sgemm_cube_ex, which keeps hi normal
           and in range.

Compared: the three GPU accumulation orders, the GPU FP16 baseline
(sgemm_cube_hgemm), and the host's FP32 SGEMM (numpy float32 matmul; numpy's
BLAS).  The reference is numpy's FP64 matmul of the same FP32 inputs.

Usage: python bench_accuracy.py [--quick] [--out FILE.json] [--md FILE.md]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

import workloads

ROOT = os.path.dirname(os.path.abspath(__file__))
ORDERS = ("elementwise", "termwise", "elementwise_cross_first")
SB = (0, 6, 11, 12)


def log(msg):
    print(f"[accuracy] {msg}", file=sys.stderr, flush=True)


def frob(C, ref):
    d = C.astype(np.float64) - ref
    n = np.linalg.norm(ref)
    return float(np.linalg.norm(d) / n) if n > 0 else float(np.linalg.norm(d))


class Runner:
    """Keeps the operands on the GPU and runs every method on them."""

    def __init__(self):
        import torch

        import paper_2507_23387_amd as sgc

        self.torch, self.sgc = torch, sgc
        self.dev = torch.device("cuda:0")

    def prescaled(self, A, B, s_b):
        torch, sgc = self.torch, self.sgc
        dA = torch.from_numpy(A).to(self.dev)
        dB = torch.from_numpy(B).to(self.dev)
        out = {f"{order}/{s_b}/pre": sgc.matmul_ex(dA, dB, scale=2.0**s_b, order=order,
                                                  prescale=True) for order in ORDERS}
        torch.cuda.synchronize()
        return {k: v.cpu().numpy() for k, v in out.items()}

    def methods(self, A, B, scales):
        torch, sgc = self.torch, self.sgc
        dA = torch.from_numpy(A).to(self.dev)
        dB = torch.from_numpy(B).to(self.dev)
        out = {"hgemm": sgc.hgemm(dA, dB)}
        for s_b in scales:
            for order in ORDERS:
                out[f"{order}/{s_b}"] = sgc.matmul(dA, dB, scale=2.0**s_b, order=order)
        torch.cuda.synchronize()
        res = {k: v.cpu().numpy() for k, v in out.items()}
        res["sgemm_fp32_host"] = A @ B
        return res


def offset_sweep(run, n, exps, seeds, out):
    rows = []
    for sym in (True, False):
        for e in exps:
            acc = {}
            for seed in seeds:
                A, B = workloads.offset_exponent_operands(n, n, n, seed, e, symmetric=sym)
                ref = A.astype(np.float64) @ B.astype(np.float64)
                for k, C in run.methods(A, B, SB).items():
                    acc.setdefault(k, []).append(frob(C, ref))
            row = {"dist": "symmetric" if sym else "nonnegative", "e": e,
                   **{k: float(np.mean(v)) for k, v in acc.items()}}
            rows.append(row)
            log(f"offset {row['dist']} e={e}: termwise/12 {row['termwise/12']:.3g} "
                f"elementwise/12 {row['elementwise/12']:.3g} sgemm {row['sgemm_fp32_host']:.3g} "
                f"hgemm {row['hgemm']:.3g}")
    out["offset"] = {"n": n, "seeds": list(seeds), "rows": rows}


def prescale_sweep(run, n, exps, seeds, out):
    rows = []
    for sym in (True, False):
        for e in exps:
            acc = {}
            for seed in seeds:
                A, B = workloads.offset_exponent_operands(n, n, n, seed, e, symmetric=sym)
                ref = A.astype(np.float64) @ B.astype(np.float64)
                res = run.prescaled(A, B, 11)
                res.update({k: v for k, v in run.methods(A, B, (11,)).items()
                            if k in ("termwise/11", "elementwise/11", "sgemm_fp32_host")})
                for k, C in res.items():
                    acc.setdefault(k, []).append(frob(C, ref))
            row = {"dist": "symmetric" if sym else "nonnegative", "e": e,
                   **{k: float(np.mean(v)) for k, v in acc.items()}}
            rows.append(row)
            log(f"prescale {row['dist']} e={e}: termwise {row['termwise/11']:.3g} -> "
                f"{row['termwise/11/pre']:.3g}")
    out["prescale"] = {"n": n, "seeds": list(seeds), "rows": rows}


def size_sweep(run, name, shapes, seeds, out):
    rows = []
    for (m, n, k) in shapes:
        acc = {}
        for seed in seeds:
            A, B = workloads.offset_exponent_operands(m, n, k, seed, 0, symmetric=True)
            ref = A.astype(np.float64) @ B.astype(np.float64)
            for key, C in run.methods(A, B, (11, 12)).items():
                acc.setdefault(key, []).append(frob(C, ref))
        row = {"m": m, "n": n, "k": k, **{key: float(np.mean(v)) for key, v in acc.items()}}
        rows.append(row)
        log(f"{name} {m}x{n}x{k}: termwise/12 {row['termwise/12']:.3g} "
            f"elementwise/12 {row['elementwise/12']:.3g} sgemm {row['sgemm_fp32_host']:.3g}")
    out[name] = {"seeds": list(seeds), "rows": rows}


def adversarial_operands(family, M, N, K, seed):
    """Inputs built to stress one part of the method (synthetic, seeded)."""
    rng = np.random.default_rng(seed)
    sign = lambda shape: rng.choice([-1.0, 1.0], size=shape)
    if family == "max_residual":
        # |a| just below the midpoint between two FP16 neighbours: the FP16
        # rounding error, and so the residual carried by lo, is near its largest.
        e = rng.integers(-8, 8, size=(M, K))
        m = 1.0 + rng.integers(0, 1024, size=(M, K)) * 2.0**-10 + 2.0**-11 * (1 - 2.0**-12)
        A = (sign((M, K)) * np.ldexp(m, e)).astype(np.float32)
        e = rng.integers(-8, 8, size=(K, N))
        m = 1.0 + rng.integers(0, 1024, size=(K, N)) * 2.0**-10 + 2.0**-11 * (1 - 2.0**-12)
        B = (sign((K, N)) * np.ldexp(m, e)).astype(np.float32)
    elif family == "cancellation":
        # Columns of A in pairs (x, -x + small), rows of B in equal pairs: every
        # dot product cancels to a small fraction of sum |a||b|.
        half = K // 2
        x = rng.uniform(0.5, 1.0, size=(M, half)) * sign((M, half))
        y = -x + rng.uniform(-1, 1, size=(M, half)) * 2.0**-10
        A = np.empty((M, K))
        A[:, 0::2], A[:, 1::2] = x, y
        b = rng.uniform(-1, 1, size=(half, N))
        B = np.repeat(b, 2, axis=0)
        A, B = A.astype(np.float32), B.astype(np.float32)
    elif family == "swamping":
        # Each row of A holds a few entries of 2^12 among entries of 2^-12:
        # small products are added to large partial sums.
        A = (rng.uniform(0.5, 1.0, size=(M, K)) * 2.0**-12 * sign((M, K)))
        big = rng.random((M, K)) < 1.0 / 64
        A[big] = rng.uniform(0.5, 1.0, size=big.sum()) * 2.0**12
        A = A.astype(np.float32)
        B = rng.uniform(-1, 1, size=(K, N)).astype(np.float32)
    elif family == "wide_exponent":
        A = (sign((M, K)) * np.ldexp(rng.uniform(1, 2, (M, K)), rng.integers(-12, 13, (M, K)))).astype(np.float32)
        B = (sign((K, N)) * np.ldexp(rng.uniform(1, 2, (K, N)), rng.integers(-12, 13, (K, N)))).astype(np.float32)
    elif family == "subnormal_hi":
        A = np.ldexp(rng.uniform(-1, 1, (M, K)), -16).astype(np.float32)
        B = rng.uniform(-1, 1, (K, N)).astype(np.float32)
    else:
        raise ValueError(family)
    return A, B


FAMILIES = ("max_residual", "cancellation", "swamping", "wide_exponent", "subnormal_hi")


def maxnorm_study(run, M, N, K, seeds, out):
    rows = []
    for fam in FAMILIES:
        acc = {}
        for seed in seeds:
            A, B = adversarial_operands(fam, M, N, K, seed)
            A64, B64 = A.astype(np.float64), B.astype(np.float64)
            ref = A64 @ B64
            absab = np.abs(A64) @ np.abs(B64)
            nz = ref != 0
            for key, C in run.methods(A, B, (11,)).items():
                d = np.abs(C.astype(np.float64) - ref)
                with np.errstate(divide="ignore", invalid="ignore"):
                    norm = float(np.max(np.where(absab > 0, d / absab, 0.0)))
                rel = float(np.max(d[nz] / np.abs(ref[nz]))) if nz.any() else 0.0
                a = acc.setdefault(key, {"max_err_over_absab": 0.0, "max_rel_err": 0.0})
                a["max_err_over_absab"] = max(a["max_err_over_absab"], norm)
                a["max_rel_err"] = max(a["max_rel_err"], rel)
        rows.append({"family": fam, **acc})
        log(f"maxnorm {fam}: termwise {acc['termwise/11']['max_err_over_absab']:.3g} "
            f"elementwise {acc['elementwise/11']['max_err_over_absab']:.3g} "
            f"sgemm {acc['sgemm_fp32_host']['max_err_over_absab']:.3g}")
    out["maxnorm"] = {"M": M, "N": N, "K": K, "seeds": list(seeds), "rows": rows}


def to_markdown(res) -> str:
    fmt = lambda x: f"{x:.2e}"
    lines = ["# Accuracy on MI355X (Sec. 6.2 experiments)", "",
             f"Generated by `python bench_accuracy.py{' --quick' if res['quick'] else ''}` on one MI355X "
             f"({res['seconds']:.0f} s).  Relative Frobenius error (Eq. err) against numpy's FP64 matmul of "
             "the same FP32 inputs, averaged over seeds.  `ew`, `tw`, `cf` = the GPU's elementwise, termwise "
             "and cross-terms-first orders at s = 2^s_b; `hgemm` = the GPU FP16 baseline; `sgemm` = the "
             f"host's FP32 SGEMM (numpy float32 matmul, {res['blas']}).", ""]
    off = res["offset"]
    for dist in ("symmetric", "nonnegative"):
        lines += [f"## Offset exponent, {dist} inputs (m = n = k = {off['n']}, seeds {off['seeds']})", "",
                  "| e | hgemm | sgemm | ew 0 | tw 0 | ew 6 | tw 6 | ew 11 | tw 11 | cf 11 | ew 12 | tw 12 | cf 12 |",
                  "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
        for r in off["rows"]:
            if r["dist"] != dist:
                continue
            cells = [r["hgemm"], r["sgemm_fp32_host"], r["elementwise/0"], r["termwise/0"],
                     r["elementwise/6"], r["termwise/6"], r["elementwise/11"], r["termwise/11"],
                     r["elementwise_cross_first/11"], r["elementwise/12"], r["termwise/12"],
                     r["elementwise_cross_first/12"]]
            lines.append(f"| {r['e']} | " + " | ".join(fmt(c) for c in cells) + " |")
        lines.append("")
    for name, title in (("mn", "Error vs m = n at k = 2816 (e = 0, symmetric)"),
                        ("k", "Error vs k at m = n = 1024 (e = 0, symmetric)"),
                        ("mkn", "Error vs m = n = k (e = 0, symmetric)")):
        sec = res[name]
        lines += [f"## {title}, seeds {sec['seeds']}", "",
                  "| m | n | k | hgemm | sgemm | ew 11 | tw 11 | cf 11 | ew 12 | tw 12 | cf 12 |",
                  "|---|---|---|---|---|---|---|---|---|---|---|"]
        for r in sec["rows"]:
            cells = [r["hgemm"], r["sgemm_fp32_host"], r["elementwise/11"], r["termwise/11"],
                     r["elementwise_cross_first/11"], r["elementwise/12"], r["termwise/12"],
                     r["elementwise_cross_first/12"]]
            lines.append(f"| {r['m']} | {r['n']} | {r['k']} | " + " | ".join(fmt(c) for c in cells) + " |")
        lines.append("")
    pre = res["prescale"]
    lines += [f"## Pre-scaled (sgemm_cube_ex, PRESCALE), s = 2^11, m = n = k = {pre['n']}, "
              f"seeds {pre['seeds']}", "",
              "| dist | e | sgemm | ew | ew pre | tw | tw pre | cf pre |",
              "|---|---|---|---|---|---|---|---|"]
    for r in pre["rows"]:
        cells = [r["sgemm_fp32_host"], r["elementwise/11"], r["elementwise/11/pre"],
                 r["termwise/11"], r["termwise/11/pre"], r["elementwise_cross_first/11/pre"]]
        lines.append(f"| {r['dist']} | {r['e']} | " + " | ".join(fmt(c) for c in cells) + " |")
    lines.append("")
    mx = res["maxnorm"]
    lines += [f"## Max-norm errors on adversarial inputs (M = {mx['M']}, N = {mx['N']}, K = {mx['K']}, "
              f"s = 2^11, worst over seeds {mx['seeds']})", "",
              "Each cell: max |C - C64| / (|A||B|) over all entries, then (in brackets) the largest "
              "|C - C64| / |C64| over entries with C64 != 0.", "",
              "| family | hgemm | sgemm | ew | tw | cf |", "|---|---|---|---|---|---|"]
    for r in mx["rows"]:
        cells = []
        for key in ("hgemm", "sgemm_fp32_host", "elementwise/11", "termwise/11", "elementwise_cross_first/11"):
            c = r[key]
            cells.append(f"{fmt(c['max_err_over_absab'])} ({fmt(c['max_rel_err'])})")
        lines.append(f"| {r['family']} | " + " | ".join(cells) + " |")
    lines.append("")
    return "\n".join(lines)


def blas_name() -> str:
    try:
        cfg = np.show_config(mode="dicts")
        return cfg["Build Dependencies"]["blas"]["name"]
    except Exception:  # noqa: BLE001 - informational only
        return "numpy's BLAS"


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--quick", action="store_true", help="fewer points and seeds")
    ap.add_argument("--out", default=None, help="write the results as JSON")
    ap.add_argument("--md", default=None, help="write the tables as markdown")
    args = ap.parse_args()
    run = Runner()
    t0 = time.perf_counter()
    res = {"quick": args.quick, "blas": blas_name()}
    if args.quick:
        offset_sweep(run, 256, (-16, -8, 0, 8), (0, 1), res)
        size_sweep(run, "mn", [(256, 256, 2816), (1024, 1024, 2816)], (0,), res)
        size_sweep(run, "k", [(256, 256, 256), (256, 256, 4096)], (0,), res)
        size_sweep(run, "mkn", [(256, 256, 256), (512, 512, 512)], (0,), res)
        maxnorm_study(run, 128, 128, 1024, (0,), res)
        prescale_sweep(run, 256, (-24, 0, 20), (0,), res)
    else:
        offset_sweep(run, 1024, tuple(range(-20, 13, 2)), (0, 1, 2, 3, 4), res)
        size_sweep(run, "mn", [(n, n, 2816) for n in (256, 512, 1024, 2048, 4096, 8192)], (0, 1, 2), res)
        size_sweep(run, "k", [(1024, 1024, k) for k in (256, 1024, 4096, 16384, 65536)], (0, 1, 2), res)
        size_sweep(run, "mkn", [(n, n, n) for n in (512, 1024, 2048, 4096)], (0, 1, 2), res)
        maxnorm_study(run, 512, 512, 8192, (0, 1, 2), res)
        prescale_sweep(run, 1024, (-28, -24, -20, -16, 0, 16, 20, 24), (0, 1, 2, 3, 4), res)
    res["seconds"] = time.perf_counter() - t0
    if args.out:
        with open(args.out, "w") as f:
            json.dump(res, f, indent=1)
    md = to_markdown(res)
    if args.md:
        with open(args.md, "w") as f:
            f.write(md)
    print(md)


if __name__ == "__main__":
    main()
