"""Benchmark: FP32-equivalent throughput of SGEMM-cube on one MI355X.

    python bench.py [--gpus 1] [--steps 50] [--warmup 10] [--workload c3]
                    [--order elementwise] [--no-cpu-baseline]

A step is one whole SGEMM-cube call on the named workload (default: the
8192^3 U[-1,1] peak-throughput case, s = 2^11, elementwise): FP32 A and B
already resident in HBM -> split (Sec. 3.3) -> three-product MFMA GEMM with
FP32 reconstruction (Eq. recover_eqn, Sec. 4.5) -> FP32 C in HBM.  It is the
same work as one sgemm_cube_ws call, issued as its two halves
(sgemm_cube_prepare + sgemm_cube_compute) so that HIP events on the launch
stream can time the dominant GEMM kernel inside the timed region.

Prints ONE JSON line.  `value` = 2MNK / t (FP32-equivalent TFLOP/s, Sec. 6.1);
`roofline` prices the GEMM kernel's 6MNK FP16 MFMA flops against the dense
FP16 MFMA peak; `cpu_baseline` times the CPU oracle on a bounded row sample of
the same workload on this host; `context` times, outside the timed region and
on the same operands, the native-FP16 baseline call of this library and the
vendor FP32 and FP16 GEMMs (torch.matmul), as reference points only.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

METRIC = "FP32-equiv TFLOP/s (2MNK/t) and % of 3-GEMM FP16 MFMA peak; max rel err"
# MI355X dense FP16 MFMA peak: 256 CU x 2.4 GHz x 4096 FLOP/clk/CU (published
# as 2.5 PFLOP/s).  The three-GEMM FP32-equivalent peak is a third of it.
FP16_PEAK_TFLOPS = 256 * 2.4e9 * 4096 / 1e12
THREE_GEMM_PEAK_TFLOPS = FP16_PEAK_TFLOPS / 3
HBM_PEAK_GBS = 8000.0
# The MFMA kernel that runs for each order: for the elementwise order the
# 256 x 256 kernel that splits A in registers (where the library chooses it:
# sgemm_cube_splits_a_in_gemm) or the one that reads the A planes (elsewhere,
# and with --unfused); either call also launches
# the unscaled 256 x 128 kernel, which reads the range flag and returns at once
# unless some |B_hi| s exceeds 65504, in which case it does the work.  For
# termwise the 256 x 128 kernel, likewise with A split in registers where the
# library chooses it, and with --split-b-in-gemm the same kernel splitting B
# (and A, where the library splits A in the GEMM) itself.  The cross-terms-first
# order has a scaled kernel and an unscaled fallback too, chosen as for the
# elementwise order.
GEMM_KERNELS = {"elementwise": "gemm_el_kernel<true, true>",
                "elementwise_unfused": "gemm_el_kernel<true, false>",
                "elementwise_unscaled": "gemm_n128_kernel<0, false, false>",
                "termwise": "gemm_n128_kernel<1, false, false>",
                "termwise_fused": "gemm_n128_kernel<1, true, false>",
                "termwise_fused_b": "gemm_n128_kernel<1, false, true>",
                "termwise_fused_ab": "gemm_n128_kernel<1, true, true>",
                "elementwise_cross_first": "gemm_n128_kernel<4, false, false>",
                "elementwise_cross_first_unscaled": "gemm_n128_kernel<3, false, false>"}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_traffic.json")


def gemm_kernel_name(kernel_key: str) -> str:
    """Kernel name of a GEMM_KERNELS key or of "elementwise_tile_" + tile_name()
    (the tile sweep: two workgroups per compute unit for 128x128x32; waves
    2 x 2, or 2 x 4 for eight)."""
    if kernel_key.startswith("elementwise_tile_"):
        dims = [int(v) for v in kernel_key.rsplit("_", 1)[1].split("x")]
        bm, bn, bk, waves = dims + [4] * (4 - len(dims))
        occ = 2 if (bm, bn, bk) == (128, 128, 32) else 1
        wm, wn = (2, 4) if waves == 8 else (2, 2)
        return f"gemm_tile_kernel<{bm}, {bn}, {bk}, {occ}, {wm}, {wn}>"
    return GEMM_KERNELS[kernel_key]


def tile_name(tile) -> str:
    """BMxBNxBK for the four-wave sweep kernels, BMxBNxBKxW otherwise."""
    return "x".join(map(str, tile if tile[3] != 4 else tile[:3]))


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _code_only(text: str) -> str:
    """C++ source without comments and with whitespace collapsed, so that a
    change of comments alone does not count as a change of the kernel."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c == '"':  # string literal (inline asm text): keep verbatim
            j = i + 1
            while j < n and text[j] != '"':
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the code (comments excluded) of the sources the GEMM kernel is
    built from: ties a committed HBM-traffic measurement to the kernel it was
    taken on."""
    h = hashlib.sha256()
    for rel in ("paper_2507_23387_amd/csrc/gemm.hip", "paper_2507_23387_amd/csrc/gemm_tile.hip",
                "paper_2507_23387_amd/csrc/gemm_common.h",
                "paper_2507_23387_amd/csrc/internal.h"):
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def traffic_entry(workload: str, order: str):
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    if data.get("kernel_source_hash") != kernel_source_hash():
        return None
    return data.get("entries", {}).get(f"{workload}/{order}")


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# Threads the CPU oracle may use: the host's available cores, capped at the
# CPU share one GPU gets on the benchmark machines.
CPU_THREAD_CAP = 16


def cpu_baseline(A, B, w, scale, order, target_s: float, kb: int):
    """Time the oracle (as it stands) on a bounded sample of output rows.

    Two calibration calls (T and 2T rows, T = threads) separate the per-call
    overhead (the oracle splits and widens all of B on every call) from the
    per-row cost; the sample is then sized to take about target_s.  Returns
    the report and the sampled rows with the oracle's values of them (the
    oracle runs with the GPU's elementwise block size kb, so they also serve
    as the parity reference)."""
    import oracle

    available = len(os.sched_getaffinity(0))
    threads = min(available, CPU_THREAD_CAP)

    def timed(n):
        rows = workloads.sample_rows(w.M, n, w.seed + n)
        t0 = time.perf_counter()
        oracle.sgemm_rows(A, B, rows, scale, order, kb=kb, threads=threads)
        return time.perf_counter() - t0

    t1 = timed(threads)
    t2 = timed(2 * threads)
    t_wave = max(t2 - t1, 1e-6)          # one more row per thread
    overhead = max(t1 - t_wave, 0.0)
    waves = int(max(1, min(w.M // threads, (target_s - overhead) / t_wave)))
    n = waves * threads
    rows = workloads.sample_rows(w.M, n, w.seed + 2)
    t0 = time.perf_counter()
    C_rows = oracle.sgemm_rows(A, B, rows, scale, order, kb=kb, threads=threads)
    t = time.perf_counter() - t0
    flops = 2.0 * len(rows) * w.N * w.K
    return {
        "value": flops / t / 1e12,
        "unit": "TFLOP/s",
        "cores": threads,
        "cores_available": available,
        "cpu_count": os.cpu_count(),
        "cpu_model": _cpu_model(),
        "kind": "oracle",
        "sample": f"{len(rows)} of {w.M} output rows of {w.name} ({order}, s=2^"
                  f"{int(np.log2(scale))}), full K={w.K} and N={w.N}; the oracle's split of "
                  f"all of B (about {overhead:.1f} s) included; {t:.1f} s wall",
        "seconds": t,
    }, rows, C_rows


def parity_report(C_gpu_rows, C_oracle_rows, A, B, rows, K):
    """Verdict of the GPU result against the oracle on sampled rows: the bar
    |C_gpu - C_oracle|_ij <= 2 K 2^-24 (|A||B|)_ij (equality where
    (|A||B|)_ij = 0, identical inf/NaN patterns) and its worst ratio."""
    g = C_gpu_rows.astype(np.float64)
    o = C_oracle_rows.astype(np.float64)
    absab = np.abs(A[rows].astype(np.float64)) @ np.abs(B.astype(np.float64))
    tol = 2.0 * K * 2.0**-24 * absab
    fin = np.isfinite(o)
    same_nonfinite = bool(np.array_equal(np.isnan(g), np.isnan(o)) and
                          np.array_equal(np.isinf(g), np.isinf(o)))
    err = np.abs(g[fin] - o[fin])
    t = tol[fin]
    ok = bool(same_nonfinite and np.all(err <= t))
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(t > 0, err / t, np.where(err > 0, np.inf, 0.0))
    return {
        "verdict": "pass" if ok else "fail",
        "bar": "|C_gpu - C_oracle| <= 2 K 2^-24 (|A||B|)",
        "rows": int(len(rows)),
        "entries": int(g.size),
        "worst_err_over_tol": float(ratio.max()) if ratio.size else 0.0,
        "max_abs_err": float(err.max()) if err.size else 0.0,
    }


def hi_only_gap(C_gpu_rows, C_oracle_rows, C_hi_rows):
    """max|C_gpu - C_oracle| / max|C_oracle - C_hi_only| on the same rows: a
    correct kernel sits far below 1 (the GPU and the oracle differ only in
    FP32 summation order), one that drops a correction term near or above 1."""
    g, o, h = (x.astype(np.float64) for x in (C_gpu_rows, C_oracle_rows, C_hi_rows))
    fin = np.isfinite(o) & np.isfinite(h)
    gap = np.abs(o - h)[fin].max()
    return float(np.abs(g - o)[fin].max() / gap) if gap > 0 else None


def _timed_ms(fn, stream, reps: int) -> float:
    """Mean duration of fn() over `reps` calls, HIP events on `stream`."""
    import torch
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def context_gemms(sgc, dA, dB, A, B, rows, stream, with_errors: bool):
    """Reference points on the same operands, outside the timed region: the
    native-FP16 MFMA baseline of this library (sgemm_cube_hgemm: FP32 in,
    fl16 conversion + HH-only GEMM), the vendor FP32 GEMM (torch.matmul on
    FP32, the call SGEMM-cube stands in for) and the vendor FP16 GEMM on
    operands already converted to FP16 (conversion not timed)."""
    import torch
    M, K = dA.shape
    N = dB.shape[1]
    flops = 2.0 * M * N * K
    out = {}
    Ch = torch.empty((M, N), dtype=torch.float32, device=dA.device)

    def hg():
        st = sgc.sgemm_cube_hgemm(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, Ch.data_ptr(), N,
                                  stream.cuda_stream)
        if st:
            raise sgc.SgemmCubeError(st, "sgemm_cube_hgemm")

    t = _timed_ms(hg, stream, 10)
    out["hgemm_call"] = {"ms": t, "tflops": flops / (t * 1e-3) / 1e12,
                         "what": "sgemm_cube_hgemm: FP32 in, fl16(A) fl16(B) on MFMA, FP32 out"}
    Cf = torch.empty((M, N), dtype=torch.float32, device=dA.device)
    t = _timed_ms(lambda: torch.matmul(dA, dB, out=Cf), stream, 10)
    out["vendor_fp32_gemm"] = {"ms": t, "tflops": flops / (t * 1e-3) / 1e12,
                               "what": "torch.matmul on FP32 tensors"}
    if with_errors:
        torch.cuda.synchronize()
        out["vendor_fp32_gemm"]["errors"] = error_report(Cf.cpu().numpy()[rows], A, B, rows)
    del Cf
    hA, hB = dA.half(), dB.half()
    Ch16 = torch.empty((M, N), dtype=torch.float16, device=dA.device)
    t = _timed_ms(lambda: torch.matmul(hA, hB, out=Ch16), stream, 10)
    out["vendor_fp16_gemm"] = {"ms": t, "tflops": flops / (t * 1e-3) / 1e12,
                               "what": "torch.matmul on FP16 tensors (conversion not timed)"}
    del hA, hB, Ch16, Ch
    return out


def error_report(C_rows, A, B, rows):
    """Context errors against an FP64 GEMM on sampled rows (Sec. 6.2 Eq. err
    plus the componentwise forms)."""
    ref = A[rows].astype(np.float64) @ B.astype(np.float64)
    absab = np.abs(A[rows].astype(np.float64)) @ np.abs(B.astype(np.float64))
    d = np.abs(C_rows.astype(np.float64) - ref)
    nz = np.abs(ref) > 0
    return {
        "max_rel_err": float(np.max(d[nz] / np.abs(ref[nz]))),
        "max_err_over_absAabsB": float(np.max(d / np.where(absab > 0, absab, 1.0))),
        "frobenius_rel_err": float(np.linalg.norm(d) / np.linalg.norm(ref)),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1,
                    help="number of GPUs; only 1 is supported (anything else exits with a message)")
    ap.add_argument("--steps", type=int, default=50, help="timed steps (one call each)")
    ap.add_argument("--warmup", type=int, default=10, help="untimed steps before them")
    ap.add_argument("--workload", default="c3",
                    help="c1 256^3, c2 4096^3, c3 8192^3 (default), c4 4096x4096x16384, "
                         "c5 16384x1024x8192, or a workload name")
    ap.add_argument("--order", default=None, help="elementwise | termwise | elementwise_cross_first")
    ap.add_argument("--scale", type=float, default=None,
                    help="s, a power of two in [1, 2^24] (default: the workload's, 2^11)")
    ap.add_argument("--stages", type=int, default=0,
                    help="elementwise only: 2 = copies overlapped with the MFMAs, 1 = copies "
                         "issued and waited for at the end of each step (0 = the library's "
                         "default), through sgemm_cube_compute_stages")
    ap.add_argument("--tile", default=None,
                    help="elementwise only: BMxBNxBK[xWAVES], time the tile-sweep kernel of "
                         "sgemm_cube_compute_tile (256x256x32, 256x128x32, 128x256x32, "
                         "128x128x32, 128x128x64 with 4 waves; 256x256x32x8) instead of the "
                         "library's GEMM")
    ap.add_argument("--unfused", action="store_true",
                    help="split A into the workspace and run the GEMM on the A planes also where "
                         "sgemm_cube would split A inside the GEMM kernel")
    ap.add_argument("--split-b-in-gemm", action="store_true",
                    help="termwise only: split B inside the GEMM kernel (sgemm_cube_compute_b "
                         "after a split pass of A, or one sgemm_cube_ex call with "
                         "SGEMM_CUBE_OPT_SPLIT_B_IN_GEMM where A is split in the GEMM too)")
    ap.add_argument("--prescale", action="store_true",
                    help="time sgemm_cube_ex with power-of-two pre-scaling (one call per step)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the oracle on the host cores")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target length of the oracle's timed sample")
    ap.add_argument("--no-errors", action="store_true",
                    help="skip the error metrics against an FP64 product")
    ap.add_argument("--no-parity", action="store_true",
                    help="skip the comparison with the oracle (short profiling runs)")
    ap.add_argument("--no-context", action="store_true",
                    help="skip the FP16-baseline and vendor-GEMM reference timings")
    ap.add_argument("--copy-mib", type=int, default=512,
                    help="size of the calibration copy (0 = skip)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the method is a "
              "single-GPU GEMM here and multi-GPU sharding is not built", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2507_23387_amd as sgc

    w = workloads.get(args.workload)
    order = args.order or w.orders[0]
    scale = args.scale or w.scales[0]
    order_code = sgc.binding.ORDERS[order]
    M, N, K = w.M, w.N, w.K
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    log(f"generating {w.name} ({M}x{N}x{K}, seed {w.seed})")
    A, B = workloads.workload_operands(w)
    dA = torch.from_numpy(A).to(dev)
    dB = torch.from_numpy(B).to(dev)
    dC = torch.empty((M, N), dtype=torch.float32, device=dev)
    ws_bytes = (sgc.sgemm_cube_ex_workspace_size(M, N, K, order_code, sgc.binding.OPT_PRESCALE)
                if args.prescale else sgc.sgemm_cube_workspace_size(M, N, K, order_code))
    ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    # A step enqueues what sgemm_cube_ws enqueues.  Where the library splits
    # A inside the GEMM kernel (sgemm_cube_splits_a_in_gemm) that is the split
    # of B (sgemm_cube_prepare with A = NULL) and sgemm_cube_compute_a; else,
    # and with --unfused or --stages, the split of both operands
    # (sgemm_cube_prepare) and the GEMM on the tiled planes.
    tile = tuple(int(v) for v in args.tile.lower().split("x")) if args.tile else None
    if tile and len(tile) == 3:
        tile = tile + (4,)
    if tile and (order != "elementwise" or tile not in sgc.binding.TILE_CONFIGS):
        print(f"--tile {args.tile}: the sweep covers the elementwise order and "
              f"{sgc.binding.TILE_CONFIGS}", file=sys.stderr)
        sys.exit(2)
    fused = (not args.unfused and not args.stages and not args.prescale and not tile and
             sgc.binding.sgemm_cube_splits_a_in_gemm(M, N, K, dA.data_ptr(), K, scale,
                                                     order_code) == 1)
    split_b = args.split_b_in_gemm
    if split_b and (order != "termwise" or args.prescale or args.stages or tile):
        print("--split-b-in-gemm: the termwise order only, without --prescale, --stages or "
              "--tile", file=sys.stderr)
        sys.exit(2)

    def prepare():
        st = sgc.sgemm_cube_prepare(M, N, K, None if fused else dA.data_ptr(), K, dB.data_ptr(),
                                    N, scale, ws.data_ptr(), ws_bytes, sh)
        if st:
            raise sgc.SgemmCubeError(st, "sgemm_cube_prepare")

    def compute():
        if fused:
            st = sgc.sgemm_cube_compute_a(M, N, K, dA.data_ptr(), K, dC.data_ptr(), N, scale,
                                          order_code, ws.data_ptr(), ws_bytes, sh)
        elif tile:
            st = sgc.binding.sgemm_cube_compute_tile(M, N, K, dC.data_ptr(), N, scale, order_code,
                                                     *tile, ws.data_ptr(), ws_bytes, sh)
        elif args.stages:
            st = sgc.binding.sgemm_cube_compute_stages(M, N, K, dC.data_ptr(), N, scale,
                                                       order_code, args.stages, ws.data_ptr(),
                                                       ws_bytes, sh)
        else:
            st = sgc.sgemm_cube_compute(M, N, K, dC.data_ptr(), N, scale, order_code,
                                        ws.data_ptr(), ws_bytes, sh)
        if st:
            raise sgc.SgemmCubeError(st, "sgemm_cube_compute")

    if split_b and fused:
        # Both operands split inside the GEMM kernel: one call, one kernel,
        # timed in the "compute" slot.
        def prepare():
            pass

        def compute():
            st = sgc.sgemm_cube_ex(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, dC.data_ptr(), N,
                                   scale, order_code, sgc.binding.OPT_SPLIT_B_IN_GEMM,
                                   ws.data_ptr(), ws_bytes, None, sh)
            if st:
                raise sgc.SgemmCubeError(st, "sgemm_cube_ex")
    elif split_b:
        # The split pass of A, then the GEMM that splits B itself.
        def prepare():
            st = sgc.sgemm_cube_prepare(M, N, K, dA.data_ptr(), K, None, N, scale, ws.data_ptr(),
                                        ws_bytes, sh)
            if st:
                raise sgc.SgemmCubeError(st, "sgemm_cube_prepare")

        def compute():
            st = sgc.binding.sgemm_cube_compute_b(M, N, K, dB.data_ptr(), N, dC.data_ptr(), N,
                                                  scale, order_code, ws.data_ptr(), ws_bytes, sh)
            if st:
                raise sgc.SgemmCubeError(st, "sgemm_cube_compute_b")

    if args.prescale:
        # The pre-scaled call has no split/compute halves: the whole call is
        # timed in the "compute" slot and the "prepare" slot is empty.
        def prepare():
            pass

        def compute():
            st = sgc.sgemm_cube_ex(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N, dC.data_ptr(), N,
                                   scale, order_code, sgc.binding.OPT_PRESCALE, ws.data_ptr(),
                                   ws_bytes, None, sh)
            if st:
                raise sgc.SgemmCubeError(st, "sgemm_cube_ex")

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        prepare()
        compute()
    torch.cuda.synchronize()

    log(f"timing {args.steps} steps")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for s in range(args.steps):
        ev[s][0].record(stream)
        prepare()
        ev[s][1].record(stream)
        compute()
        ev[s][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = ev[0][0].elapsed_time(ev[-1][2])
    split_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    gemm_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    step_times = np.array([e[0].elapsed_time(e[2]) for e in ev])
    ms_per_step = total_ms / args.steps
    flops = 2.0 * M * N * K
    value = flops / (ms_per_step * 1e-3) / 1e12
    log(f"{ms_per_step:.4f} ms/step (split {split_ms:.4f}, gemm {gemm_ms:.4f}); "
        f"{value:.1f} TFLOP/s FP32-equivalent = {100 * value / THREE_GEMM_PEAK_TFLOPS:.1f}% "
        f"of the 3-GEMM peak; wall {wall * 1e3 / args.steps:.4f} ms/step")

    # A plain device copy of known size, outside the timed region: the
    # rocprofv3 FETCH_SIZE / WRITE_SIZE counters of this dispatch calibrate
    # the same counters read for the GEMM kernel.
    # Its bandwidth (bytes read + written) is also the practical ceiling the
    # HBM-bound split is compared with.
    copy_gbs = None
    if args.copy_mib > 0:
        n = args.copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        for _ in range(5):
            dst.copy_(src)
        c1.record(stream)
        torch.cuda.synchronize()
        copy_gbs = 2 * 4 * n * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
        del src, dst

    gemm_tflops = 3 * flops / (gemm_ms * 1e-3) / 1e12
    kernel_key = order
    # The range flag: the workspace's first two words are equal after a split
    # of B that found |B_hi| s > 65504 (s > 2^15 routes there too).
    hdr = ws[:8].view(torch.int32).cpu()
    unscaled = bool(hdr[0] == hdr[1]) or scale > 32768.0
    if order == "elementwise":
        if unscaled:
            kernel_key = "elementwise_unscaled"
        elif tile:
            kernel_key = "elementwise_tile_" + tile_name(tile)
        elif not fused:
            kernel_key = "elementwise_unfused"
    elif order == "elementwise_cross_first" and unscaled:
        kernel_key = "elementwise_cross_first_unscaled"
    elif order == "termwise" and split_b:
        kernel_key = "termwise_fused_ab" if fused else "termwise_fused_b"
    elif order == "termwise" and fused:
        kernel_key = "termwise_fused"
    traffic = traffic_entry(w.name, kernel_key)
    roofline = {
        "bound": "mfma",
        "kernel": gemm_kernel_name(kernel_key),
        "achieved": gemm_tflops,
        "peak": FP16_PEAK_TFLOPS,
        "unit": "TFLOP/s",
        "frac": gemm_tflops / FP16_PEAK_TFLOPS,
        "traffic": traffic,
        "algorithmic_flops_per_launch": 3 * flops,
        "avg_launch_ms": gemm_ms,
    }
    # 4 B read + 2 x 2 B written per element split (B only when A is split in
    # the GEMM kernel, A only when B is).
    split_bytes = 8.0 * ((0 if fused else M * K) + (0 if split_b else K * N))
    extra = {
        "pct_of_3gemm_peak": 100 * value / THREE_GEMM_PEAK_TFLOPS,
        "three_gemm_peak_tflops": THREE_GEMM_PEAK_TFLOPS,
        "split_ms": split_ms,
        "split_gbs": split_bytes / (split_ms * 1e-3) / 1e9 if split_bytes else None,
        "device_copy_gbs": copy_gbs,
        "gemm_ms": gemm_ms,
        "step_ms": {"median": float(np.median(step_times)), "min": float(step_times.min()),
                    "max": float(step_times.max())},
        "wall_ms_per_step": wall * 1e3 / args.steps,
    }

    import oracle

    kb = sgc.sgemm_cube_block_k()
    C_gpu = dC.cpu().numpy()  # the result of the last timed step

    if not args.no_errors:
        log("context errors on sampled rows vs FP64 (both orders and the FP16 baseline)")
        rows = workloads.sample_rows(M, 8, w.seed + 3)
        extra["errors"] = {}
        for o in ("elementwise", "termwise"):
            if o == order and not args.prescale:
                Cn = C_gpu[rows]
            else:
                Co_dev = sgc.matmul(dA, dB, scale, o)
                torch.cuda.synchronize()
                Cn = Co_dev.cpu().numpy()[rows]
                del Co_dev
            extra["errors"][o] = error_report(Cn, A, B, rows)
        Ch = sgc.hgemm(dA, dB)
        torch.cuda.synchronize()
        extra["errors"]["hgemm_fp16"] = error_report(Ch.cpu().numpy()[rows], A, B, rows)
        del Ch
        extra["max_rel_err"] = error_report(C_gpu[rows], A, B, rows)["max_rel_err"]

    if not args.no_context:
        log("context: FP16 baseline and vendor GEMM timings")
        rows = workloads.sample_rows(M, 8, w.seed + 3)
        extra["context"] = context_gemms(sgc, dA, dB, A, B, rows, stream, not args.no_errors)

    cpu = None
    parity = None
    oracle_fn = oracle.sgemm_prescaled if args.prescale else oracle.sgemm
    if args.no_parity:
        if not args.no_cpu_baseline:
            log(f"cpu baseline (oracle) ~{args.cpu_seconds:.0f} s")
            cpu = cpu_baseline(A, B, w, scale, order, args.cpu_seconds, kb)[0]
    elif not args.no_cpu_baseline:
        log(f"cpu baseline (oracle) ~{args.cpu_seconds:.0f} s")
        if args.prescale:
            # The oracle's pre-scaled product has no row-sampled form; time the
            # plain oracle and check parity on band rows below.
            cpu, prow, C_or = cpu_baseline(A, B, w, scale, order, args.cpu_seconds, kb)
            prow = workloads.band_rows(M, w.seed)
            C_or = oracle_fn(A[prow], B, scale, order, kb=kb)
        else:
            cpu, prow, C_or = cpu_baseline(A, B, w, scale, order, args.cpu_seconds, kb)
    else:
        prow = workloads.band_rows(M, w.seed)
        C_or = oracle_fn(A[prow], B, scale, order, kb=kb)
    if not args.no_parity:
        log(f"parity of the timed result against the oracle on {len(prow)} rows")
        parity = parity_report(C_gpu[prow], C_or, A, B, prow, K)
        # The distance to the oracle's hi-only product on one row per 256-row band.
        brow = workloads.band_rows(M, w.seed + 1)
        C_band = oracle_fn(A[brow], B, scale, order, kb=kb)
        C_hi = oracle_fn(A[brow], B, scale, "hi_only", kb=kb)
        parity["band_rows"] = int(len(brow))
        parity["band_verdict"] = parity_report(C_gpu[brow], C_band, A, B, brow, K)["verdict"]
        parity["max_err_over_hi_only_gap"] = hi_only_gap(C_gpu[brow], C_band, C_hi)
        if (parity["band_verdict"] != "pass" or
                not (parity["max_err_over_hi_only_gap"] or 0) <= 0.1):
            parity["verdict"] = "fail"

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 MFMA products, f32 accumulation (f32 in/out)",
        "data": "synthetic",
        "config": {"workload": w.name, "M": M, "N": N, "K": K, "seed": w.seed,
                   "distribution": w.dist, "scale": scale, "order": order,
                   **({"prescale": True} if args.prescale else {}),
                   "split_of_a": "in the GEMM kernel" if fused else "separate pass",
                   "split_of_b": "in the GEMM kernel" if split_b else "separate pass",
                   **({"stages": args.stages} if args.stages else {}),
                   **({"tile": tile_name(tile)} if tile else {})},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "parity": parity,
        **extra,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
