"""Sustained rate of v_mfma_f32_16x16x32_f16 with register-held operands on one MI355X.

    python bench_ceiling.py [--workgroups 1024] [--iters 4000] [--reps 20] [--smi]

Runs sgemm_cube_mfma_loop (a diagnostic entry point of libsgemmcube: each wave
issues 64 * iters MFMAs from operands held in registers, no memory traffic in
the loop) on several kinds of FP16 operand data and prints a markdown table:
ms per launch (HIP events, median of --reps launches after 3 warm-up
launches), TFLOP/s, and the fraction of the published dense FP16 peak
(2516.6 TFLOP/s = 256 CU x 2.4 GHz x 4096 FLOP/clk).  The board's power limit
lowers the clock by how much energy the operands cost, so this rate is the
practical ceiling for the GEMM kernels, whose operands are random data.
With --smi, `amd-smi metric -p -c` is sampled while each case runs for about
two seconds, and the mean socket power and GFX clock are added.
"""
from __future__ import annotations

import argparse
import os
import re
import subprocess
import sys
import threading
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP16_PEAK_TFLOPS = 256 * 2.4e9 * 4096 / 1e12
OPERAND_VALUES = 32768  # FP16 values read by every workgroup (64 KiB)


def operand_data(kind: str, seed: int = 1) -> np.ndarray:
    """FP16 operand values as uint16 bit patterns."""
    rng = np.random.default_rng(seed)
    if kind == "uniform":
        v = rng.uniform(-1.0, 1.0, OPERAND_VALUES)
    elif kind == "normal":
        v = rng.standard_normal(OPERAND_VALUES)
    elif kind == "constant":
        v = np.full(OPERAND_VALUES, 0.5)
    elif kind == "zero":
        v = np.zeros(OPERAND_VALUES)
    else:
        raise ValueError(kind)
    return v.astype(np.float16).view(np.uint16)


class SmiSampler:
    """Background sampler of socket power (W) and mean GFX clock (MHz)."""

    def __init__(self, period: float = 0.3):
        self.period = period
        self.samples = []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            try:
                out = subprocess.run(["amd-smi", "metric", "-p", "-c"], capture_output=True,
                                     text=True, timeout=5).stdout
            except (OSError, subprocess.TimeoutExpired):
                return
            p = re.search(r"SOCKET_POWER:\s*([\d.]+)", out)
            clks = [float(c) for c in re.findall(r"\bCLK:\s*([\d.]+)\s*MHz", out)[:8]]
            if p and clks:
                self.samples.append((float(p.group(1)), sum(clks) / len(clks)))
            time.sleep(self.period)

    def __enter__(self):
        self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._thread.join(timeout=10)

    def summary(self):
        # The driver refreshes its values about once a second: drop the first
        # second's samples, taken while the load was ramping up.
        s = self.samples[3:] or self.samples
        if not s:
            return None, None
        return float(np.mean([p for p, _ in s])), float(np.mean([c for _, c in s]))


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workgroups", type=int, default=1024)
    ap.add_argument("--iters", type=int, default=4000)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--kinds", default="uniform,normal,constant,zero")
    ap.add_argument("--smi", action="store_true")
    args = ap.parse_args()

    import torch

    import paper_2507_23387_amd as sgc

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    out = torch.empty(args.workgroups * 256, dtype=torch.float32, device=dev)
    flop = args.workgroups * 4 * args.iters * 64 * 16 * 16 * 32 * 2.0

    print(f"sgemm_cube_mfma_loop: {args.workgroups} workgroups x 4 waves x {args.iters} x 64 "
          f"MFMAs = {flop / 1e12:.2f} TFLOP per launch\n")
    head = "| operands | ms per launch | TFLOP/s | % of 2516.6 |"
    sep = "|---|---|---|---|"
    if args.smi:
        head += " socket power W | mean GFX clock MHz |"
        sep += "---|---|"
    print(head)
    print(sep, flush=True)
    for kind in args.kinds.split(","):
        ops = torch.from_numpy(operand_data(kind).view(np.int16).copy()).to(dev)

        def launch():
            st = sgc.sgemm_cube_mfma_loop(args.workgroups, args.iters, ops.data_ptr(),
                                          ops.numel() * 2, out.data_ptr(), out.numel() * 4,
                                          stream.cuda_stream)
            if st:
                raise sgc.SgemmCubeError(st, "sgemm_cube_mfma_loop")

        for _ in range(3):
            launch()
        torch.cuda.synchronize()
        times = []
        for _ in range(args.reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            e1.synchronize()
            times.append(e0.elapsed_time(e1))
        ms = float(np.median(times))
        tf = flop / (ms * 1e-3) / 1e12
        row = f"| {kind} | {ms:.3f} | {tf:.1f} | {100 * tf / FP16_PEAK_TFLOPS:.1f}% |"
        if args.smi:
            with SmiSampler() as smi:
                t_end = time.perf_counter() + 2.0
                while time.perf_counter() < t_end:
                    for _ in range(10):
                        launch()
                    torch.cuda.synchronize()
            p, c = smi.summary()
            row += f" {p:.0f} | {c:.0f} |" if p is not None else " n/a | n/a |"
        print(row, flush=True)


if __name__ == "__main__":
    main()
