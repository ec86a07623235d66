"""Summaries of rocprofv3 runs of bench.py, for the files under profiles/.

    python bench_profile.py stats DIR
        kernel statistics of a `rocprofv3 --kernel-trace --stats` run
        (DIR/**/*kernel_stats.csv) as a markdown table
    python bench_profile.py traffic FETCH_DIR WRITE_DIR --workload W --order O
                            [--copy-mib 512] [--source profiles/FILE.md]
        HBM traffic of the GEMM kernel from two `rocprofv3 --pmc` passes
        (FETCH_SIZE, then WRITE_SIZE), each scaled by what the same counter
        reads for bench.py's plain device copy of --copy-mib MiB; writes the
        entry into profiles/gemm_traffic.json (tied to the hash of the GEMM
        kernel's sources) and prints a markdown summary
    python bench_profile.py busy DIR
        MFMA busy fraction and average shader clock per GEMM dispatch from a
        `--pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES` pass
    python bench_profile.py lds_l2 DIR
        LDS bank conflicts and L2 hit rate per GEMM dispatch from a
        `--pmc SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS TCC_HIT_sum
        TCC_MISS_sum` pass

Reads only the CSV files rocprofv3 wrote; runs nothing on the GPU.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402  (kernel-name table, source hash, traffic file)
import workloads  # noqa: E402

SIMDS = 1024  # 256 CUs x 4 SIMDs
XCDS = 8


def _rows(directory: str, suffix: str):
    files = sorted(glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {directory}")
    out = []
    for f in files:
        with open(f, newline="") as fh:
            out.extend(csv.DictReader(fh))
    return out


def short(name: str) -> str:
    """Kernel name without the namespace and argument list."""
    n = name
    for pre in ("void ", "(anonymous namespace)::", "sgc::"):
        n = n.replace(pre, "")
    return n.split("(")[0][:60]


def stats(directory: str) -> str:
    rows = _rows(directory, "kernel_stats.csv")
    lines = ["| kernel | calls | avg us | min us | max us | share |",
             "|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"| {short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{float(r['Percentage']):.1f}% |")
    return "\n".join(lines)


def counters(directory: str, counter: str):
    """{kernel: [value per dispatch]} of one counter (KiB for *_SIZE)."""
    per = defaultdict(dict)
    for r in _rows(directory, "counter_collection.csv"):
        if r["Counter_Name"] != counter:
            continue
        per[r["Kernel_Name"]][int(r["Dispatch_Id"])] = float(r["Counter_Value"])
    return {k: [v[d] for d in sorted(v)] for k, v in per.items()}


def _find(per: dict, needle: str):
    hits = [k for k in per if needle in k]
    if not hits:
        raise SystemExit(f"no kernel matching {needle!r} in {sorted(per)}")
    return per[hits[0]]


def traffic(fetch_dir, write_dir, workload, order, copy_mib, source=None):
    w = workloads.get(workload)
    fetch = counters(fetch_dir, "FETCH_SIZE")
    write = counters(write_dir, "WRITE_SIZE")
    copy_kib = copy_mib * 1024.0
    # The calibration copy is the largest device copy of the run (the other
    # copies are small transfers torch makes around it).
    f_copy = max(_find(fetch, "copyBuffer"))
    w_copy = max(_find(write, "copyBuffer"))
    f_scale = copy_kib / f_copy
    w_scale = copy_kib / w_copy
    kname = bench.gemm_kernel_name(order).split("<")[0]
    tmpl = bench.gemm_kernel_name(order).split("<")[1].rstrip(">")
    key = f"{kname}<{tmpl}"  # template argument as in the mangled-free name
    gf = [v for k, vs in fetch.items() if kname in k and f"<{tmpl}" in k for v in vs]
    gw = [v for k, vs in write.items() if kname in k and f"<{tmpl}" in k for v in vs]
    if not gf or not gw:
        raise SystemExit(f"no dispatches of {key} in {sorted(fetch)}")
    fb = sum(gf) / len(gf) * 1024 * f_scale
    wb = sum(gw) / len(gw) * 1024 * w_scale
    M, N, K = w.M, w.N, w.K
    alg_read = 2 * 2 * (M * K + K * N)  # four FP16 planes
    alg = alg_read + 4 * M * N
    entry = {"bytes": fb + wb, "fetch_bytes": fb, "write_bytes": wb,
             "algorithmic_bytes": alg, "fetch_scale": f_scale, "write_scale": w_scale,
             "source": source or f"profiles/hbm_traffic_{workload}_{order}.md"}
    try:
        with open(bench.TRAFFIC_FILE) as fh:
            data = json.load(fh)
    except (OSError, ValueError):
        data = {}
    h = bench.kernel_source_hash()
    if data.get("kernel_source_hash") != h:
        data = {"kernel_source_hash": h, "entries": {}}
    data["entries"][f"{workload}/{order}"] = entry
    with open(bench.TRAFFIC_FILE, "w") as fh:
        json.dump(data, fh, indent=1)
        fh.write("\n")

    def fmt(vs):
        return ", ".join(f"{v:.0f}" for v in vs)

    lines = ["| kernel | FETCH_SIZE (KiB per dispatch) | WRITE_SIZE (KiB per dispatch) |",
             "|---|---|---|"]
    for k in sorted(set(fetch) | set(write)):
        lines.append(f"| {short(k)} | {fmt(fetch.get(k, []))} | {fmt(write.get(k, []))} |")
    lines += [
        "",
        f"Calibration: the plain {copy_mib} MiB device copy reads {f_copy:.0f} KiB FETCH_SIZE "
        f"and {w_copy:.0f} KiB WRITE_SIZE for {copy_kib:.0f} KiB moved each way, so FETCH_SIZE "
        f"is scaled by {f_scale:.4f} and WRITE_SIZE by {w_scale:.4f}.",
        "",
        f"GEMM kernel per launch: fetched {fb / 1e9:.3f} GB, written {wb / 1e9:.3f} GB; "
        f"algorithmic {alg_read / 1e9:.3f} GB read (four FP16 planes) + "
        f"{4 * M * N / 1e9:.3f} GB written (C); fetch / algorithmic read = "
        f"{fb / alg_read:.1f}x.",
        "",
        f"Kernel code hash (comments excluded): {h}",
    ]
    return "\n".join(lines)


def busy(directory: str) -> str:
    act = counters(directory, "GRBM_GUI_ACTIVE")
    mfma = counters(directory, "SQ_VALU_MFMA_BUSY_CYCLES")
    durs = {}
    for r in _rows(directory, "counter_collection.csv"):
        durs.setdefault(r["Kernel_Name"], {})[int(r["Dispatch_Id"])] = (
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    lines = ["| kernel | dispatch | duration us | active cycles (per XCD) | avg clock GHz | "
             "MFMA busy |", "|---|---|---|---|---|---|"]
    for k in sorted(act):
        if "gemm" not in k or k not in mfma:
            continue
        ds = sorted(durs[k])
        for d, a, m in zip(ds, act[k], mfma[k]):
            t = durs[k][d]
            if t < 50e-6:
                continue
            cyc = a / XCDS
            lines.append(f"| {short(k)} | {d} | {t * 1e6:.1f} | {cyc:.4g} | {cyc / t / 1e9:.3f} | "
                         f"{100 * m / (cyc * SIMDS):.1f}% |")
    return "\n".join(lines)


def lds_l2(directory: str) -> str:
    """LDS bank conflicts and L2 hit rate per GEMM dispatch from a
    `--pmc SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS TCC_HIT_sum
    TCC_MISS_sum` pass."""
    conf = counters(directory, "SQ_LDS_BANK_CONFLICT")
    active = counters(directory, "SQ_LDS_IDX_ACTIVE")
    insts = counters(directory, "SQ_INSTS_LDS")
    hit = counters(directory, "TCC_HIT_sum")
    miss = counters(directory, "TCC_MISS_sum")
    lines = ["| kernel | LDS instructions | LDS bank-conflict cycles | conflict / LDS active | "
             "L2 hits | L2 misses | L2 hit rate |", "|---|---|---|---|---|---|---|"]
    for k in sorted(conf):
        if "gemm" not in k or k not in hit:
            continue
        for c, a, n, h, m in zip(conf[k], active[k], insts[k], hit[k], miss[k]):
            if n < 1e6:
                continue
            lines.append(f"| {short(k)} | {n:.4g} | {c:.4g} | {100 * c / max(a, 1):.2f}% | "
                         f"{h:.4g} | {m:.4g} | {100 * h / max(h + m, 1):.1f}% |")
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("dir")
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("--workload", default="square8192_uniform")
    b.add_argument("--order", default="elementwise")
    b.add_argument("--copy-mib", type=int, default=512)
    b.add_argument("--source", default=None,
                   help="the profiles/ summary the entry cites (default "
                        "profiles/hbm_traffic_<workload>_<order>.md)")
    c = sub.add_parser("busy")
    c.add_argument("dir")
    d = sub.add_parser("lds_l2")
    d.add_argument("dir")
    args = ap.parse_args()
    if args.cmd == "stats":
        print(stats(args.dir))
    elif args.cmd == "traffic":
        print(traffic(args.fetch_dir, args.write_dir, workloads.get(args.workload).name,
                      args.order, args.copy_mib, args.source))
    elif args.cmd == "busy":
        print(busy(args.dir))
    else:
        print(lds_l2(args.dir))


if __name__ == "__main__":
    main()
