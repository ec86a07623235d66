"""bench_profile.py, which turns rocprofv3 CSV output into the summaries and
the HBM-traffic entries under profiles/: its arithmetic on small synthetic
CSV files of rocprofv3's column layout (no GPU needed)."""
import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import bench_profile  # noqa: E402

GEMM = ("void sgc::(anonymous namespace)::gemm_el_kernel<true, false>(unsigned short*, "
        "unsigned short*, unsigned short const*, unsigned short const*, unsigned int const*, int, "
        "int, int, float*, long, int, int, float, float, float const*, long, int)")
COPY = "__amd_rocclr_copyBuffer"
COLS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id",
        "Grid_Size", "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size",
        "Scratch_Size", "VGPR_Count", "Accum_VGPR_Count", "SGPR_Count", "Counter_Name",
        "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(directory, rows):
    """rows: (dispatch, kernel, counter, value, duration_ns)."""
    os.makedirs(directory, exist_ok=True)
    with open(os.path.join(directory, "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f, quoting=csv.QUOTE_NONNUMERIC)
        w.writerow(COLS)
        for d, k, c, v, ns in rows:
            start = 10**9 + 10**7 * d
            w.writerow([d, d, "Agent 1", 1, 1, 1, 1, 1, k, 256, 0, 0, 0, 0, 0, c, float(v), start,
                        start + ns])


def test_busy_gives_clock_and_mfma_fraction(tmp_path):
    d = str(tmp_path / "busy")
    cyc = 1.0e6  # per XCD
    _write(d, [(3, GEMM, "GRBM_GUI_ACTIVE", 8 * cyc, 500_000),
               (3, GEMM, "SQ_VALU_MFMA_BUSY_CYCLES", 0.5 * cyc * 1024, 500_000),
               (3, GEMM, "SQ_BUSY_CYCLES", 1.0, 500_000),
               (4, GEMM, "GRBM_GUI_ACTIVE", 8 * cyc, 20_000),  # under 50 us: skipped
               (4, GEMM, "SQ_VALU_MFMA_BUSY_CYCLES", 1.0, 20_000)])
    out = bench_profile.busy(d).splitlines()
    assert len(out) == 3
    assert out[2] == "| gemm_el_kernel<true, false> | 3 | 500.0 | 1e+06 | 2.000 | 50.0% |"


def test_lds_l2_gives_conflicts_and_hit_rate(tmp_path):
    d = str(tmp_path / "lds")
    _write(d, [(2, GEMM, "SQ_LDS_BANK_CONFLICT", 250.0, 10**6),
               (2, GEMM, "SQ_LDS_IDX_ACTIVE", 1000.0, 10**6),
               (2, GEMM, "SQ_INSTS_LDS", 2.0e6, 10**6),
               (2, GEMM, "TCC_HIT_sum", 800.0, 10**6),
               (2, GEMM, "TCC_MISS_sum", 200.0, 10**6)])
    out = bench_profile.lds_l2(d).splitlines()
    assert out[2] == "| gemm_el_kernel<true, false> | 2e+06 | 250 | 25.00% | 800 | 200 | 80.0% |"


def test_traffic_scales_by_the_calibration_copy_and_writes_the_entry(tmp_path, monkeypatch):
    traffic_file = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(traffic_file))
    copy_mib = 512
    copy_kib = copy_mib * 1024.0
    fd, wd = str(tmp_path / "fetch"), str(tmp_path / "write")
    # The copy's FETCH_SIZE reads half the bytes moved, WRITE_SIZE all of them.
    _write(fd, [(1, COPY, "FETCH_SIZE", copy_kib / 2, 10**5), (2, COPY, "FETCH_SIZE", 4.0, 10),
                (5, GEMM, "FETCH_SIZE", 1.0e6, 10**6), (6, GEMM, "FETCH_SIZE", 3.0e6, 10**6)])
    _write(wd, [(1, COPY, "WRITE_SIZE", copy_kib, 10**5),
                (5, GEMM, "WRITE_SIZE", 2.0e5, 10**6), (6, GEMM, "WRITE_SIZE", 2.0e5, 10**6)])
    text = bench_profile.traffic(fd, wd, "square8192_uniform", "elementwise_unfused", copy_mib,
                                 source="profiles/x.md")
    data = json.loads(traffic_file.read_text())
    assert data["kernel_source_hash"] == bench.kernel_source_hash()
    e = data["entries"]["square8192_uniform/elementwise_unfused"]
    assert e["fetch_scale"] == pytest.approx(2.0) and e["write_scale"] == pytest.approx(1.0)
    assert e["fetch_bytes"] == pytest.approx(2.0e6 * 1024 * 2.0)   # mean KiB x 1024 x scale
    assert e["write_bytes"] == pytest.approx(2.0e5 * 1024)
    assert e["bytes"] == pytest.approx(e["fetch_bytes"] + e["write_bytes"])
    n = 8192
    assert e["algorithmic_bytes"] == 4 * n * n * 2 + 4 * n * n
    assert e["source"] == "profiles/x.md"
    assert "scaled by 2.0000" in text
    # The entry is what bench.py reports for that workload and kernel.
    assert bench.traffic_entry("square8192_uniform", "elementwise_unfused") == e
