"""bench.py end to end on the GPU, in a child process: it prints exactly one
JSON line with the fields the benchmark contract names (metric, value, unit,
steps, warm-up, ms per step, the roofline object of the dominant kernel, the
CPU-oracle baseline, the parity verdict), and the figures agree with each
other.  The 256^3 workload keeps the run short."""
import json
import os
import subprocess
import sys

import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_prints_one_consistent_json_line(gpu):
    log("bench.py --workload c1 in a child process")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "c1",
                        "--steps", "3", "--warmup", "1", "--cpu-seconds", "1",
                        "--copy-mib", "64"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-4000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    cfg = d["config"]
    assert cfg["workload"] == "square256_uniform" and (cfg["M"], cfg["N"], cfg["K"]) == (256,) * 3
    assert d["unit"] == "TFLOP/s" and d["n_gpus"] == 1 and d["data"] == "synthetic"
    assert (d["steps"], d["warmup"]) == (3, 1)
    assert d["higher_is_better"] is True and d["scaling"] == "weak" and d["vs_baseline"] is None
    # value = 2 M N K / (ms per step)
    assert d["ms_per_step"] > 0
    assert d["value"] == pytest.approx(2 * 256**3 / (d["ms_per_step"] * 1e-3) / 1e12, rel=1e-6)
    roof = d["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s"
    assert roof["peak"] == pytest.approx(256 * 2.4e9 * 4096 / 1e12)
    assert roof["achieved"] > 0 and roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"])
    # 6 M N K FP16 MFMA flops per launch over the kernel's event-timed average
    assert roof["achieved"] == pytest.approx(6 * 256**3 / (roof["avg_launch_ms"] * 1e-3) / 1e12,
                                             rel=1e-6)
    assert roof["traffic"] is None or {"bytes", "fetch_bytes", "write_bytes"} <= set(roof["traffic"])
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "TFLOP/s" and cpu["value"] > 0
    assert cpu["cores"] >= 1 and isinstance(cpu["sample"], str)
    assert d["parity"]["verdict"] == "pass"
