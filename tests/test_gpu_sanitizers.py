"""The C-ABI's host code under the host AddressSanitizer and
UndefinedBehaviorSanitizer with real device work: tests/sanitize/abi_check.cpp
in its "gpu" mode drives every entry point (all orders, the pool-allocating,
caller-workspace and fixed-workspace calls, prepare/compute, compute_a,
compute_stages, the pre-scaled call with its range report, the split and
the FP16 baseline) on ragged and padded shapes, on the null stream and on a
created stream, and checks each C against an FP64 GEMM within
4 K 2^-24 (|A||B|)_ij.  The program is built by __graft_entry__.build()
(paper_2507_23387_amd.build.build_sanitized) beforehand."""
import os
import subprocess

import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "sanitize", "abi_check")


def test_every_entry_point_under_host_sanitizers(gpu):
    assert os.path.exists(EXE), f"{EXE} is not built: run __graft_entry__.build()"
    log("abi_check gpu under ASan/UBSan")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:protect_shadow_gap=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    proc = subprocess.run([EXE, "gpu"], capture_output=True, text=True, env=env, timeout=100)
    assert proc.returncode == 0, proc.stderr[-4000:]
    assert "abi_check gpu: all checks passed" in proc.stdout
