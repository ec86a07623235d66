"""Host AddressSanitizer + UndefinedBehaviorSanitizer runs (no GPU needed).

- The oracle (oracle/oracle.c) with tests/sanitize/oracle_check.c, built by
  gcc with -fsanitize=address,undefined: conversions over a strided walk of
  all 2^32 patterns and every FP16 pattern, the split with padded leading
  dimensions, every order of the GEMM on ragged shapes with one and several
  OpenMP threads, K = 0, empty shapes and argument errors.
- The C-ABI's host code (validation, workspace carving, queries) through
  tests/sanitize/abi_check.cpp, linked with the library's sources built with
  the sanitizers on their host pass (paper_2507_23387_amd.build.build_sanitized),
  in its "cpu" mode: every call returns before device work.  The "gpu" mode of
  the same program runs in tests/test_gpu_sanitizers.py.

Both programs are built into a temporary directory from the current sources."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    proc = subprocess.run(cmd, capture_output=True, text=True, env=ENV, **kw)
    assert proc.returncode == 0, (cmd, proc.stdout[-2000:], proc.stderr[-4000:])
    return proc.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_check")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fno-fast-math", "-ffp-contract=off",
          "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
          "-static-libasan", os.path.join(SAN, "oracle_check.c"),
          os.path.join(ROOT, "oracle", "oracle.c"), "-o", exe, "-lm"])
    for threads in ("1", "4"):
        out = subprocess.run([exe], capture_output=True, text=True,
                             env=dict(ENV, OMP_NUM_THREADS=threads), timeout=300)
        assert out.returncode == 0, out.stderr[-4000:]
        assert "all checks passed" in out.stdout


def test_abi_host_code_under_asan_ubsan(tmp_path):
    from paper_2507_23387_amd import build as hip_build

    exe = hip_build.build_sanitized(out_dir=str(tmp_path))
    out = _run([exe, "cpu"], timeout=120)
    assert "abi_check cpu: all checks passed" in out
