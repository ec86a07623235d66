"""Host logic of bench.py (no GPU needed): the one-GPU guard, the comment-blind
hash that ties a committed HBM-traffic measurement to the kernel code, and the
rule that the traffic figure is withheld once that code has changed."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""  # no JSON line for a run that did not happen


def test_code_only_ignores_comments_and_layout():
    a = """
    // a line comment
    int f(int x) {  /* block
       comment */ return x + 1; }
    """
    b = "int f(int x){return x+1;}"
    c = "int f(int x) { return x + 2; }"
    assert bench._code_only(a) == bench._code_only("int f(int x) { return x + 1; }")
    # Whitespace between tokens is collapsed, not removed: the two spellings
    # differ, which only makes the hash stricter.
    assert bench._code_only(a) != bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(c)


def test_code_only_keeps_string_literals_verbatim():
    # Inline asm lives in string literals: a comment marker inside one is code.
    src = 'asm volatile("s_waitcnt vmcnt(0) // not a comment");  // a comment'
    out = bench._code_only(src)
    assert '"s_waitcnt vmcnt(0) // not a comment"' in out
    assert "a comment" not in out.replace("not a comment", "")
    assert bench._code_only('x = "a\\"b"; // c') == 'x = "a\\"b";'


def test_kernel_source_hash_is_stable():
    h = bench.kernel_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
    assert bench.kernel_source_hash() == h


@pytest.fixture()
def traffic_file(tmp_path, monkeypatch):
    path = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(path))
    return path


def test_traffic_entry_requires_the_current_kernel_hash(traffic_file):
    entry = {"bytes": 1.0, "fetch_bytes": 0.5, "write_bytes": 0.5}
    data = {"kernel_source_hash": bench.kernel_source_hash(),
            "entries": {"square8192_uniform/elementwise": entry}}
    traffic_file.write_text(json.dumps(data))
    assert bench.traffic_entry("square8192_uniform", "elementwise") == entry
    assert bench.traffic_entry("square8192_uniform", "termwise") is None

    data["kernel_source_hash"] = "0" * 16  # measured on other kernel code
    traffic_file.write_text(json.dumps(data))
    assert bench.traffic_entry("square8192_uniform", "elementwise") is None


def test_traffic_entry_missing_or_malformed_file(traffic_file):
    assert bench.traffic_entry("square8192_uniform", "elementwise") is None
    traffic_file.write_text("{not json")
    assert bench.traffic_entry("square8192_uniform", "elementwise") is None


def test_committed_traffic_file_is_consistent():
    # Whether its hash matches the current kernels decides only whether the
    # bench line reports it; its figures must add up either way.
    with open(os.path.join(ROOT, "profiles", "gemm_traffic.json")) as f:
        data = json.load(f)
    assert len(data["kernel_source_hash"]) == 16
    e = data["entries"]["square8192_uniform/elementwise"]
    assert e["bytes"] == pytest.approx(e["fetch_bytes"] + e["write_bytes"])
    # Four FP16 planes of 8192 x 8192 read, C written once in FP32.
    assert e["algorithmic_bytes"] == 4 * 8192 * 8192 * 2 + 8192 * 8192 * 4
