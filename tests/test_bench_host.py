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
    for key, e in data["entries"].items():
        assert e["bytes"] == pytest.approx(e["fetch_bytes"] + e["write_bytes"]), key
        assert os.path.exists(os.path.join(ROOT, e["source"])), (key, e["source"])
    # The default bench line's kernel at 8192^3 (A split in a pass of its own):
    # four FP16 planes of 8192 x 8192 read, C written once in FP32.
    e = data["entries"]["square8192_uniform/elementwise_unfused"]
    assert e["algorithmic_bytes"] == 4 * 8192 * 8192 * 2 + 8192 * 8192 * 4


def test_parity_report_passes_within_the_bar_and_fails_outside():
    import numpy as np

    rng = np.random.default_rng(1)
    A = rng.uniform(-1, 1, (6, 50)).astype(np.float32)
    B = rng.uniform(-1, 1, (50, 7)).astype(np.float32)
    rows = np.array([1, 4])
    ref = (A[rows].astype(np.float64) @ B.astype(np.float64)).astype(np.float32)
    absab = np.abs(A[rows].astype(np.float64)) @ np.abs(B.astype(np.float64))
    tol = 2 * 50 * 2.0**-24 * absab
    r = bench.parity_report(ref, ref, A, B, rows, 50)
    assert r["verdict"] == "pass" and r["worst_err_over_tol"] == 0 and r["entries"] == 14
    near = (ref.astype(np.float64) + 0.5 * tol).astype(np.float32)
    assert bench.parity_report(near, ref, A, B, rows, 50)["verdict"] == "pass"
    far = (ref.astype(np.float64) + 3.0 * tol).astype(np.float32)
    r = bench.parity_report(far, ref, A, B, rows, 50)
    assert r["verdict"] == "fail" and r["worst_err_over_tol"] > 2
    nan = ref.copy()
    nan[0, 0] = np.nan
    assert bench.parity_report(nan, ref, A, B, rows, 50)["verdict"] == "fail"


def test_hi_only_gap():
    import numpy as np

    o = np.array([[1.0, 2.0]], np.float32)
    h = np.array([[1.5, 2.0]], np.float32)
    assert bench.hi_only_gap(o, o, h) == 0.0
    assert bench.hi_only_gap(o + np.float32(0.25), o, h) == 0.5
    assert bench.hi_only_gap(o, o, o) is None


def test_tile_keys_name_the_sweep_kernels():
    from paper_2507_23387_amd import binding

    names = set()
    for tile in binding.TILE_CONFIGS:
        key = "elementwise_tile_" + bench.tile_name(tile)
        name = bench.gemm_kernel_name(key)
        assert name.startswith(f"gemm_tile_kernel<{tile[0]}, {tile[1]}, {tile[2]}, ")
        names.add(name)
    assert len(names) == len(binding.TILE_CONFIGS)
    # Four-wave keys keep the three-field form the committed profiles use.
    assert bench.tile_name((256, 256, 32, 4)) == "256x256x32"
    assert bench.gemm_kernel_name("elementwise_tile_256x256x32") == \
        "gemm_tile_kernel<256, 256, 32, 1, 2, 2>"
    assert bench.gemm_kernel_name("elementwise_tile_128x128x32") == \
        "gemm_tile_kernel<128, 128, 32, 2, 2, 2>"
    assert bench.tile_name((256, 256, 32, 8)) == "256x256x32x8"
    assert bench.gemm_kernel_name("elementwise_tile_256x256x32x8") == \
        "gemm_tile_kernel<256, 256, 32, 1, 2, 4>"


def _mangled_prefix(name: str) -> bytes:
    """Itanium-mangled form of 'kernel<args>' as it appears in the library's
    kernel symbols: each int argument Li<n>E, each bool Lb<0|1>E."""
    kernel, args = name.split("<", 1)
    out = kernel + "I"
    for a in args.rstrip(">").split(","):
        a = a.strip()
        out += {"true": "Lb1E", "false": "Lb0E"}.get(a, f"Li{a}E")
    return (out + "E").encode()


def test_roofline_kernel_names_are_kernels_of_the_library():
    """Every kernel name bench.py reports (and keys the committed traffic
    entries by) names a kernel the built library contains, so the rocprofv3
    summaries and the roofline line refer to the code that runs."""
    from paper_2507_23387_amd import binding

    data = open(binding.LIB_PATH, "rb").read()
    names = set(bench.GEMM_KERNELS.values())
    names |= {bench.gemm_kernel_name("elementwise_tile_" + bench.tile_name(t))
              for t in binding.TILE_CONFIGS}
    for name in sorted(names):
        assert _mangled_prefix(name) in data, name
    assert _mangled_prefix("gemm_n128_kernel<5, false, false>") not in data


def test_error_report_on_a_hand_computed_case():
    import numpy as np

    # A = [[1, 2], [3, -4]], B = I: ref = A; C off by +0.5 in one entry, and a
    # zero reference entry (excluded from the relative error).
    A = np.array([[1.0, 2.0], [3.0, -4.0], [0.0, 0.0]], np.float32)
    B = np.eye(2, dtype=np.float32)
    rows = np.array([0, 1, 2])
    C = A.copy()
    C[1, 1] = -3.5
    r = bench.error_report(C, A, B, rows)
    assert r["max_rel_err"] == 0.5 / 4.0
    assert r["max_err_over_absAabsB"] == 0.5 / 4.0
    assert r["frobenius_rel_err"] == pytest.approx(0.5 / np.sqrt(1 + 4 + 9 + 16))
