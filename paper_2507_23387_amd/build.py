"""Build libsgemmcube.so (all HIP kernels + the C-ABI) for gfx950, in-tree.

    python -m paper_2507_23387_amd.build [-v]

hipcc cross-compiles without a GPU.  Flags:
  --offload-arch=gfx950            CDNA4 only, no other targets
  -O3 -std=c++17 -fPIC -shared
  -Xclang -target-feature -Xclang -packed-fp32-ops
                                   no packed-FP32 VALU instructions (the host
                                   pass warns that it does not know the
                                   feature; that is harmless)
No fast-math and no denormal flushing: the split relies on IEEE RN-even
conversion with FP16 and FP32 denormals kept.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libsgemmcube.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    "-fvisibility=hidden",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


# Extra flags per source file.  The GEMM kernels: the "iterative-minreg"
# machine scheduler keeps the 256 accumulators of the 256 x 256 kernels in
# place (the default strategy shuffles them between AGPRs and VGPRs inside the
# main loop, which more than doubles the kernel's time).
_MINREG = ["-mllvm", "-amdgpu-sched-strategy=iterative-minreg"]
FILE_FLAGS = {
    "gemm.hip": _MINREG,
    "gemm_tile.hip": _MINREG,
}

# Host AddressSanitizer + UndefinedBehaviorSanitizer for the checking build
# (build_sanitized): on the host pass only, each flag behind -Xarch_host; the
# device code is compiled exactly as in the library.
SANITIZE_HOST = [
    "-Xarch_host", "-fsanitize=address",
    "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=all",
    "-Xarch_host", "-fno-omit-frame-pointer",
    "-Xarch_host", "-g",
]
SANITIZE_DIR = os.path.join(ROOT, "tests", "sanitize")

_NOISE = "is not a recognized feature for this target"


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    errlines = [l for l in proc.stderr.splitlines() if _NOISE not in l]
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(errlines))
    if verbose and errlines:
        print("\n".join(errlines))


def _compile_all(jobs, verbose):
    """Run the compile commands concurrently (one hipcc process each)."""
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 8))
    with ThreadPoolExecutor(max_workers=workers) as pool:
        for f in [pool.submit(_run, cmd, verbose) for cmd in jobs]:
            f.result()


def _includes():
    return ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile every source to an object (with its FILE_FLAGS) and link them."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    jobs, objs = [], []
    for src in sources():
        name = os.path.basename(src)
        obj = os.path.join(objdir, name + ".o")
        jobs.append([HIPCC, *compile_flags, *FILE_FLAGS.get(name, []), *extra_flags, *_includes(),
                     "-c", src, "-o", obj])
        objs.append(obj)
    _compile_all(jobs, verbose)
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", LIB + ".tmp"], verbose)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def build_sanitized(out_dir: str | None = None, verbose: bool = False) -> str:
    """Build tests/sanitize/abi_check: the library's sources with SANITIZE_HOST
    on their host pass, linked statically into the program that drives every
    entry point.  The device code is the library's (same flags, same gfx950
    kernels).  Returns the path of the executable."""
    default_dir = os.path.join(SANITIZE_DIR, "_build")
    out_dir = out_dir or default_dir
    os.makedirs(out_dir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f not in ("-shared", "-fvisibility=hidden")]
    jobs, objs = [], []
    for src in [*sources(), os.path.join(SANITIZE_DIR, "abi_check.cpp")]:
        name = os.path.basename(src)
        obj = os.path.join(out_dir, name + ".o")
        lang = ["-x", "hip"] if name.endswith(".cpp") else []
        jobs.append([HIPCC, *compile_flags, *FILE_FLAGS.get(name, []), *SANITIZE_HOST,
                     *_includes(), *lang, "-c", src, "-o", obj])
        objs.append(obj)
    _compile_all(jobs, verbose)
    # The objects stay in out_dir; the default executable goes beside its
    # source (build folders do not travel with the tree).
    exe = os.path.join(SANITIZE_DIR if out_dir == default_dir else out_dir, "abi_check")
    _run([HIPCC, "--offload-arch=gfx950", *SANITIZE_HOST, *objs, "-o", exe + ".tmp"], verbose)
    os.replace(exe + ".tmp", exe)
    return exe


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
