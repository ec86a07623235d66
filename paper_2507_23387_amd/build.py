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
    "gemm_fused.hip": _MINREG,
}

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


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile every source to an object (with its FILE_FLAGS) and link them."""
    incs = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    objs = []
    for src in sources():
        name = os.path.basename(src)
        obj = os.path.join(objdir, name + ".o")
        _run([HIPCC, *compile_flags, *FILE_FLAGS.get(name, []), *extra_flags, *incs, "-c", src,
              "-o", obj], verbose)
        objs.append(obj)
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", LIB + ".tmp"], verbose)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
