"""The boundary is a C ABI: a plain C11 program (tests/c_abi/use_from_c.c)
includes include/sgemm_cube.h, links against the built libsgemmcube.so and
runs the calls that need no GPU (queries, argument validation)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2507_23387_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_header_and_library_work_from_c(tmp_path):
    assert os.path.exists(os.path.join(LIBDIR, "libsgemmcube.so")), "build the library first"
    exe = tmp_path / "use_from_c"
    cmd = ["gcc", "-std=c11", "-Wall", "-Werror=implicit-function-declaration",
           "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
           "-D__HIP_PLATFORM_AMD__", os.path.join(ROOT, "tests", "c_abi", "use_from_c.c"),
           "-L", LIBDIR, "-lsgemmcube", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, LD_LIBRARY_PATH=LIBDIR + os.pathsep + os.environ.get("LD_LIBRARY_PATH", ""))
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120, env=env)
    assert r.returncode == 0, (r.stdout, r.stderr[-3000:])
    assert r.stdout.strip() == "0"
