"""Concurrent host threads, each on its own stream, calling sgemm_cube and
sgemm_cube_ws from the first call of a fresh process (tests/threads_child.py):
every output must equal, bit for bit, the same call made alone, and that
result meets the parity bar against the oracle.  The header states that the
entry points are thread-safe; the library's only shared state is set up once
per device (the workspace pool, the kernels' LDS limits) and the range-flag
stamp counter."""
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from tests import threads_child as child
from tests.gpu_util import log
from tests.helpers import abs_ab, assert_parity

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_concurrent_threads_match_the_call_made_alone(gpu, tmp_path):
    import torch

    from paper_2507_23387_amd import binding

    out = tmp_path / "threads.npz"
    log(f"{len(child.CASES)} host threads x {child.REPS} calls in a child process")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "threads_child.py"),
                        str(out)], capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert r.stdout.strip().endswith("ok")
    got = np.load(out)
    kb = binding.sgemm_cube_block_k()
    for i, (M, N, K, order) in enumerate(child.CASES):
        A, B = child.operands(i)
        log(f"thread case {i}: {M}x{N}x{K} {order}")
        C = binding.matmul(torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda(),
                           scale=child.SCALE, order=order)
        torch.cuda.synchronize()
        ref = C.cpu().numpy()
        assert np.isfinite(ref).all()
        for rep in range(child.REPS):
            c = got[f"c{i}_r{rep}"]
            assert np.array_equal(c.view(np.uint32), ref.view(np.uint32)), (i, rep)
        Co = oracle.sgemm(A, B, child.SCALE, order, kb=kb)
        assert_parity(ref, Co, K, abs_ab(A, B), f"thread case {i}")
