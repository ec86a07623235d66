"""SGEMM_CUBE_ERR_ALLOC: sgemm_cube takes its workspace from a library-owned
stream-ordered pool; when device memory cannot hold it the call returns
SGEMM_CUBE_ERR_ALLOC before any device work, leaves C untouched and leaves no
error behind, so the next call on the same thread works.

The operands are real device buffers (so a call that wrongly went ahead would
only compute, never touch memory it does not own); device memory is then
filled with torch allocations until less than half of the workspace is free."""
import pytest

from tests.gpu_util import log

pytestmark = pytest.mark.gpu

GIB = 1 << 30


def _fill_device_memory(torch, keep_free):
    """Allocate blocks until the device has less than keep_free bytes free."""
    held = []
    chunk = 32 * GIB
    while chunk >= 64 << 20:
        free, _ = torch.cuda.mem_get_info()
        if free < keep_free:
            break
        size = min(chunk, free - keep_free // 2)
        try:
            held.append(torch.empty(size, dtype=torch.uint8, device="cuda"))
        except torch.OutOfMemoryError:
            chunk //= 2
    return held


def test_exhausted_device_memory_gives_err_alloc(gpu):
    import torch

    from paper_2507_23387_amd import binding

    M = N = K = 16384
    need = binding.sgemm_cube_workspace_size(M, N, K)
    assert need >= 2 * GIB
    A = torch.zeros((M, K), dtype=torch.float32, device="cuda")
    B = torch.zeros((K, N), dtype=torch.float32, device="cuda")
    C = torch.full((M, N), 7.0, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    torch.cuda.synchronize()
    log(f"filling device memory below {need // 2} bytes free")
    held = _fill_device_memory(torch, need // 2)
    try:
        free, total = torch.cuda.mem_get_info()
        log(f"free {free} of {total} bytes, workspace {need}")
        assert free < need
        st = binding.sgemm_cube(M, N, K, A.data_ptr(), K, B.data_ptr(), N, C.data_ptr(), N,
                                2048.0, binding.ELEMENTWISE, stream)
        torch.cuda.synchronize()
        assert binding.sgemm_cube_status_string(st) == "SGEMM_CUBE_ERR_ALLOC"
        assert bool((C[::1024, ::1024] == 7.0).all())       # C untouched
    finally:
        del held
        torch.cuda.empty_cache()
    # The library works again, and the failed allocation left no error for the
    # launch checks of this call to pick up.
    m, n, k = 300, 200, 128
    a = torch.randn((m, k), device="cuda")
    b = torch.randn((k, n), device="cuda")
    c1 = torch.full((m, n), float("nan"), device="cuda")
    assert binding.sgemm_cube(m, n, k, a.data_ptr(), k, b.data_ptr(), n, c1.data_ptr(), n,
                              2048.0, binding.ELEMENTWISE, stream) == 0
    ws = binding.workspace(m, n, k)
    c2 = torch.full((m, n), float("nan"), device="cuda")
    assert binding.sgemm_cube_ws(m, n, k, a.data_ptr(), k, b.data_ptr(), n, c2.data_ptr(), n,
                                 2048.0, binding.ELEMENTWISE, ws.data_ptr(), ws.numel(),
                                 stream) == 0
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
