"""Child process of tests/test_gpu_threads.py: host threads call the library
at the same time, each on its own stream, from the first call of the
process on (so the library's once-per-device set-up -- the workspace pool,
each kernel's LDS limit -- runs concurrently too).  Saves every output to
the .npz file named on the command line; the parent checks them."""
import os
import sys
import threading

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

# (M, N, K, order): each thread its own shape and order, covering the 256 x 256
# kernel with A split in the GEMM and on planes, the 256 x 128 kernels, and
# the cross-terms-first pair.
CASES = [(300, 260, 320, "elementwise"), (513, 1024, 192, "termwise"),
         (1024, 700, 256, "elementwise_cross_first"), (129, 2100, 128, "termwise"),
         (640, 4200, 96, "elementwise"), (200, 132, 4096, "termwise")]
REPS = 6
SCALE = 2048.0


def operands(i):
    import workloads

    M, N, K, _ = CASES[i]
    return workloads.make_operands(M, N, K, 100 + i, "uniform_pm1")


def main(out_path):
    import numpy as np
    import torch

    from paper_2507_23387_amd import binding

    torch.cuda.init()
    jobs = []
    for i, (M, N, K, order) in enumerate(CASES):
        A, B = operands(i)
        dA = torch.from_numpy(A).cuda()
        dB = torch.from_numpy(B).cuda()
        Cs = [torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
              for _ in range(REPS)]
        nbytes = binding.sgemm_cube_workspace_size(M, N, K, binding.ORDERS[order])
        ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device="cuda")
        jobs.append((M, N, K, binding.ORDERS[order], dA, dB, Cs, ws, nbytes, torch.cuda.Stream()))
    torch.cuda.synchronize()
    start = threading.Barrier(len(jobs))
    status = [[] for _ in jobs]

    def worker(i):
        M, N, K, order, dA, dB, Cs, ws, nbytes, stream = jobs[i]
        h = stream.cuda_stream
        start.wait()
        for r in range(REPS):
            if r % 2 == 0:
                st = binding.sgemm_cube(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                        Cs[r].data_ptr(), N, SCALE, order, h)
            else:
                st = binding.sgemm_cube_ws(M, N, K, dA.data_ptr(), K, dB.data_ptr(), N,
                                           Cs[r].data_ptr(), N, SCALE, order, ws.data_ptr(),
                                           nbytes, h)
            status[i].append(st)
        stream.synchronize()

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
        assert not t.is_alive(), "a worker thread did not finish"
    torch.cuda.synchronize()
    bad = [(i, s) for i, sts in enumerate(status) for s in sts if s != 0]
    assert len(status[0]) == REPS and not bad, f"statuses {status}"
    np.savez(out_path, **{f"c{i}_r{r}": job[6][r].cpu().numpy()
                          for i, job in enumerate(jobs) for r in range(REPS)})
    print("ok", flush=True)


if __name__ == "__main__":
    main(sys.argv[1])
