"""Helpers for the GPU tests: move numpy operands to the device, call the
library through its C-ABI binding, bring results back."""
from __future__ import annotations

import sys

import numpy as np


def log(msg: str):
    """Name the case before a GPU step, flushed, so a crash still says where."""
    print(f"[gpu-test] {msg}", file=sys.stderr, flush=True)


def to_dev(x: np.ndarray, device="cuda"):
    import torch

    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def padded(x: np.ndarray, ld: int, device="cuda", offset: int = 0):
    """Device copy of a row-major matrix stored with leading dimension ld,
    starting `offset` elements into its allocation (misaligns the base)."""
    import torch

    rows, cols = x.shape
    buf = torch.full((offset + max(rows, 1) * ld,), float("nan"), dtype=torch.float32,
                     device=device)
    view = buf[offset:offset + rows * ld].view(rows, ld) if rows else buf[:0].view(0, ld)
    view[:, :cols].copy_(torch.from_numpy(np.ascontiguousarray(x)))
    return buf, view


def gemm(A: np.ndarray, B: np.ndarray, scale: float, order: str):
    """Run sgemm_cube on contiguous copies of A, B; return C as numpy."""
    import torch

    from paper_2507_23387_amd import binding

    C = binding.matmul(to_dev(A), to_dev(B), scale=scale, order=order)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def hgemm(A: np.ndarray, B: np.ndarray):
    import torch

    from paper_2507_23387_amd import binding

    C = binding.hgemm(to_dev(A), to_dev(B))
    torch.cuda.synchronize()
    return C.cpu().numpy()


def split(X: np.ndarray, scale: float):
    import torch

    from paper_2507_23387_amd import binding

    hi, lo = binding.split(to_dev(X.astype(np.float32)), scale)
    torch.cuda.synchronize()
    return hi.cpu().numpy().view(np.uint16), lo.cpu().numpy().view(np.uint16)
