"""FP32-accuracy GEMM from three FP16 MFMA products on MI355X (gfx950).

Implements the SGEMM-cube method of arXiv 2507.23387: FP32 operands split into
an FP16 high word and a scaled FP16 residual (Sec. 3.3), the product rebuilt
from three FP16 GEMMs with FP32 accumulation (Eq. recover_eqn), in the
elementwise, termwise or cross-terms-first order (Sec. 4.5), with optional
power-of-two pre-scaling and a range report (sgemm_cube_ex).  All computation
happens in the HIP kernels of ``libsgemmcube.so``; ``binding`` is the ctypes
layer over its C-ABI (include/sgemm_cube.h).

The names below resolve on first use, so that ``paper_2507_23387_amd.build``
(which compiles the library) imports on a checkout where the library is not
built yet.  Using any of them without the built library raises ImportError:
there is no fallback.
"""
_EXPORTS = (
    "ELEMENTWISE",
    "TERMWISE",
    "ELEMENTWISE_CROSS_FIRST",
    "SgemmCubeError",
    "hgemm",
    "matmul",
    "matmul_ex",
    "sgemm_cube",
    "sgemm_cube_block_k",
    "sgemm_cube_compute",
    "sgemm_cube_compute_a",
    "sgemm_cube_compute_b",
    "sgemm_cube_compute_stages",
    "sgemm_cube_compute_tile",
    "sgemm_cube_ex",
    "sgemm_cube_ex_workspace_size",
    "sgemm_cube_hgemm",
    "sgemm_cube_noalloc",
    "sgemm_cube_prepare",
    "sgemm_cube_split",
    "sgemm_cube_splits_a_in_gemm",
    "sgemm_cube_status_string",
    "sgemm_cube_workspace_size",
    "sgemm_cube_ws",
    "split",
    "workspace",
)

__all__ = list(_EXPORTS)


def __getattr__(name):
    if name in _EXPORTS or name == "binding":
        import importlib

        # Raises ImportError if libsgemmcube.so is missing.
        binding = importlib.import_module(__name__ + ".binding")
        return binding if name == "binding" else getattr(binding, name)
    raise AttributeError(f"module {__name__!r} has no attribute {name!r}")
