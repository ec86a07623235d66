// Launcher of the diagnostic register-only MFMA loop (ceiling.hip), used by
// the C-ABI layer.  Not installed; the public interface is
// include/sgemm_cube.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sgc {

// Enqueue the loop on `workgroups` workgroups of 256 threads, `iters`
// iterations of 64 MFMAs per wave; the 64 KiB at `operands` are read, out
// receives workgroups x 256 floats.  Arguments already validated.
hipError_t launch_mfma_loop(int64_t workgroups, int64_t iters, const uint16_t* operands,
                            float* out, hipStream_t stream);

}  // namespace sgc
