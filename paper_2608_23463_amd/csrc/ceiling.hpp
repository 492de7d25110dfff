// Matrix-core ceiling probe (measurement aid, not on the layer's path).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pf {

// Enqueues n_workgroups workgroups of four waves; each wave runs iters x 8
// independent bf16 MFMAs (32x32x16) on register operands and writes one float
// per thread to out[n_workgroups * 256].
hipError_t launch_mfma_ceiling(float* out, int64_t n_workgroups, int iters, hipStream_t stream);

}  // namespace pf
