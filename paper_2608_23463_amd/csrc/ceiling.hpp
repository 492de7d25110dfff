// Matrix-core and HBM-read ceiling probes (measurement aids, not on the layer's path).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pf {

// Enqueues n_workgroups workgroups of four waves; each wave runs iters x 8
// independent bf16 MFMAs (32x32x16) on register operands and writes one float
// per thread to out[n_workgroups * 256].
hipError_t launch_mfma_ceiling(float* out, int64_t n_workgroups, int iters, hipStream_t stream);

// Enqueues n_workgroups workgroups of four waves that read bytes (a multiple
// of 16) of src with grid-strided 16-byte loads; workgroup w writes the XOR of
// every 32-bit word it read to out[w].
hipError_t launch_read_ceiling(const void* src, size_t bytes, unsigned* out, int64_t n_workgroups,
                               hipStream_t stream);

}  // namespace pf
