// Measured ceiling of the matrix cores (measurement aid, not on the layer's
// path): every wave issues a long run of independent bf16 MFMAs with no
// memory traffic, so the achieved rate is what the kernels' main loops could
// reach at best on this device, next to the vendor's dense bf16 peak.
#include <hip/hip_runtime.h>

#include "ceiling.hpp"
#include "common.hpp"

namespace pf {

constexpr int kCeilChains = 8;  // independent accumulators per wave

__global__ void __launch_bounds__(256) mfma_ceiling_kernel(float* __restrict__ out, int iters) {
  const int lane = threadIdx.x & 63;
  bf16x8 a, b;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    a[e] = (bf16)(0.001f * (float)((lane + e) & 7));
    b[e] = (bf16)(0.002f * (float)((lane * 3 + e) & 7));
  }
  f32x16 acc[kCeilChains];
#pragma unroll
  for (int c = 0; c < kCeilChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[c][r] = 0.0f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kCeilChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < kCeilChains; ++c)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[c][r];
  out[(size_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
}

hipError_t launch_mfma_ceiling(float* out, int64_t n_workgroups, int iters, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_ceiling_kernel, dim3((unsigned)n_workgroups), dim3(256), 0, stream, out, iters);
  return hipGetLastError();
}

}  // namespace pf

