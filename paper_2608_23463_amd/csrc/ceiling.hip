// Measured ceilings (measurement aids, not on the layer's path):
// - matrix cores: every wave issues a long run of independent bf16 MFMAs with
//   no memory traffic, so the achieved rate is what the kernels' main loops
//   could reach at best on this device, next to the vendor's dense bf16 peak;
// - HBM reads: a grid-strided stream of 16-byte loads with nothing else to
//   do, the rate a read-bound kernel (the decode attention) can reach at best,
//   next to the vendor's HBM figure.
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

constexpr int kReadInFlight = 4;  // 16-byte loads in flight per lane

__global__ void __launch_bounds__(256) read_ceiling_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                           unsigned* __restrict__ out) {
  unsigned acc = 0;
  const int64_t stride = (int64_t)gridDim.x * 256 * kReadInFlight;
  for (int64_t i = (int64_t)blockIdx.x * 256 * kReadInFlight + threadIdx.x; i < n16; i += stride) {
    u32x4 v[kReadInFlight];
#pragma unroll
    for (int u = 0; u < kReadInFlight; ++u) {
      const int64_t j = i + (int64_t)u * 256;
      v[u] = j < n16 ? src[j] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kReadInFlight; ++u) acc ^= v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc ^= (unsigned)__shfl_xor((int)acc, off);
  __shared__ unsigned part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) out[blockIdx.x] = part[0] ^ part[1] ^ part[2] ^ part[3];
}

hipError_t launch_read_ceiling(const void* src, size_t bytes, unsigned* out, int64_t n_workgroups,
                               hipStream_t stream) {
  hipLaunchKernelGGL(read_ceiling_kernel, dim3((unsigned)n_workgroups), dim3(256), 0, stream,
                     static_cast<const u32x4*>(src), (int64_t)(bytes / 16), out);
  return hipGetLastError();
}

}  // namespace pf

