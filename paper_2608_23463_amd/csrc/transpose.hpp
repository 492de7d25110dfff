// out[c, r] = in[r, c] through 64x64 LDS tiles (shared by the backward's
// operand transposes and the fp32 prefill's transposed cache values).
#pragma once

#include "common.hpp"

namespace pf {

// out[c, r] = in[r, c] for r < R, c < C (row strides ld_in, ld_out), through
// 64x64 LDS tiles: 16-byte coalesced reads along c, 16-byte writes along r.
// With `part`, the tile also leaves the column sums of its 64 rows in
// part[blockIdx.y][c] (fixed order: a thread's 16-byte run, then a butterfly
// over the runs of one column), the first stage of a bias gradient.
// blockIdx.z selects a batch entry: in/out advance by in_bs/out_bs elements.
// With R_out > R the output columns R .. R_out-1 are written as zeros (the
// grid then covers R_out rows).
template <typename T>
__global__ void __launch_bounds__(256) transpose_kernel(const T* __restrict__ in, int64_t ld_in, int64_t R, int C,
                                                        T* __restrict__ out, int64_t ld_out, float* __restrict__ part,
                                                        int64_t in_bs = 0, int64_t out_bs = 0, int64_t R_out = 0) {
  constexpr int kV = 16 / sizeof(T);
  constexpr int kRuns = 64 / kV;  // runs per column; consecutive threads
  __shared__ T tile[64][64 + 2];
  in += (int64_t)blockIdx.z * in_bs;
  out += (int64_t)blockIdx.z * out_bs;
  const int64_t r0 = (int64_t)blockIdx.y * 64;
  const int c0 = blockIdx.x * 64;
  const int tid = threadIdx.x;
  for (int i = tid; i < 64 * 64 / kV; i += 256) {
    const int rr = i / (64 / kV), cc = (i % (64 / kV)) * kV;
    const int64_t r = r0 + rr;
    const int c = c0 + cc;
    T v[kV];
    if (r < R && c + kV <= C) {
      const u32x4 raw = ld16(in + r * ld_in + c);
      const T* e = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int k = 0; k < kV; ++k) v[k] = e[k];
    } else {
#pragma unroll
      for (int k = 0; k < kV; ++k) v[k] = (r < R && c + k < C) ? in[r * ld_in + c + k] : (T)0.0f;
    }
#pragma unroll
    for (int k = 0; k < kV; ++k) tile[rr][cc + k] = v[k];
  }
  __syncthreads();
  for (int i = tid; i < 64 * 64 / kV; i += 256) {
    const int cc = i / kRuns, rr = (i % kRuns) * kV;
    const int c = c0 + cc;
    const int64_t r = r0 + rr;
    T v[kV];
#pragma unroll
    for (int k = 0; k < kV; ++k) v[k] = tile[rr + k][cc];
    if (part) {  // block-uniform; rows past R and columns past C hold zeros
      float sum = 0.0f;
#pragma unroll
      for (int k = 0; k < kV; ++k) sum += to_f32(v[k]);
#pragma unroll
      for (int off = 1; off < kRuns; off <<= 1) sum += __shfl_xor(sum, off);
      if (rr == 0 && c < C) part[(int64_t)blockIdx.y * C + c] = sum;
    }
    if (c >= C) continue;
    const int64_t rw = R_out > R ? R_out : R;  // rows read past R are zeros
    if (r + kV <= rw) {
      st16(out + (int64_t)c * ld_out + r, *reinterpret_cast<const u32x4*>(v));
    } else {
      for (int k = 0; r + k < rw; ++k) out[(int64_t)c * ld_out + r + k] = v[k];
    }
  }
}

}  // namespace pf
