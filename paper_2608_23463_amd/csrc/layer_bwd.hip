// ProxyFormer layer backward: the chain rule through every forward step, in
// reverse order, from the activations the forward saved.
//
//  1. gate: dG = dY * Delta * s(1 - s) with s = sigmoid(G) (elementwise), then
//     one GEMM [dG W_gx | dG W_gd] whose epilogue forms dX = dY + dG W_gx (fp32
//     accumulator) and dDelta = s * dY + dG W_gd; dW_g = dG^T [X, Delta].
//     With residual-add injection (Eq. 11) dDelta = dY and dX starts at dY.
//  2. decompression levels 1..M (reverse of Eq. 17): dW_dj = dT^T U_j,
//     dU_j = dT W_dj; the top level's epilogue undoes the token-causal shift.
//  3. output map: dO = dHbar W_o (written per head in both layouts for the
//     attention backward), dW_o = dHbar^T O.
//  4. attention backward (separate dK/dV and dQ kernels, no atomics).
//  5. projections: dW_{q,k,v} = d{Q,K,V}^T H; dH = dH_out + dQ W_q + dK W_k
//     + dV W_v accumulated in fp32, rounded once (this is dH_in, Eq. 8).
//  6. compression levels M..1 (reverse of Eq. 16): dW_cj = dZ_j^T V_j and
//     dV_j = dZ_j W_cj; level 1 adds into the fp32 dX and rounds it once.
// Bias gradients are column sums, reduced in two fixed-order stages. In bf16
// every GEMM whose reduction runs over tokens (the weight gradients) reads its
// token-major operands as they are, through LDS transpose reads, so no
// transposed copy of an activation is made. In fp32 those operands are
// transposed once into workspace when they have kTransposeMinRows rows or
// more and a transposed row of them spans at most 8 MiB (the transpose of the
// output-gradient operand also leaves the bias column sums), and read through
// the register-transposing GEMM otherwise.
#include <algorithm>

#include "attention.hpp"
#include "epilogues.hpp"
#include "layer.hpp"
#include "runner.hpp"
#include "transpose.hpp"

namespace pf {

// dG = dY * Delta * s * (1 - s), s = sigmoid(G); 8 elements per thread.
template <typename T>
__global__ void __launch_bounds__(256) gate_bwd_prep_kernel(const T* __restrict__ dy, const T* __restrict__ delta,
                                                            const T* __restrict__ g, T* __restrict__ dg, int64_t n8) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < n8; c += stride) {
    float a[8], b[8], z[8], o[8];
    load8(dy + c * 8, a);
    load8(delta + c * 8, b);
    load8(g + c * 8, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float s = sigmoidf(z[e]);
      o[e] = a[e] * b[e] * s * (1.0f - s);
    }
    store8(dg + c * 8, o);
  }
}

// Eq. 13 backward, one wave per row: N = X rstd, dS = dY N, dT = dY,
// dN = dY (1 + S) and the RMSNorm's dX = rstd (dN - N mean(dN N)).
// [dS | dT] go to dst [rows, 2d], dX to dx32 (fp32; the compression's data
// gradient is added to it later). The row mean takes a first pass (per-lane
// runs of 8, then a butterfly), the outputs a second.
template <typename T>
__global__ void __launch_bounds__(256) affine_bwd_prep_kernel(const T* __restrict__ dy, const T* __restrict__ x,
                                                              const T* __restrict__ s, const float* __restrict__ rstd,
                                                              T* __restrict__ dst, float* __restrict__ dx32,
                                                              int64_t rows, int d) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int64_t base = row * d;
  const float rs = rstd[row];
  float acc = 0.0f;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float g[8], xv[8], sv[8];
    load8(dy + base + c, g);
    load8(x + base + c, xv);
    load8(s + base + c, sv);
#pragma unroll
    for (int e = 0; e < 8; ++e) acc = fmaf(g[e] * (1.0f + sv[e]), xv[e] * rs, acc);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  const float mean = acc / (float)d;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float g[8], xv[8], sv[8], ds[8], dx[8];
    load8(dy + base + c, g);
    load8(x + base + c, xv);
    load8(s + base + c, sv);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float n = xv[e] * rs;
      ds[e] = g[e] * n;
      dx[e] = rs * (g[e] * (1.0f + sv[e]) - n * mean);
    }
    store8(dst + row * 2 * d + c, ds);
    store8(dst + row * 2 * d + d + c, g);
    store8(dx32 + base + c, dx);
  }
}

// Per-head gate backward, one wave per row (4 rows per workgroup): the
// head sums dG_h = sum over the head's channels of dY * Delta, times
// sigmoid'(G_h) (partials per run of 8 channels through LDS, summed in run
// order), then dDelta = dY sigmoid(G_h(c)) + dG W_gd and the fp32 dX = dY +
// dG W_gx, with dG in fp32 and the gate rows read per run; dG in the
// activation type (row stride ldg) for the weight gradient.
// d <= 4096, nh <= 64, d / nh a multiple of 8.
template <typename T>
__global__ void __launch_bounds__(256) head_gate_bwd_kernel(const T* __restrict__ dy, const T* __restrict__ delta,
                                                            const float* __restrict__ gh, const T* __restrict__ wg,
                                                            T* __restrict__ ddelta, float* __restrict__ dx32,
                                                            T* __restrict__ dgh, int64_t rows, int d, int nh,
                                                            int ldg) {
  __shared__ float part[4][512];
  __shared__ float dgs[4][64];
  __shared__ float sgs[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  const bool live = row < rows;  // every wave reaches the barriers
  const int runs = d / 8, rph = d / nh / 8;  // runs per row, runs per head
  const int64_t base = row * d;
  if (live) {
    for (int run = lane; run < runs; run += 64) {
      float a[8], b[8];
      load8(dy + base + run * 8, a);
      load8(delta + base + run * 8, b);
      float p = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) p = fmaf(a[e], b[e], p);
      part[w][run] = p;
    }
  }
  __syncthreads();
  if (live && lane < nh) {
    float acc = 0.0f;
    for (int k = 0; k < rph; ++k) acc += part[w][lane * rph + k];
    const float sg = sigmoidf(gh[row * nh + lane]);
    const float dg = acc * sg * (1.0f - sg);
    dgs[w][lane] = dg;
    sgs[w][lane] = sg;
    dgh[row * ldg + lane] = from_f32<T>(dg);
  }
  __syncthreads();
  if (!live) return;
  for (int run = lane; run < runs; run += 64) {
    const int c0 = run * 8, h = run / rph;
    float a[8], dd[8], dx[8];
    load8(dy + base + c0, a);
    const float sg = sgs[w][h];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      dd[e] = a[e] * sg;
      dx[e] = a[e];
    }
    for (int k = 0; k < nh; ++k) {
      const float g = dgs[w][k];
      float wx[8], wd[8];
      load8(wg + (int64_t)k * 2 * d + c0, wx);
      load8(wg + (int64_t)k * 2 * d + d + c0, wd);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        dx[e] = fmaf(g, wx[e], dx[e]);
        dd[e] = fmaf(g, wd[e], dd[e]);
      }
    }
    store8(ddelta + base + c0, dd);
    store8(dx32 + base + c0, dx);
  }
}

// Column sums in two fixed-order stages: partial sums over row chunks, then
// the sum of the partials in chunk order.
template <typename T>
__global__ void __launch_bounds__(256) colsum_partial_kernel(const T* __restrict__ in, int64_t rows, int n,
                                                             int64_t ld, int64_t rows_per_chunk,
                                                             float* __restrict__ part) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  const int chunk = blockIdx.y;
  if (c >= n) return;
  const int64_t r0 = (int64_t)chunk * rows_per_chunk;
  const int64_t r1 = std::min<int64_t>(rows, r0 + rows_per_chunk);
  float s = 0.0f;
  for (int64_t r = r0; r < r1; ++r) s += to_f32(in[r * ld + c]);
  part[(int64_t)chunk * n + c] = s;
}

// The same partial sums, 8 columns per thread (16-byte loads; n and ld
// multiples of 8) over four independent row streams combined in a fixed
// order, so the sums stay deterministic.
template <typename T>
__global__ void __launch_bounds__(256) colsum_partial8_kernel(const T* __restrict__ in, int64_t rows, int n,
                                                              int64_t ld, int64_t rows_per_chunk,
                                                              float* __restrict__ part) {
  const int c = (blockIdx.x * blockDim.x + threadIdx.x) * 8;
  const int chunk = blockIdx.y;
  if (c >= n) return;
  const int64_t r0 = (int64_t)chunk * rows_per_chunk;
  const int64_t r1 = std::min<int64_t>(rows, r0 + rows_per_chunk);
  float s[4][8];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int e = 0; e < 8; ++e) s[u][e] = 0.0f;
  int64_t r = r0;
  for (; r + 4 <= r1; r += 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      float v[8];
      load8(in + (r + u) * ld + c, v);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[u][e] += v[e];
    }
  }
  for (; r < r1; ++r) {
    float v[8];
    load8(in + r * ld + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) s[0][e] += v[e];
  }
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (s[0][e] + s[1][e]) + (s[2][e] + s[3][e]);
  store8(part + (int64_t)chunk * n + c, o);
}

__global__ void __launch_bounds__(256) colsum_final_kernel(const float* __restrict__ part, int chunks, int n,
                                                           float* __restrict__ out) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= n) return;
  float s = 0.0f;
  for (int k = 0; k < chunks; ++k) s += part[(int64_t)k * n + c];
  out[c] = s;
}

// Gate dgrad epilogue: columns [0, d) are dG W_gx, columns [d, 2d) dG W_gd.
template <typename T>
struct EpiGateDgrad {
  const T* dy;
  const T* g;
  float* dx32;
  T* ddelta;
  int d;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (c < d) {
      const int64_t i = (int64_t)r * d + c;
      dx32[i] = to_f32(dy[i]) + v;
    } else {
      const int64_t i = (int64_t)r * d + (c - d);
      ddelta[i] = from_f32<T>(to_f32(dy[i]) * sigmoidf(to_f32(g[i])) + v);
    }
  }
  // Two-phase form (the direct kernel's epilogue reads ahead): pre() loads
  // dY, and G for the dDelta half.
  struct Col {};
  struct Pre {
    Raw8<T> a, z;
  };
  __device__ __forceinline__ void col(int, Col&) const {}
  __device__ __forceinline__ void pre(int r, int c, Pre& q) const {
    const int64_t i = (int64_t)r * d + (c < d ? c : c - d);
    raw_load8(dy + i, q.a);
    if (c >= d) raw_load8(g + i, q.z);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v, const Col&, const Pre& q) const {
    float a[8], o[8];
    raw_to_f32(q.a, a);
    if (c < d) {
      const int64_t i = (int64_t)r * d + c;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = a[e] + v[e];
      store8(dx32 + i, o);
    } else {
      const int64_t i = (int64_t)r * d + (c - d);
      float z[8];
      raw_to_f32(q.z, z);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = a[e] * sigmoidf(z[e]) + v[e];
      store8(ddelta + i, o);
    }
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    float a[8], o[8];
    if (c < d) {  // d is a multiple of 8, so a chunk never straddles the halves
      const int64_t i = (int64_t)r * d + c;
      load8(dy + i, a);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = a[e] + v[e];
      store8(dx32 + i, o);
    } else {
      const int64_t i = (int64_t)r * d + (c - d);
      float z[8];
      load8(dy + i, a);
      load8(g + i, z);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = a[e] * sigmoidf(z[e]) + v[e];
      store8(ddelta + i, o);
    }
  }
};

// Gradient of S back to the rows of the W_o output: in token-causal mode
// dHbar[r - 1] = dS[r] within a sequence and the last proxy (which feeds no
// block) gets zero; the row r = b*m writes that zero.
template <typename T>
struct EpiUnshift {
  T* out;
  int m, ld, shift;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (!shift) {
      out[(int64_t)r * ld + c] = from_f32<T>(v);
      return;
    }
    const int i = r % m;
    if (i > 0)
      out[(int64_t)(r - 1) * ld + c] = from_f32<T>(v);
    else
      out[(int64_t)(r + m - 1) * ld + c] = from_f32<T>(0.0f);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    if (!shift) {
      store8(out + (int64_t)r * ld + c, v);
      return;
    }
    const int i = r % m;
    if (i > 0) {
      store8(out + (int64_t)(r - 1) * ld + c, v);
    } else {
      const float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      store8(out + (int64_t)(r + m - 1) * ld + c, z);
    }
  }
};

// fp32 accumulation across several GEMMs into `acc`; the first may start from
// `add` (dtype T) instead of the accumulator, the last writes the rounded sum
// to `out` (and `out2`) instead of the accumulator.
template <typename T>
struct EpiAccum {
  float* acc;
  int64_t ld;
  const T* add;
  int first;
  T* out;
  T* out2;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    const int64_t i = (int64_t)r * ld + c;
    const float t = v + (first ? (add ? to_f32(add[i]) : 0.0f) : acc[i]);
    if (out) {
      out[i] = from_f32<T>(t);
      if (out2) out2[i] = from_f32<T>(t);
    } else {
      acc[i] = t;
    }
  }
  // Two-phase form: pre() loads the addend (`add` or the accumulator).
  struct Col {};
  struct Pre {
    Raw8<T> a;
    Raw8<float> f;
  };
  __device__ __forceinline__ void col(int, Col&) const {}
  __device__ __forceinline__ void pre(int r, int c, Pre& q) const {
    const int64_t i = (int64_t)r * ld + c;
    if (!first)
      raw_load8(acc + i, q.f);
    else if (add)
      raw_load8(add + i, q.a);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v, const Col&, const Pre& q) const {
    float b[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (!first)
      raw_to_f32(q.f, b);
    else if (add)
      raw_to_f32(q.a, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] += v[e];
    finish(r, c, b);
  }
  __device__ __forceinline__ void finish(int r, int c, const float* t) const {
    const int64_t i = (int64_t)r * ld + c;
    if (out) {
      store8(out + i, t);
      if (out2) store8(out2 + i, t);
    } else {
      store8(acc + i, t);
    }
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    const int64_t i = (int64_t)r * ld + c;
    float t[8], b[8];
    if (first) {
      if (add) {
        load8(add + i, b);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) b[e] = 0.0f;
      }
    } else {
      load8(acc + i, b);
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] = v[e] + b[e];
    if (out) {
      store8(out + i, t);
      if (out2) store8(out2 + i, t);
    } else {
      store8(acc + i, t);
    }
  }
};

template <typename T>
static void transpose(Runner& run, const char* label, const T* in, int64_t ld_in, int64_t R, int C, T* out,
                      int64_t ld_out, float* part = nullptr) {
  if (run.dry || R <= 0 || C <= 0) return;
  run.launch(label, [&] {
    hipLaunchKernelGGL((transpose_kernel<T>), dim3((C + 63) / 64, (unsigned)((R + 63) / 64)), dim3(256), 0,
                       run.stream, in, ld_in, R, C, out, ld_out, part);
    return hipGetLastError();
  });
}

template <typename T>
static void colsum(Runner& run, const char* label, const T* in, int64_t rows, int n, int64_t ld, float* part,
                   float* out) {
  if (!out || run.dry) return;
  const int chunks = (int)std::max<int64_t>(1, std::min<int64_t>(kColsumChunks, (rows + 63) / 64));
  const int64_t rpc = (rows + chunks - 1) / chunks;
  run.launch(label, [&] {
    if (n % 8 == 0 && ld % 8 == 0)
      hipLaunchKernelGGL((colsum_partial8_kernel<T>), dim3((n / 8 + 255) / 256, chunks), dim3(256), 0, run.stream,
                         in, rows, n, ld, rpc, part);
    else
      hipLaunchKernelGGL((colsum_partial_kernel<T>), dim3((n + 255) / 256, chunks), dim3(256), 0, run.stream, in,
                         rows, n, ld, rpc, part);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((n + 255) / 256), dim3(256), 0, run.stream, part, chunks, n, out);
    return hipGetLastError();
  });
}

// Remaining stages of a bias gradient whose per-64-row partial sums a
// transpose left in `part` (ceil(rows / 64) chunks): the chunks are summed
// in groups of consecutive chunks into part2, then the groups in order.
static void colsum_final(Runner& run, const char* label, int64_t rows, int n, const float* part, float* part2,
                         float* out) {
  if (!out || run.dry) return;
  const int chunks = (int)((rows + 63) / 64);
  const int groups = std::min(chunks, 64);
  const int64_t per = (chunks + groups - 1) / groups;
  run.launch(label, [&] {
    hipLaunchKernelGGL((colsum_partial_kernel<float>), dim3((n + 255) / 256, groups), dim3(256), 0, run.stream, part,
                       (int64_t)chunks, n, (int64_t)n, per, part2);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((n + 255) / 256), dim3(256), 0, run.stream, part2, groups, n, out);
    return hipGetLastError();
  });
}

// dW (fp32 [M, N] with row stride ldo) = sum over rows r of A[r, m] * B[r, n]:
// both operands are row-major [rows, *] activations, i.e. contiguous along
// the output dimensions. Over many rows both are first transposed into
// tr_a / tr_b ([M, rows] and [N, rows], rows padded to a multiple of 8) so the
// product runs on K-contiguous operands; `a_t` passes an A already
// transposed into tr_a by the caller. With `db`, the column sums of A (a
// bias gradient) are formed too, from the transpose's tiles when there is one.
template <typename T>
static void wgrad(Runner& run, const char* label, const T* a, int64_t lda, const T* b, int64_t ldb, int M, int N,
                  int64_t rows, float* out, int64_t ldo, T* tr_a, T* tr_b, bool a_t = false, float* db = nullptr,
                  float* part = nullptr, float* part2 = nullptr) {
  GemmProblem pr{};
  pr.M = M;
  pr.N = N;
  pr.K = (int)rows;
  if constexpr (sizeof(T) == 2) {
    // bf16: the direct kernel reads both row-major operands through LDS
    // transpose reads; no transposed copies
    if (db) colsum<T>(run, "bias_colsum", a, rows, M, lda, part, db);
    if (!out) return;
    pr.a = a;
    pr.lda = lda;
    pr.b = b;
    pr.ldb = ldb;
    run.gemm<T, LAYOUT_MN, LAYOUT_MN>(label, pr, EpiF32{out, ldo, 0});
    return;
  }
  const bool tr = wgrad_transposes(rows, sizeof(T));
  if (out && tr && !a_t) {
    transpose<T>(run, "transpose", a, lda, rows, M, tr_a, round8(rows), db ? part : nullptr);
    if (db) colsum_final(run, "bias_colsum", rows, M, part, part2, db);
  } else if (db) {
    colsum<T>(run, "bias_colsum", a, rows, M, lda, part, db);
  }
  if (!out) return;
  if (tr) {
    const int64_t ldt = round8(rows);
    transpose<T>(run, "transpose", b, ldb, rows, N, tr_b, ldt);
    pr.a = tr_a;
    pr.lda = ldt;
    pr.b = tr_b;
    pr.ldb = ldt;
    run.gemm<T, LAYOUT_K, LAYOUT_K>(label, pr, EpiF32{out, ldo, 0});
    return;
  }
  pr.a = a;
  pr.lda = lda;
  pr.b = b;
  pr.ldb = ldb;
  run.gemm<T, LAYOUT_MN, LAYOUT_MN>(label, pr, EpiF32{out, ldo, 0});
}

// dA [rows, N] = G [rows, K] W [K, N] for a weight W stored [K (out), N (in)]:
// the weight is read contiguous along N (LAYOUT_MN), or, over many rows,
// transposed once into tr_w ([N, K]) for the direct kernel.
template <typename T, class Epi>
static void dgrad(Runner& run, const char* label, const T* g, int64_t ldg, const void* w, int64_t ldw, int64_t rows,
                  int N, int K, const Epi& epi, T* tr_w) {
  GemmProblem pr{};
  pr.a = g;
  pr.lda = ldg;
  pr.M = (int)rows;
  pr.N = N;
  pr.K = K;
  if (rows >= kTransposeMinRows) {
    transpose<T>(run, "transpose", reinterpret_cast<const T*>(w), ldw, K, N, tr_w, K);
    pr.b = tr_w;
    pr.ldb = K;
    run.gemm<T, LAYOUT_K, LAYOUT_K>(label, pr, epi);
    return;
  }
  pr.b = w;
  pr.ldb = ldw;
  run.gemm<T, LAYOUT_K, LAYOUT_MN>(label, pr, epi);
}

template <typename T>
static void backward_impl(Runner& run, const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                          const void* x, const char* saved, const void* dy, const void* dh_out, void* dx, void* dh_in,
                          const pf_layer_grads* gr, char* ws) {
  const LayerActs A = layer_acts(d, true);
  const LayerWs W = layer_ws_layout(d, true);
  auto S = [&](size_t off) { return reinterpret_cast<const T*>(saved + off); };
  auto WT = [&](size_t off) { return reinterpret_cast<T*>(ws + off); };
  auto WF = [&](size_t off) { return reinterpret_cast<float*>(ws + off); };
  float* part = WF(W.colsum);
  float* part2 = WF(W.colsum2);
  T* tra = WT(W.tr_a);
  T* trb = WT(W.tr_b);
  T* trw = WT(W.tr_w);
  const int64_t BL = (int64_t)d.B * d.L;
  const int64_t Bm = (int64_t)d.B * d.m;
  const int df = d.d_f, dp = d.d_p;
  const T* dyp = reinterpret_cast<const T*>(dy);
  const T* xp = reinterpret_cast<const T*>(x);

  // 1. injection: gated (Eq. 12), affine (Eq. 13) or residual add (Eq. 11:
  //    dDelta = dX = dY)
  const bool add_inject = cfg->injection == PF_INJECT_ADD;
  if (cfg->injection == PF_INJECT_AFFINE) {
    run.launch("affine_bwd_prep", [&] {
      hipLaunchKernelGGL((affine_bwd_prep_kernel<T>), dim3((unsigned)((BL + 3) / 4)), dim3(256), 0, run.stream, dyp,
                         xp, S(A.g), reinterpret_cast<const float*>(saved + A.rstd), WT(W.dst), WF(W.dx32), BL, df);
      return hipGetLastError();
    });
    // dDelta = [dS | dT] W_a
    dgrad<T>(run, "affine_dgrad_gemm", WT(W.dst), 2 * df, w->affine.w, df, BL, df, 2 * df,
             EpiLinear<T>{WT(W.ddelta), df, nullptr, nullptr, 0, nullptr}, trw);
    // dW_a = [dS | dT]^T Delta, one half (and its bias columns) at a time
    float* dwa = reinterpret_cast<float*>(gr->affine.dw);
    float* dba = reinterpret_cast<float*>(gr->affine.db);
    for (int half = 0; half < 2; ++half)
      wgrad<T>(run, "affine_wgrad_gemm", WT(W.dst) + half * df, 2 * df, S(A.delta), df, df, df, BL,
               dwa ? dwa + (int64_t)half * df * df : nullptr, df, tra, trb, false, dba ? dba + half * df : nullptr,
               part, part2);
  } else if (cfg->injection == PF_INJECT_GATED_HEAD) {
    const int ldg = (int)round8(d.nh);
    run.launch("head_gate_bwd", [&] {
      hipLaunchKernelGGL((head_gate_bwd_kernel<T>), dim3((unsigned)((BL + 3) / 4)), dim3(256), 0, run.stream, dyp,
                         S(A.delta), reinterpret_cast<const float*>(saved + A.gh),
                         reinterpret_cast<const T*>(w->gate.w), WT(W.ddelta), WF(W.dx32), WT(W.dgh), BL, df, d.nh,
                         ldg);
      return hipGetLastError();
    });
    // dW_g = dG^T [X | Delta]: dG is transposed once for both halves
    float* dwg = reinterpret_cast<float*>(gr->gate.dw);
    wgrad<T>(run, "head_gate_wgrad_gemm", WT(W.dgh), ldg, xp, df, d.nh, df, BL, dwg, 2 * df, tra, trb, false,
             reinterpret_cast<float*>(gr->gate.db), part, part2);
    wgrad<T>(run, "head_gate_wgrad_gemm", WT(W.dgh), ldg, S(A.delta), df, d.nh, df, BL, dwg ? dwg + df : nullptr,
             2 * df, tra, trb, dwg != nullptr);
  } else if (!add_inject) {
    run.launch("gate_bwd_prep", [&] {
      const int64_t n8 = BL * df / 8;
      const int blocks = (int)std::min<int64_t>((n8 + 255) / 256, 16384);
      hipLaunchKernelGGL((gate_bwd_prep_kernel<T>), dim3(blocks), dim3(256), 0, run.stream, dyp, S(A.delta), S(A.g),
                         WT(W.dg), n8);
      return hipGetLastError();
    });
    dgrad<T>(run, "gate_dgrad_gemm", WT(W.dg), df, w->gate.w, 2 * df, BL, 2 * df, df,
             EpiGateDgrad<T>{dyp, S(A.g), WF(W.dx32), WT(W.ddelta), df}, trw);
    float* dwg = reinterpret_cast<float*>(gr->gate.dw);
    // dG is transposed once for both halves of dW_g
    wgrad<T>(run, "gate_wgrad_gemm", WT(W.dg), df, xp, df, df, df, BL, dwg, 2 * df, tra, trb, false,
             reinterpret_cast<float*>(gr->gate.db), part, part2);
    wgrad<T>(run, "gate_wgrad_gemm", WT(W.dg), df, S(A.delta), df, df, df, BL, dwg ? dwg + df : nullptr, 2 * df, tra,
             trb, dwg != nullptr);
  }

  // 2. decompression levels 1..M (reverse of Eq. 17)
  const T* dT = add_inject ? dyp : WT(W.ddelta);  // dU_0 = dDelta
  for (int j = 0; j < d.M; ++j) {
    const int64_t rows = (int64_t)d.B * d.R[j + 1];
    const int kd = d.k[j] * d.d[j];
    const int dn = d.d[j + 1];
    const T* u_in = j == d.M - 1 ? S(A.s) : S(A.u[j + 1]);
    wgrad<T>(run, "decompress_wgrad_gemm", dT, kd, u_in, dn, kd, dn, rows,
             reinterpret_cast<float*>(gr->decompress[j].dw), dn, tra, trb, false,
             reinterpret_cast<float*>(gr->decompress[j].db), part, part2);
    if (j == d.M - 1) {
      dgrad<T>(run, "decompress_dgrad_gemm", dT, kd, w->decompress[j].w, dn, rows, dn, kd,
               EpiUnshift<T>{WT(W.dhbar), (int)d.m, dp, cfg->mask == PF_TOKEN_CAUSAL ? 1 : 0}, trw);
    } else {
      dgrad<T>(run, "decompress_dgrad_gemm", dT, kd, w->decompress[j].w, dn, rows, dn, kd,
               EpiLinear<T>{WT(W.du[j + 1]), dn, nullptr, nullptr, 0, nullptr}, trw);
      dT = WT(W.du[j + 1]);
    }
  }

  // 3. output map of the interaction
  if (d.ld_t != d.m) {
    const size_t tb = (size_t)d.B * d.nh * d.dh * d.ld_t * sizeof(T);
    run.launch("fill_zero", [&] { return fill_zero(WT(W.dOt), tb, run.stream); });
  }
  dgrad<T>(run, "o_dgrad_gemm", WT(W.dhbar), dp, w->o.w, dp, Bm, dp, dp,
           EpiHeads<T>{WT(W.dO), WT(W.dOt), nullptr, (int)d.m, d.dh, d.nh, d.ld_t}, trw);
  wgrad<T>(run, "o_wgrad_gemm", WT(W.dhbar), dp, S(A.o), dp, dp, dp, Bm, reinterpret_cast<float*>(gr->o.dw), dp, tra,
           trb, false, reinterpret_cast<float*>(gr->o.db), part, part2);

  // 4. attention (Eq. 9)
  AttnBwdParams ap{};
  ap.q = S(A.q);
  ap.k = S(A.k);
  ap.q_lo = d.split ? S(A.q_lo) : nullptr;
  ap.k_lo = d.split ? S(A.k_lo) : nullptr;
  ap.v = S(A.v);
  ap.qt = S(A.qt);
  ap.kt = S(A.kt);
  ap.o = S(A.o);
  ap.do_ = WT(W.dO);
  ap.dot = WT(W.dOt);
  ap.lse = reinterpret_cast<const float*>(saved + A.lse);
  ap.delta = WF(W.delta_rs);
  ap.dq = WT(W.dq);
  ap.dk = WT(W.dk);
  ap.dv = WT(W.dv);
  ap.m = (int)d.m;
  ap.n_heads = d.nh;
  ap.ld_t = d.ld_t;
  ap.causal = cfg->mask != PF_BIDIRECTIONAL;
  ap.scale = (float)(1.0 / std::sqrt((double)d.dh));
  ap.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
  run.launch("attention_bwd", [&] { return launch_attention_bwd<T>(ap, d.B, d.dh, run.stream); });

  // 5. projections of H (and the residual update of Eq. 8)
  const T* dqkv[3] = {WT(W.dq), WT(W.dk), WT(W.dv)};
  const pf_linear* maps[3] = {&w->q, &w->k, &w->v};
  const pf_linear_grad* grads[3] = {&gr->q, &gr->k, &gr->v};
  for (int i = 0; i < 3; ++i) {
    wgrad<T>(run, "qkv_wgrad_gemm", dqkv[i], dp, S(A.h), dp, dp, dp, Bm, reinterpret_cast<float*>(grads[i]->dw), dp,
             tra, trb, false, reinterpret_cast<float*>(grads[i]->db), part, part2);
  }
  for (int i = 0; i < 3; ++i) {
    EpiAccum<T> e{WF(W.dh32), dp, reinterpret_cast<const T*>(dh_out), i == 0, i == 2 ? WT(W.dh) : nullptr,
                  i == 2 ? reinterpret_cast<T*>(dh_in) : nullptr};
    dgrad<T>(run, "qkv_dgrad_gemm", dqkv[i], dp, maps[i]->w, dp, Bm, dp, dp, e, trw);
  }

  // 6. compression levels M..1 (reverse of Eq. 16)
  const T* dz = WT(W.dh);
  for (int j = d.M - 1; j >= 0; --j) {
    const int64_t rows = (int64_t)d.B * d.R[j + 1];
    const int kd = d.k[j] * d.d[j];
    const int dn = d.d[j + 1];
    const T* v_in = j == 0 ? xp : S(A.z[j]);
    wgrad<T>(run, "compress_wgrad_gemm", dz, dn, v_in, kd, dn, kd, rows,
             reinterpret_cast<float*>(gr->compress[j].dw), kd, tra, trb, false,
             reinterpret_cast<float*>(gr->compress[j].db), part, part2);
    if (j == 0) {
      // dX = (dY + dG W_gx, in dx32) or dY, plus this level's data gradient
      EpiAccum<T> e = add_inject ? EpiAccum<T>{WF(W.dx32), kd, dyp, 1, reinterpret_cast<T*>(dx), nullptr}
                                 : EpiAccum<T>{WF(W.dx32), kd, nullptr, 0, reinterpret_cast<T*>(dx), nullptr};
      dgrad<T>(run, "compress_dgrad_gemm", dz, dn, w->compress[j].w, kd, rows, kd, dn, e, trw);
    } else {
      dgrad<T>(run, "compress_dgrad_gemm", dz, dn, w->compress[j].w, kd, rows, kd, dn,
               EpiLinear<T>{WT(W.dz[j]), kd, nullptr, nullptr, 0, nullptr}, trw);
      dz = WT(W.dz[j]);
    }
  }
}

template <typename T>
hipError_t layer_backward_run(const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                              const void* x, const void*, const char* saved, const void* dy, const void* dh_out,
                              void* dx, void* dh_in, const pf_layer_grads* gr, char* ws, hipStream_t stream) {
  const LayerWs W = layer_ws(d, true);
  Runner run(false, stream, reinterpret_cast<float*>(ws + W.gemm));
  backward_impl<T>(run, d, cfg, w, x, saved, dy, dh_out, dx, dh_in, gr, ws);
  return run.err;
}

size_t layer_backward_gemm_ws(const LayerDims& d) {
  pf_layer_config cfg{};
  cfg.mask = PF_TOKEN_CAUSAL;
  cfg.injection = d.inject;
  pf_layer_weights w{};
  // every weight gradient requested, so every GEMM is planned
  static float dummy;
  pf_layer_grads gr{};
  for (int j = 0; j < PF_MAX_LEVELS; ++j) gr.compress[j].dw = gr.decompress[j].dw = &dummy;
  gr.q.dw = gr.k.dw = gr.v.dw = gr.o.dw = gr.gate.dw = gr.affine.dw = &dummy;
  Runner run(true);
  if (d.esize == 2)
    backward_impl<bf16>(run, d, &cfg, &w, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &gr, nullptr);
  else
    backward_impl<float>(run, d, &cfg, &w, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, &gr, nullptr);
  return run.gemm_need;
}

template hipError_t layer_backward_run<bf16>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                             const void*, const void*, const char*, const void*, const void*, void*,
                                             void*, const pf_layer_grads*, char*, hipStream_t);
template hipError_t layer_backward_run<float>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                              const void*, const void*, const char*, const void*, const void*, void*,
                                              void*, const pf_layer_grads*, char*, hipStream_t);

}  // namespace pf
