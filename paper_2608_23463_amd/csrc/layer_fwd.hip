// ProxyFormer layer forward (Algorithm 1): planning of sizes and buffers,
// and the sequence of kernels that computes X^(l), H^(l) from X^(l-1), H^(l-1).
//
//  1. compression, one GEMM per level (Eq. 7, 15-16); the block partition of
//     Eq. 2 and the grouping of Eq. 16 are zero-copy views of row-major data,
//     and the last level's epilogue adds b_c and H_in (Eq. 8) and writes H.
//  2. Q, K, V projections of H, written per head (V key-contiguous). In bf16
//     mode with extended precision H, the level outputs Z_j, Q and K keep a
//     bf16 low part as well (two-term split), and the GEMMs that read them
//     multiply [hi | lo] by [W | W]: the attention logits then carry ~16
//     mantissa bits.
//  3. causal flash attention over the m proxies (Eq. 9).
//  4. output map W_o -> contextualised proxies S.
//  5. decompression, one GEMM per level from level M down to 1 (Eq. 10, 17),
//     reading S, which the W_o epilogue wrote already shifted (block i
//     receives proxy i-1 in token-causal mode).
//  6. gate GEMM over [X, Delta] with the injection X + sigmoid(G) * Delta in
//     its epilogue (Eq. 12).
#include <algorithm>

#include "attention.hpp"
#include "epilogues.hpp"
#include "fused_gate.hpp"
#include "layer.hpp"
#include "runner.hpp"

namespace pf {

__global__ void fill_zero_kernel(u32x4* p, size_t n16) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) p[i] = u32x4{0u, 0u, 0u, 0u};
}

hipError_t fill_zero(void* p, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16;  // every buffer here is a multiple of 16 bytes
  const int blocks = (int)std::min<size_t>((n16 + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, reinterpret_cast<u32x4*>(p), n16);
  return hipGetLastError();
}

// b'[p][n] = b_g[n] (or 0) for every position p: the fused gate's bias when
// the decompression has no bias.
template <typename T>
__global__ void __launch_bounds__(256) gate_bias_broadcast_kernel(const T* __restrict__ bg, float* __restrict__ out,
                                                                   int k, int n) {
  const int64_t total = (int64_t)k * n;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256)
    out[i] = bg ? to_f32(bg[i % n]) : 0.0f;
}

__global__ void pad_rows_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, int64_t L_in,
                                int64_t L_pad, int64_t row16, int64_t total) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t c = i % row16, r = i / row16;
    const int64_t b = r / L_pad, t = r - b * L_pad;
    dst[i] = t < L_in ? src[(b * L_in + t) * row16 + c] : u32x4{0u, 0u, 0u, 0u};
  }
}

hipError_t pad_rows(const void* src, void* dst, int B, int64_t L_in, int64_t L_pad, int64_t row_bytes,
                    hipStream_t stream) {
  const int64_t row16 = row_bytes / 16, total = (int64_t)B * L_pad * row16;
  if (total == 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(pad_rows_kernel, dim3(blocks), dim3(256), 0, stream, reinterpret_cast<const u32x4*>(src),
                     reinterpret_cast<u32x4*>(dst), L_in, L_pad, row16, total);
  return hipGetLastError();
}

hipError_t unpad_rows(const void* src, void* dst, int B, int64_t L_in, int64_t L_pad, int64_t row_bytes,
                      hipStream_t stream) {
  return hipMemcpy2DAsync(dst, (size_t)(L_in * row_bytes), src, (size_t)(L_pad * row_bytes),
                          (size_t)(L_in * row_bytes), (size_t)B, hipMemcpyDeviceToDevice, stream);
}

__global__ void permute_patches_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst, int64_t L, int w,
                                       int p, int64_t row16, int64_t total, int scatter) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t P = (int64_t)p * p, pw = w / p;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int64_t c = i % row16, r = i / row16;
    const int64_t b = r / L, j = r - b * L;
    const int64_t blk = j / P, u = j - blk * P;
    const int64_t t = ((blk / pw) * p + u / p) * w + (blk % pw) * p + u % p;  // raster index
    if (scatter)
      dst[(b * L + t) * row16 + c] = src[i];
    else
      dst[i] = src[(b * L + t) * row16 + c];
  }
}

hipError_t permute_patches(const void* src, void* dst, int B, int64_t L, int w, int p, int64_t row_bytes,
                           bool scatter, hipStream_t stream) {
  const int64_t row16 = row_bytes / 16, total = (int64_t)B * L * row16;
  if (total == 0) return hipSuccess;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(permute_patches_kernel, dim3(blocks), dim3(256), 0, stream, reinterpret_cast<const u32x4*>(src),
                     reinterpret_cast<u32x4*>(dst), L, w, p, row16, total, scatter ? 1 : 0);
  return hipGetLastError();
}

// Eq. 13: rstd[r] = 1 / sqrt(mean(x[r]^2) + eps), one wave per row (fp32
// sum of squares: per-lane runs of 8, then a butterfly over the wave).
template <typename T>
__global__ void __launch_bounds__(256) rstd_rows_kernel(const T* __restrict__ x, float* __restrict__ rstd,
                                                        int64_t rows, int d, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* xr = x + row * d;
  float ss = 0.0f;
  for (int c = lane * 8; c < d; c += 64 * 8) {
    float v[8];
    load8(xr + c, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) ss = fmaf(v[e], v[e], ss);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  if (lane == 0) rstd[row] = 1.0f / sqrtf(ss / (float)d + eps);
}

// Per-head gate (Eq. 12 with one gate per head): y = x + sigmoid(G[r, h(c)])
// * delta for runs of 8 channels (d / n_heads is a multiple of 8, so a run
// stays inside one head).
template <typename T>
__global__ void __launch_bounds__(256) head_gate_combine_kernel(const T* __restrict__ x, const T* __restrict__ delta,
                                                                const float* __restrict__ gh, T* __restrict__ y,
                                                                int64_t rows, int d, int nh) {
  // A row is tpr runs of 8; a block covers rpb rows at a time (one row in
  // passes of 256 runs when tpr > 256). The run and its head are fixed per
  // thread, so the loop carries no division.
  const int tpr = d / 8;
  const int rpb = tpr <= 256 ? 256 / tpr : 1;
  const int lr = tpr <= 256 ? (int)threadIdx.x / tpr : 0;
  if (lr >= rpb) return;
  const int j0 = tpr <= 256 ? (int)threadIdx.x - lr * tpr : (int)threadIdx.x;
  const int gs = d / nh;
  for (int64_t r = (int64_t)blockIdx.x * rpb + lr; r < rows; r += (int64_t)gridDim.x * rpb) {
    const T* xr = x + r * d;
    const T* dr = delta + r * d;
    T* yr = y + r * d;
    for (int j = j0; j < tpr; j += 256) {
      const float s = sigmoidf(gh[r * nh + (j * 8) / gs]);
      float a[8], b[8], o[8];
      load8(xr + j * 8, a);
      load8(dr + j * 8, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = fmaf(s, b[e], a[e]);
      store8(yr + j * 8, o);
    }
  }
}

// W_a [2d, d] (s rows, then t rows) -> rows interleaved s_0, t_0, s_1, t_1,
// ..., so the affine GEMM's columns 2c and 2c+1 are s and t of channel c.
template <typename T>
__global__ void __launch_bounds__(256) affine_interleave_kernel(const T* __restrict__ w, const T* __restrict__ b,
                                                                T* __restrict__ w_il, T* __restrict__ b_il, int d) {
  const int64_t total = (int64_t)2 * d * d;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int rr = (int)(i / d), cc = (int)(i % d);
    const int src = (rr & 1) ? d + (rr >> 1) : (rr >> 1);
    w_il[i] = w[(int64_t)src * d + cc];
    if (cc == 0) b_il[rr] = b ? b[src] : (T)0.0f;
  }
}

int layer_dims(const pf_layer_config* c, LayerDims* d, const char** why) {
  *why = nullptr;
  if (!c) return *why = "config is NULL", PF_ERR_INVALID_ARG;
  if (c->dtype != PF_FP32 && c->dtype != PF_BF16) return *why = "dtype must be PF_FP32 or PF_BF16", PF_ERR_INVALID_ARG;
  if (c->mask < PF_TOKEN_CAUSAL || c->mask > PF_BIDIRECTIONAL) return *why = "unknown mask mode", PF_ERR_INVALID_ARG;
  if (c->injection < PF_INJECT_GATED || c->injection > PF_INJECT_GATED_HEAD)
    return *why = "unknown injection mode", PF_ERR_INVALID_ARG;
  if (c->precision != PF_PRECISION_EXTENDED && c->precision != PF_PRECISION_BF16)
    return *why = "precision must be PF_PRECISION_EXTENDED or PF_PRECISION_BF16", PF_ERR_INVALID_ARG;
  if (c->gate_fusion != PF_GATE_SEPARATE && c->gate_fusion != PF_GATE_FUSED)
    return *why = "gate_fusion must be PF_GATE_SEPARATE or PF_GATE_FUSED", PF_ERR_INVALID_ARG;
  if (c->batch < 1 || c->seq_len < 1) return *why = "batch and seq_len must be >= 1", PF_ERR_INVALID_ARG;
  if (c->n_levels < 1 || c->n_levels > PF_MAX_LEVELS) return *why = "n_levels must be in 1..4", PF_ERR_INVALID_ARG;
  if (c->d_fine < 1 || c->d_proxy < 1 || c->n_heads < 1 || c->head_dim < 1)
    return *why = "widths and head counts must be >= 1", PF_ERR_INVALID_ARG;
  if ((int64_t)c->n_heads * c->head_dim != c->d_proxy) return *why = "n_heads * head_dim must equal d_proxy", PF_ERR_INVALID_ARG;
  d->B = c->batch;
  d->inject = c->injection;
  d->L_in = c->seq_len;
  d->d_f = c->d_fine;
  d->d_p = c->d_proxy;
  d->nh = c->n_heads;
  d->dh = c->head_dim;
  d->M = c->n_levels;
  d->P = 1;
  for (int j = 0; j < d->M; ++j) {
    if (c->factors[j] < 1) return *why = "every factor k_j must be >= 1", PF_ERR_INVALID_ARG;
    d->k[j] = c->factors[j];
    d->P *= c->factors[j];
    if (d->P > (1 << 20)) return *why = "block size P too large", PF_ERR_INVALID_ARG;
  }
  // m = ceil(L / P) blocks (Sec. 3.1); a partial last block is zero-padded
  d->L = (d->L_in + d->P - 1) / d->P * d->P;
  d->img_w = 0;
  d->patch = 0;
  if (c->image_width < 0) return *why = "image_width must be >= 0", PF_ERR_INVALID_ARG;
  if (c->image_width > 0) {  // 2-D partition (Sec. 3.9)
    if (d->M != 1) return *why = "the 2-D partition takes one level (P = p * p)", PF_ERR_UNSUPPORTED;
    int p = 1;
    while ((int64_t)(p + 1) * (p + 1) <= d->P) ++p;
    if ((int64_t)p * p != d->P) return *why = "the 2-D partition needs P = p * p", PF_ERR_INVALID_ARG;
    if (d->L_in % c->image_width != 0) return *why = "seq_len must be image_width * height", PF_ERR_INVALID_ARG;
    const int64_t h = d->L_in / c->image_width;
    if (c->image_width % p != 0 || h % p != 0)
      return *why = "image width and height must be multiples of the patch side", PF_ERR_INVALID_ARG;
    d->img_w = c->image_width;
    d->patch = p;
  }
  d->d[0] = d->d_f;
  for (int j = 1; j < d->M; ++j) d->d[j] = c->level_dims[j - 1] > 0 ? c->level_dims[j - 1] : d->d_p;
  d->d[d->M] = d->d_p;
  d->R[0] = d->L;
  for (int j = 1; j <= d->M; ++j) d->R[j] = d->R[j - 1] / d->k[j - 1];
  d->m = d->R[d->M];
  if ((int64_t)d->B * d->L > INT32_MAX) return *why = "batch * seq_len exceeds 2^31 - 1 rows", PF_ERR_UNSUPPORTED;
  d->ld_t = (int)((d->m + 63) / 64 * 64);
  d->esize = c->dtype == PF_BF16 ? 2 : 4;
  d->split = d->esize == 2 && c->precision == PF_PRECISION_EXTENDED;
  d->fused_gate = false;  // set below once the level widths are known
  // the attention kernels address one head's tensors ([m, d_head] rows,
  // [d_head, ld_t] transposed) through 32-bit buffer offsets
  if ((int64_t)d->ld_t * c->head_dim * d->esize >= ((int64_t)1 << 31))
    return *why = "one head's proxy tensors exceed 2 GiB (m * head_dim * element size)", PF_ERR_UNSUPPORTED;
  for (int j = 0; j <= d->M; ++j)
    if (d->d[j] % 8 != 0) return *why = "every channel width must be a multiple of 8", PF_ERR_UNSUPPORTED;
  // A GEMM tile reaches up to 256 rows of an operand through one 32-bit
  // buffer range whose out-of-range offset is 2^31, so an operand row (a
  // level's grouped row of k_j * d_{j-1} elements, the gate's 2 * d_fine) may
  // span at most 8 MiB.
  for (int j = 0; j < d->M; ++j)
    if ((int64_t)d->k[j] * d->d[j] * d->esize > kMaxGemmRowBytes)
      return *why = "a grouped row k_j * d_{j-1} * element size exceeds 8 MiB", PF_ERR_UNSUPPORTED;
  if ((int64_t)2 * d->d_f * d->esize > kMaxGemmRowBytes)
    return *why = "2 * d_fine * element size exceeds 8 MiB", PF_ERR_UNSUPPORTED;
  // the projections read H with its low part beside it ([H_hi | H_lo] rows)
  if ((int64_t)2 * d->d_p * d->esize > kMaxGemmRowBytes)
    return *why = "2 * d_proxy * element size exceeds 8 MiB", PF_ERR_UNSUPPORTED;
  if (d->dh != 64 && d->dh != 128) return *why = "head_dim must be 64 or 128", PF_ERR_UNSUPPORTED;
  d->fused_gate = c->gate_fusion == PF_GATE_FUSED && d->esize == 2 && c->injection == PF_INJECT_GATED &&
                  fused_gate_supported(d->d_f, d->d[1]);
  if (c->injection == PF_INJECT_GATED_HEAD && (d->d_f % d->nh != 0 || (d->d_f / d->nh) % 8 != 0))
    return *why = "the per-head gate needs d_fine / n_heads to be a multiple of 8", PF_ERR_UNSUPPORTED;
  if (c->injection == PF_INJECT_GATED_HEAD && (d->d_f > 4096 || d->nh > 64))
    return *why = "the per-head gate takes d_fine <= 4096 and n_heads <= 64", PF_ERR_UNSUPPORTED;
  return PF_OK;
}

LayerActs layer_acts(const LayerDims& d, bool bwd) {
  LayerActs a{};
  size_t off = 0;
  const size_t es = d.esize;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t prox = (size_t)d.B * d.m * d.d_p * es;
  const size_t headt = (size_t)d.B * d.nh * d.dh * d.ld_t * es;
  const bool split = d.split;
  for (int j = 1; j < d.M; ++j) {
    a.z[j] = take((size_t)d.B * d.R[j] * d.d[j] * es);
    a.z_lo[j] = take(split ? (size_t)d.B * d.R[j] * d.d[j] * es : 0);
  }
  a.h = bwd ? take(prox) : 0;
  a.h_lo = take(split ? prox : 0);
  a.q = take(prox);
  a.k = take(prox);
  a.q_lo = take(split && bwd ? prox : 0);  // the backward's split logits
  a.k_lo = take(split && bwd ? prox : 0);
  // the forward attention reads Q pre-scaled; the backward reads Q itself
  a.qs = bwd ? take(prox) : a.q;
  // the forward attention's fp8 correction rows: 2 dh bytes per head row,
  // the size of a bf16 row
  a.qx = take(split ? prox : 0);
  a.kx = take(split ? prox : 0);
  a.v = bwd ? take(prox) : 0;
  a.qt = bwd ? take(headt) : 0;
  a.kt = bwd ? take(headt) : 0;
  a.vt = take(headt);
  a.o = take(prox);
  a.lse = take((size_t)d.B * d.nh * d.m * 4);
  a.s = take(prox);
  for (int j = 1; j < d.M; ++j) a.u[j] = take((size_t)d.B * d.R[j] * d.d[j] * es);
  // Delta is materialised for the injections that read it after the
  // decompression, and for the backward; residual addition writes Y from the
  // decompression's epilogue, and the fused gate keeps Delta in registers
  const bool need_delta = d.inject != PF_INJECT_ADD && (bwd || !d.fused_gate);
  a.delta = take(need_delta ? (size_t)d.B * d.L * d.d_f * es : 0);
  a.g = bwd && (d.inject == PF_INJECT_GATED || d.inject == PF_INJECT_AFFINE) ? take((size_t)d.B * d.L * d.d_f * es)
                                                                               : 0;
  const bool affine = d.inject == PF_INJECT_AFFINE;
  a.rstd = take(affine ? (size_t)d.B * d.L * 4 : 0);
  a.gh = take(d.inject == PF_INJECT_GATED_HEAD ? (size_t)d.B * d.L * d.nh * 4 : 0);
  a.aff_w = take(affine ? (size_t)2 * d.d_f * d.d_f * es : 0);
  a.aff_b = take(affine ? (size_t)2 * d.d_f * es : 0);
  a.bytes = off;
  return a;
}

LayerWs layer_ws_layout(const LayerDims& d, bool bwd) {
  LayerWs w{};
  size_t off = 0;
  const size_t es = d.esize;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t prox = (size_t)d.B * d.m * d.d_p * es;
  const size_t tok = (size_t)d.B * d.L * d.d_f * es;
  if (!bwd) {
    w.acts = take(layer_acts(d, false).bytes);
    w.gate_c = take(d.fused_gate ? (size_t)d.k[0] * d.d_f * d.d[1] * es : 0);
    w.gate_b = take(d.fused_gate ? (size_t)d.k[0] * d.d_f * 4 : 0);
  } else {
    const size_t prox32 = (size_t)d.B * d.m * d.d_p * 4;
    w.dg = take(tok);
    w.ddelta = take(tok);
    w.dx32 = take((size_t)d.B * d.L * d.d_f * 4);
    for (int j = 1; j < d.M; ++j) w.du[j] = take((size_t)d.B * d.R[j] * d.d[j] * es);
    w.dhbar = take(prox);
    w.dO = take(prox);
    w.dOt = take((size_t)d.B * d.nh * d.dh * d.ld_t * es);
    w.delta_rs = take((size_t)d.B * d.nh * d.m * 4);
    w.dq = take(prox);
    w.dk = take(prox);
    w.dv = take(prox);
    w.dh32 = take(prox32);
    w.dh = take(prox);
    for (int j = 1; j < d.M; ++j) w.dz[j] = take((size_t)d.B * d.R[j] * d.d[j] * es);
    // widest bias: max over every linear map's output width
    int64_t widest = std::max<int64_t>(2 * d.d_f, d.d_p);
    for (int j = 0; j < d.M; ++j) widest = std::max<int64_t>(widest, (int64_t)d.k[j] * d.d[j]);
    // bias-gradient partials: kColsumChunks row chunks, or one per 64 rows
    // when the column sums come out of a transpose
    size_t part = (size_t)kColsumChunks * widest;
    auto tp = [&](int64_t rows, int64_t cols) {
      if (wgrad_transposes(rows, es)) part = std::max(part, (size_t)((rows + 63) / 64 * cols));
    };
    tp((int64_t)d.B * d.L, d.d_f);
    for (int j = 0; j < d.M; ++j) {
      tp((int64_t)d.B * d.R[j + 1], (int64_t)d.k[j] * d.d[j]);
      tp((int64_t)d.B * d.R[j + 1], d.d[j + 1]);
    }
    tp((int64_t)d.B * d.m, d.d_p);
    w.colsum = take(part * 4);
    w.colsum2 = take((size_t)64 * widest * 4);
    // transposed operands: every large gradient / activation operand is at
    // most [B*L, d_f] elements (plus row padding to a multiple of 8)
    size_t tr = 0, trw = 0;
    auto op = [&](int64_t rows, int64_t cols) {
      if (wgrad_transposes(rows, es)) tr = std::max(tr, (size_t)(round8(rows) * cols) * es);
    };
    auto wt = [&](int64_t out, int64_t in) { trw = std::max(trw, (size_t)(out * in) * es); };
    op((int64_t)d.B * d.L, d.d_f);
    wt(d.d_f, 2 * (int64_t)d.d_f);
    for (int j = 0; j < d.M; ++j) {
      const int64_t rows = (int64_t)d.B * d.R[j + 1];
      op(rows, (int64_t)d.k[j] * d.d[j]);
      op(rows, d.d[j + 1]);
      wt((int64_t)d.k[j] * d.d[j], d.d[j + 1]);
    }
    op((int64_t)d.B * d.m, d.d_p);
    wt(d.d_p, d.d_p);
    w.tr_a = take(tr);
    w.tr_b = take(tr);
    w.tr_w = take(trw);
  }
  if (bwd && d.inject == PF_INJECT_AFFINE) w.dst = take(2 * tok);
  if (bwd && d.inject == PF_INJECT_GATED_HEAD) w.dgh = take((size_t)d.B * d.L * round8(d.nh) * es);
  if (d.staged()) {
    w.x_pad = take(tok);
    w.y_pad = take(tok);
    w.dy_pad = bwd ? take(tok) : 0;
  }
  w.gemm = off;
  w.bytes = off;
  return w;
}

LayerWs layer_ws(const LayerDims& d, bool bwd) {
  LayerWs w = layer_ws_layout(d, bwd);
  w.bytes = w.gemm + align256(layer_gemm_ws_bytes(d, bwd));
  return w;
}

template <typename T>
static void forward_impl(Runner& run, const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                         const void* x, const void* h_in, void* x_out, void* h_out, char* act, bool saving,
                         char* ws) {
  const LayerActs A = layer_acts(d, saving);
  auto P = [&](size_t off) { return reinterpret_cast<T*>(act + off); };
  const int64_t rows_m = (int64_t)d.B * d.m;

  const bool split = d.split;

  // 1. compression cascade (Eq. 7, 16) and the residual proxy update (Eq. 8).
  //    Levels after the first read their input as [hi | lo] against [W | W].
  const T* zin = reinterpret_cast<const T*>(x);
  const T* zin_lo = nullptr;
  for (int j = 0; j < d.M; ++j) {
    GemmProblem pr{};
    const int kd = d.k[j] * d.d[j];
    pr.a = zin;
    pr.lda = kd;
    pr.b = w->compress[j].w;
    pr.ldb = kd;
    pr.M = (int)(d.B * d.R[j + 1]);
    pr.N = d.d[j + 1];
    pr.K = kd;
    if (zin_lo) {
      pr.a2 = zin_lo;
      pr.lda2 = kd;
      pr.a_ksplit = kd;
      pr.b2 = w->compress[j].w;
      pr.ldb2 = kd;
      pr.b_ksplit = kd;
      pr.K = 2 * kd;
    }
    EpiLinear<T> e{};
    e.bias = reinterpret_cast<const T*>(w->compress[j].b);
    if (j == d.M - 1) {
      e.out = reinterpret_cast<T*>(h_out);
      e.ldo = d.d_p;
      e.add = reinterpret_cast<const T*>(h_in);
      e.ld_add = d.d_p;
      e.out2 = saving ? P(A.h) : nullptr;
      e.out_lo = split ? P(A.h_lo) : nullptr;
    } else {
      e.out = P(A.z[j + 1]);
      e.ldo = d.d[j + 1];
      e.out_lo = split ? P(A.z_lo[j + 1]) : nullptr;
    }
    run.gemm<T, LAYOUT_K, LAYOUT_K>("compress_gemm", pr, e);
    zin = e.out;
    zin_lo = e.out_lo;
  }

  // 2. projections of H into per-head Q, K (row layout, hi and lo parts) and
  //    V (key-contiguous); Q and K read H as [hi | lo]
  const T* hbuf = reinterpret_cast<const T*>(h_out);
  if (d.ld_t != d.m) {
    // padding columns of the transposed tensors must read as zero
    const size_t tb = (size_t)d.B * d.nh * d.dh * d.ld_t * sizeof(T);
    run.launch("fill_zero", [&] { return fill_zero(P(A.vt), tb, run.stream); });
    if (saving) {
      run.launch("fill_zero", [&] { return fill_zero(P(A.qt), tb, run.stream); });
      run.launch("fill_zero", [&] { return fill_zero(P(A.kt), tb, run.stream); });
    }
  }
  const pf_linear* proj[3] = {&w->q, &w->k, &w->v};
  // Q goes to the attention pre-scaled by log2(e)/sqrt(d_head) (scores in
  // exp2 units); the unscaled Q is kept only for the backward
  const float qscale = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
  T* outs[3] = {saving ? P(A.q) : nullptr, P(A.k), saving ? P(A.v) : nullptr};
  T* outs_t[3] = {saving ? P(A.qt) : nullptr, saving ? P(A.kt) : nullptr, P(A.vt)};
  // the low parts of Q and K are kept for the backward; the forward
  // attention reads the fp8 correction rows
  T* outs_lo[3] = {split && saving ? P(A.q_lo) : nullptr, split && saving ? P(A.k_lo) : nullptr, nullptr};
  for (int i = 0; i < 3; ++i) {
    GemmProblem pr{};
    pr.a = hbuf;
    pr.lda = d.d_p;
    pr.b = proj[i]->w;
    pr.ldb = d.d_p;
    pr.M = (int)rows_m;
    pr.N = d.d_p;
    pr.K = d.d_p;
    if (split && i < 2) {  // Q and K read H as [hi | lo]
      pr.a2 = P(A.h_lo);
      pr.lda2 = d.d_p;
      pr.a_ksplit = d.d_p;
      pr.b2 = proj[i]->w;
      pr.ldb2 = d.d_p;
      pr.b_ksplit = d.d_p;
      pr.K = 2 * d.d_p;
    }
    EpiHeads<T> e{outs[i], outs_t[i], reinterpret_cast<const T*>(proj[i]->b), (int)d.m, d.dh, d.nh, d.ld_t,
                  outs_lo[i]};
    if (i == 0) {
      e.outs = P(A.qs);
      e.scale = qscale;
    }
    if (split && i < 2) {
      e.outx = reinterpret_cast<uint8_t*>(act + (i == 0 ? A.qx : A.kx));
      e.xmode = i == 0 ? 1 : 2;
    }
    run.gemm<T, LAYOUT_K, LAYOUT_K>("qkv_gemm", pr, e);
  }

  // 3. attention over the proxies (Eq. 9)
  AttnParams ap{};
  ap.q = P(A.qs);
  ap.k = P(A.k);
  ap.qx = split ? act + A.qx : nullptr;
  ap.kx = split ? act + A.kx : nullptr;
  ap.vt = P(A.vt);
  ap.o = P(A.o);
  ap.lse = reinterpret_cast<float*>(act + A.lse);
  ap.m = (int)d.m;
  ap.n_heads = d.nh;
  ap.ld_t = d.ld_t;
  ap.causal = cfg->mask != PF_BIDIRECTIONAL;
  run.launch("attention_fwd", [&] { return launch_attention_fwd<T>(ap, d.B, d.dh, run.stream); });

  // 4. output map of the interaction; in token-causal mode its epilogue also
  //    applies the shift, so S holds proxy i-1 at row i (zero at row 0)
  {
    GemmProblem pr{};
    pr.a = P(A.o);
    pr.lda = d.d_p;
    pr.b = w->o.w;
    pr.ldb = d.d_p;
    pr.M = (int)rows_m;
    pr.N = d.d_p;
    pr.K = d.d_p;
    const T* bo = reinterpret_cast<const T*>(w->o.b);
    if (cfg->mask == PF_TOKEN_CAUSAL) {
      run.gemm<T, LAYOUT_K, LAYOUT_K>("o_gemm", pr, EpiShift<T>{P(A.s), bo, (int)d.m, d.d_p});
    } else {
      run.gemm<T, LAYOUT_K, LAYOUT_K>("o_gemm", pr, EpiLinear<T>{P(A.s), d.d_p, bo, nullptr, 0, nullptr});
    }
  }

  // 5. decompression, level M down to 1 (Eq. 10, 17). With residual-add
  // injection (Eq. 11) the last level's epilogue adds X and writes Y itself:
  // its [B R_1, k_1 d_fine] output is X_out byte for byte.
  const bool add_inject = cfg->injection == PF_INJECT_ADD;
  const bool fuse = d.fused_gate;
  for (int j = d.M - 1; j >= (fuse ? 1 : 0); --j) {  // a fused level 1 runs with the gate below
    GemmProblem pr{};
    pr.a = j == d.M - 1 ? P(A.s) : P(A.u[j + 1]);
    pr.lda = d.d[j + 1];
    pr.b = w->decompress[j].w;
    pr.ldb = d.d[j + 1];
    pr.M = (int)(d.B * d.R[j + 1]);
    pr.N = d.k[j] * d.d[j];
    pr.K = d.d[j + 1];
    const T* bias = reinterpret_cast<const T*>(w->decompress[j].b);
    if (j == 0 && add_inject) {
      EpiLinear<T> e{reinterpret_cast<T*>(x_out), pr.N, bias, reinterpret_cast<const T*>(x), pr.N, nullptr};
      run.gemm<T, LAYOUT_K, LAYOUT_K>("decompress_gemm", pr, e);
      continue;
    }
    T* out = j == 0 ? P(A.delta) : P(A.u[j]);
    EpiLinear<T> e{out, pr.N, bias, nullptr, 0, nullptr};
    run.gemm<T, LAYOUT_K, LAYOUT_K>("decompress_gemm", pr, e);
  }

  // 6. affine modulation (Eq. 13): [S | T] = Delta W_a^T + b_a with s and t
  //    interleaved per channel, Y = (1 + S) * X * rstd + T in the epilogue
  if (cfg->injection == PF_INJECT_AFFINE) {
    const int64_t rows = (int64_t)d.B * d.L;
    float* rstd = reinterpret_cast<float*>(act + A.rstd);
    run.launch("affine_rstd", [&] {
      hipLaunchKernelGGL((rstd_rows_kernel<T>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, run.stream,
                         reinterpret_cast<const T*>(x), rstd, rows, d.d_f, kAffineEps);
      return hipGetLastError();
    });
    run.launch("affine_interleave", [&] {
      const int64_t total = (int64_t)2 * d.d_f * d.d_f;
      hipLaunchKernelGGL((affine_interleave_kernel<T>), dim3((unsigned)std::min<int64_t>((total + 255) / 256, 4096)),
                         dim3(256), 0, run.stream, reinterpret_cast<const T*>(w->affine.w),
                         reinterpret_cast<const T*>(w->affine.b), P(A.aff_w), P(A.aff_b), d.d_f);
      return hipGetLastError();
    });
    GemmProblem pr{};
    pr.a = P(A.delta);
    pr.lda = d.d_f;
    pr.b = P(A.aff_w);
    pr.ldb = d.d_f;
    pr.M = (int)rows;
    pr.N = 2 * d.d_f;
    pr.K = d.d_f;
    EpiAffine<T> e{reinterpret_cast<const T*>(x), rstd, P(A.aff_b), reinterpret_cast<T*>(x_out),
                   saving ? P(A.g) : nullptr, d.d_f};
    run.gemm<T, LAYOUT_K, LAYOUT_K>("affine_gemm", pr, e);
    return;
  }

  // 6. per-head gate: G = [X, Delta] W_g^T + b_g (N = n_heads, fp32), then
  //    Y = X + sigmoid(G[head]) * Delta
  if (cfg->injection == PF_INJECT_GATED_HEAD) {
    const int64_t rows = (int64_t)d.B * d.L;
    float* gh = reinterpret_cast<float*>(act + A.gh);
    GemmProblem pr{};
    pr.a = x;
    pr.lda = d.d_f;
    pr.a2 = P(A.delta);
    pr.lda2 = d.d_f;
    pr.a_ksplit = d.d_f;
    pr.b = w->gate.w;
    pr.ldb = 2 * d.d_f;
    pr.M = (int)rows;
    pr.N = d.nh;
    pr.K = 2 * d.d_f;
    run.gemm<T, LAYOUT_K, LAYOUT_K>("head_gate_gemm", pr, EpiBiasF32<T>{gh, d.nh, reinterpret_cast<const T*>(w->gate.b)});
    run.launch("head_gate_combine", [&] {
      const int tpr = d.d_f / 8, rpb = tpr <= 256 ? 256 / tpr : 1;
      hipLaunchKernelGGL((head_gate_combine_kernel<T>), dim3((unsigned)std::min<int64_t>((rows + rpb - 1) / rpb, 16384)),
                         dim3(256), 0, run.stream, reinterpret_cast<const T*>(x), P(A.delta), gh,
                         reinterpret_cast<T*>(x_out), rows, d.d_f, d.nh);
      return hipGetLastError();
    });
    return;
  }

  // 5+6. level-1 decompression fused with the gated injection (Eq. 10, 12):
  //    C[p] = W_gd W_d1[p] and b'[p] = b_g + W_gd b_d1[p] for every position
  //    p < k_1, then one kernel forms Delta and G per tile and writes Y
  if constexpr (sizeof(T) == 2) {
    if (fuse) {
      const LayerWs W = layer_ws_layout(d, false);
      const int k1 = d.k[0], d1 = d.d[1];
      const T* wg = reinterpret_cast<const T*>(w->gate.w);
      T* cmat = reinterpret_cast<T*>(ws ? ws + W.gate_c : nullptr);
      float* bprime = reinterpret_cast<float*>(ws ? ws + W.gate_b : nullptr);
      {
        GemmProblem pc{};
        pc.a = wg ? wg + d.d_f : nullptr;  // W_gd: columns d_f .. 2 d_f of W_g
        pc.lda = 2 * d.d_f;
        pc.b = w->decompress[0].w;  // W_d1[p] read [c][n] (contiguous along n)
        pc.ldb = d1;
        pc.M = d.d_f;
        pc.N = d1;
        pc.K = d.d_f;
        pc.batch = k1;
        pc.batch_b = (int64_t)d.d_f * d1;
        run.gemm<T, LAYOUT_K, LAYOUT_MN>("gate_fold_gemm", pc, EpiStacked<T>{cmat, d1, d.d_f});
      }
      const T* bg = reinterpret_cast<const T*>(w->gate.b);
      const bool have_bd = w->decompress[0].b != nullptr;
      if (have_bd || run.dry) {  // the sizing run plans this GEMM whatever the bias
        GemmProblem pb{};
        pb.a = w->decompress[0].b;  // b_d1 viewed [k_1, d_f]
        pb.lda = d.d_f;
        pb.b = wg ? wg + d.d_f : nullptr;
        pb.ldb = 2 * d.d_f;
        pb.M = k1;
        pb.N = d.d_f;
        pb.K = d.d_f;
        run.gemm<T, LAYOUT_K, LAYOUT_K>("gate_fold_bias_gemm", pb, EpiBiasF32<T>{bprime, d.d_f, bg});
      }
      if (!have_bd) {
        run.launch("gate_fold_bias", [&] {
          const int64_t total = (int64_t)k1 * d.d_f;
          hipLaunchKernelGGL((gate_bias_broadcast_kernel<T>), dim3((unsigned)std::min<int64_t>((total + 255) / 256, 1024)),
                             dim3(256), 0, run.stream, bg, bprime, k1, d.d_f);
          return hipGetLastError();
        });
      }
      FusedGateParams fp{};
      fp.s = reinterpret_cast<const bf16*>(d.M == 1 ? P(A.s) : P(A.u[1]));
      fp.x = reinterpret_cast<const bf16*>(x);
      fp.wc = reinterpret_cast<const bf16*>(cmat);
      fp.wd = reinterpret_cast<const bf16*>(w->decompress[0].w);
      fp.wg = reinterpret_cast<const bf16*>(wg);
      fp.bias_g = bprime;
      fp.bias_d = reinterpret_cast<const bf16*>(w->decompress[0].b);
      fp.y = reinterpret_cast<bf16*>(x_out);
      fp.delta_out = saving ? reinterpret_cast<bf16*>(P(A.delta)) : nullptr;
      fp.g_out = saving ? reinterpret_cast<bf16*>(P(A.g)) : nullptr;
      fp.M = (int)(d.B * d.R[1]);
      fp.k = k1;
      fp.N = d.d_f;
      fp.Ks = d1;
      fp.lda_s = d1;
      fp.lda_x = (int64_t)k1 * d.d_f;
      fp.ldb_g = 2 * (int64_t)d.d_f;
      run.launch("fused_gate", [&] { return launch_fused_gate(fp, run.stream); });
      return;
    }
  }

  // 6. gated injection (Eq. 12)
  if (!add_inject) {
    GemmProblem pr{};
    pr.a = x;
    pr.lda = d.d_f;
    pr.a2 = P(A.delta);
    pr.lda2 = d.d_f;
    pr.a_ksplit = d.d_f;
    pr.b = w->gate.w;
    pr.ldb = 2 * d.d_f;
    pr.M = (int)(d.B * d.L);
    pr.N = d.d_f;
    pr.K = 2 * d.d_f;
    EpiGate<T> e{reinterpret_cast<const T*>(x), P(A.delta), reinterpret_cast<const T*>(w->gate.b),
                 reinterpret_cast<T*>(x_out), saving ? P(A.g) : nullptr, d.d_f};
    run.gemm<T, LAYOUT_K, LAYOUT_K>("gate_gemm", pr, e);
  }
}

template <typename T>
hipError_t layer_forward_run(const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                             const void* x, const void* h_in, void* x_out, void* h_out, char* acts, bool saving,
                             char* ws, hipStream_t stream) {
  const LayerWs W = layer_ws(d, false);
  Runner run(false, stream, reinterpret_cast<float*>(ws + W.gemm));
  forward_impl<T>(run, d, cfg, w, x, h_in, x_out, h_out, acts, saving, ws);
  return run.err;
}

size_t layer_forward_gemm_ws(const LayerDims& d) {
  pf_layer_config cfg{};
  cfg.mask = PF_TOKEN_CAUSAL;
  cfg.injection = d.inject;
  pf_layer_weights w{};
  Runner run(true);
  if (d.esize == 2)
    forward_impl<bf16>(run, d, &cfg, &w, nullptr, nullptr, nullptr, nullptr, nullptr, true, nullptr);
  else
    forward_impl<float>(run, d, &cfg, &w, nullptr, nullptr, nullptr, nullptr, nullptr, true, nullptr);
  return run.gemm_need;
}

template hipError_t layer_forward_run<bf16>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                            const void*, const void*, void*, void*, char*, bool, char*,
                                            hipStream_t);
template hipError_t layer_forward_run<float>(const LayerDims&, const pf_layer_config*, const pf_layer_weights*,
                                             const void*, const void*, void*, void*, char*, bool, char*,
                                             hipStream_t);

}  // namespace pf
