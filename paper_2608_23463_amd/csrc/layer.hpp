// Host-side planning shared by the layer entry points: derived sizes and the
// byte layout of the saved-activation region and the workspace.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "../../include/proxyformer.h"

namespace pf {

constexpr int kPlanCUs = 256;  // MI355X compute units; fixes split-K plans (and workspace sizes)

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct LayerDims {
  int B;
  int64_t L;        // tokens per sequence the kernels see: m * P (the last block zero-padded)
  int64_t L_in;     // tokens per sequence of the caller's tensors (<= L)
  int d_f, d_p, nh, dh;
  int M;            // levels
  int k[PF_MAX_LEVELS];
  int d[PF_MAX_LEVELS + 1];       // d[0] = d_fine ... d[M] = d_proxy
  int64_t R[PF_MAX_LEVELS + 1];   // rows per sequence after j levels; R[0] = L, R[M] = m
  int64_t P, m;
  int ld_t;         // row stride of transposed per-head tensors (m rounded up to 64)
  int esize;        // bytes per activation element
  int img_w, patch; // 2-D partition: image width and patch side (0 for sequences)
  int inject;       // pf_injection
  bool split;       // bf16 low parts on the proxy path (PF_PRECISION_EXTENDED in bf16 mode)
  bool fused_gate;  // level-1 decompression and the gate run as one kernel (bf16, gated injection)
  // the caller's token tensors go through workspace copies (padded or patch-ordered)
  bool staged() const { return L_in != L || img_w > 0; }
};

// Byte offsets of every activation inside the region that holds them
// (the caller's `saved` buffer, or the workspace when saved is NULL).
// With PF_PRECISION_EXTENDED in bf16 mode the proxy path upstream of the
// attention logits (Z_j, H, Q, K) also keeps the low part of a two-term bf16
// split (the *_lo buffers): a proxy sums P * d_fine products, so its
// magnitude, and the logits', grow with the compression fan-in, and one bf16
// rounding there moves a sharp softmax by several percent. The forward
// attention reads the Q and K remainders as fp8 correction rows (qx, kx);
// the bf16 low parts of Q and K are kept only for the backward. In fp32 mode
// and with PF_PRECISION_BF16 the *_lo, qx and kx buffers are empty.
struct LayerActs {
  size_t z[PF_MAX_LEVELS];    // Z_j, j = 1..M-1: compression level outputs [B*R_j, d_j]
  size_t z_lo[PF_MAX_LEVELS];
  size_t h;                   // H = H_in + c [B*m, d_p] (copy kept for the backward)
  size_t h_lo;
  size_t q, k, v;             // [B, h, m, dh]
  size_t q_lo, k_lo;
  size_t qs;                  // Q * log2(e)/sqrt(d_head) for the forward attention [B, h, m, dh]
                              // (the same buffer as q unless activations are saved)
  size_t qx, kx;              // extended precision: fp8 correction rows of scaled Q and of K
                              // [B, h, m, 2 dh] bytes (see EpiHeads)
  size_t qt, kt, vt;          // [B, h, dh, ld_t]
  size_t o;                   // [B*m, d_p]
  size_t lse;                 // [B, h, m] fp32
  size_t s;                   // S [B*m, d_p]: the contextualised proxy each block receives
  size_t u[PF_MAX_LEVELS];    // U_j, j = 1..M-1: decompression level outputs [B*R_j, d_j]
  size_t delta;               // [B*L, d_f] (absent for residual addition, and in a forward with the fused gate)
  size_t g;                   // gate pre-activation G, or s of Eq. 13 [B*L, d_f]
  size_t rstd;                // Eq. 13: 1 / RMS of every X row, fp32 [B*L]
  size_t gh;                  // per-head gate pre-activation, fp32 [B*L, n_heads]
  size_t aff_w, aff_b;        // Eq. 13: W_a, b_a with s and t rows interleaved [2 d_f, d_f], [2 d_f]
  size_t bytes;
};

struct LayerWs {
  size_t gate_c, gate_b;     // fused gate: C [k_1 d_f, d_1] and b' [k_1, d_f] fp32
  size_t acts;      // forward activations when saved == NULL
  size_t gemm;      // split-K partials
  // backward scratch
  size_t dg, ddelta;          // dG, dDelta [B*L, d_f]
  size_t dx32;                // fp32 accumulator of dX [B*L, d_f]
  size_t du[PF_MAX_LEVELS];   // dU_j j = 1..M-1 [B*R_j, d_j]
  size_t dhbar;               // gradient of the W_o output (shift undone) [B*m, d_p]
  size_t dO, dOt;             // [B, h, m, dh], [B, h, dh, ld_t]
  size_t delta_rs;            // rowsum(dO * O) [B, h, m] fp32
  size_t dq, dk, dv;          // [B*m, d_p]
  size_t dh32;                // fp32 accumulator of dH [B*m, d_p]
  size_t dh;                  // dH in the activation dtype [B*m, d_p]
  size_t dz[PF_MAX_LEVELS];   // dZ_j j = 1..M-1 [B*R_j, d_j]
  size_t colsum;              // bias-gradient partial column sums
  size_t colsum2;             // second-stage partials (64 groups)
  size_t tr_a, tr_b;          // transposed GEMM operands of the large weight gradients [cols, rows]
  size_t tr_w;                // a transposed weight [in, out] for the large data gradients
  // staged token tensors (L_in < L: zero-padded to L tokens; 2-D partition:
  // in patch order)
  size_t x_pad;               // X with zero padding [B*L, d_f]
  size_t y_pad;               // forward: X_out; backward: dX [B*L, d_f]
  size_t dy_pad;              // backward: dY with zero padding [B*L, d_f]
  size_t dst;                 // Eq. 13 backward: [dS | dT] [B*L, 2 d_f]
  size_t dgh;                 // per-head gate backward: dG [B*L, round8(n_heads)]
  size_t bytes;
};

constexpr int kColsumChunks = 512;
// Weight and data gradients over at least this many rows run on transposed
// (K-contiguous) operand copies through the direct GEMM kernel.
constexpr int64_t kTransposeMinRows = 8192;
// fp32 weight gradients: a transposed copy's rows are runs of `rows` tokens,
// and a K-contiguous GEMM operand row may span at most 8 MiB (256 tile rows
// in one 32-bit buffer range), so longer runs keep the M/N-contiguous loads.
inline bool wgrad_transposes(int64_t rows, int64_t esize) {
  return rows >= kTransposeMinRows && rows * esize <= ((int64_t)1 << 23);
}
inline int64_t round8(int64_t v) { return (v + 7) / 8 * 8; }

// dst[b, t] = t < L_in ? src[b, t] : 0 for t < L_pad, rows of row_bytes (a
// multiple of 16) with per-sequence strides L_in and L_pad rows.
hipError_t pad_rows(const void* src, void* dst, int B, int64_t L_in, int64_t L_pad, int64_t row_bytes,
                    hipStream_t stream);
// dst[b, t] = src[b, t] for t < L_in (the first L_in of L_pad rows per sequence).
hipError_t unpad_rows(const void* src, void* dst, int B, int64_t L_in, int64_t L_pad, int64_t row_bytes,
                      hipStream_t stream);

// 2-D partition: position j of the patch-ordered sequence holds raster
// token perm(j) of an image of width w with p x p patches. Gather:
// dst[b, j] = src[b, perm(j)]; scatter: dst[b, perm(j)] = src[b, j].
hipError_t permute_patches(const void* src, void* dst, int B, int64_t L, int w, int p, int64_t row_bytes,
                           bool scatter, hipStream_t stream);

// Validates cfg; on failure returns a status and writes a message.
int layer_dims(const pf_layer_config* cfg, LayerDims* d, const char** why);
LayerActs layer_acts(const LayerDims& d, bool for_backward);
// Workspace offsets without the split-K region (gemm == bytes == end of the
// fixed buffers); layer_ws adds the split-K region sized by a dry run.
LayerWs layer_ws_layout(const LayerDims& d, bool for_backward);
LayerWs layer_ws(const LayerDims& d, bool for_backward);
size_t layer_forward_gemm_ws(const LayerDims& d);
size_t layer_backward_gemm_ws(const LayerDims& d);

template <typename T>
hipError_t layer_forward_run(const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                             const void* x, const void* h_in, void* x_out, void* h_out, char* acts,
                             bool saving, char* ws, hipStream_t stream);

template <typename T>
hipError_t layer_backward_run(const LayerDims& d, const pf_layer_config* cfg, const pf_layer_weights* w,
                              const void* x, const void* h_in, const char* saved, const void* dy,
                              const void* dh_out, void* dx, void* dh_in, const pf_layer_grads* gr,
                              char* ws, hipStream_t stream);

size_t layer_gemm_ws_bytes(const LayerDims& d, bool for_backward);

}  // namespace pf
