// Causal multi-head attention over the proxy sequence (Eq. 9) for gfx950.
#pragma once

#include "common.hpp"

namespace pf {

// Per-head tensors of one layer call. Heads are laid out [B, h, rows, d_head]
// ("row" tensors) or [B, h, d_head, ld_t] ("transposed" tensors, the proxy
// index contiguous with row stride ld_t >= m, a multiple of 64 whose padding
// columns hold zeros).
struct AttnParams {
  const void* q;    // [B, h, m, dh]
  const void* k;    // [B, h, m, dh]
  const void* q_lo; // optional low parts of the two-term split of Q and K
  const void* k_lo; //   (bf16 only): logits use Qh Kh + Ql Kh + Qh Kl
  const void* vt;   // [B, h, dh, ld_t]
  void* o;          // [B*m, h*dh] row-major (heads are column slices)
  float* lse;       // [B, h, m] natural-log log-sum-exp of the scaled scores
  int m, n_heads, ld_t;
  int causal;       // 1: key j visible to query i iff j <= i
  float scale_log2; // log2(e) / sqrt(dh)
};

template <typename T>
hipError_t launch_attention_fwd(const AttnParams& p, int batch, int head_dim, hipStream_t stream);

// Backward of Eq. 9 given dO and the forward's O and LSE. Row tensors q, k, v,
// do_ and transposed tensors qt, kt, dot (layouts as above). Writes dq, dk, dv
// in the activation dtype as [B*m, h*dh] row-major (heads are column slices);
// each value is accumulated in fp32 and rounded once. delta is scratch
// [B, h, m] fp32 for rowsum(dO * O).
struct AttnBwdParams {
  const void* q;
  const void* k;
  const void* q_lo;  // optional, as in AttnParams
  const void* k_lo;
  const void* v;
  const void* qt;
  const void* kt;
  const void* o;     // [B*m, h*dh]
  const void* do_;   // [B, h, m, dh]
  const void* dot;   // [B, h, dh, ld_t]
  const float* lse;
  float* delta;
  void* dq;
  void* dk;
  void* dv;
  int m, n_heads, ld_t;
  int causal;
  float scale_log2;
  float scale;
};

template <typename T>
hipError_t launch_attention_bwd(const AttnBwdParams& p, int batch, int head_dim, hipStream_t stream);

}  // namespace pf
