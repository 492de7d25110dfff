// Causal multi-head attention over the proxy sequence (Eq. 9) for gfx950.
#pragma once

#include "common.hpp"

namespace pf {

// Physical 16-byte chunk of logical chunk c in row r of an LDS tile whose
// rows hold C chunks (C a power of two). A 16-byte read serves 16 lanes per
// pass over 64 banks, i.e. 16 chunk slots of 256 bytes, and the fragment
// reads put 16 consecutive rows (same logical chunk) in one pass: the XOR
// term walks through all C chunks as r steps over the 16 / C rows that share
// a 256-byte span, so the 16 rows land on 16 different slots.
template <int C>
__device__ __forceinline__ int lds_swz(int r, int c) {
  static_assert(C >= 4 && (C & (C - 1)) == 0, "rows of 4, 8, 16, ... chunks");
  return C >= 16 ? c ^ (r & 15) : c ^ ((r / (16 / C)) & (C - 1));
}

// acc + 2^-8 A B^T for one 32x32 block of fp8 e5m2 operands over 64 K
// elements: lane l supplies row l % 32 of A and of B, bytes
// [32 (l / 32), +32) of the block's 64 (the same convention on both sides,
// so the products pair up whatever order the hardware takes them in; checked
// on the device against a host product). The 2^-8 is B's block scale.
typedef int i32x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ f32x16 mfma_bf8_scaled(const i32x8& a, const i32x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 1, 1, 0, 127, 0, 119);
}

// Value of lane l ^ 32 (the other half of the wave), through the VALU.
__device__ __forceinline__ float other_half(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __builtin_bit_cast(float, (__lane_id() < 32) ? r[1] : r[0]);
}

// P^T operand of one 16-key MFMA step taken from a 32x32 S^T accumulator
// (keys on rows, queries on lanes). The accumulator gives a lane runs of 4
// keys: registers 8*s2 .. 8*s2+7 hold keys 16*s2 + {0..3, 8..11} in the lower
// lane half and 16*s2 + {4..7, 12..15} in the upper half. One
// v_permlane32_swap per register pair exchanges keys 8..11 (lower half) with
// keys 4..7 (upper half), so lane group g holds keys 16*s2 + 8*g .. +7 in order,
// the operand layout whose matching V^T fragment is one contiguous 16-byte
// read (bf16 operands).
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  // one v_cvt_pk_bf16_f32 (round to nearest even)
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
__device__ __forceinline__ bf16x8 pt_frag_bf16(const f32x16& s, int s2) {
  const int r0 = s2 * 8;
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(s[r0 + 2 * i], s[r0 + 2 * i + 1]);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const auto x = __builtin_amdgcn_permlane32_swap(w[i], w[i + 2], false, false);
    w[i] = x[0];
    w[i + 2] = x[1];
  }
  return __builtin_bit_cast(bf16x8, w);
}

// Per-head tensors of one layer call. Heads are laid out [B, h, rows, d_head]
// ("row" tensors) or [B, h, d_head, ld_t] ("transposed" tensors, the proxy
// index contiguous with row stride ld_t >= m, a multiple of 64 whose padding
// columns hold zeros).
struct AttnParams {
  const void* q;    // [B, h, m, dh], pre-scaled by log2(e) / sqrt(dh)
  const void* k;    // [B, h, m, dh]
  const void* qx;   // optional (bf16 only): fp8 e5m2 correction rows [B, h, m, 2 dh]
  const void* kx;   //   of the split logits, whose products are 256 (Ql Kh + Qh Kl)
  const void* vt;   // [B, h, dh, ld_t]
  void* o;          // [B*m, h*dh] row-major (heads are column slices)
  float* lse;       // [B, h, m] natural-log log-sum-exp of the scores Q.K / sqrt(dh)
  int m, n_heads, ld_t;
  int causal;       // 1: key j visible to query i iff j <= i
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
  const void* q_lo;  // optional bf16 low parts of the split (logits Qh Kh + Ql Kh + Qh Kl)
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
