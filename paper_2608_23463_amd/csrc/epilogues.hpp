// GEMM epilogues used by the layer and decode paths. Each is a functor
// epi(row, col, acc) applied to one fp32 result of C = A B^T.
#pragma once

#include "common.hpp"

namespace pf {

// out[r, c] = acc + bias[c] (+ add[r, c]); optional second copy out2.
// out_lo (bf16 only, optional): low part of the two-term split of the result.
template <typename T>
struct EpiLinear {
  T* out;
  int64_t ldo;
  const T* bias;
  const T* add;
  int64_t ld_add;
  T* out2;
  T* out_lo;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    if (add) v += to_f32(add[(int64_t)r * ld_add + c]);
    const T o = from_f32<T>(v);
    out[(int64_t)r * ldo + c] = o;
    if (out2) out2[(int64_t)r * ldo + c] = o;
    if (out_lo) out_lo[(int64_t)r * ldo + c] = from_f32<T>(split_lo(v));
  }
  struct Col {
    Raw8<T> b;
  };
  struct Pre {
    Raw8<T> a;
  };
  __device__ __forceinline__ void col(int c, Col& k) const {
    if (bias) raw_load8(bias + c, k.b);
  }
  __device__ __forceinline__ void pre(int r, int c, Pre& q) const {
    if (add) raw_load8(add + (int64_t)r * ld_add + c, q.a);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0, const Col& k, const Pre& q) const {
    float v[8], t[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e];
    if (bias) {
      raw_to_f32(k.b, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += t[e];
    }
    if (add) {
      raw_to_f32(q.a, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += t[e];
    }
    finish(r, c, v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float v[8], t[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e];
    if (bias) {
      load8(bias + c, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += t[e];
    }
    if (add) {
      load8(add + (int64_t)r * ld_add + c, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += t[e];
    }
    finish(r, c, v);
  }
  __device__ __forceinline__ void finish(int r, int c, const float* v) const {
    float t[8];
    store8(out + (int64_t)r * ldo + c, v);
    if (out2) store8(out2 + (int64_t)r * ldo + c, v);
    if (out_lo) {
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = split_lo(v[e]);
      store8(out_lo + (int64_t)r * ldo + c, t);
    }
  }
};

// Splits a [B*m, h*dh] projection into per-head tensors: row r = b*m + i,
// column c = head*dh + e. `out` is [B, h, m, dh], `out_t` is [B, h, dh, ld_t].
// Optionally also a scaled copy (v * scale) in the row layout, `outs`.
template <typename T>
struct EpiHeads {
  T* out;
  T* out_t;
  const T* bias;
  int m, dh, n_heads, ld_t;
  T* out_lo;  // optional low part of the split, row layout
  T* outs = nullptr;
  float scale = 1.0f;
  // fp8 (e5m2) operand of the attention's correction product, rows of 2 dh
  // bytes [B, h, m, 2 dh] (bf16 only). With hi = bf16(x) and lo = x - hi of
  // the value x the attention reads (x = v * scale for Q, v for K):
  // xmode 1 writes [fp8(256 lo) | fp8(hi)], xmode 2 writes [fp8(hi) |
  // fp8(256 lo)], so the dot product of a Q row and a K row is
  // 256 (Ql Kh + Qh Kl).
  uint8_t* outx = nullptr;
  int xmode = 0;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    const T o = from_f32<T>(v);
    const int b = r / m, i = r - b * m;
    const int hd = c / dh, e = c - hd * dh;
    const int64_t bh = (int64_t)b * n_heads + hd;
    if (out) out[(bh * m + i) * dh + e] = o;
    if (out_t) out_t[(bh * dh + e) * ld_t + i] = o;
    if (out_lo) out_lo[(bh * m + i) * dh + e] = from_f32<T>(split_lo(v));
    if (outs) outs[(bh * m + i) * dh + e] = from_f32<T>(v * scale);
    if (outx) {
      const float x = xmode == 1 ? v * scale : v;
      const float hi = (float)(bf16)x, lo = (x - hi) * 256.0f;
      uint8_t* row = outx + (bh * m + i) * 2 * dh;
      row[e] = (uint8_t)pack_bf8x4(xmode == 1 ? lo : hi, 0.0f, 0.0f, 0.0f);
      row[dh + e] = (uint8_t)pack_bf8x4(xmode == 1 ? hi : lo, 0.0f, 0.0f, 0.0f);
    }
  }
  struct Col {
    Raw8<T> b;
  };
  struct Pre {};
  __device__ __forceinline__ void col(int c, Col& k) const {
    if (bias) raw_load8(bias + c, k.b);
  }
  __device__ __forceinline__ void pre(int, int, Pre&) const {}
  __device__ __forceinline__ void vec8(int r, int c, const float* v0, const Col& k, const Pre&) const {
    float v[8], t[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (bias) raw_to_f32(k.b, t);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e] + t[e];
    finish(r, c, v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float v[8], t[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (bias) load8(bias + c, t);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e] + t[e];
    finish(r, c, v);
  }
  // 8 consecutive channels stay inside one head (dh is a multiple of 8)
  __device__ __forceinline__ void finish(int r, int c, const float* v) const {
    const int b = r / m, i = r - b * m;
    const int hd = c / dh, e0 = c - hd * dh;
    const int64_t bh = (int64_t)b * n_heads + hd;
    if (out) store8(out + (bh * m + i) * dh + e0, v);
    if (out_lo) {
      float t[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) t[e] = split_lo(v[e]);
      store8(out_lo + (bh * m + i) * dh + e0, t);
    }
    if (outs) {
      float s[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] = v[e] * scale;
      store8(outs + (bh * m + i) * dh + e0, s);
    }
    if (out_t) {
#pragma unroll
      for (int e = 0; e < 8; ++e) out_t[(bh * dh + e0 + e) * ld_t + i] = from_f32<T>(v[e]);
    }
    if (outx) {
      float hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = xmode == 1 ? v[e] * scale : v[e];
        hi[e] = (float)(bf16)x;
        lo[e] = (x - hi[e]) * 256.0f;
      }
      const float* first = xmode == 1 ? lo : hi;
      const float* second = xmode == 1 ? hi : lo;
      uint8_t* row = outx + (bh * m + i) * 2 * dh;
      typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
      *reinterpret_cast<u32x2_t*>(row + e0) =
          u32x2_t{pack_bf8x4(first[0], first[1], first[2], first[3]), pack_bf8x4(first[4], first[5], first[6], first[7])};
      *reinterpret_cast<u32x2_t*>(row + dh + e0) = u32x2_t{pack_bf8x4(second[0], second[1], second[2], second[3]),
                                                           pack_bf8x4(second[4], second[5], second[6], second[7])};
    }
  }
};

// Output map of the interaction with the token-causal shift folded in: row
// r = b*m + i of H-bar goes to row r + 1 of S (the proxy block i + 1 receives);
// the row i = m - 1 has no receiver and instead clears row b*m (block 0
// receives zero). Every row of S is written exactly once.
template <typename T>
struct EpiShift {
  T* out;
  const T* bias;
  int m, ld;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    const int i = r % m;
    if (i < m - 1)
      out[(int64_t)(r + 1) * ld + c] = from_f32<T>(v);
    else
      out[(int64_t)(r - i) * ld + c] = from_f32<T>(0.0f);
  }
  struct Col {
    Raw8<T> b;
  };
  struct Pre {};
  __device__ __forceinline__ void col(int c, Col& k) const {
    if (bias) raw_load8(bias + c, k.b);
  }
  __device__ __forceinline__ void pre(int, int, Pre&) const {}
  __device__ __forceinline__ void vec8(int r, int c, const float* v0, const Col& k, const Pre&) const {
    float v[8], t[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (bias) raw_to_f32(k.b, t);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e] + t[e];
    finish(r, c, v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float v[8], t[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (bias) load8(bias + c, t);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e] + t[e];
    finish(r, c, v);
  }
  __device__ __forceinline__ void finish(int r, int c, const float* v) const {
    const int i = r % m;
    if (i < m - 1) {
      store8(out + (int64_t)(r + 1) * ld + c, v);
    } else {
      const float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      store8(out + (int64_t)(r - i) * ld + c, z);
    }
  }
};

// Gated injection (Eq. 12): G = acc + b_g; Y = X + sigmoid(G) * Delta.
template <typename T>
struct EpiGate {
  const T* x;
  const T* delta;
  const T* bias;
  T* y;
  T* gsave;
  int64_t ld;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    const int64_t i = (int64_t)r * ld + c;
    const float xv = to_f32(x[i]);
    const float dv = to_f32(delta[i]);
    y[i] = from_f32<T>(xv + sigmoidf(v) * dv);
    if (gsave) gsave[i] = from_f32<T>(v);
  }
  // Two-phase form: col() reads the bias, pre() the 8 values of X and Delta.
  struct Col {
    Raw8<T> b;
  };
  struct Pre {
    Raw8<T> x8, d8;
  };
  __device__ __forceinline__ void col(int c, Col& k) const {
    if (bias) raw_load8(bias + c, k.b);
  }
  __device__ __forceinline__ void pre(int r, int c, Pre& q) const {
    const int64_t i = (int64_t)r * ld + c;
    raw_load8(x + i, q.x8);
    raw_load8(delta + i, q.d8);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0, const Col& k, const Pre& q) const {
    float xv[8], dv[8], bv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    raw_to_f32(q.x8, xv);
    raw_to_f32(q.d8, dv);
    if (bias) raw_to_f32(k.b, bv);
    finish(r, c, v0, xv, dv, bv);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float xv[8], dv[8], bv[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int64_t i = (int64_t)r * ld + c;
    load8(x + i, xv);
    load8(delta + i, dv);
    if (bias) load8(bias + c, bv);
    finish(r, c, v0, xv, dv, bv);
  }
  __device__ __forceinline__ void finish(int r, int c, const float* v0, const float* xv, const float* dv,
                                         const float* bv) const {
    float g[8], yv[8];
    const int64_t i = (int64_t)r * ld + c;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      g[e] = v0[e] + bv[e];
      yv[e] = xv[e] + sigmoidf(g[e]) * dv[e];
    }
    store8(y + i, yv);
    if (gsave) store8(gsave + i, g);
  }
};

// out[(z M + r) ldo + c] = acc for batch z = blockIdx.y of a batched GEMM:
// the batches' [M, N] results stacked along rows.
template <typename T>
struct EpiStacked {
  T* out;
  int64_t ldo;
  int M;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    out[((int64_t)blockIdx.y * M + r) * ldo + c] = from_f32<T>(v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    store8(out + ((int64_t)blockIdx.y * M + r) * ldo + c, v);
  }
};

// fp32 out[r, c] = acc + bias[c] (bias in the activation type, optional).
template <typename T>
struct EpiBiasF32 {
  float* out;
  int ldo;
  const T* bias;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    out[(int64_t)r * ldo + c] = v + (bias ? to_f32(bias[c]) : 0.0f);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
#pragma unroll
    for (int e = 0; e < 8; ++e) (*this)(r, c + e, v[e]);
  }
};

constexpr float kAffineEps = 1e-6f;  // RMSNorm epsilon of Eq. 13

// Affine modulation (Eq. 13) on the GEMM [S | T] = Delta W_a^T + b_a with s
// and t interleaved per channel (columns 2c, 2c+1): y[r, c] = (1 + s) *
// x[r, c] * rstd[r] + t; optionally s is kept for the backward. The GEMM's
// N = 2 d_fine is a multiple of 16 (d_fine % 8 == 0), so every store goes
// through vec8 and covers 4 whole channels; the scalar form is never called.
template <typename T>
struct EpiAffine {
  const T* x;
  const float* rstd;
  const T* bias;  // interleaved [2 d_fine]
  T* y;
  T* ssave;       // [rows, d_fine] or NULL
  int d;
  __device__ __forceinline__ void operator()(int, int, float) const {}
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    const int ch = c >> 1;
    const int64_t i = (int64_t)r * d + ch;
    float b[8], xv[4], yv[4], sv[4];
    load8(bias + c, b);
    load4(x + i, xv);
    const float rs = rstd[r];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float s = v[2 * e] + b[2 * e], t = v[2 * e + 1] + b[2 * e + 1];
      sv[e] = s;
      yv[e] = fmaf(1.0f + s, xv[e] * rs, t);
    }
    store4(y + i, yv);
    if (ssave) store4(ssave + i, sv);
  }
};

// fp32 store with optional accumulation into what is there (fixed order:
// one writer per element per launch, launches ordered on the stream).
struct EpiF32 {
  float* out;
  int64_t ldo;
  int accumulate;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    float* p = out + (int64_t)r * ldo + c;
    *p = accumulate ? *p + v : v;
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float* p = out + (int64_t)r * ldo + c;
    if ((ldo & 3) != 0) {
      for (int e = 0; e < 8; ++e) (*this)(r, c + e, v0[e]);
      return;
    }
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e];
    if (accumulate) {
      float t[8];
      load8(p, t);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += t[e];
    }
    store8(p, v);
  }
};

}  // namespace pf
