// GEMM epilogues used by the layer and decode paths. Each is a functor
// epi(row, col, acc) applied to one fp32 result of C = A B^T.
#pragma once

#include "common.hpp"

namespace pf {

// out[r, c] = acc + bias[c] (+ add[r, c]); optional second copy out2.
template <typename T>
struct EpiLinear {
  T* out;
  int64_t ldo;
  const T* bias;
  const T* add;
  int64_t ld_add;
  T* out2;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    if (add) v += to_f32(add[(int64_t)r * ld_add + c]);
    const T o = from_f32<T>(v);
    out[(int64_t)r * ldo + c] = o;
    if (out2) out2[(int64_t)r * ldo + c] = o;
  }
};

// Splits a [B*m, h*dh] projection into per-head tensors: row r = b*m + i,
// column c = head*dh + e. `out` is [B, h, m, dh], `out_t` is [B, h, dh, ld_t].
template <typename T>
struct EpiHeads {
  T* out;
  T* out_t;
  const T* bias;
  int m, dh, n_heads, ld_t;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    const T o = from_f32<T>(v);
    const int b = r / m, i = r - b * m;
    const int hd = c / dh, e = c - hd * dh;
    const int64_t bh = (int64_t)b * n_heads + hd;
    if (out) out[(bh * m + i) * dh + e] = o;
    if (out_t) out_t[(bh * dh + e) * ld_t + i] = o;
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
};

}  // namespace pf
