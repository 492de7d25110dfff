// Flash-style causal multi-head attention over proxies (Eq. 9), forward.
//
// One workgroup = 4 waves = 128 queries of one (sequence, head); each wave owns
// 32 queries. Keys/values stream through LDS 64 at a time (double buffered).
// A wave computes the transposed score tile S^T = K Q^T with MFMA so that each
// lane holds one query column: the online-softmax statistics of a query live
// in one lane pair (lane, lane ^ 32), and only the running maximum needs one
// cross-half exchange per tile. The probabilities P^T stay in registers and
// feed O^T += V^T P^T directly as the B operand; V arrives key-contiguous
// (the producing GEMM writes V transposed), so the A fragments are plain LDS
// reads. Exponentials use exp2 with log2(e)/sqrt(d_head) folded into the
// score scale. With SPLIT, Q and K arrive as bf16 hi/lo pairs and the scores
// are Kh Qh + Kl Qh + Kh Ql (three MFMAs into one accumulator), so a sharp
// softmax is not moved by one bf16 rounding of its logits. Masked scores are
// -inf and contribute exactly zero, so a query
// never depends on later proxies (bit-exact causality).
#include "attention.hpp"

namespace pf {

template <typename T, int DH, bool SPLIT>
struct AttnFwdShape {
  static constexpr int kVec = 16 / sizeof(T);
  static constexpr int kKT = 64;                    // keys per tile
  static constexpr int kKStride = DH + kVec;        // K tile row stride
  static constexpr int kVStride = kKT + kVec;       // V^T tile row stride
  static constexpr int kKElems = kKT * kKStride;
  static constexpr int kKParts = SPLIT ? 2 : 1;     // K hi (and lo) tiles
  static constexpr int kVOff = kKParts * kKElems;
  static constexpr int kStage = kVOff + DH * kVStride;
  static constexpr int kKLoads = kKT * DH / (256 * kVec);
  static constexpr int kVLoads = DH * kKT / (256 * kVec);
};

template <typename T>
struct Quad;  // four consecutive elements
template <>
struct Quad<bf16> {
  typedef uint2 type;
};
template <>
struct Quad<float> {
  typedef u32x4 type;
};

template <typename T, int DH, bool SPLIT>
__global__ void __launch_bounds__(256) attn_fwd_kernel(const AttnParams p) {
  typedef AttnFwdShape<T, DH, SPLIT> S;
  typedef Mma<T> MM;
  __shared__ __attribute__((aligned(16))) T smem[2 * S::kStage];

  const int nqt = (p.m + 127) / 128;
  const int qt = nqt - 1 - (int)blockIdx.x;  // longest causal rows first
  const int bh = blockIdx.y;
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;
  const int q0 = qt * 128;
  const int qw0 = q0 + wave * 32;
  const int myq = qw0 + col;

  const T* qp = reinterpret_cast<const T*>(p.q) + (int64_t)bh * p.m * DH;
  const T* kp = reinterpret_cast<const T*>(p.k) + (int64_t)bh * p.m * DH;
  const T* qlp = SPLIT ? reinterpret_cast<const T*>(p.q_lo) + (int64_t)bh * p.m * DH : nullptr;
  const T* klp = SPLIT ? reinterpret_cast<const T*>(p.k_lo) + (int64_t)bh * p.m * DH : nullptr;
  const T* vtp = reinterpret_cast<const T*>(p.vt) + (int64_t)bh * DH * p.ld_t;

  typename MM::frag qf[DH / 16], qfl[SPLIT ? DH / 16 : 1];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (myq < p.m) {
      qf[kk] = MM::load(qp + (int64_t)myq * DH + kk * 16 + g * 8);
      if constexpr (SPLIT) qfl[kk] = MM::load(qlp + (int64_t)myq * DH + kk * 16 + g * 8);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        qf[kk][i] = (T)0.0f;
        if constexpr (SPLIT) qfl[kk][i] = (T)0.0f;
      }
    }
  }

  const int kv_end = p.causal ? min(p.m, q0 + 128) : p.m;
  const int ntiles = (kv_end + S::kKT - 1) / S::kKT;

  u32x4 rk[S::kKParts][S::kKLoads], rv[S::kVLoads];
  auto fetch = [&](int kt0) {
    constexpr int kc = DH / S::kVec;
#pragma unroll
    for (int part = 0; part < S::kKParts; ++part) {
      const T* src = part == 0 ? kp : klp;
#pragma unroll
      for (int i = 0; i < S::kKLoads; ++i) {
        const int v = tid + i * 256;
        const int key = kt0 + v / kc;
        u32x4 val = {0u, 0u, 0u, 0u};
        if (key < p.m) val = ld16(src + (int64_t)key * DH + (v % kc) * S::kVec);
        rk[part][i] = val;
      }
    }
    constexpr int vc = S::kKT / S::kVec;
#pragma unroll
    for (int i = 0; i < S::kVLoads; ++i) {
      const int v = tid + i * 256;
      rv[i] = ld16(vtp + (int64_t)(v / vc) * p.ld_t + kt0 + (v % vc) * S::kVec);
    }
  };
  auto stash = [&](T* st) {
    constexpr int kc = DH / S::kVec;
#pragma unroll
    for (int part = 0; part < S::kKParts; ++part)
#pragma unroll
      for (int i = 0; i < S::kKLoads; ++i) {
        const int v = tid + i * 256;
        st16(st + part * S::kKElems + (v / kc) * S::kKStride + (v % kc) * S::kVec, rk[part][i]);
      }
    constexpr int vc = S::kKT / S::kVec;
#pragma unroll
    for (int i = 0; i < S::kVLoads; ++i) {
      const int v = tid + i * 256;
      st16(st + S::kVOff + (v / vc) * S::kVStride + (v % vc) * S::kVec, rv[i]);
    }
  };

  f32x16 oacc[DH / 32];
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[cb][r] = 0.0f;
  float mrun = -INFINITY, lrun = 0.0f;

  fetch(0);
  stash(smem);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int kt0 = t * S::kKT;
    const bool more = t + 1 < ntiles;
    if (more) fetch(kt0 + S::kKT);
    const T* sk = smem + (t & 1) * S::kStage;
    const T* sv = sk + S::kVOff;
    const bool active = !p.causal || kt0 <= qw0 + 31;  // uniform across the wave
    if (active) {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < DH / 16; ++kk) {
          const int off = (kb * 32 + col) * S::kKStride + kk * 16 + g * 8;
          const typename MM::frag kh = MM::load(sk + off);
          s[kb] = MM::mma(kh, qf[kk], s[kb]);
          if constexpr (SPLIT) {
            s[kb] = MM::mma(MM::load(sk + S::kKElems + off), qf[kk], s[kb]);
            s[kb] = MM::mma(kh, qfl[kk], s[kb]);
          }
        }
      }
      const bool need_mask = (p.causal && kt0 + S::kKT - 1 > qw0) || kt0 + S::kKT > p.m;
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float v = s[kb][r] * p.scale_log2;
          if (need_mask) {
            const int key = kt0 + kb * 32 + acc_row(r, lane);
            if (key >= p.m || (p.causal && key > myq)) v = -INFINITY;
          }
          s[kb][r] = v;
          mt = fmaxf(mt, v);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      const float mnew = fmaxf(mrun, mt);
      const float alpha = fast_exp2(mrun - mnew);
      mrun = mnew;
      float ls = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = fast_exp2(s[kb][r] - mnew);
          s[kb][r] = e;
          ls += e;
        }
      lrun = lrun * alpha + ls;
#pragma unroll
      for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          float pv[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) pv[i] = s[kb][s2 * 8 + i];
          const typename MM::frag pb = MM::pack(pv);
#pragma unroll
          for (int cb = 0; cb < DH / 32; ++cb) {
            const T* vrow = sv + (cb * 32 + col) * S::kVStride + kb * 32 + s2 * 16 + g * 4;
            typename MM::frag va;
            typedef typename Quad<T>::type QT;
            const QT lo = *reinterpret_cast<const QT*>(vrow);
            const QT hi = *reinterpret_cast<const QT*>(vrow + 8);
            *reinterpret_cast<QT*>(&va) = lo;
            *(reinterpret_cast<QT*>(&va) + 1) = hi;
            oacc[cb] = MM::mma(va, pb, oacc[cb]);
          }
        }
    }
    if (more) stash(smem + ((t + 1) & 1) * S::kStage);
    __syncthreads();
  }

  const float ltot = lrun + __shfl_xor(lrun, 32);
  if (myq < p.m) {
    const float inv = 1.0f / ltot;
    T* orow = reinterpret_cast<T*>(p.o) + ((int64_t)b * p.m + myq) * ((int64_t)p.n_heads * DH) + h * DH;
#pragma unroll
    for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[cb * 32 + acc_row(r, lane)] = from_f32<T>(oacc[cb][r] * inv);
    if (g == 0) p.lse[(int64_t)bh * p.m + myq] = (mrun + __log2f(ltot)) * 0.69314718055994531f;
  }
}

template <typename T>
hipError_t launch_attention_fwd(const AttnParams& p, int batch, int head_dim, hipStream_t stream) {
  if (p.m <= 0) return hipSuccess;
  dim3 grid((p.m + 127) / 128, batch * p.n_heads);
  const bool split = sizeof(T) == 2 && p.q_lo && p.k_lo;
  if (head_dim == 64) {
    if (split)
      hipLaunchKernelGGL((attn_fwd_kernel<T, 64, sizeof(T) == 2>), grid, dim3(256), 0, stream, p);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<T, 64, false>), grid, dim3(256), 0, stream, p);
  } else {
    if (split)
      hipLaunchKernelGGL((attn_fwd_kernel<T, 128, sizeof(T) == 2>), grid, dim3(256), 0, stream, p);
    else
      hipLaunchKernelGGL((attn_fwd_kernel<T, 128, false>), grid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

template hipError_t launch_attention_fwd<bf16>(const AttnParams&, int, int, hipStream_t);
template hipError_t launch_attention_fwd<float>(const AttnParams&, int, int, hipStream_t);

}  // namespace pf
