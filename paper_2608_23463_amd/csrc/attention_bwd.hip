// Backward of the causal multi-head proxy attention (Eq. 9).
//
// With P = softmax(S), S = Q K^T / sqrt(d_head) + M and D_i = sum_c dO_ic O_ic:
//   dV = P^T dO,  dP = dO V^T,  dS = P * (dP - D),  dQ = dS K / sqrt(d_head),
//   dK = dS^T Q / sqrt(d_head).
// P is recomputed from the forward's log-sum-exp. Two kernels, no atomics,
// so every gradient is written once and results are deterministic:
//  - attn_bwd_dkdv_kernel: a workgroup owns 128 keys (4 waves x 32, one key
//    per lane); it walks the query tiles that can see those keys and
//    accumulates dV^T += dO^T P and dK^T += Q^T dS in registers.
//  - attn_bwd_dq_kernel: a workgroup owns 128 queries (one per lane) and walks
//    the visible key tiles, accumulating dQ^T += K^T dS^T.
// Probabilities and dS stay in registers and feed the next MFMA directly as
// its B operand (same key/query permutation on both operands, as in the
// forward kernel). The transposed operands (Q^T, K^T, dO^T) are produced
// key/query-contiguous by the GEMM epilogues, so every MFMA fragment is a
// plain LDS read. With SPLIT (bf16 hi/lo parts of Q and K) the recomputed
// scores are Qh Kh + Ql Kh + Qh Kl, matching the forward's logits.
#include "attention.hpp"

namespace pf {

template <typename T>
struct QuadB;
template <>
struct QuadB<bf16> {
  typedef uint2 type;
};
template <>
struct QuadB<float> {
  typedef u32x4 type;
};

// Fragment of a "transposed" LDS tile: row `row`, permuted columns
// base + 4g + {0..3} and base + 8 + 4g + {0..3}.
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag tfrag(const T* rowp, int base, int g) {
  typedef typename QuadB<T>::type QT;
  typename Mma<T>::frag f;
  *reinterpret_cast<QT*>(&f) = *reinterpret_cast<const QT*>(rowp + base + 4 * g);
  *(reinterpret_cast<QT*>(&f) + 1) = *reinterpret_cast<const QT*>(rowp + base + 8 + 4 * g);
  return f;
}

// Copy a [rows][cols] tile (cols contiguous, global row stride ld) into LDS
// rows of `stride` elements; rows >= valid_rows (or columns >= valid_cols)
// read as zero. cols is a multiple of 16 / sizeof(T).
template <typename T, int ROWS, int COLS>
__device__ __forceinline__ void tile_to_lds(T* lds, int stride, const T* g, int64_t ld, int valid_rows,
                                            int valid_cols, int tid) {
  constexpr int kVec = 16 / sizeof(T);
  constexpr int kChunks = ROWS * COLS / kVec;
  for (int c = tid; c < kChunks; c += 256) {
    const int r = c / (COLS / kVec), col = (c % (COLS / kVec)) * kVec;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r < valid_rows && col < valid_cols) v = ld16(g + (int64_t)r * ld + col);
    st16(lds + r * stride + col, v);
  }
}

// D = rowsum(dO * O) per (sequence, head, query); one wave per row.
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_bwd_delta_kernel(const T* __restrict__ dO, const T* __restrict__ O,
                                                             float* __restrict__ delta, int m, int nh, int64_t nrows) {
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (b*nh + h)*m + i
  const int lane = threadIdx.x & 63;
  if (row >= nrows) return;
  const int64_t bh = row / m, i = row % m;
  const int64_t b = bh / nh, h = bh % nh;
  const T* dor = dO + row * DH;
  const T* orow = O + (b * m + i) * ((int64_t)nh * DH) + h * DH;
  float s = 0.0f;
  for (int c = lane; c < DH; c += 64) s += to_f32(dor[c]) * to_f32(orow[c]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) delta[row] = s;
}

template <typename T, int DH, bool SPLIT>
__global__ void __launch_bounds__(256) attn_bwd_dkdv_kernel(const AttnBwdParams p) {
  typedef Mma<T> MM;
  constexpr int kVec = 16 / sizeof(T);
  constexpr int QT = 64;                 // queries per tile
  constexpr int RS = DH + kVec;          // row-layout tile stride
  constexpr int TS = QT + kVec;          // transposed tile stride
  __shared__ __attribute__((aligned(16))) T s_q[QT * RS];
  __shared__ __attribute__((aligned(16))) T s_ql[SPLIT ? QT * RS : 8];
  __shared__ __attribute__((aligned(16))) T s_do[QT * RS];
  __shared__ __attribute__((aligned(16))) T s_qt[DH * TS];
  __shared__ __attribute__((aligned(16))) T s_dot[DH * TS];
  __shared__ float s_lse[QT], s_d[QT];

  const int bh = blockIdx.y;
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;
  const int k0 = blockIdx.x * 128;
  const int kw0 = k0 + wave * 32;
  const int mykey = kw0 + col;
  const int m = p.m;
  const int64_t hoff = (int64_t)bh * m * DH;
  const int64_t toff = (int64_t)bh * DH * p.ld_t;
  const T* qg = reinterpret_cast<const T*>(p.q) + hoff;
  const T* kg = reinterpret_cast<const T*>(p.k) + hoff;
  const T* vg = reinterpret_cast<const T*>(p.v) + hoff;
  const T* dog = reinterpret_cast<const T*>(p.do_) + hoff;
  const T* qtg = reinterpret_cast<const T*>(p.qt) + toff;
  const T* dotg = reinterpret_cast<const T*>(p.dot) + toff;
  const T* qlg = SPLIT ? reinterpret_cast<const T*>(p.q_lo) + hoff : nullptr;
  const T* klg = SPLIT ? reinterpret_cast<const T*>(p.k_lo) + hoff : nullptr;

  // this wave's keys and values as B operands (column = key)
  typename MM::frag kf[DH / 16], kfl[SPLIT ? DH / 16 : 1], vf[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (mykey < m) {
      kf[kk] = MM::load(kg + (int64_t)mykey * DH + kk * 16 + g * 8);
      vf[kk] = MM::load(vg + (int64_t)mykey * DH + kk * 16 + g * 8);
      if constexpr (SPLIT) kfl[kk] = MM::load(klg + (int64_t)mykey * DH + kk * 16 + g * 8);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        kf[kk][i] = vf[kk][i] = (T)0.0f;
        if constexpr (SPLIT) kfl[kk][i] = (T)0.0f;
      }
    }
  }
  f32x16 dvt[DH / 32], dkt[DH / 32];
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) dvt[cb][r] = dkt[cb][r] = 0.0f;

  const int nqt = (m + QT - 1) / QT;
  const int qt_begin = p.causal ? k0 / QT : 0;
  for (int qt = qt_begin; qt < nqt; ++qt) {
    const int q0 = qt * QT;
    const int vq = min(QT, m - q0);
    __syncthreads();
    tile_to_lds<T, QT, DH>(s_q, RS, qg + (int64_t)q0 * DH, DH, vq, DH, tid);
    if constexpr (SPLIT) tile_to_lds<T, QT, DH>(s_ql, RS, qlg + (int64_t)q0 * DH, DH, vq, DH, tid);
    tile_to_lds<T, QT, DH>(s_do, RS, dog + (int64_t)q0 * DH, DH, vq, DH, tid);
    tile_to_lds<T, DH, QT>(s_qt, TS, qtg + q0, p.ld_t, DH, p.ld_t - q0, tid);
    tile_to_lds<T, DH, QT>(s_dot, TS, dotg + q0, p.ld_t, DH, p.ld_t - q0, tid);
    if (tid < QT) {
      const bool ok = q0 + tid < m;
      s_lse[tid] = ok ? p.lse[(int64_t)bh * m + q0 + tid] * 1.4426950408889634f : 0.0f;
      s_d[tid] = ok ? p.delta[(int64_t)bh * m + q0 + tid] : 0.0f;
    }
    __syncthreads();
    if (p.causal && q0 + QT - 1 < kw0) continue;  // every query of the tile precedes this wave's keys
#pragma unroll
    for (int qb = 0; qb < QT / 32; ++qb) {
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk) {
        const int off = (qb * 32 + col) * RS + kk * 16 + g * 8;
        const typename MM::frag qh = MM::load(s_q + off);
        s = MM::mma(qh, kf[kk], s);
        if constexpr (SPLIT) {
          s = MM::mma(MM::load(s_ql + off), kf[kk], s);
          s = MM::mma(qh, kfl[kk], s);
        }
        dp = MM::mma(MM::load(s_do + off), vf[kk], dp);
      }
      float pr[16], dsr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ql = qb * 32 + acc_row(r, lane);
        const int q = q0 + ql;
        const bool ok = q < m && mykey < m && (!p.causal || mykey <= q);
        const float pv = ok ? fast_exp2(s[r] * p.scale_log2 - s_lse[ql]) : 0.0f;
        pr[r] = pv;
        dsr[r] = pv * (dp[r] - s_d[ql]);
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const typename MM::frag pb = MM::pack(&pr[s2 * 8]);
        const typename MM::frag db = MM::pack(&dsr[s2 * 8]);
#pragma unroll
        for (int cb = 0; cb < DH / 32; ++cb) {
          const int crow = (cb * 32 + col) * TS;
          dvt[cb] = MM::mma(tfrag<T>(s_dot + crow, qb * 32 + s2 * 16, g), pb, dvt[cb]);
          dkt[cb] = MM::mma(tfrag<T>(s_qt + crow, qb * 32 + s2 * 16, g), db, dkt[cb]);
        }
      }
    }
  }

  if (mykey < m) {
    const int64_t orow = ((int64_t)b * m + mykey) * ((int64_t)p.n_heads * DH) + h * DH;
#pragma unroll
    for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = cb * 32 + acc_row(r, lane);
        reinterpret_cast<T*>(p.dv)[orow + c] = from_f32<T>(dvt[cb][r]);
        reinterpret_cast<T*>(p.dk)[orow + c] = from_f32<T>(dkt[cb][r] * p.scale);
      }
  }
}

template <typename T, int DH, bool SPLIT>
__global__ void __launch_bounds__(256) attn_bwd_dq_kernel(const AttnBwdParams p) {
  typedef Mma<T> MM;
  constexpr int kVec = 16 / sizeof(T);
  constexpr int KT = 64;
  constexpr int RS = DH + kVec;
  constexpr int TS = KT + kVec;
  __shared__ __attribute__((aligned(16))) T s_k[KT * RS];
  __shared__ __attribute__((aligned(16))) T s_kl[SPLIT ? KT * RS : 8];
  __shared__ __attribute__((aligned(16))) T s_v[KT * RS];
  __shared__ __attribute__((aligned(16))) T s_kt[DH * TS];

  const int nqtiles = (p.m + 127) / 128;
  const int qtile = nqtiles - 1 - (int)blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, col = lane & 31;
  const int q0 = qtile * 128;
  const int qw0 = q0 + wave * 32;
  const int myq = qw0 + col;
  const int m = p.m;
  const int64_t hoff = (int64_t)bh * m * DH;
  const int64_t toff = (int64_t)bh * DH * p.ld_t;
  const T* qg = reinterpret_cast<const T*>(p.q) + hoff;
  const T* kg = reinterpret_cast<const T*>(p.k) + hoff;
  const T* vg = reinterpret_cast<const T*>(p.v) + hoff;
  const T* dog = reinterpret_cast<const T*>(p.do_) + hoff;
  const T* ktg = reinterpret_cast<const T*>(p.kt) + toff;
  const T* qlg = SPLIT ? reinterpret_cast<const T*>(p.q_lo) + hoff : nullptr;
  const T* klg = SPLIT ? reinterpret_cast<const T*>(p.k_lo) + hoff : nullptr;

  typename MM::frag qf[DH / 16], qfl[SPLIT ? DH / 16 : 1], dof[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (myq < m) {
      qf[kk] = MM::load(qg + (int64_t)myq * DH + kk * 16 + g * 8);
      dof[kk] = MM::load(dog + (int64_t)myq * DH + kk * 16 + g * 8);
      if constexpr (SPLIT) qfl[kk] = MM::load(qlg + (int64_t)myq * DH + kk * 16 + g * 8);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        qf[kk][i] = dof[kk][i] = (T)0.0f;
        if constexpr (SPLIT) qfl[kk][i] = (T)0.0f;
      }
    }
  }
  const float lse2 = myq < m ? p.lse[(int64_t)bh * m + myq] * 1.4426950408889634f : 0.0f;
  const float dlt = myq < m ? p.delta[(int64_t)bh * m + myq] : 0.0f;
  f32x16 dqt[DH / 32];
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqt[cb][r] = 0.0f;

  const int kv_end = p.causal ? min(m, q0 + 128) : m;
  const int ntiles = (kv_end + KT - 1) / KT;
  for (int t = 0; t < ntiles; ++t) {
    const int kt0 = t * KT;
    const int vk = min(KT, m - kt0);
    __syncthreads();
    tile_to_lds<T, KT, DH>(s_k, RS, kg + (int64_t)kt0 * DH, DH, vk, DH, tid);
    if constexpr (SPLIT) tile_to_lds<T, KT, DH>(s_kl, RS, klg + (int64_t)kt0 * DH, DH, vk, DH, tid);
    tile_to_lds<T, KT, DH>(s_v, RS, vg + (int64_t)kt0 * DH, DH, vk, DH, tid);
    tile_to_lds<T, DH, KT>(s_kt, TS, ktg + kt0, p.ld_t, DH, p.ld_t - kt0, tid);
    __syncthreads();
    if (p.causal && kt0 > qw0 + 31) continue;
#pragma unroll
    for (int kb = 0; kb < KT / 32; ++kb) {
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk) {
        const int off = (kb * 32 + col) * RS + kk * 16 + g * 8;
        const typename MM::frag kh = MM::load(s_k + off);
        s = MM::mma(kh, qf[kk], s);
        if constexpr (SPLIT) {
          s = MM::mma(MM::load(s_kl + off), qf[kk], s);
          s = MM::mma(kh, qfl[kk], s);
        }
        dp = MM::mma(MM::load(s_v + off), dof[kk], dp);
      }
      float dsr[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kt0 + kb * 32 + acc_row(r, lane);
        const bool ok = key < m && myq < m && (!p.causal || key <= myq);
        const float pv = ok ? fast_exp2(s[r] * p.scale_log2 - lse2) : 0.0f;
        dsr[r] = pv * (dp[r] - dlt);
      }
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        const typename MM::frag db = MM::pack(&dsr[s2 * 8]);
#pragma unroll
        for (int cb = 0; cb < DH / 32; ++cb)
          dqt[cb] = MM::mma(tfrag<T>(s_kt + (cb * 32 + col) * TS, kb * 32 + s2 * 16, g), db, dqt[cb]);
      }
    }
  }
  if (myq < m) {
    const int64_t orow = ((int64_t)b * m + myq) * ((int64_t)p.n_heads * DH) + h * DH;
#pragma unroll
    for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        reinterpret_cast<T*>(p.dq)[orow + cb * 32 + acc_row(r, lane)] = from_f32<T>(dqt[cb][r] * p.scale);
  }
}

template <typename T>
hipError_t launch_attention_bwd(const AttnBwdParams& p, int batch, int head_dim, hipStream_t stream) {
  if (p.m <= 0) return hipSuccess;
  const int64_t rows = (int64_t)batch * p.n_heads * p.m;
  const dim3 dgrid((unsigned)((rows + 3) / 4));
  const dim3 kgrid((p.m + 127) / 128, batch * p.n_heads);
  const bool split = sizeof(T) == 2 && p.q_lo && p.k_lo;
  if (head_dim == 64) {
    hipLaunchKernelGGL((attn_bwd_delta_kernel<T, 64>), dgrid, dim3(256), 0, stream,
                       reinterpret_cast<const T*>(p.do_), reinterpret_cast<const T*>(p.o), p.delta, p.m, p.n_heads, rows);
    if (split) {
      hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, 64, sizeof(T) == 2>), kgrid, dim3(256), 0, stream, p);
      hipLaunchKernelGGL((attn_bwd_dq_kernel<T, 64, sizeof(T) == 2>), kgrid, dim3(256), 0, stream, p);
    } else {
      hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, 64, false>), kgrid, dim3(256), 0, stream, p);
      hipLaunchKernelGGL((attn_bwd_dq_kernel<T, 64, false>), kgrid, dim3(256), 0, stream, p);
    }
  } else {
    hipLaunchKernelGGL((attn_bwd_delta_kernel<T, 128>), dgrid, dim3(256), 0, stream,
                       reinterpret_cast<const T*>(p.do_), reinterpret_cast<const T*>(p.o), p.delta, p.m, p.n_heads, rows);
    if (split) {
      hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, 128, sizeof(T) == 2>), kgrid, dim3(256), 0, stream, p);
      hipLaunchKernelGGL((attn_bwd_dq_kernel<T, 128, sizeof(T) == 2>), kgrid, dim3(256), 0, stream, p);
    } else {
      hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, 128, false>), kgrid, dim3(256), 0, stream, p);
      hipLaunchKernelGGL((attn_bwd_dq_kernel<T, 128, false>), kgrid, dim3(256), 0, stream, p);
    }
  }
  return hipGetLastError();
}

template hipError_t launch_attention_bwd<bf16>(const AttnBwdParams&, int, int, hipStream_t);
template hipError_t launch_attention_bwd<float>(const AttnBwdParams&, int, int, hipStream_t);

}  // namespace pf
