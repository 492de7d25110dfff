// Prefill: the parallel form of the generation block (Eq. 19-20) over a chunk
// of T tokens per sequence, with the cache update of Eq. 21 for the chunk's
// complete blocks. It gives what T streaming decode steps give.
//
// Token t of the chunk sits in block t / P. Its output attends to two key
// sets, each under its own softmax: the tokens of its own block up to itself
// (A_x) and the cached proxies of every block before its own, i.e. the n0
// rows already cached plus the chunk's blocks 0 .. t/P - 1 (A_h). Launches:
//  1. rmsnorm_rows_kernel: u = RMSNorm(x) * gamma, one wave per token.
//  2. GEMMs from u: Q and K into per-head row tensors, V into a per-head
//     token-contiguous tensor (the MFMA operand layout of the value product),
//     alpha = sigmoid(u W_alpha^T + b) into fp32.
//  3. the append of the chunk's complete blocks (the decode path's
//     compression and K/V proxy GEMMs), so the cache holds every row a token
//     of the chunk may see.
//  4. fp32 only: a transposed copy of the cached values (rows 0 .. n0 +
//     T/P - 1), the operand layout the fp32 value product reads with 16-byte
//     chunks. The bf16 path reads the cached values in place, row-major like
//     the keys, through LDS transpose reads.
//  5. gen_attn_kernel: per (sequence, head, 128 tokens), the local phase
//     then the cache phase, each a flash-style loop over 64-key tiles staged
//     through LDS; A = A_x + alpha * A_h.
//  6. y = x + A W_o^T + b_o (GEMM with the residual in its epilogue).
//  7. the tokens of an unfinished last block (T % P of them) are copied into
//     the local slots, so decoding continues at j = T % P.
#include <algorithm>
#include <cmath>

#include "attention.hpp"
#include "decode.hpp"
#include "epilogues.hpp"
#include "layer.hpp"
#include "runner.hpp"
#include "transpose.hpp"

namespace pf {

// ---- RMSNorm rows ----------------------------------------------------------------

// u[r] = x[r] / sqrt(mean(x[r]^2) + eps) * gamma, one wave per row, the sum of
// squares in fp32 (per-lane runs of 8, then a butterfly over the wave).
// d * sizeof(T) <= 4096, so a lane holds at most four runs of 8.
template <typename T>
__global__ void __launch_bounds__(256) rmsnorm_rows_kernel(const T* __restrict__ x, const T* __restrict__ gamma,
                                                           T* __restrict__ u, int64_t rows, int d, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* xr = x + row * d;
  float v[4][8];
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < d) {
      load8(xr + c, v[i]);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(v[i][e], v[i][e], ss);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
  const float rs = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = (lane + 64 * i) * 8;
    if (c < d) {
      float g[8], o[8];
      load8(gamma + c, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = v[i][e] * rs * g[e];
      store8(u + row * d + c, o);
    }
  }
}

// alpha = sigmoid(acc + bias) into fp32 [rows, h] (Eq. 20's gate per head).
template <typename T>
struct EpiSigmoidF32 {
  float* out;
  int ldo;
  const T* bias;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    out[(int64_t)r * ldo + c] = sigmoidf(v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
#pragma unroll
    for (int e = 0; e < 8; ++e) (*this)(r, c + e, v0[e]);
  }
};

// ---- attention over the two key sets ------------------------------------------------

struct GenAttnParams {
  const void* q;       // [B, h, T, dh], scaled by log2(e) / sqrt(dh)
  const void* k;       // [B, h, T, dh]
  const void* vt;      // [B, h, dh, ld_t], columns T .. ld_t-1 zero
  const void* v;       // bf16: [B, h, T, dh] (in place of vt)
  const void* kc;      // [B, h, n_cap, dh] cache keys
  const void* vc;      // bf16: [B, h, n_cap, dh] cached values (in place of vct)
  const void* vct;     // [B, h, dh, ld_c] cached values, columns n_keys .. ld_c-1 zero
  const float* alpha;  // [B*T, h]
  void* out;           // [B*T, h*dh] A = A_x + alpha * A_h
  int T, nh, ld_t, ld_c, P;
  int n0;              // cached rows before the chunk
  int n_keys;          // cached rows after the chunk's append
  int64_t n_cap;
};

template <typename T, int DH>
struct GenShape {
  static constexpr int kKT = 64;                          // keys per tile
  static constexpr int kRowBytes = DH * (int)sizeof(T);   // K tile row: one key
  static constexpr int kVRowBytes = kKT * (int)sizeof(T); // V^T tile row: one channel
  static constexpr int kKTile = kKT * kRowBytes;
  static constexpr int kVTile = DH * kVRowBytes;
  static constexpr int kStage = kKTile + kVTile;
  static constexpr int kInstsPerWave = kStage / 1024 / 4;  // 1 KB direct loads per wave and stage
  static constexpr int kNS = 2;
  static_assert(kKTile % 1024 == 0 && kVTile % 1024 == 0 && (kStage / 1024) % 4 == 0, "stage splits into wave loads");
};


// Chunk swizzle of a row-major value tile read through LDS transpose reads:
// a read pass covers 4 consecutive rows (keys) at 4 consecutive chunks, so
// the key moves rows by 64 bytes within each 256-byte bank window.
template <int NC>
__device__ __forceinline__ int vtr_swz(int r, int c) {
  static_assert(NC == 8 || NC >= 16, "rows of 128 bytes or of 256 bytes and more");
  return NC == 8 ? c ^ (((r >> 1) & 1) * 4) : c ^ ((r & 3) * 4);
}


// One softmax over the keys lo .. hi (inclusive, per lane; hi < lo: none) of
// the 64-key tiles t_first .. t_last. Keys come from kp (rows of DH, nkeys
// readable rows), values from vtp (DH rows of stride ld_v). The wave's 32
// queries (lane pairs l, l ^ 32) have windows bounded by wlo_min <= lo <=
// wlo_max and whi_min <= hi <= whi_max, which decide tiles skipped and tiles
// masked. On return o holds the normalised result (zero without any key).
// Follows the online softmax of the proxy attention forward; scores are the
// transposed tile S^T = K Q^T, so a lane holds one query.
// With VROW (bf16) the values are row-major like the keys (vtp: rows of DH,
// nkeys readable rows; ld_v unused) and their MFMA operands come from LDS
// transpose reads; otherwise vtp holds V^T (DH rows of stride ld_v).
template <typename T, int DH, bool VROW = false>
__device__ __forceinline__ void gen_phase(char* smem, const char* kp, int nkeys, const char* vtp, int ld_v,
                                          int t_first, int t_last, int lo, int hi, int wlo_min, int wlo_max,
                                          int whi_min, int whi_max, const typename Mma<T>::frag (&qf)[DH / 16],
                                          f32x16 (&o)[DH / 32]) {
  typedef GenShape<T, DH> S;
  typedef Mma<T> MM;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, col = lane & 31;
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[cb][r] = 0.0f;
  // Online softmax in exp2 units (Q arrives scaled by log2(e)/sqrt(d_head)),
  // with the reference maximum of the proxy attention forward: mref is set
  // from a real maximum on a lane pair's first tile with a visible key and
  // kept while the running sums stay below 2^64; the score MFMAs start at
  // -mref, so each probability is one exp2 of an MFMA result.
  float mref = -INFINITY, lrun = 0.0f;
  f32x16 negm, zero;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    negm[r] = 0.0f;
    zero[r] = 0.0f;
  }
  bool have_ref = false;  // wave-uniform
  constexpr float kSumLimit = 18446744073709551616.0f;  // 2^64
  const int ntiles = t_last - t_first + 1;

  auto issue = [&](int t, int stage) {
    const int kt0 = (t_first + t) * S::kKT;
    char* st = smem + stage * S::kStage;
    const rsrc_t rk = make_rsrc_uniform(kp + (int64_t)kt0 * S::kRowBytes, (uint32_t)max(0, nkeys - kt0) * S::kRowBytes);
    const rsrc_t rv = VROW ? make_rsrc_uniform(vtp + (int64_t)kt0 * S::kRowBytes,
                                               (uint32_t)max(0, nkeys - kt0) * S::kRowBytes)
                           : make_rsrc_uniform(vtp + (int64_t)kt0 * sizeof(T),
                                               (uint32_t)((int64_t)DH * ld_v * sizeof(T) - (int64_t)kt0 * sizeof(T)));
#pragma unroll
    for (int j = 0; j < S::kInstsPerWave; ++j) {
      const int i = wave * S::kInstsPerWave + j;  // wave-uniform
      const int off = i * 1024;
      uint32_t vo;
      rsrc_t r;
      if (off < S::kKTile) {  // K: row = key
        r = rk;
        const int row = off / S::kRowBytes + lane / (S::kRowBytes / 16);
        vo = (uint32_t)(row * S::kRowBytes + lds_swz<S::kRowBytes / 16>(row, lane % (S::kRowBytes / 16)) * 16);
      } else if constexpr (VROW) {  // V: row = key, like K
        r = rv;
        const int row = (off - S::kKTile) / S::kRowBytes + lane / (S::kRowBytes / 16);
        vo = (uint32_t)(row * S::kRowBytes + vtr_swz<S::kRowBytes / 16>(row, lane % (S::kRowBytes / 16)) * 16);
      } else {  // V^T: row = channel, stride ld_v
        r = rv;
        const int row = (off - S::kKTile) / S::kVRowBytes + lane / (S::kVRowBytes / 16);
        vo = (uint32_t)((int64_t)row * ld_v * sizeof(T) + lds_swz<S::kVRowBytes / 16>(row, lane % (S::kVRowBytes / 16)) * 16);
      }
      buf_ld16_lds(r, vo, st + off);
    }
  };

  lds_barrier();  // every wave is done with the LDS of the previous phase
  if (ntiles > 0) issue(0, 0);
  for (int t = 0; t < ntiles; ++t) {
    const int kt0 = (t_first + t) * S::kKT;
    wait_vmcnt<0>();
    lds_barrier();  // tile t landed for all; every wave is done with tile t-1
    if (t + 1 < ntiles) issue(t + 1, (t + 1) & 1);
    const char* sk = smem + (t & 1) * S::kStage;
    const char* sv = sk + S::kKTile;
    const bool active = kt0 <= whi_max && kt0 + S::kKT - 1 >= wlo_min && whi_max >= wlo_min;
    if (!active) continue;  // wave-uniform
    const bool need_mask = kt0 < wlo_max || kt0 + S::kKT - 1 > whi_min;  // some lane sees part of the tile
    // S^T = K Q^T + c0 for the tile's 64 keys, keys outside [lo, hi] at -inf
    auto scores = [&](f32x16 (&s)[2], const f32x16& c0) {
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = c0;
        const int kr = kb * 32 + col;
        const char* krow = sk + kr * S::kRowBytes;
#pragma unroll
        for (int kk = 0; kk < DH / 16; ++kk) {
          typename MM::frag kh;
          if constexpr (sizeof(T) == 2) {
            kh = *reinterpret_cast<const typename MM::frag*>(krow + lds_swz<S::kRowBytes / 16>(kr, kk * 2 + g) * 16);
          } else {
            const int c0i = kk * 4 + g * 2;
            const f32x4 a = *reinterpret_cast<const f32x4*>(krow + lds_swz<S::kRowBytes / 16>(kr, c0i) * 16);
            const f32x4 b = *reinterpret_cast<const f32x4*>(krow + lds_swz<S::kRowBytes / 16>(kr, c0i + 1) * 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              kh[e] = a[e];
              kh[e + 4] = b[e];
            }
          }
          s[kb] = MM::mma(kh, qf[kk], s[kb]);
        }
      }
      __builtin_amdgcn_s_setprio(0);
      if (need_mask) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = kt0 + kb * 32 + acc_row(r, lane);
            s[kb][r] = (key < lo || key > hi) ? -INFINITY : s[kb][r];
          }
      }
    };
    // probabilities in place (exp2 of score - shift), summed in four chains
    auto exponentiate = [&](f32x16 (&s)[2], float shift) {
      float ls[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float e = fast_exp2(s[kb][r] - shift);
          s[kb][r] = e;
          ls[r & 3] += e;
        }
      return (ls[0] + ls[1]) + (ls[2] + ls[3]);
    };
    f32x16 s[2];
    float tsum = 0.0f;
    bool redo = !have_ref;
    if (have_ref) {
      scores(s, negm);
      tsum = exponentiate(s, 0.0f);
      redo = __builtin_amdgcn_ballot_w64(!(lrun + tsum <= kSumLimit)) != 0;
    }
    if (redo) {  // wave-uniform: first active tile, a sum past the limit, or a lane's first key
      scores(s, zero);
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kb][r]);
      mt = fmaxf(mt, other_half(mt));
      const float ltot = lrun + other_half(lrun);
      const float mnew = fmaxf(mt, mref + fmaxf(0.0f, __log2f(ltot)));
      // nothing is accumulated while a lane has no reference
      const float a = mref == -INFINITY ? 0.0f : fast_exp2(mref - mnew);
      lrun *= a;
#pragma unroll
      for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[cb][r] *= a;
      mref = mnew;
#pragma unroll
      for (int r = 0; r < 16; ++r) negm[r] = -mnew;
      have_ref = true;
      // a lane that has seen no key keeps mref = -inf: its scores are all
      // -inf here (probability 0), and on a later tile its first visible key
      // gives an infinite sum, which brings it back here
      tsum = exponentiate(s, mnew == -INFINITY ? 0.0f : mnew);
    }
    lrun += tsum;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        typename MM::frag pb;
        if constexpr (sizeof(T) == 2) {
          pb = pt_frag_bf16(s[kb], s2);
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) pb[i] = s[kb][s2 * 8 + i];
        }
        const int c0 = kb * 32 + s2 * 16 + g * 8;
        const int c4 = kb * 32 + s2 * 16 + g * 4;
#pragma unroll
        for (int cb = 0; cb < DH / 32; ++cb) {
          const int dd = cb * 32 + col;
          const char* vrow = sv + dd * S::kVRowBytes;
          typename MM::frag va;
          if constexpr (VROW) {
            // keys c0 .. c0+7 of channel dd: two transpose reads, lane i of a
            // 16-lane group addressing key c0 (+4) + i / 4 at channels
            // 4 (i % 4) .. +3 of the group's 16
            const int ch = cb * 32 + (lane & 16) + 4 * (lane & 3);
            const int k1 = c0 + ((lane & 15) >> 2);
            auto addr = [&](int key) {
              return sv + key * S::kRowBytes + vtr_swz<S::kRowBytes / 16>(key, ch / 8) * 16 + ((ch / 4) & 1) * 8;
            };
            const auto lo = __builtin_bit_cast(bf16x4, lds_read_tr16(addr(k1)));
            const auto hi = __builtin_bit_cast(bf16x4, lds_read_tr16(addr(k1 + 4)));
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              va[e] = lo[e];
              va[e + 4] = hi[e];
            }
          } else if constexpr (sizeof(T) == 2) {
            va = *reinterpret_cast<const typename MM::frag*>(vrow + lds_swz<S::kVRowBytes / 16>(dd, c0 / 8) * 16);
          } else {
            const f32x4 a = *reinterpret_cast<const f32x4*>(vrow + lds_swz<S::kVRowBytes / 16>(dd, c4 / 4) * 16);
            const f32x4 b = *reinterpret_cast<const f32x4*>(vrow + lds_swz<S::kVRowBytes / 16>(dd, c4 / 4 + 2) * 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              va[e] = a[e];
              va[e + 4] = b[e];
            }
          }
          o[cb] = MM::mma(va, pb, o[cb]);
        }
      }
    __builtin_amdgcn_s_setprio(0);
  }
  const float ltot = lrun + other_half(lrun);
  const float inv = ltot > 0.0f ? 1.0f / ltot : 0.0f;
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[cb][r] *= inv;
}

// One workgroup = 4 waves = 128 tokens of one (sequence, head), 32 per wave.
template <typename T, int DH>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(DH == 64 ? 2 : 1)))
    gen_attn_kernel(const GenAttnParams p) {
  typedef GenShape<T, DH> S;
  typedef Mma<T> MM;
  // bf16 values stay row-major and reach the MFMA through LDS transpose reads
  constexpr bool kRow = sizeof(T) == 2;
  __shared__ __attribute__((aligned(1024))) char smem[S::kNS * S::kStage];

  // 1-D grid over (head, token tile); each XCD gets a contiguous run so the
  // tiles of one head share an L2 while they stream the same cache rows
  const int nqt = (p.T + 127) / 128;
  int bh, qt;
  {
    const int total = (int)gridDim.x;
    const int q = total / kNumXcd, rem = total % kNumXcd;
    const int wg = blockIdx.x, xcd = wg % kNumXcd, local = wg / kNumXcd;
    const int t = (xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q) + local;
    bh = t / nqt;
    qt = t % nqt;
  }
  const int b = bh / p.nh, h = bh % p.nh;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, col = lane & 31;
  const int last = p.T - 1;
  const int q0 = qt * 128, qw0 = q0 + wave * 32;
  const int myq = qw0 + col;
  // padding lanes past the chunk compute with the last token and store nothing
  const int qc = min(myq, last), qw0c = min(qw0, last), qw1c = min(qw0 + 31, last), q1c = min(q0 + 127, last);

  typename MM::frag qf[DH / 16];
  const T* qp = reinterpret_cast<const T*>(p.q) + ((int64_t)bh * p.T + qc) * DH;
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) qf[kk] = MM::load(qp + kk * 16 + g * 8);
  const float alpha = p.alpha[((int64_t)b * p.T + qc) * p.nh + h];

  // local phase: keys blk(t)*P .. t of the chunk
  f32x16 ox[DH / 32];
  {
    const char* kp = reinterpret_cast<const char*>(p.k) + (int64_t)bh * p.T * S::kRowBytes;
    const char* vtp = kRow ? reinterpret_cast<const char*>(p.v) + (int64_t)bh * p.T * S::kRowBytes
                           : reinterpret_cast<const char*>(p.vt) + (int64_t)bh * DH * p.ld_t * (int64_t)sizeof(T);
    const int lo = (qc / p.P) * p.P;
    gen_phase<T, DH, kRow>(smem, kp, p.T, vtp, p.ld_t, ((q0 / p.P) * p.P) / S::kKT, q1c / S::kKT, lo, qc,
                     (qw0c / p.P) * p.P, (qw1c / p.P) * p.P, qw0c, qw1c, qf, ox);
  }
  // cache phase: rows 0 .. n0 + blk(t) - 1
  f32x16 oc[DH / 32];
  {
    const char* kp = reinterpret_cast<const char*>(p.kc) + (int64_t)bh * p.n_cap * S::kRowBytes;
    const char* vtp = kRow ? reinterpret_cast<const char*>(p.vc) + (int64_t)bh * p.n_cap * S::kRowBytes
                           : reinterpret_cast<const char*>(p.vct) + (int64_t)bh * DH * p.ld_c * (int64_t)sizeof(T);
    const int hmax = p.n0 + q1c / p.P - 1;
    gen_phase<T, DH, kRow>(smem, kp, p.n_keys, vtp, p.ld_c, 0, hmax >= 0 ? hmax / S::kKT : -1, 0, p.n0 + qc / p.P - 1, 0,
                     0, p.n0 + qw0c / p.P - 1, p.n0 + qw1c / p.P - 1, qf, oc);
  }
  if (myq < p.T) {
    T* orow = reinterpret_cast<T*>(p.out) + ((int64_t)b * p.T + myq) * ((int64_t)p.nh * DH) + h * DH;
#pragma unroll
    for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[cb * 32 + acc_row(r, lane)] = from_f32<T>(fmaf(alpha, oc[cb][r], ox[cb][r]));
  }
}

// Tokens start .. start+rem-1 of every sequence into the local slots 0 ..
// rem-1: x into x_blk [B, P, d], K into k_loc and V into v_loc [B, h, P, dh].
// Value (bh, t, e) sits at v[bh * v_bh + t * v_t + e * v_e] (per-head rows,
// or the token-contiguous transposed copy).
template <typename T>
__global__ void __launch_bounds__(256) prefill_tail_kernel(const T* __restrict__ x, const T* __restrict__ k,
                                                           const T* __restrict__ v, T* __restrict__ x_blk,
                                                           T* __restrict__ k_loc, T* __restrict__ v_loc, int B,
                                                           int T_, int nh, int dh, int64_t P, int start, int rem,
                                                           int64_t v_bh, int64_t v_t, int64_t v_e) {
  const int d = nh * dh;
  const int64_t total = (int64_t)B * rem * d;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
    const int c = (int)(i % d);
    const int s = (int)((i / d) % rem);
    const int b = (int)(i / ((int64_t)rem * d));
    const int h = c / dh, e = c - h * dh;
    const int64_t bh = (int64_t)b * nh + h;
    x_blk[((int64_t)b * P + s) * d + c] = x[((int64_t)b * T_ + start + s) * d + c];
    k_loc[(bh * P + s) * dh + e] = k[(bh * T_ + start + s) * dh + e];
    v_loc[(bh * P + s) * dh + e] = v[bh * v_bh + (start + s) * v_t + e * v_e];
  }
}

// ---- sizes ------------------------------------------------------------------------

static int64_t round64(int64_t v) { return (v + 63) / 64 * 64; }

const char* prefill_limits(const DecodeDims& d, int64_t T, int64_t n_cap) {
  if (T < 0) return "n_tokens must be >= 0";
  if (n_cap < 0) return "n_cap must be >= 0";
  if ((int64_t)d.B * T >= ((int64_t)1 << 31)) return "batch * n_tokens must stay below 2^31";
  if ((int64_t)d.B * d.nh > 65535) return "batch * n_heads must be at most 65535";
  const int64_t es = d.esize;
  if ((int64_t)d.dh * round64(T) * es >= ((int64_t)1 << 31))
    return "one head's token-contiguous values (head_dim * n_tokens) must stay below 2 GiB";
  if ((int64_t)d.dh * round64(std::max<int64_t>(n_cap, 1)) * es >= ((int64_t)1 << 31))
    return "one head's cached keys or values (head_dim * n_cap) must stay below 2 GiB";
  return nullptr;
}

template <typename T>
static void prefill_impl(Runner& run, const DecodeDims& d, const pf_decode_weights* w, const pf_decode_state& st,
                         const void* x, int64_t n_tok, void* y, char* ws, const PrefillWs& W);

static size_t prefill_gemm_need(const DecodeDims& d, int64_t T, const PrefillWs& W) {
  Runner dry(true);
  pf_decode_weights nw{};
  pf_decode_state ns{};
  if (d.esize == 2)
    prefill_impl<bf16>(dry, d, &nw, ns, nullptr, T, nullptr, nullptr, W);
  else
    prefill_impl<float>(dry, d, &nw, ns, nullptr, T, nullptr, nullptr, W);
  return dry.gemm_need;
}

PrefillWs prefill_ws(const DecodeDims& d, int64_t T, int64_t n_cap) {
  PrefillWs w{};
  size_t off = decode_ws(d).bytes;  // the chunk's append uses the decode workspace
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t es = d.esize;
  const size_t rows = (size_t)d.B * T;
  w.ld_t = round64(T);
  w.ld_c = round64(std::max<int64_t>(n_cap, 1));
  w.u = take(rows * d.d * es);
  w.q = take(rows * d.d * es);
  w.k = take(rows * d.d * es);
  // bf16 keeps V per head in rows and reads the cached values in place; fp32
  // keeps V^T and a transposed copy of the cached values
  const bool vrow = d.esize == 2;
  w.vt = take(vrow ? rows * d.d * es : (size_t)d.B * d.nh * d.dh * w.ld_t * es);
  w.alpha = take(rows * d.nh * 4);
  w.vct = take(vrow ? 0 : (size_t)d.B * d.nh * d.dh * w.ld_c * es);
  const int64_t nblk = T / d.P;
  w.xc = take(nblk > 0 && T % d.P != 0 ? (size_t)d.B * nblk * d.P * d.d * es : 0);
  w.gemm = off;
  w.bytes = off + align256(prefill_gemm_need(d, T, w));
  return w;
}

// ---- launch sequence ----------------------------------------------------------------

template <typename T>
static void prefill_impl(Runner& run, const DecodeDims& d, const pf_decode_weights* w, const pf_decode_state& st,
                         const void* x, int64_t n_tok, void* y, char* ws, const PrefillWs& W) {
  const int Tn = (int)n_tok;
  const int rows = d.B * Tn;
  auto P_ = [&](size_t off) { return reinterpret_cast<T*>(ws + off); };
  T* u = run.dry ? nullptr : P_(W.u);
  T* q = run.dry ? nullptr : P_(W.q);
  T* k = run.dry ? nullptr : P_(W.k);
  T* vt = run.dry ? nullptr : P_(W.vt);
  float* alpha = run.dry ? nullptr : reinterpret_cast<float*>(ws + W.alpha);
  T* vct = run.dry ? nullptr : P_(W.vct);
  const T* xin = reinterpret_cast<const T*>(x);

  // 1. u = RMSNorm(x) * gamma
  run.launch("prefill_norm", [&] {
    hipLaunchKernelGGL((rmsnorm_rows_kernel<T>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, run.stream, xin,
                       reinterpret_cast<const T*>(w->rms_gamma), u, (int64_t)rows, d.d, d.eps);
    return hipGetLastError();
  });

  // 2. projections: Q, K per head (row tensors), V per head (bf16) or
  //    token-contiguous (fp32), alpha
  constexpr bool vrow = sizeof(T) == 2;
  if (!vrow && W.ld_t != Tn) {  // padding columns of V^T must read as zero
    const size_t tb = (size_t)d.B * d.nh * d.dh * W.ld_t * sizeof(T);
    run.launch("fill_zero", [&] { return fill_zero(vt, tb, run.stream); });
  }
  const pf_linear* proj[3] = {&w->q, &w->k, &w->v};
  // Q goes to the attention pre-scaled by log2(e)/sqrt(d_head): scores in
  // exp2 units
  T* outs[3] = {nullptr, k, vrow ? vt : nullptr};
  T* outs_t[3] = {nullptr, nullptr, vrow ? nullptr : vt};
  for (int i = 0; i < 3; ++i) {
    GemmProblem pr{};
    pr.a = u;
    pr.lda = d.d;
    pr.b = proj[i]->w;
    pr.ldb = d.d;
    pr.M = rows;
    pr.N = d.d;
    pr.K = d.d;
    EpiHeads<T> e{outs[i], outs_t[i], reinterpret_cast<const T*>(proj[i]->b), Tn, d.dh, d.nh, (int)W.ld_t, nullptr};
    if (i == 0) {
      e.outs = q;
      e.scale = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
    }
    run.gemm<T, LAYOUT_K, LAYOUT_K>("prefill_qkv_gemm", pr, e);
  }
  {
    GemmProblem pr{};
    pr.a = u;
    pr.lda = d.d;
    pr.b = w->alpha.w;
    pr.ldb = d.d;
    pr.M = rows;
    pr.N = d.nh;
    pr.K = d.d;
    run.gemm<T, LAYOUT_K, LAYOUT_K>("prefill_alpha_gemm", pr,
                                    EpiSigmoidF32<T>{alpha, d.nh, reinterpret_cast<const T*>(w->alpha.b)});
  }

  // 3. append the chunk's complete blocks (Eq. 21)
  const int64_t nblk = n_tok / d.P;
  if (!run.dry && nblk > 0 && run.ok()) {
    const void* xb = x;
    if (n_tok % d.P != 0) {  // gather the complete blocks into one [B, nblk*P, d] view
      const size_t width = (size_t)nblk * d.P * d.d * sizeof(T);
      run.launch("prefill_gather", [&] {
        return hipMemcpy2DAsync(ws + W.xc, width, x, (size_t)n_tok * d.d * sizeof(T), width, d.B,
                                hipMemcpyDeviceToDevice, run.stream);
      });
      xb = ws + W.xc;
    }
    if (run.ok()) {
      const DecodePos np{};
      run.err = cache_append_run<T>(d, decode_ws(d), w, st, np, xb, nblk, ws, run.stream);
    }
  }

  // 4. fp32: cached values of rows 0 .. n_keys-1, transposed with row stride
  //    ld_c (the columns up to the next multiple of 64 are zeros; W.ld_c,
  //    sized from the capacity, bounds it)
  const int64_t n_keys = st.n + nblk;
  const int64_t ld_c = round64(std::max<int64_t>(n_keys, 1));
  if (!vrow && n_keys > 0) {
    run.launch("prefill_cache_vt", [&] {
      const dim3 grid((d.dh + 63) / 64, (unsigned)(ld_c / 64), (unsigned)(d.B * d.nh));
      hipLaunchKernelGGL((transpose_kernel<T>), grid, dim3(256), 0, run.stream,
                         reinterpret_cast<const T*>(st.v_cache), (int64_t)d.dh, n_keys, d.dh, vct, ld_c,
                         (float*)nullptr, st.n_cap * d.dh, (int64_t)d.dh * ld_c, ld_c);
      return hipGetLastError();
    });
  }

  // 5. attention over the chunk's blocks and the cache; A overwrites u
  GenAttnParams ap{};
  ap.q = q;
  ap.k = k;
  ap.vt = vrow ? nullptr : vt;
  ap.v = vrow ? vt : nullptr;
  ap.kc = st.k_cache;
  ap.vc = vrow ? st.v_cache : nullptr;
  ap.vct = vrow ? nullptr : vct;
  ap.alpha = alpha;
  ap.out = u;
  ap.T = Tn;
  ap.nh = d.nh;
  ap.ld_t = (int)W.ld_t;
  ap.ld_c = (int)ld_c;
  ap.P = (int)d.P;
  ap.n0 = (int)st.n;
  ap.n_keys = (int)n_keys;
  ap.n_cap = st.n_cap;
  run.launch("prefill_attn", [&] {
    const dim3 grid((unsigned)(((Tn + 127) / 128) * d.B * d.nh));
    if (d.dh == 64)
      hipLaunchKernelGGL((gen_attn_kernel<T, 64>), grid, dim3(256), 0, run.stream, ap);
    else
      hipLaunchKernelGGL((gen_attn_kernel<T, 128>), grid, dim3(256), 0, run.stream, ap);
    return hipGetLastError();
  });

  // 7 (before the output map, which may not alias x anyway): the unfinished
  // block into the local slots
  const int rem = (int)(n_tok - nblk * d.P);
  if (rem > 0) {
    run.launch("prefill_tail", [&] {
      const int64_t total = (int64_t)d.B * rem * d.d;
      const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 4096);
      hipLaunchKernelGGL((prefill_tail_kernel<T>), dim3(blocks), dim3(256), 0, run.stream, xin, k, vt,
                         reinterpret_cast<T*>(st.x_blk), reinterpret_cast<T*>(st.k_loc),
                         reinterpret_cast<T*>(st.v_loc), d.B, Tn, d.nh, d.dh, d.P, (int)(nblk * d.P), rem,
                         vrow ? (int64_t)Tn * d.dh : (int64_t)d.dh * W.ld_t, vrow ? (int64_t)d.dh : (int64_t)1,
                         vrow ? (int64_t)1 : W.ld_t);
      return hipGetLastError();
    });
  }

  // 6. y = x + A W_o^T + b_o
  {
    GemmProblem pr{};
    pr.a = u;
    pr.lda = d.d;
    pr.b = w->o.w;
    pr.ldb = d.d;
    pr.M = rows;
    pr.N = d.d;
    pr.K = d.d;
    EpiLinear<T> e{reinterpret_cast<T*>(y), d.d, reinterpret_cast<const T*>(w->o.b), xin, d.d, nullptr, nullptr};
    run.gemm<T, LAYOUT_K, LAYOUT_K>("prefill_out_gemm", pr, e);
  }
}

template <typename T>
hipError_t prefill_run(const DecodeDims& d, const pf_decode_weights* w, const pf_decode_state& st, const void* x,
                       int64_t n_tok, void* y, char* ws, hipStream_t stream) {
  if (n_tok <= 0) return hipSuccess;
  const PrefillWs W = prefill_ws(d, n_tok, st.n_cap);
  Runner run(false, stream, reinterpret_cast<float*>(ws + W.gemm));
  prefill_impl<T>(run, d, w, st, x, n_tok, y, ws, W);
  return run.err;
}

template hipError_t prefill_run<bf16>(const DecodeDims&, const pf_decode_weights*, const pf_decode_state&,
                                      const void*, int64_t, void*, char*, hipStream_t);
template hipError_t prefill_run<float>(const DecodeDims&, const pf_decode_weights*, const pf_decode_state&,
                                       const void*, int64_t, void*, char*, hipStream_t);

}  // namespace pf
