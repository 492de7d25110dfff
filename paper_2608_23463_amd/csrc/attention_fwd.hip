// Flash-style causal multi-head attention over proxies (Eq. 9), forward.
//
// One workgroup = 4 waves = 128 queries of one (sequence, head); each wave owns
// 32 queries. Key and value tiles of 64 keys arrive in LDS through direct
// (buffer -> LDS) loads into a ring of NS stages with XOR-swizzled 16-byte
// chunks, so fragment reads are conflict-free 16-byte reads. A wave computes
// the transposed score tile S^T = K Q^T with MFMA, so each lane holds one
// query column: the online-softmax statistics of a query live in one lane
// pair (lane, lane ^ 32). Q arrives pre-scaled by log2(e)/sqrt(d_head), so
// scores are in exp2 units; the score MFMAs start their accumulators at
// minus the query's reference maximum, so each probability is one exp2 of an
// MFMA result, with no per-score scaling or shift. The reference is a real
// maximum taken on the wave's first tile and kept while the running sums stay
// below 2^64 (no per-tile maximum); a tile that would exceed that is redone
// against a new reference. P^T stays in registers: one v_permlane32_swap per
// pair of packed values turns the accumulator layout (runs of 4 keys) into
// MFMA operands of 8 consecutive keys, so V^T (key-contiguous, written
// transposed by the producing GEMM) is read as 16-byte chunks. With SPLIT
// (bf16 extended precision) the scores are Kh Qh + (Kl Qh + Kh Ql) with Qh, Kh
// the bf16 values and Ql, Kl their rounding remainders, so a sharp softmax is
// not moved by one bf16 rounding of its logits. The correction products come
// from fp8 e5m2 rows [256 Ql | Qh] and [Kh | 256 Kl] written by the Q and K
// projections: per 32-key block one fp8 MFMA per 64 bytes of the row (half
// the matrix time of two bf16 products), whose block scale removes the 256.
// The correction is ~2^-8 of the logit, so its fp8 rounding (2^-3) leaves the
// logits exact to ~2^-11 of |q||k| (one bf16 rounding: ~2^-8); e5m2's range
// (2^-14 .. 57344 normal) holds Q and K rows of any practical magnitude.
// Masked scores are -inf and contribute exactly zero, so a query never
// depends on later proxies (bit-exact causality).
#include "attention.hpp"

namespace pf {

template <typename T, int DH, bool SPLIT, int NS>
struct AttnFwdShape {
  static constexpr int kKT = 64;                         // keys per tile
  static constexpr int kRowBytes = DH * (int)sizeof(T);  // K tile row: one key
  static constexpr int kVRowBytes = kKT * (int)sizeof(T);  // V^T tile row: one channel
  static constexpr int kKTile = kKT * kRowBytes;
  static constexpr int kVTile = DH * kVRowBytes;
  static constexpr int kKParts = SPLIT ? 2 : 1;
  static constexpr int kStage = kKParts * kKTile + kVTile;  // bytes
  static constexpr int kInsts = kStage / 1024;             // 1 KB direct loads per stage
  static constexpr int kInstsPerWave = kInsts / 4;
  static constexpr int kNS = NS;  // ring depth
  static_assert(kRowBytes >= 128 && kVRowBytes >= 128, "rows of at least 8 chunks");
  static_assert(kKTile % 1024 == 0 && kVTile % 1024 == 0 && kInsts % 4 == 0, "stage splits into wave loads");
};


template <typename T, int DH, bool SPLIT, int NS, int OCC>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(OCC)))
    attn_fwd_kernel(const AttnParams p) {
  static_assert(!SPLIT || sizeof(T) == 2, "the split takes bf16 operands");
  constexpr int kXB = 2 * DH / 64;  // fp8 blocks of 64 bytes per correction row
  typedef AttnFwdShape<T, DH, SPLIT, NS> S;
  typedef Mma<T> MM;
  __shared__ __attribute__((aligned(1024))) char smem[S::kNS * S::kStage];

  // 1-D grid over (head, query tile). Consecutive workgroups go to different
  // XCDs (round robin over 8), so the id is remapped to give every XCD a
  // contiguous run of tiles: the query tiles of one head share an L2 while
  // they stream the same keys. Longest causal rows first within a head.
  const int nqt = (p.m + 127) / 128;
  int bh, qt;
  {
    const int total = (int)gridDim.x;
    const int q = total / kNumXcd, rem = total % kNumXcd;
    const int wg = blockIdx.x, xcd = wg % kNumXcd, local = wg / kNumXcd;
    const int t = (xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q) + local;
    bh = t / nqt;
    qt = nqt - 1 - t % nqt;
  }
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, col = lane & 31;
  const int q0 = qt * 128;
  const int qw0 = q0 + wave * 32;
  const int myq = qw0 + col;

  const char* kp = reinterpret_cast<const char*>(p.k) + (int64_t)bh * p.m * S::kRowBytes;
  // the second K tile (SPLIT): the fp8 correction rows, 2 dh bytes like a
  // bf16 key row
  const char* klp = SPLIT ? reinterpret_cast<const char*>(p.kx) + (int64_t)bh * p.m * S::kRowBytes : nullptr;
  const char* vtp = reinterpret_cast<const char*>(p.vt) + (int64_t)bh * DH * p.ld_t * (int64_t)sizeof(T);
  const T* qp = reinterpret_cast<const T*>(p.q) + (int64_t)bh * p.m * DH;

  typename MM::frag qf[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (myq < p.m) {
      qf[kk] = MM::load(qp + (int64_t)myq * DH + kk * 16 + g * 8);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) qf[kk][i] = (T)0.0f;
    }
  }
  // fp8 correction operand of this lane's query: bytes [32 g, +32) of each
  // 64-byte block of its row
  i32x8 qx[SPLIT ? kXB : 1];
  if constexpr (SPLIT) {
    const char* qxr = reinterpret_cast<const char*>(p.qx) + ((int64_t)bh * p.m + (myq < p.m ? myq : 0)) * 2 * DH;
#pragma unroll
    for (int xb = 0; xb < kXB; ++xb) {
      const u32x4 lo = *reinterpret_cast<const u32x4*>(qxr + xb * 64 + 32 * g);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(qxr + xb * 64 + 32 * g + 16);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        qx[xb][e] = myq < p.m ? (int)lo[e] : 0;
        qx[xb][e + 4] = myq < p.m ? (int)hi[e] : 0;
      }
    }
  }

  const int kv_end = p.causal ? min(p.m, q0 + 128) : p.m;
  const int ntiles = (kv_end + S::kKT - 1) / S::kKT;

  // Direct loads of one stage: this wave's kInstsPerWave 1 KB blocks. Block
  // i of the stage covers bytes [i KB, i+1 KB): the K tile(s), then V^T.
  auto issue = [&](int t, int stage) {
    const int kt0 = t * S::kKT;
    char* st = smem + stage * S::kStage;
    const uint32_t krows = (uint32_t)max(0, p.m - kt0) * S::kRowBytes;  // keys past m read as zero
    const rsrc_t rk = make_rsrc_uniform(kp + (int64_t)kt0 * S::kRowBytes, krows);
    const rsrc_t rkl = SPLIT ? make_rsrc_uniform(klp + (int64_t)kt0 * S::kRowBytes, krows) : rk;
    const rsrc_t rv = make_rsrc_uniform(vtp + (int64_t)kt0 * sizeof(T),
                                        (uint32_t)((int64_t)DH * p.ld_t * sizeof(T) - (int64_t)kt0 * sizeof(T)));
#pragma unroll
    for (int j = 0; j < S::kInstsPerWave; ++j) {
      const int i = wave * S::kInstsPerWave + j;  // wave-uniform
      const int off = i * 1024;
      uint32_t vo;
      rsrc_t r;
      if (off < S::kKParts * S::kKTile) {  // K: row = key, contiguous rows
        r = off < S::kKTile ? rk : rkl;
        const int row = (off % S::kKTile) / S::kRowBytes + lane / (S::kRowBytes / 16);
        vo = (uint32_t)(row * S::kRowBytes + lds_swz<S::kRowBytes / 16>(row, lane % (S::kRowBytes / 16)) * 16);
      } else {  // V^T: row = channel, stride ld_t
        r = rv;
        const int row = (off - S::kKParts * S::kKTile) / S::kVRowBytes + lane / (S::kVRowBytes / 16);
        vo = (uint32_t)((int64_t)row * p.ld_t * sizeof(T) + lds_swz<S::kVRowBytes / 16>(row, lane % (S::kVRowBytes / 16)) * 16);
      }
      buf_ld16_lds(r, vo, st + off);
    }
  };

  f32x16 oacc[DH / 32];
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[cb][r] = 0.0f;
  // Online softmax in exp2 units (Q arrives scaled by log2(e)/sqrt(d_head)).
  // mref is the reference maximum of this lane's query, the same in both
  // lanes of the pair; lrun the lane's partial sum of exp2(score - mref).
  // negm holds -mref in every slot and starts the score accumulators, so the
  // MFMAs deliver score - mref and each probability is one exp2. The
  // reference is set from a real maximum on the wave's first tile and kept
  // while the running sums stay below 2^64; a tile that would push one past
  // it (a score more than ~64 above the reference) is redone with a new
  // reference. Rescaling by a power of the reference shift is exact up to
  // rounding, so the result does not depend on when it happens.
  float lrun = 0.0f;
  float mref = -INFINITY;
  f32x16 negm, zero;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    negm[r] = 0.0f;
    zero[r] = 0.0f;
  }
  bool have_ref = false;  // wave-uniform
  constexpr float kSumLimit = 18446744073709551616.0f;  // 2^64

#pragma unroll
  for (int s0 = 0; s0 < S::kNS - 1; ++s0)
    if (s0 < ntiles) issue(s0, s0);

  for (int t = 0; t < ntiles; ++t) {
    const int kt0 = t * S::kKT;
    // tile t has landed for this wave (younger: the tiles after it), then for all
    if constexpr (S::kNS == 3) {
      if (t + 1 < ntiles)
        wait_vmcnt<S::kInstsPerWave>();
      else
        wait_vmcnt<0>();
    } else {
      wait_vmcnt<0>();
    }
    lds_barrier();  // also: every wave is done with tile t-1, whose stage is refilled next
    if (t + S::kNS - 1 < ntiles) issue(t + S::kNS - 1, (t + S::kNS - 1) % S::kNS);
    const char* sk = smem + (t % S::kNS) * S::kStage;
    const char* sv = sk + S::kKParts * S::kKTile;
    const bool active = !p.causal || kt0 <= qw0 + 31;  // uniform across the wave
    if (active) {
      const bool need_mask = (p.causal && kt0 + S::kKT - 1 > qw0) || kt0 + S::kKT > p.m;  // wave-uniform
      const int klim = p.causal ? min(myq, p.m - 1) : p.m - 1;  // last visible key
      // S^T = K Q^T + c0 for 64 keys (two 32-key blocks) x this wave's 32
      // queries, masked entries -inf. The matrix phases run at raised wave
      // priority, so the SIMD's other wave (in its softmax phase) fills the
      // issue slots between MFMAs.
      auto scores = [&](f32x16 (&s)[2], const f32x16& c0) {
        // every fragment read is issued before the first MFMA
        typename MM::frag kh[2][DH / 16];
        i32x8 kx[2][SPLIT ? kXB : 1];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const int kr = kb * 32 + col;  // key row of this lane's A fragment
          const char* krow = sk + kr * S::kRowBytes;
          if constexpr (SPLIT) {
#pragma unroll
            for (int xb = 0; xb < kXB; ++xb) {
              const u32x4 lo = *reinterpret_cast<const u32x4*>(
                  krow + S::kKTile + lds_swz<S::kRowBytes / 16>(kr, xb * 4 + 2 * g) * 16);
              const u32x4 hi = *reinterpret_cast<const u32x4*>(
                  krow + S::kKTile + lds_swz<S::kRowBytes / 16>(kr, xb * 4 + 2 * g + 1) * 16);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                kx[kb][xb][e] = (int)lo[e];
                kx[kb][xb][e + 4] = (int)hi[e];
              }
            }
          }
#pragma unroll
          for (int kk = 0; kk < DH / 16; ++kk) {
            if constexpr (sizeof(T) == 2) {
              const int off = lds_swz<S::kRowBytes / 16>(kr, kk * 2 + g) * 16;
              kh[kb][kk] = *reinterpret_cast<const typename MM::frag*>(krow + off);
            } else {
              const int c0i = kk * 4 + g * 2;
              const f32x4 lo = *reinterpret_cast<const f32x4*>(krow + lds_swz<S::kRowBytes / 16>(kr, c0i) * 16);
              const f32x4 hi = *reinterpret_cast<const f32x4*>(krow + lds_swz<S::kRowBytes / 16>(kr, c0i + 1) * 16);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                kh[kb][kk][e] = lo[e];
                kh[kb][kk][e + 4] = hi[e];
              }
            }
          }
        }
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kk = 0; kk < DH / 16; ++kk)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb) {
            s[kb] = MM::mma(kh[kb][kk], qf[kk], kk == 0 ? c0 : s[kb]);
          }
        if constexpr (SPLIT) {
#pragma unroll
          for (int xb = 0; xb < kXB; ++xb)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) s[kb] = mfma_bf8_scaled(kx[kb][xb], qx[xb], s[kb]);
        }
        __builtin_amdgcn_s_setprio(0);
        if (need_mask) {  // selects, no per-element branches
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int key = kt0 + kb * 32 + acc_row(r, lane);
              s[kb][r] = key > klim ? -INFINITY : s[kb][r];
            }
        }
      };
      // probabilities in place, summed in four chains
      auto exponentiate = [&](f32x16 (&s)[2], float shift) {
        float ls[4];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float e = fast_exp2(s[kb][r] - shift);
            s[kb][r] = e;
            ls[r & 3] = kb == 0 && r < 4 ? e : ls[r & 3] + e;
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
      if (redo) {  // wave-uniform: first tile, or a sum past the limit
        scores(s, zero);
        float mt = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kb][r]);
        mt = fmaxf(mt, other_half(mt));
        // the pair's sum so far in reference units: a shift by its
        // exponent brings it back near 1 when no score of this tile does
        const float ltot = lrun + other_half(lrun);
        const float mnew = fmaxf(mt, mref + fmaxf(0.0f, __log2f(ltot)));
        const float alpha = fast_exp2(mref - mnew);  // 0 while there is no reference
        lrun *= alpha;
#pragma unroll
        for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
        mref = mnew;
#pragma unroll
        for (int r = 0; r < 16; ++r) negm[r] = -mnew;
        have_ref = true;
        tsum = exponentiate(s, mnew);
      }
      lrun += tsum;
      __builtin_amdgcn_s_setprio(1);
      // O^T += V^T P^T, 16 keys per MFMA
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          // bf16: after the swap lane group g holds keys 16*s2 + 8*g .. +7;
          // fp32: no swap, slots 0-3 / 4-7 are keys 16*s2 + 4*g + {0..3} / + 8,
          // each run one 16-byte chunk of V^T.
          typename MM::frag pb;
          if constexpr (sizeof(T) == 2) {
            pb = pt_frag_bf16(s[kb], s2);
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) pb[i] = s[kb][s2 * 8 + i];
          }
          const int c0 = kb * 32 + s2 * 16 + g * 8;  // bf16: first key of this lane's 8
          const int c4 = kb * 32 + s2 * 16 + g * 4;  // fp32: first key of the lane's first run
#pragma unroll
          for (int cb = 0; cb < DH / 32; ++cb) {
            const int d = cb * 32 + col;
            const char* vrow = sv + d * S::kVRowBytes;
            typename MM::frag va;
            if constexpr (sizeof(T) == 2) {
              va = *reinterpret_cast<const typename MM::frag*>(vrow + lds_swz<S::kVRowBytes / 16>(d, c0 / 8) * 16);
            } else {
              const f32x4 lo = *reinterpret_cast<const f32x4*>(vrow + lds_swz<S::kVRowBytes / 16>(d, c4 / 4) * 16);
              const f32x4 hi = *reinterpret_cast<const f32x4*>(vrow + lds_swz<S::kVRowBytes / 16>(d, c4 / 4 + 2) * 16);
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                va[e] = lo[e];
                va[e + 4] = hi[e];
              }
            }
            oacc[cb] = MM::mma(va, pb, oacc[cb]);
          }
        }
    }
  }

  __builtin_amdgcn_s_setprio(0);
  const float ltot = lrun + other_half(lrun);
  if (myq < p.m) {
    const float inv = 1.0f / ltot;
    T* orow = reinterpret_cast<T*>(p.o) + ((int64_t)b * p.m + myq) * ((int64_t)p.n_heads * DH) + h * DH;
#pragma unroll
    for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) orow[cb * 32 + acc_row(r, lane)] = from_f32<T>(oacc[cb][r] * inv);
    if (g == 0) p.lse[(int64_t)bh * p.m + myq] = (mref + __log2f(ltot)) * 0.69314718055994531f;
  }
}

// Ring depth and the occupancy the register allocation targets (waves per
// SIMD). Two stages and a target of 2 measured best for d_head = 64 (a
// target of 3 caps registers at 168 and schedules worse).
template <typename T, int DH, bool SPLIT>
struct AttnFwdCfg {
  static constexpr int kNS = 2;
  static constexpr int kOcc = DH == 64 ? 2 : 1;
};

template <typename T, int DH, bool SPLIT>
static hipError_t launch_fwd_cfg(const AttnParams& p, dim3 grid, hipStream_t stream) {
  typedef AttnFwdCfg<T, DH, SPLIT> C;
  hipLaunchKernelGGL((attn_fwd_kernel<T, DH, SPLIT, C::kNS, C::kOcc>), grid, dim3(256), 0, stream, p);
  return hipGetLastError();
}

template <typename T, int DH>
static hipError_t launch_fwd_dh(const AttnParams& p, dim3 grid, hipStream_t stream) {
  if constexpr (sizeof(T) == 2) {
    if (p.qx && p.kx) return launch_fwd_cfg<T, DH, true>(p, grid, stream);
  }
  return launch_fwd_cfg<T, DH, false>(p, grid, stream);
}

template <typename T>
hipError_t launch_attention_fwd(const AttnParams& p, int batch, int head_dim, hipStream_t stream) {
  if (p.m <= 0) return hipSuccess;  // one head's tensors are below 2 GiB (checked by layer_dims)
  dim3 grid(((p.m + 127) / 128) * batch * p.n_heads);
  if (head_dim == 64) return launch_fwd_dh<T, 64>(p, grid, stream);
  return launch_fwd_dh<T, 128>(p, grid, stream);
}

template hipError_t launch_attention_fwd<bf16>(const AttnParams&, int, int, hipStream_t);
template hipError_t launch_attention_fwd<float>(const AttnParams&, int, int, hipStream_t);

}  // namespace pf
