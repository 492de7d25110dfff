// Backward of the causal multi-head proxy attention (Eq. 9).
//
// With P = softmax(S), S = Q K^T / sqrt(d_head) + M and D_i = sum_c dO_ic O_ic:
//   dV = P^T dO,  dP = dO V^T,  dS = P * (dP - D),  dQ = dS K / sqrt(d_head),
//   dK = dS^T Q / sqrt(d_head).
// P is recomputed from the forward's log-sum-exp. Two kernels, no atomics,
// so every gradient is written once and results are deterministic:
//  - attn_bwd_dkdv_kernel: a workgroup owns 128 keys (4 waves x 32, one key
//    per lane column); it walks the 32-query tiles that can see those keys
//    and accumulates dV^T += dO^T P and dK^T += Q^T dS in registers.
//  - attn_bwd_dq_kernel: a workgroup owns 128 queries and walks the visible
//    32-key tiles, accumulating dQ^T += K^T dS^T.
// Tiles stream into LDS through direct (buffer -> LDS) loads into a ring of
// stages, 16-byte chunks XOR-swizzled per row, as in the forward kernel:
// row-layout tiles (Q, dO or K, V: one position per row) feed the score
// MFMAs, transposed tiles (Q^T, dO^T or K^T, written position-contiguous by
// the producing GEMM epilogues) feed the gradient MFMAs. P and dS stay in
// registers and become the gradient MFMAs' other operand through one
// v_permlane32_swap per register pair (bf16), so the matching transposed
// fragment is one 16-byte read. With SPLIT (bf16 hi/lo parts of Q and K)
// the recomputed scores are Qh Kh + Ql Kh + Qh Kl, matching the forward's
// logits. Workgroups are dealt XCD-contiguous per head (the head's tiles are
// shared in one L2), longest causal range first.
#include "attention.hpp"

namespace pf {

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

// Tile geometry shared by both kernels: kT positions (queries for dK/dV,
// keys for dQ) per tile; a row-layout tile has one position per row (DH
// channels), a transposed tile one channel per row (kT positions).
template <typename T, int DH, bool SPLIT>
struct BwdShape {
  static constexpr int kT = 32;
  static constexpr int kRowB = DH * (int)sizeof(T);   // row-layout row bytes
  static constexpr int kTRowB = kT * (int)sizeof(T);  // transposed row bytes
  static constexpr int kRowTile = kT * kRowB;
  static constexpr int kTTile = DH * kTRowB;
  static constexpr int kParts = SPLIT ? 2 : 1;        // hi (and lo) parts of Q or K
  static constexpr int kRowInsts = kRowTile / 1024;   // 1 KB direct loads per tile
  static constexpr int kTInsts = kTTile / 1024;
  static_assert(kRowTile % 1024 == 0 && kTTile % 1024 == 0, "tiles split into 1 KB loads");
  static_assert(kRowB >= 128 && kTRowB >= 64, "rows of at least 4 chunks");
};


// A-operand fragment of a row-layout tile: row r, k-step kk (bf16: logical
// chunk 2 kk + g; fp32: chunks 4 kk + 2 g and the next).
template <typename T, int kRowB>
__device__ __forceinline__ typename Mma<T>::frag row_frag(const char* tile, int r, int kk, int g) {
  constexpr int C = kRowB / 16;
  const char* row = tile + r * kRowB;
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const bf16x8*>(row + lds_swz<C>(r, kk * 2 + g) * 16);
  } else {
    const f32x4 lo = *reinterpret_cast<const f32x4*>(row + lds_swz<C>(r, kk * 4 + g * 2) * 16);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(row + lds_swz<C>(r, kk * 4 + g * 2 + 1) * 16);
    typename Mma<T>::frag f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = lo[e];
      f[e + 4] = hi[e];
    }
    return f;
  }
}

// Operand of positions 16 s2 .. 16 s2 + 15 of a 32x32 accumulator (positions
// on rows): bf16 lane group g holds positions 16 s2 + 8 g .. + 7 after the
// swap; fp32 slots 0-3 / 4-7 are positions 16 s2 + 4 g + {0..3} / + 8.
template <typename T>
__device__ __forceinline__ typename Mma<T>::frag acc_operand(const f32x16& s, int s2) {
  if constexpr (sizeof(T) == 2) {
    return pt_frag_bf16(s, s2);
  } else {
    typename Mma<T>::frag f;
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = s[s2 * 8 + i];
    return f;
  }
}

// The matching fragment of a transposed tile: channel row d.
template <typename T, int kTRowB>
__device__ __forceinline__ typename Mma<T>::frag t_frag(const char* tile, int d, int s2, int g) {
  constexpr int C = kTRowB / 16;
  const char* row = tile + d * kTRowB;
  if constexpr (sizeof(T) == 2) {
    return *reinterpret_cast<const bf16x8*>(row + lds_swz<C>(d, s2 * 2 + g) * 16);
  } else {
    const f32x4 lo = *reinterpret_cast<const f32x4*>(row + lds_swz<C>(d, s2 * 4 + g) * 16);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(row + lds_swz<C>(d, s2 * 4 + g + 2) * 16);
    typename Mma<T>::frag f;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = lo[e];
      f[e + 4] = hi[e];
    }
    return f;
  }
}

// Direct loads of one row-layout tile block (1 KB) and one transposed tile
// block: lane -> (row, physical chunk); the global side fetches the logical
// chunk that lands there.
template <int kRowB>
__device__ __forceinline__ uint32_t row_voff(int blk, int lane) {
  constexpr int C = kRowB / 16;
  const int r = blk * (1024 / kRowB) + lane / C, pc = lane % C;
  return (uint32_t)(r * kRowB + lds_swz<C>(r, pc) * 16);
}
template <int kTRowB>
__device__ __forceinline__ uint32_t t_voff(int blk, int lane, int64_t ld_bytes) {
  constexpr int C = kTRowB / 16;
  const int r = blk * (1024 / kTRowB) + lane / C, pc = lane % C;
  return (uint32_t)(r * ld_bytes + lds_swz<C>(r, pc) * 16);
}

// Stages of kInsts 1 KB loads are dealt to the four waves in contiguous
// runs of kPer (the last wave takes the remainder).
template <int kInsts>
struct StageDeal {
  static constexpr int kPer = (kInsts + 3) / 4;
  static_assert(kInsts - 3 * kPer > 0 && kPer < 64, "every wave loads, within the vmcnt range");
};
// Waits until at most one younger stage of this wave's loads is in flight.
template <int kInsts>
__device__ __forceinline__ void wait_one_younger(int wave) {
  constexpr int kPer = StageDeal<kInsts>::kPer;
  if (wave == 3)
    wait_vmcnt<kInsts - 3 * kPer>();
  else
    wait_vmcnt<kPer>();
}

// Four consecutive outputs (4 channels of one row), one 8- or 16-byte store.
__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  uint2 w;
  w.x = pack_bf16x2(a, b);
  w.y = pack_bf16x2(c, d);
  *reinterpret_cast<uint2*>(p) = w;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *reinterpret_cast<f32x4*>(p) = v;
}

// Writes a DH x 32 accumulator (channels on rows, this lane's position on
// the column) times `scale` to row `orow` of a [B*m, h*DH] gradient.
template <typename T, int DH>
__device__ __forceinline__ void store_rowgrad(T* out, int64_t orow, const f32x16 (&acc)[DH / 32], float scale,
                                              int lane) {
#pragma unroll
  for (int cb = 0; cb < DH / 32; ++cb)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int c = cb * 32 + acc_row(r4 * 4, lane);  // rows r4*4 .. +3 are 4 consecutive channels
      store4(out + orow + c, acc[cb][r4 * 4] * scale, acc[cb][r4 * 4 + 1] * scale, acc[cb][r4 * 4 + 2] * scale,
             acc[cb][r4 * 4 + 3] * scale);
    }
}

// XCD-contiguous deal of a 1-D grid over (head, block): consecutive
// workgroup ids go round robin over the XCDs, so the id is remapped to give
// every XCD a contiguous run of (head, block) pairs.
__device__ __forceinline__ int xcd_order() {
  const int total = (int)gridDim.x;
  const int q = total / kNumXcd, rem = total % kNumXcd;
  const int wg = blockIdx.x, xcd = wg % kNumXcd, local = wg / kNumXcd;
  return (xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q) + local;
}

template <typename T, int DH, bool SPLIT>
struct DkdvCfg {
  typedef BwdShape<T, DH, SPLIT> S;
  // stage (bytes): Q | Q_lo | dO | Q^T | dO^T | LSE (1 KB) | D (1 KB)
  static constexpr int oDO = S::kParts * S::kRowTile;
  static constexpr int oQT = oDO + S::kRowTile;
  static constexpr int oDOT = oQT + S::kTTile;
  static constexpr int oL = oDOT + S::kTTile;
  static constexpr int oD = oL + 1024;
  static constexpr int kStage = oD + 1024;
  static constexpr int kInsts = (S::kParts + 1) * S::kRowInsts + 2 * S::kTInsts + 2;
  static constexpr int kNS = (DH == 64 && 3 * kStage <= 160 * 1024) ? 3 : 2;
};

template <typename T, int DH, bool SPLIT>
__global__ void __launch_bounds__(256) attn_bwd_dkdv_kernel(const AttnBwdParams p) {
  typedef BwdShape<T, DH, SPLIT> S;
  typedef DkdvCfg<T, DH, SPLIT> C;
  typedef Mma<T> MM;
  constexpr int QT = S::kT, NS = C::kNS;
  constexpr int es = (int)sizeof(T);
  __shared__ __attribute__((aligned(1024))) char smem[NS * C::kStage];

  const int nkb = (p.m + 127) / 128;
  const int t0 = xcd_order();
  const int bh = t0 / nkb, kblk = t0 % nkb;  // key block 0 sees the most queries
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, col = lane & 31;
  const int m = p.m;
  const int k0 = kblk * 128;
  const int kw0 = k0 + wave * 32;
  const int mykey = kw0 + col;
  const int64_t hoff = (int64_t)bh * m * DH;

  // this wave's keys and values as B operands (column = key)
  typename MM::frag kf[DH / 16], kfl[SPLIT ? DH / 16 : 1], vf[DH / 16];
  {
    const T* kg = reinterpret_cast<const T*>(p.k) + hoff;
    const T* vg = reinterpret_cast<const T*>(p.v) + hoff;
    const T* klg = SPLIT ? reinterpret_cast<const T*>(p.k_lo) + hoff : nullptr;
    const int kr = min(mykey, m - 1);  // rows past m are zeroed below
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      kf[kk] = MM::load(kg + (int64_t)kr * DH + kk * 16 + g * 8);
      vf[kk] = MM::load(vg + (int64_t)kr * DH + kk * 16 + g * 8);
      if constexpr (SPLIT) kfl[kk] = MM::load(klg + (int64_t)kr * DH + kk * 16 + g * 8);
      if (mykey >= m) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          kf[kk][i] = vf[kk][i] = (T)0.0f;
          if constexpr (SPLIT) kfl[kk][i] = (T)0.0f;
        }
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
  const int ntiles = nqt - qt_begin;
  const char* qg = reinterpret_cast<const char*>(p.q) + hoff * es;
  const char* qlg = SPLIT ? reinterpret_cast<const char*>(p.q_lo) + hoff * es : nullptr;
  const char* dog = reinterpret_cast<const char*>(p.do_) + hoff * es;
  const int64_t toff = (int64_t)bh * DH * p.ld_t * es;
  const char* qtg = reinterpret_cast<const char*>(p.qt) + toff;
  const char* dotg = reinterpret_cast<const char*>(p.dot) + toff;
  const int64_t ld_b = (int64_t)p.ld_t * es;

  // Direct loads of one stage: wave w issues loads [w kPer, (w + 1) kPer)
  // of the stage (wave-uniform index, scalar branches).
  auto issue = [&](int t, int stage) {
    const int q0 = (qt_begin + t) * QT;
    char* st = smem + stage * C::kStage;
    const uint32_t rows_b = (uint32_t)(m - q0) * S::kRowB;  // rows past m read as zero
    const uint32_t t_b = (uint32_t)((int64_t)DH * ld_b - (int64_t)q0 * es);
    const uint32_t v_b = (uint32_t)(m - q0) * 4u;
    const rsrc_t rq = make_rsrc_uniform(qg + (int64_t)q0 * S::kRowB, rows_b);
    const rsrc_t rql = SPLIT ? make_rsrc_uniform(qlg + (int64_t)q0 * S::kRowB, rows_b) : rq;
    const rsrc_t rdo = make_rsrc_uniform(dog + (int64_t)q0 * S::kRowB, rows_b);
    const rsrc_t rqt = make_rsrc_uniform(qtg + (int64_t)q0 * es, t_b);
    const rsrc_t rdot = make_rsrc_uniform(dotg + (int64_t)q0 * es, t_b);
    const rsrc_t rl = make_rsrc_uniform(p.lse + (int64_t)bh * m + q0, v_b);
    const rsrc_t rd = make_rsrc_uniform(p.delta + (int64_t)bh * m + q0, v_b);
    constexpr int kRowAll = (S::kParts + 1) * S::kRowInsts;
    constexpr int kPer = StageDeal<C::kInsts>::kPer;
#pragma unroll
    for (int jj = 0; jj < kPer; ++jj) {
      const int i = wave * kPer + jj;  // wave-uniform
      if (i >= C::kInsts) continue;
      if (i < kRowAll) {
        const int part = i / S::kRowInsts;
        buf_ld16_lds(part == 0 ? rq : (SPLIT && part == 1 ? rql : rdo), row_voff<S::kRowB>(i % S::kRowInsts, lane),
                     st + i * 1024);
      } else if (i < kRowAll + 2 * S::kTInsts) {
        const int j = i - kRowAll;
        buf_ld16_lds(j < S::kTInsts ? rqt : rdot, t_voff<S::kTRowB>(j % S::kTInsts, lane, ld_b),
                     st + C::oQT + j * 1024);
      } else {
        const bool is_l = i == C::kInsts - 2;
        buf_ld16_lds(is_l ? rl : rd, lane < QT / 4 ? (uint32_t)lane * 16u : kOOB, st + (is_l ? C::oL : C::oD));
      }
    }
  };

#pragma unroll
  for (int s0 = 0; s0 < NS - 1; ++s0)
    if (s0 < ntiles) issue(s0, s0);
  for (int t = 0; t < ntiles; ++t) {
    // tile t has landed for this wave (younger: at most one more stage), then for all
    if (NS == 3 && t + 1 < ntiles)
      wait_one_younger<C::kInsts>(wave);
    else
      wait_vmcnt<0>();
    lds_barrier();  // also: every wave is done with the stage refilled next
    if (t + NS - 1 < ntiles) issue(t + NS - 1, (t + NS - 1) % NS);
    const int q0 = (qt_begin + t) * QT;
    if (p.causal && q0 + QT - 1 < kw0) continue;  // every query of the tile precedes this wave's keys
    const char* st = smem + (t % NS) * C::kStage;
    // S = Q K^T and dP = dO V^T: 32 queries (rows) x this wave's 32 keys
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.0f;
    // fragments one k-step ahead of their MFMAs; the fences keep the
    // compiler from hoisting every read of the tile (register pressure)
    typename MM::frag fq[2], fql[2], fo[2];
    auto ld = [&](int kk, int u) {
      fq[u] = row_frag<T, S::kRowB>(st, col, kk, g);
      if constexpr (SPLIT) fql[u] = row_frag<T, S::kRowB>(st + S::kRowTile, col, kk, g);
      fo[u] = row_frag<T, S::kRowB>(st + C::oDO, col, kk, g);
    };
    ld(0, 0);
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      const int u = kk & 1;
      if (kk + 1 < DH / 16) ld(kk + 1, u ^ 1);
      s = MM::mma(fq[u], kf[kk], s);
      if constexpr (SPLIT) {
        s = MM::mma(fql[u], kf[kk], s);
        s = MM::mma(fq[u], kfl[kk], s);
      }
      dp = MM::mma(fo[u], vf[kk], dp);
      __builtin_amdgcn_sched_barrier(0);
    }
    // LSE and D of this lane's 16 query rows: four runs of four queries
    const float* sl = reinterpret_cast<const float*>(st + C::oL);
    const float* sd = reinterpret_cast<const float*>(st + C::oD);
    const bool need_mask = (p.causal && q0 < kw0 + 31) || q0 + QT > m;
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(sl + acc_row(r4 * 4, lane));
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(sd + acc_row(r4 * 4, lane));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = r4 * 4 + e;
        float pv = fast_exp2(fmaf(s[r], p.scale_log2, -l4[e] * 1.4426950408889634f));
        if (need_mask) {
          const int q = q0 + acc_row(r, lane);
          pv = (q < m && (!p.causal || mykey <= q)) ? pv : 0.0f;
        }
        s[r] = pv;
        dp[r] = pv * (dp[r] - d4[e]);
      }
    }
    // dV^T += dO^T P and dK^T += Q^T dS, 16 queries per MFMA
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const typename MM::frag pb = acc_operand<T>(s, s2);
      const typename MM::frag db = acc_operand<T>(dp, s2);
#pragma unroll
      for (int cb = 0; cb < DH / 32; ++cb) {
        const int d = cb * 32 + col;
        dvt[cb] = MM::mma(t_frag<T, S::kTRowB>(st + C::oDOT, d, s2, g), pb, dvt[cb]);
        dkt[cb] = MM::mma(t_frag<T, S::kTRowB>(st + C::oQT, d, s2, g), db, dkt[cb]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if (mykey < m) {
    const int64_t orow = ((int64_t)b * m + mykey) * ((int64_t)p.n_heads * DH) + h * DH;
    store_rowgrad<T, DH>(reinterpret_cast<T*>(p.dv), orow, dvt, 1.0f, lane);
    store_rowgrad<T, DH>(reinterpret_cast<T*>(p.dk), orow, dkt, p.scale, lane);
  }
}

template <typename T, int DH, bool SPLIT>
struct DqCfg {
  typedef BwdShape<T, DH, SPLIT> S;
  // stage (bytes): K | K_lo | V | K^T
  static constexpr int oV = S::kParts * S::kRowTile;
  static constexpr int oKT = oV + S::kRowTile;
  static constexpr int kStage = oKT + S::kTTile;
  static constexpr int kInsts = (S::kParts + 1) * S::kRowInsts + S::kTInsts;
  static constexpr int kNS = (DH == 64 && 3 * kStage <= 160 * 1024) ? 3 : 2;
};

template <typename T, int DH, bool SPLIT>
__global__ void __launch_bounds__(256) attn_bwd_dq_kernel(const AttnBwdParams p) {
  typedef BwdShape<T, DH, SPLIT> S;
  typedef DqCfg<T, DH, SPLIT> C;
  typedef Mma<T> MM;
  constexpr int KT = S::kT, NS = C::kNS;
  constexpr int es = (int)sizeof(T);
  __shared__ __attribute__((aligned(1024))) char smem[NS * C::kStage];

  const int nqb = (p.m + 127) / 128;
  const int t0 = xcd_order();
  const int bh = t0 / nqb, qblk = nqb - 1 - t0 % nqb;  // the last query block sees the most keys
  const int b = bh / p.n_heads, h = bh % p.n_heads;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, col = lane & 31;
  const int m = p.m;
  const int q0 = qblk * 128;
  const int qw0 = q0 + wave * 32;
  const int myq = qw0 + col;
  const int64_t hoff = (int64_t)bh * m * DH;

  // this wave's queries as B operands (column = query)
  typename MM::frag qf[DH / 16], qfl[SPLIT ? DH / 16 : 1], dof[DH / 16];
  {
    const T* qg = reinterpret_cast<const T*>(p.q) + hoff;
    const T* dog = reinterpret_cast<const T*>(p.do_) + hoff;
    const T* qlg = SPLIT ? reinterpret_cast<const T*>(p.q_lo) + hoff : nullptr;
    const int qr = min(myq, m - 1);
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      qf[kk] = MM::load(qg + (int64_t)qr * DH + kk * 16 + g * 8);
      dof[kk] = MM::load(dog + (int64_t)qr * DH + kk * 16 + g * 8);
      if constexpr (SPLIT) qfl[kk] = MM::load(qlg + (int64_t)qr * DH + kk * 16 + g * 8);
      if (myq >= m) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          qf[kk][i] = dof[kk][i] = (T)0.0f;
          if constexpr (SPLIT) qfl[kk][i] = (T)0.0f;
        }
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
  const char* kg = reinterpret_cast<const char*>(p.k) + hoff * es;
  const char* klg = SPLIT ? reinterpret_cast<const char*>(p.k_lo) + hoff * es : nullptr;
  const char* vg = reinterpret_cast<const char*>(p.v) + hoff * es;
  const char* ktg = reinterpret_cast<const char*>(p.kt) + (int64_t)bh * DH * p.ld_t * es;
  const int64_t ld_b = (int64_t)p.ld_t * es;

  auto issue = [&](int t, int stage) {
    const int kt0 = t * KT;
    char* st = smem + stage * C::kStage;
    const uint32_t rows_b = (uint32_t)(m - kt0) * S::kRowB;
    const uint32_t t_b = (uint32_t)((int64_t)DH * ld_b - (int64_t)kt0 * es);
    const rsrc_t rk = make_rsrc_uniform(kg + (int64_t)kt0 * S::kRowB, rows_b);
    const rsrc_t rkl = SPLIT ? make_rsrc_uniform(klg + (int64_t)kt0 * S::kRowB, rows_b) : rk;
    const rsrc_t rv = make_rsrc_uniform(vg + (int64_t)kt0 * S::kRowB, rows_b);
    const rsrc_t rkt = make_rsrc_uniform(ktg + (int64_t)kt0 * es, t_b);
    constexpr int kRowAll = (S::kParts + 1) * S::kRowInsts;
    constexpr int kPer = StageDeal<C::kInsts>::kPer;
#pragma unroll
    for (int jj = 0; jj < kPer; ++jj) {
      const int i = wave * kPer + jj;  // wave-uniform
      if (i >= C::kInsts) continue;
      if (i < kRowAll) {
        const int part = i / S::kRowInsts;
        buf_ld16_lds(part == 0 ? rk : (SPLIT && part == 1 ? rkl : rv), row_voff<S::kRowB>(i % S::kRowInsts, lane),
                     st + i * 1024);
      } else {
        buf_ld16_lds(rkt, t_voff<S::kTRowB>(i - kRowAll, lane, ld_b), st + i * 1024);
      }
    }
  };

#pragma unroll
  for (int s0 = 0; s0 < NS - 1; ++s0)
    if (s0 < ntiles) issue(s0, s0);
  for (int t = 0; t < ntiles; ++t) {
    if (NS == 3 && t + 1 < ntiles)
      wait_one_younger<C::kInsts>(wave);
    else
      wait_vmcnt<0>();
    lds_barrier();
    if (t + NS - 1 < ntiles) issue(t + NS - 1, (t + NS - 1) % NS);
    const int kt0 = t * KT;
    if (p.causal && kt0 > qw0 + 31) continue;  // every key of the tile follows this wave's queries
    const char* st = smem + (t % NS) * C::kStage;
    // S^T = K Q^T and dP^T = V dO^T: 32 keys (rows) x this wave's 32 queries
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.0f;
    typename MM::frag fk[2], fkl[2], fv[2];
    auto ld = [&](int kk, int u) {
      fk[u] = row_frag<T, S::kRowB>(st, col, kk, g);
      if constexpr (SPLIT) fkl[u] = row_frag<T, S::kRowB>(st + S::kRowTile, col, kk, g);
      fv[u] = row_frag<T, S::kRowB>(st + C::oV, col, kk, g);
    };
    ld(0, 0);
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      const int u = kk & 1;
      if (kk + 1 < DH / 16) ld(kk + 1, u ^ 1);
      s = MM::mma(fk[u], qf[kk], s);
      if constexpr (SPLIT) {
        s = MM::mma(fkl[u], qf[kk], s);
        s = MM::mma(fk[u], qfl[kk], s);
      }
      dp = MM::mma(fv[u], dof[kk], dp);
      __builtin_amdgcn_sched_barrier(0);
    }
    const bool need_mask = (p.causal && kt0 + KT - 1 > qw0) || kt0 + KT > m;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float pv = fast_exp2(fmaf(s[r], p.scale_log2, -lse2));
      if (need_mask) {
        const int key = kt0 + acc_row(r, lane);
        pv = (key < m && myq < m && (!p.causal || key <= myq)) ? pv : 0.0f;
      }
      s[r] = pv * (dp[r] - dlt);  // dS^T
    }
    // dQ^T += K^T dS^T, 16 keys per MFMA
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const typename MM::frag db = acc_operand<T>(s, s2);
#pragma unroll
      for (int cb = 0; cb < DH / 32; ++cb)
        dqt[cb] = MM::mma(t_frag<T, S::kTRowB>(st + C::oKT, cb * 32 + col, s2, g), db, dqt[cb]);
    }
  }
  if (myq < m) {
    const int64_t orow = ((int64_t)b * m + myq) * ((int64_t)p.n_heads * DH) + h * DH;
    store_rowgrad<T, DH>(reinterpret_cast<T*>(p.dq), orow, dqt, p.scale, lane);
  }
}

template <typename T, int DH, bool SPLIT>
static void launch_bwd_cfg(const AttnBwdParams& p, int batch, hipStream_t stream) {
  const unsigned blocks = (unsigned)(((p.m + 127) / 128) * batch * p.n_heads);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, DH, SPLIT>), dim3(blocks), dim3(256), 0, stream, p);
  hipLaunchKernelGGL((attn_bwd_dq_kernel<T, DH, SPLIT>), dim3(blocks), dim3(256), 0, stream, p);
}

template <typename T>
hipError_t launch_attention_bwd(const AttnBwdParams& p, int batch, int head_dim, hipStream_t stream) {
  if (p.m <= 0) return hipSuccess;  // one head's tensors are below 2 GiB (checked by layer_dims)
  const int64_t rows = (int64_t)batch * p.n_heads * p.m;
  const dim3 dgrid((unsigned)((rows + 3) / 4));
  const bool split = sizeof(T) == 2 && p.q_lo && p.k_lo;
  constexpr bool kSplit = sizeof(T) == 2;
  if (head_dim == 64) {
    hipLaunchKernelGGL((attn_bwd_delta_kernel<T, 64>), dgrid, dim3(256), 0, stream,
                       reinterpret_cast<const T*>(p.do_), reinterpret_cast<const T*>(p.o), p.delta, p.m, p.n_heads, rows);
    if (split)
      launch_bwd_cfg<T, 64, kSplit>(p, batch, stream);
    else
      launch_bwd_cfg<T, 64, false>(p, batch, stream);
  } else {
    hipLaunchKernelGGL((attn_bwd_delta_kernel<T, 128>), dgrid, dim3(256), 0, stream,
                       reinterpret_cast<const T*>(p.do_), reinterpret_cast<const T*>(p.o), p.delta, p.m, p.n_heads, rows);
    if (split)
      launch_bwd_cfg<T, 128, kSplit>(p, batch, stream);
    else
      launch_bwd_cfg<T, 128, false>(p, batch, stream);
  }
  return hipGetLastError();
}

template hipError_t launch_attention_bwd<bf16>(const AttnBwdParams&, int, int, hipStream_t);
template hipError_t launch_attention_bwd<float>(const AttnBwdParams&, int, int, hipStream_t);

}  // namespace pf
