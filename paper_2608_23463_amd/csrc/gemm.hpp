// Tiled MFMA GEMM for gfx950 with pluggable epilogues.
//
// Computes C[m][n] = sum_k A(m, k) * B(n, k) for m < M, n < N, k < K and hands
// every fp32 result to an epilogue functor epi(row, col, value).
//  A(m,k): LAYOUT_K  -> A[m * lda + k]  (row-major, reduction contiguous)
//          LAYOUT_MN -> A[k * lda + m]  (reduction strided)
//  B(n,k): LAYOUT_K  -> B[n * ldb + k]  (a weight stored [out, in])
//          LAYOUT_MN -> B[k * ldb + n]
// Optional concatenation along K, handled in the tile loader (LAYOUT_K
// operands): for k >= a_ksplit the A values come from A2
// (A2[m * lda2 + k - a_ksplit]), and for k >= b_ksplit the B values from B2.
// Used for the gate input [X, Delta], and for the split-precision products
// [X_hi | X_lo] [W | W]^T = X W^T to ~16 mantissa bits.
// Split-K: gridDim.z slices of the reduction range, each slice handing its
// partial sums to the epilogue (normally a store into an fp32 workspace,
// reduced afterwards in a fixed order, so results are deterministic).
//
// Design: a workgroup owns a BM x BN tile, WM x WN waves each own a
// (BM/WM) x (BN/WN) sub-tile made of 32x32 MFMA tiles. K advances BK at a
// time through two LDS buffers; the next K slice is fetched from global
// memory into registers while the current one is multiplied. Operands in
// LAYOUT_MN are transposed in registers (VEC x VEC blocks) before they are
// written to LDS, so LDS always holds rows contiguous along K and every lane
// reads its MFMA fragment with 16-byte LDS reads. Rows are padded by 16 bytes
// so that the 32 rows a fragment read touches fall in distinct banks.
// Workgroups are dealt to the 8 XCDs round-robin; the tile index is remapped
// so that each XCD works on a contiguous band of tiles (shared L2), and
// within the band GROUP_M row tiles are visited per column sweep.
#pragma once

#include <algorithm>
#include <type_traits>

#include "common.hpp"

namespace pf {

enum { LAYOUT_K = 0, LAYOUT_MN = 1 };

// Longest operand row (bytes) a GEMM takes: a tile addresses up to 256 rows
// through one 32-bit buffer range that must stay below the out-of-range
// offset kOOB = 2^31.
constexpr int64_t kMaxGemmRowBytes = (int64_t)1 << 23;

struct GemmParams {
  const void* a;
  int64_t lda;
  const void* a2;
  int64_t lda2;
  int a_ksplit;        // K index where A2 starts (>= K: unused)
  const void* b;
  int64_t ldb;
  const void* b2;
  int64_t ldb2;
  int b_ksplit;        // K index where B2 starts (>= K: unused)
  int M, N, K;
  int k_slice;         // reduction length per gridDim.z slice (multiple of BK)
  int tiles_m, tiles_n;
  int group_m;
  int64_t batch_a, batch_b;  // element offsets of batch blockIdx.y in A and B (direct kernel)
};

template <typename T, int BM, int BN, int BK, int WM, int WN>
struct GemmShape {
  static constexpr int kThreads = WM * WN * kWave;
  static constexpr int kVec = 16 / sizeof(T);  // elements per 16-byte access
  static constexpr int kStride = BK + kVec;    // LDS row stride (elements)
  static constexpr int kTM = BM / WM, kTN = BN / WN;
  static constexpr int kFM = kTM / 32, kFN = kTN / 32;
  static constexpr int kALoads = BM * BK / (kThreads * kVec);
  static constexpr int kBLoads = BN * BK / (kThreads * kVec);
  static constexpr int kStageElems = (BM + BN) * kStride;
  static constexpr size_t kLdsBytes = 2 * kStageElems * sizeof(T);
  static_assert(BK % 16 == 0, "BK must hold whole k16 steps");
  static_assert(kTM % 32 == 0 && kTN % 32 == 0, "wave tile must be whole 32x32 MFMA tiles");
  static_assert((BM * BK) % (kThreads * kVec) == 0, "A tile must split evenly");
  static_assert((BN * BK) % (kThreads * kVec) == 0, "B tile must split evenly");
};

// ---- tile loaders: global -> registers -> LDS ------------------------------
//
// Both loaders use buffer loads: the per-thread byte offsets inside a tile are
// computed once; each K step only rebuilds the (scalar) descriptor whose base
// is the tile's first element and whose byte range ends at the operand's
// edge, so out-of-range rows and K rows read as zero in hardware.

// Rows of the tile are contiguous along K in global memory.
template <typename T, int ROWS, int BK, int NT, bool IS_A>
struct LoaderK {
  static constexpr int kVec = 16 / sizeof(T);
  static constexpr int kChunks = BK / kVec;  // 16-byte chunks per row
  static constexpr int kLoads = ROWS * BK / (NT * kVec);

  uint32_t voff[kLoads];  // byte offset of each chunk from the tile's first element
  int kc[kLoads];         // K offset (elements) of each chunk inside the tile
  const char* src1;       // row row0 of the primary source
  const char* src2;       // row row0 of the source after the K split
  int64_t ld_bytes;
  uint32_t row_bytes_valid;  // bytes spanned by the valid rows of the tile
  int ksplit;

  __device__ __forceinline__ void init(const GemmParams& p, int row0, int rows_total, int tid) {
    const int64_t ld = IS_A ? p.lda : p.ldb;
    ld_bytes = ld * (int64_t)sizeof(T);
    src1 = reinterpret_cast<const char*>(IS_A ? p.a : p.b) + row0 * ld_bytes;
    const void* s2 = IS_A ? p.a2 : p.b2;
    src2 = s2 ? reinterpret_cast<const char*>(s2) + row0 * ld_bytes : nullptr;  // same row stride
    ksplit = IS_A ? p.a_ksplit : p.b_ksplit;
    const int valid = max(0, min(ROWS, rows_total - row0));
    row_bytes_valid = (uint32_t)(valid * ld_bytes);
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int v = tid + i * NT;
      kc[i] = (v % kChunks) * kVec;
      voff[i] = (uint32_t)((v / kChunks) * ld_bytes + kc[i] * (int)sizeof(T));
    }
  }

  // One K step [k0, k0 + BK) clipped to kend.
  __device__ __forceinline__ void fetch(u32x4 (&r)[kLoads], int k0, int kend) const {
    const bool partial = k0 + BK > kend;
    if (k0 + BK <= ksplit || k0 >= ksplit) {
      const bool second = k0 >= ksplit;
      const int krel = second ? k0 - ksplit : k0;
      const rsrc_t rs = make_rsrc((second ? src2 : src1) + (int64_t)krel * sizeof(T),
                                  row_bytes_valid - (uint32_t)(krel * sizeof(T)));
      if (!partial) {
#pragma unroll
        for (int i = 0; i < kLoads; ++i) r[i] = buf_ld16(rs, voff[i]);
      } else {
#pragma unroll
        for (int i = 0; i < kLoads; ++i) r[i] = buf_ld16(rs, k0 + kc[i] < kend ? voff[i] : kOOB);
      }
    } else {
      // the tile straddles the split: read each chunk from its source
      const rsrc_t r1 = make_rsrc(src1 + (int64_t)k0 * sizeof(T), row_bytes_valid - (uint32_t)(k0 * sizeof(T)));
      const rsrc_t r2 = make_rsrc(src2 + (int64_t)(k0 - ksplit) * (int64_t)sizeof(T),
                                  row_bytes_valid + (uint32_t)((ksplit - k0) * sizeof(T)));
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        const int k = k0 + kc[i];
        const bool ok = k < kend;
        const u32x4 a = buf_ld16(r1, ok && k < ksplit ? voff[i] : kOOB);
        const u32x4 b = buf_ld16(r2, ok && k >= ksplit ? voff[i] : kOOB);
        r[i] = a | b;
      }
    }
  }

  static __device__ __forceinline__ void stash(const u32x4 (&r)[kLoads], T* lds, int stride, int tid) {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) {
      const int v = tid + i * NT;
      st16(lds + (v / kChunks) * stride + (v % kChunks) * kVec, r[i]);
    }
  }
};

// Tile rows are contiguous along M (or N) in global memory: element (row, k)
// sits at base[k * ld + row]. Each thread fetches VEC x VEC blocks and
// transposes them in registers.
template <typename T, int ROWS, int BK, int NT, bool IS_A>
struct LoaderMN {
  static constexpr int kVec = 16 / sizeof(T);
  static constexpr int kRowBlocks = ROWS / kVec;
  static constexpr int kTotalBlocks = ROWS * BK / (kVec * kVec);
  static constexpr int kBlocks = (kTotalBlocks + NT - 1) / NT;  // blocks per thread (some idle)
  static constexpr int kLoads = kBlocks * kVec;
  static_assert(ROWS % kVec == 0 && BK % kVec == 0, "tile must hold whole VEC x VEC blocks");

  uint32_t voff[kLoads];
  const char* src;
  int64_t ld_bytes;

  __device__ __forceinline__ void init(const GemmParams& p, int row0, int rows_total, int tid) {
    const int64_t ld = IS_A ? p.lda : p.ldb;
    ld_bytes = ld * (int64_t)sizeof(T);
    src = reinterpret_cast<const char*>(IS_A ? p.a : p.b) + (int64_t)row0 * sizeof(T);
#pragma unroll
    for (int bi = 0; bi < kBlocks; ++bi) {
      const int blk = tid + bi * NT;
      const int row = (blk % kRowBlocks) * kVec;
      const int kb = (blk / kRowBlocks) * kVec;
      const bool active = ((kTotalBlocks % NT == 0) || blk < kTotalBlocks) && row0 + row < rows_total;
#pragma unroll
      for (int t = 0; t < kVec; ++t)
        voff[bi * kVec + t] = active ? (uint32_t)((kb + t) * ld_bytes + row * (int)sizeof(T)) : kOOB;
    }
  }

  __device__ __forceinline__ void fetch(u32x4 (&r)[kLoads], int k0, int kend) const {
    // the range covers this step's K rows below kend only, so it stays below
    // kOOB (idle blocks) however long K is
    const rsrc_t rs = make_rsrc(src + (int64_t)k0 * ld_bytes, (uint32_t)(max(0, min(BK, kend - k0)) * ld_bytes));
#pragma unroll
    for (int i = 0; i < kLoads; ++i) r[i] = buf_ld16(rs, voff[i]);
  }

  static __device__ __forceinline__ void stash(const u32x4 (&r)[kLoads], T* lds, int stride, int tid) {
#pragma unroll
    for (int bi = 0; bi < kBlocks; ++bi) {
      const int blk = tid + bi * NT;
      if ((kTotalBlocks % NT) != 0 && blk >= kTotalBlocks) continue;
      const int row = (blk % kRowBlocks) * kVec;
      const int kb = (blk / kRowBlocks) * kVec;
      const u32x4* in = &r[bi * kVec];
      if constexpr (sizeof(T) == 2) {
        // 8x8 block of 16-bit values: in[t] = k-row t, halves = rows.
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          u32x4 o;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t x = in[2 * w][c >> 1];
            const uint32_t y = in[2 * w + 1][c >> 1];
            o[w] = (c & 1) ? ((x >> 16) | (y & 0xffff0000u)) : ((x & 0xffffu) | (y << 16));
          }
          st16(lds + (row + c) * stride + kb, o);
        }
      } else {
        // 4x4 block of 32-bit values.
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          u32x4 o;
#pragma unroll
          for (int w = 0; w < 4; ++w) o[w] = in[w][c];
          st16(lds + (row + c) * stride + kb, o);
        }
      }
    }
  }
};

template <typename T, int ROWS, int BK, int NT, bool IS_A, int LAYOUT>
using Loader = typename std::conditional<LAYOUT == LAYOUT_K, LoaderK<T, ROWS, BK, NT, IS_A>,
                                         LoaderMN<T, ROWS, BK, NT, IS_A>>::type;

// Tile index remap: contiguous bands per XCD, GROUP_M-row column sweeps.
__device__ __forceinline__ void tile_coords(const GemmParams& p, int& tm, int& tn) {
  const int T = p.tiles_m * p.tiles_n;
  const int wg = blockIdx.x;
  const int q = T / kNumXcd, rem = T % kNumXcd;
  const int xcd = wg % kNumXcd, local = wg / kNumXcd;
  const int t = (xcd < rem ? xcd * (q + 1) : rem * (q + 1) + (xcd - rem) * q) + local;
  const int gsz = p.group_m * p.tiles_n;
  const int g = t / gsz;
  const int first_m = g * p.group_m;
  const int gm = min(p.tiles_m - first_m, p.group_m);
  const int w = t % gsz;
  tm = first_m + w % gm;
  tn = w / gm;
}

// Optional two-phase epilogue protocol. An epilogue that defines the types
// Col and Pre with methods col(c, Col&), pre(r, c, Pre&) and
// vec8(r, c, v, const Col&, const Pre&) has its column data (a bias) read
// once per thread and its row data (tensors it combines with) read for a
// whole group of chunks before any result is formed or stored. Global loads
// and stores share one in-order counter, so reads issued before the stores
// are never held up behind them.
struct NoData {};
template <class Epi, class = void>
struct EpiCol {
  typedef NoData type;
};
template <class Epi>
struct EpiCol<Epi, std::void_t<typename Epi::Col>> {
  typedef typename Epi::Col type;
};
template <class Epi, class = void>
struct EpiPre {
  typedef NoData type;
};
template <class Epi>
struct EpiPre<Epi, std::void_t<typename Epi::Pre>> {
  typedef typename Epi::Pre type;
};
template <class Epi>
constexpr bool kEpiTwoPhase = !std::is_same<typename EpiCol<Epi>::type, NoData>::value;
template <class Epi>
__device__ __forceinline__ void epi_col(const Epi& e, int c, typename EpiCol<Epi>::type& col) {
  if constexpr (kEpiTwoPhase<Epi>) e.col(c, col);
}
template <class Epi>
__device__ __forceinline__ void epi_pre(const Epi& e, int r, int c, typename EpiPre<Epi>::type& pre) {
  if constexpr (kEpiTwoPhase<Epi>) e.pre(r, c, pre);
}
template <class Epi>
__device__ __forceinline__ void epi_vec8(const Epi& e, int r, int c, const float* v,
                                         const typename EpiCol<Epi>::type& col,
                                         const typename EpiPre<Epi>::type& pre) {
  if constexpr (kEpiTwoPhase<Epi>)
    e.vec8(r, c, v, col, pre);
  else
    e.vec8(r, c, v);
}

// Epilogue through LDS, one band of kTM rows (one wave row) at a time: the
// waves of that band park their fp32 accumulators in LDS, then every thread
// takes 8 consecutive columns of a row and hands them to the epilogue, so
// its global reads and writes are 16-byte and coalesced along rows.
template <class S, int BM, int BN, int WM, class Epi>
__device__ __forceinline__ void gemm_store(f32x16 (&acc)[S::kFM][S::kFN], float* stage, const GemmParams& p, int m0,
                                           int n0, int wm, int wn, int lane, int tid, const Epi& epi) {
  constexpr int kSRow = BN + 8;  // +32 bytes: the two lane halves hit disjoint banks
  constexpr int kChunks = S::kTM * BN / 8;
  // A thread's 8 columns are the same in every chunk it takes.
  static_assert(S::kThreads % (BN / 8) == 0, "chunk columns must be fixed per thread");
  typename EpiCol<Epi>::type colv;
  if (p.N >= 8) epi_col(epi, min(n0 + (tid % (BN / 8)) * 8, p.N - 8), colv);
#pragma unroll 1
  for (int band = 0; band < WM; ++band) {
    lds_barrier();  // LDS only: earlier stores may stay in flight
    if (wm == band) {
#pragma unroll
      for (int i = 0; i < S::kFM; ++i)
#pragma unroll
        for (int j = 0; j < S::kFN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            stage[(i * 32 + acc_row(r, lane)) * kSRow + wn * S::kTN + j * 32 + (lane & 31)] = acc[i][j][r];
    }
    lds_barrier();
    // Two phases per group of chunks: every global read the epilogue needs
    // (Epi::pre) is issued first, then the values are combined and stored,
    // so a thread keeps kGroup loads in flight instead of one.
    // The reads are unconditional (coordinates clamped into the matrix; a
    // clamped chunk's values are not used), so no branch separates a load
    // from its use and the compiler keeps them all in flight. An epilogue
    // with reads therefore needs N >= 8.
    static_assert(kChunks % S::kThreads == 0, "chunks must split evenly over threads");
    constexpr int kPerThread = kChunks / S::kThreads;
    constexpr int kGroupMax = S::kThreads > 256 ? 2 : 4;  // 8-wave tiles have half the registers
    constexpr int kGroup = kPerThread < kGroupMax ? kPerThread : kGroupMax;
    static_assert(kPerThread % kGroup == 0, "chunk groups must tile the band");
#pragma unroll 1
    for (int c0 = 0; c0 < kPerThread; c0 += kGroup) {
      typename EpiPre<Epi>::type pre[kGroup];
      bool full[kGroup];
#pragma unroll
      for (int u = 0; u < kGroup; ++u) {
        const int c = tid + (c0 + u) * S::kThreads;
        const int rl = c / (BN / 8), cl = (c % (BN / 8)) * 8;
        const int row = m0 + band * S::kTM + rl, col = n0 + cl;
        full[u] = row < p.M && col + 8 <= p.N;
        epi_pre(epi, min(row, p.M - 1), min(col, p.N - 8), pre[u]);
      }
#pragma unroll
      for (int u = 0; u < kGroup; ++u) {
        const int c = tid + (c0 + u) * S::kThreads;
        const int rl = c / (BN / 8), cl = (c % (BN / 8)) * 8;
        const int row = m0 + band * S::kTM + rl, col = n0 + cl;
        if (row >= p.M || col >= p.N) continue;
        float v[8];
        const f32x4 a = *reinterpret_cast<const f32x4*>(stage + rl * kSRow + cl);
        const f32x4 b = *reinterpret_cast<const f32x4*>(stage + rl * kSRow + cl + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = a[e];
          v[e + 4] = b[e];
        }
        if (full[u]) {
          epi_vec8(epi, row, col, v, colv, pre[u]);
        } else {
          for (int e = 0; col + e < p.N; ++e) epi(row, col + e, v[e]);
        }
      }
    }
  }
}

// Wave-local epilogue of the direct kernel: each wave writes its own
// kTM x kTN tile, kRows rows per step, through a private LDS region, with
// no workgroup barrier, so a wave that finishes its MFMAs stores while the
// others still multiply. The epilogue's global reads (Epi::pre) run kAhead
// steps ahead of their use; their coordinates are clamped into the matrix
// (a clamped chunk's values are not used), which needs N >= 8.
template <class S, int kRows, class Epi>
__device__ __forceinline__ void gemm_store_wave(f32x16 (&acc)[S::kFM][S::kFN], float* region, const GemmParams& p,
                                                int row0, int col0, int lane, const Epi& epi) {
  constexpr int kTN = S::kTN;
  constexpr int kSRow = kTN + 8;               // rows r and r + 4 land on disjoint banks
  constexpr int kCpr = kTN / 8;                // 8-column chunks per row
  constexpr int kRowsPerPass = kWave / kCpr;   // rows one wave instruction covers
  constexpr int kPer = kRows / kRowsPerPass;   // chunks per lane per step
  constexpr int kHalves = 32 / kRows;          // steps per 32-row MFMA block
  constexpr int kSteps = S::kFM * kHalves;
  constexpr int kAhead = 2;
  static_assert((kRows == 16 || kRows == 8) && kCpr <= kWave && kRows % kRowsPerPass == 0, "wave tile width");
  const int cl = (lane % kCpr) * 8;
  const int rl0 = lane / kCpr;
  const int col = col0 + cl;
  typename EpiCol<Epi>::type colv;
  if (p.N >= 8) epi_col(epi, min(col, p.N - 8), colv);
  typename EpiPre<Epi>::type pre[kAhead + 1][kPer];
  auto issue = [&](int step, typename EpiPre<Epi>::type (&q)[kPer]) {
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int row = row0 + step * kRows + rl0 + u * kRowsPerPass;
      epi_pre(epi, min(row, p.M - 1), min(col, p.N - 8), q[u]);
    }
  };
#pragma unroll
  for (int a = 0; a < kAhead; ++a)
    if (a < kSteps && p.N >= 8) issue(a, pre[a]);
#pragma unroll
  for (int step = 0; step < kSteps; ++step) {
    const int i = step / kHalves, h = step % kHalves;
    if (step + kAhead < kSteps && p.N >= 8) issue(step + kAhead, pre[(step + kAhead) % (kAhead + 1)]);
    // Block i holds rows 8 (r / 4) + 4 (lane / 32) + r % 4 in register r, so
    // registers [h kRows / 2, (h + 1) kRows / 2) are rows [h kRows, (h + 1) kRows).
#pragma unroll
    for (int j = 0; j < S::kFN; ++j)
#pragma unroll
      for (int r = h * kRows / 2; r < (h + 1) * kRows / 2; ++r)
        region[(acc_row(r, lane) - h * kRows) * kSRow + j * 32 + (lane & 31)] = acc[i][j][r];
    // The region is private to the wave: LDS completion is the only ordering needed.
    asm volatile("" ::: "memory");
    wait_lgkmcnt0();
    asm volatile("" ::: "memory");
    float v[kPer][8];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const float* src = region + (rl0 + u * kRowsPerPass) * kSRow + cl;
      const f32x4 a = *reinterpret_cast<const f32x4*>(src);
      const f32x4 b = *reinterpret_cast<const f32x4*>(src + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[u][e] = a[e];
        v[u][e + 4] = b[e];
      }
    }
    asm volatile("" ::: "memory");
    wait_lgkmcnt0();
    asm volatile("" ::: "memory");
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int row = row0 + step * kRows + rl0 + u * kRowsPerPass;
      if (row >= p.M || col >= p.N) continue;
      if (col + 8 <= p.N) {
        epi_vec8(epi, row, col, v[u], colv, pre[step % (kAhead + 1)][u]);
      } else {
        for (int e = 0; col + e < p.N; ++e) epi(row, col + e, v[u][e]);
      }
    }
  }
}

// Pins the instruction order of kSteps MFMA k-steps, each made of kMfma
// MFMAs with the kReads fragment reads of the following k-step riding on
// its first MFMAs (masks: 0x100 DS read, 0x008 MFMA), so LDS latency hides
// behind matrix work.
template <int kReads, int kMfma, int kSteps>
__device__ __forceinline__ void pin_substeps() {
  constexpr int kLead = kReads < kMfma ? kReads : kMfma;
#pragma unroll
  for (int st = 0; st < kSteps; ++st) {
#pragma unroll
    for (int t = 0; t < kLead; ++t) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    if (kReads > kLead) __builtin_amdgcn_sched_group_barrier(0x100, kReads - kLead, 0);
    if (kMfma > kLead) __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kLead, 0);
  }
}

// Pins the instruction order of one BK slice: the reads of step 0, then
// pin_substeps over the remaining steps and the last step's MFMAs.
template <int kReads, int kMfma, int kSteps>
__device__ __forceinline__ void pin_kstep_schedule() {
  __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
  pin_substeps<kReads, kMfma, kSteps - 1>();
  __builtin_amdgcn_sched_group_barrier(0x008, kMfma, 0);
}

// Occupancy: the two LDS stages of the 256x256 tile admit one workgroup per
// CU, so the kernel declares that and lets the compiler keep the prefetched
// fragments in registers instead of scheduling for more waves.
template <typename T, int BM, int BN, int BK, int WM, int WN, int LA, int LB, class Epi>
__global__ void __launch_bounds__(WM* WN* kWave)
    __attribute__((amdgpu_waves_per_eu(1, (BM >= 256 ? 1 : 2))))
    gemm_kernel(const GemmParams p, const Epi epi) {
  typedef GemmShape<T, BM, BN, BK, WM, WN> S;
  typedef Loader<T, BM, BK, S::kThreads, true, LA> LdA;
  typedef Loader<T, BN, BK, S::kThreads, false, LB> LdB;
  typedef Mma<T> MM;
  __shared__ __attribute__((aligned(16))) T smem[2 * S::kStageElems];

  int tm, tn;
  tile_coords(p, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = blockIdx.z * p.k_slice;
  const int kend = min(p.K, kbeg + p.k_slice);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  f32x16 acc[S::kFM][S::kFN];
#pragma unroll
  for (int i = 0; i < S::kFM; ++i)
#pragma unroll
    for (int j = 0; j < S::kFN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  LdA lda_;
  LdB ldb_;
  lda_.init(p, m0, p.M, tid);
  ldb_.init(p, n0, p.N, tid);
  u32x4 ra[LdA::kLoads], rb[LdB::kLoads];
  const int nk = (kend - kbeg + BK - 1) / BK;
  if (nk > 0) {
    lda_.fetch(ra, kbeg, kend);
    ldb_.fetch(rb, kbeg, kend);
    LdA::stash(ra, smem, S::kStride, tid);
    LdB::stash(rb, smem + BM * S::kStride, S::kStride, tid);
  }
  __syncthreads();

  const int frow = lane & 31;
  const int fk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    T* cur = smem + (kt & 1) * S::kStageElems;
    const bool more = kt + 1 < nk;
    if (more) {
      lda_.fetch(ra, kbeg + (kt + 1) * BK, kend);
      ldb_.fetch(rb, kbeg + (kt + 1) * BK, kend);
    }
    const T* sa = cur + (wm * S::kTM + frow) * S::kStride + fk;
    const T* sb = cur + (BM + wn * S::kTN + frow) * S::kStride + fk;
    // fragments of k16 step s + 1 are read from LDS while step s multiplies
    typename MM::frag fa[2][S::kFM], fb[2][S::kFN];
#pragma unroll
    for (int i = 0; i < S::kFM; ++i) fa[0][i] = MM::load(sa + i * 32 * S::kStride);
#pragma unroll
    for (int j = 0; j < S::kFN; ++j) fb[0][j] = MM::load(sb + j * 32 * S::kStride);
#pragma unroll
    for (int st = 0; st < BK / 16; ++st) {
      const int cb = st & 1, nb = cb ^ 1;
      if (st + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < S::kFM; ++i) fa[nb][i] = MM::load(sa + i * 32 * S::kStride + (st + 1) * 16);
#pragma unroll
        for (int j = 0; j < S::kFN; ++j) fb[nb][j] = MM::load(sb + j * 32 * S::kStride + (st + 1) * 16);
      }
#pragma unroll
      for (int i = 0; i < S::kFM; ++i)
#pragma unroll
        for (int j = 0; j < S::kFN; ++j) acc[i][j] = MM::mma(fa[cb][i], fb[cb][j], acc[i][j]);
    }
    if constexpr (sizeof(T) == 2) pin_kstep_schedule<S::kFM + S::kFN, S::kFM * S::kFN, BK / 16>();
    if (more) {
      T* nxt = smem + ((kt + 1) & 1) * S::kStageElems;
      LdA::stash(ra, nxt, S::kStride, tid);
      LdB::stash(rb, nxt + BM * S::kStride, S::kStride, tid);
    }
    __syncthreads();
  }

  static_assert((size_t)S::kTM * (BN + 8) * sizeof(float) <= S::kLdsBytes, "epilogue band must fit in LDS");
  gemm_store<S, BM, BN, WM>(acc, reinterpret_cast<float*>(smem), p, m0, n0, wm, wn, lane, tid, epi);
}

// Direct-to-LDS GEMM. Each wave issues buffer_load_dwordx4 ... lds: a wave
// instruction fills 1 KB of a tile (64 lanes x 16 bytes) and no registers
// hold prefetched data. An operand contiguous along K (LAYOUT_K) lands as
// ROWS rows of BK elements; one contiguous along M or N (LAYOUT_MN, bf16) as
// BK rows of ROWS elements, and its MFMA fragments (8 consecutive k of one
// row or column) come from two LDS transpose reads (ds_read_b64_tr_b16),
// so weight and data gradients need no transposed copies in HBM. 16-byte
// chunks are XOR-swizzled by row so every fragment read pass hits 64
// distinct banks without padding. The loads for tile k+1 go out right after
// the single barrier of step k, into the other LDS stage, and land while
// step k multiplies. The K concatenation point, if any, falls on a BK
// boundary.
template <typename T, int ROWS, int BK, int LAYOUT, int WAVES>
struct DirectOp {
  static constexpr bool kMN = LAYOUT == LAYOUT_MN;
  static constexpr int kRowElems = kMN ? ROWS : BK;
  static constexpr int kTileRows = kMN ? BK : ROWS;
  static constexpr int kRowBytes = kRowElems * (int)sizeof(T);
  static constexpr int kCpr = kRowBytes / 16;            // 16-byte chunks per row
  static constexpr int kRowsPerInst = kWave / kCpr;      // rows one wave instruction fills
  static constexpr int kInsts = kTileRows / (kRowsPerInst * WAVES);  // loads per thread per stage
  static constexpr int kElems = kTileRows * kRowElems;
  static_assert(!kMN || sizeof(T) == 2, "transpose reads take 16-bit elements");
  static_assert(kMN ? kCpr >= 16 : (kCpr == 8 || kCpr == 4), "swizzle covers these row widths");
  static_assert(kInsts >= 1 && kTileRows % (kRowsPerInst * WAVES) == 0, "tile rows split evenly over waves");
  // Physical chunk of logical chunk c in row r is c ^ key(r). K-major: a
  // 16-byte read pass serves 16 lanes (16 consecutive rows at one logical
  // chunk) over 64 banks, i.e. 16 slots of 16 bytes; rows of 8 chunks put
  // two rows in each 256-byte span, so the key steps every second row and
  // the 16 rows land on 16 distinct slots (a key of r & 7 would put rows r
  // and r + 8 on one slot). M/N-major: a transpose-read pass touches 4
  // consecutive rows (k) at 4 consecutive chunks; the key moves each row by
  // 64 bytes.
  static __device__ __forceinline__ int key(int r) {
    if constexpr (kMN) return (r & 3) * 4;
    return kCpr == 8 ? ((r >> 1) & 7) : ((r >> 2) & 3);
  }
};

template <typename T, int BM, int BN, int BK, int WM, int WN, int NS, int LA = LAYOUT_K, int LB = LAYOUT_K>
struct DirectShape {
  typedef GemmShape<T, BM, BN, BK, WM, WN> S;
  static constexpr int kWaves = WM * WN;
  typedef DirectOp<T, BM, BK, LA, WM * WN> OA;
  typedef DirectOp<T, BN, BK, LB, WM * WN> OB;
  static constexpr int kNia = OA::kInsts;
  static constexpr int kNib = OB::kInsts;
  static constexpr int kLoads = kNia + kNib;           // loads per thread per stage
  static constexpr int kStage = OA::kElems + OB::kElems;  // elements per stage
  static constexpr size_t kMainBytes = (size_t)NS * kStage * sizeof(T);
  // fp32 staging of 16 rows of every wave's tile (the wave-local epilogue)
  static constexpr size_t kEpiRegion16 = (size_t)kWaves * 16 * (S::kTN + 8) * sizeof(float);
  static constexpr size_t kLdsBytes = kMainBytes;
  static_assert(NS >= 2 && kLoads * (NS - 1) < 64, "outstanding loads must fit the vmcnt counter");
  static_assert(kLdsBytes <= 160 * 1024, "LDS budget of one workgroup");
};

typedef short pf_v4i16 __attribute__((ext_vector_type(4)));
// LDS transpose read: within each 16-lane group, lane i supplies the address
// of 4 consecutive 16-bit elements and lane l receives element l % 4 of the
// lanes l / 4, 4 + l / 4, 8 + l / 4, 12 + l / 4, in that order.
__device__ __forceinline__ pf_v4i16 lds_read_tr16(const void* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) pf_v4i16*)(const_cast<void*>(p)));
}

// Waits until at most `pending` stages of loads (kLoads each) are in flight.
template <int L, int NP>
__device__ __forceinline__ void wait_stages(int pending) {
  if constexpr (NP == 0) {
    wait_vmcnt<0>();
  } else {
    if (pending >= NP)
      wait_vmcnt<NP * L>();
    else
      wait_stages<L, NP - 1>(pending);
  }
}

// FAST (K-major operands whose slices hold whole BK tiles): the buffer
// descriptors of A, A2, B and B2 are built once per workgroup, their ranges
// clamp the tile rows, and a K step only moves the scalar offset of the loads.
template <typename T, int BM, int BN, int BK, int WM, int WN, int NS, class Epi, int LA = LAYOUT_K,
          int LB = LAYOUT_K, bool FAST = false>
__global__ void __launch_bounds__(WM* WN* kWave)
    __attribute__((amdgpu_waves_per_eu(WM* WN / 4, (BM >= 256 ? 1 : 2) * WM * WN / 4)))
    gemm_direct_kernel(const GemmParams p, const Epi epi) {
  typedef DirectShape<T, BM, BN, BK, WM, WN, NS, LA, LB> D;
  typedef typename D::S S;
  typedef typename D::OA OA;
  typedef typename D::OB OB;
  typedef Mma<T> MM;
  constexpr int kVec = 16 / (int)sizeof(T);  // elements per chunk
  __shared__ __attribute__((aligned(1024))) char smem_raw[D::kLdsBytes];
  T* smem = reinterpret_cast<T*>(smem_raw);

  int tm, tn;
  tile_coords(p, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = blockIdx.z * p.k_slice;
  const int kend = min(p.K, kbeg + p.k_slice);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // scalar: LDS bases go to M0
  const int wm = wave / WN, wn = wave % WN;

  const int64_t lda_b = p.lda * (int64_t)sizeof(T), ldb_b = p.ldb * (int64_t)sizeof(T);
  // per-lane byte offsets inside a tile (rows r, swizzled chunk)
  uint32_t voa[OA::kInsts], vob[OB::kInsts];
  int kca[OA::kInsts], kcb[OB::kInsts];
  {
    const int lr_a = lane / OA::kCpr, lc_a = lane % OA::kCpr;
#pragma unroll
    for (int i = 0; i < OA::kInsts; ++i) {
      const int r = (wave * OA::kInsts + i) * OA::kRowsPerInst + lr_a;
      const int gc = lc_a ^ OA::key(r);
      kca[i] = gc * kVec;
      voa[i] = (uint32_t)(r * lda_b + gc * 16);
    }
    const int lr_b = lane / OB::kCpr, lc_b = lane % OB::kCpr;
#pragma unroll
    for (int i = 0; i < OB::kInsts; ++i) {
      const int r = (wave * OB::kInsts + i) * OB::kRowsPerInst + lr_b;
      const int gc = lc_b ^ OB::key(r);
      kcb[i] = gc * kVec;
      vob[i] = (uint32_t)(r * ldb_b + gc * 16);
    }
  }
  // K-major: the tile is BM (BN) rows from m0 (n0), a stage advances along
  // each row. M/N-major: the tile is BK rows of the operand starting at row
  // k0, each read from column m0 (n0); only the rows below kend and the
  // columns below M (N) of the last row are in range.
  // batch blockIdx.y of a batched problem starts at its own A and B
  const char* a1 = reinterpret_cast<const char*>(p.a) + (int64_t)blockIdx.y * p.batch_a * (int64_t)sizeof(T) +
                   (OA::kMN ? m0 * (int64_t)sizeof(T) : m0 * lda_b);
  const char* a2 = p.a2 ? reinterpret_cast<const char*>(p.a2) + (OA::kMN ? m0 * (int64_t)sizeof(T) : m0 * lda_b)
                        : nullptr;
  const char* b1 = reinterpret_cast<const char*>(p.b) + (int64_t)blockIdx.y * p.batch_b * (int64_t)sizeof(T) +
                   (OB::kMN ? n0 * (int64_t)sizeof(T) : n0 * ldb_b);
  const char* b2 = p.b2 ? reinterpret_cast<const char*>(p.b2) + (OB::kMN ? n0 * (int64_t)sizeof(T) : n0 * ldb_b)
                        : nullptr;
  const uint32_t a_rows = (uint32_t)(max(0, min(BM, p.M - m0)) * lda_b);
  const uint32_t b_rows = (uint32_t)(max(0, min(BN, p.N - n0)) * ldb_b);
  const int a_cols = max(0, min(BM, p.M - m0)), b_cols = max(0, min(BN, p.N - n0));

  // Loads [i0, i1) of one stage (A's loads, then B's), so a stage can be
  // issued at once or spread over the k-steps of a tile.
  auto issue_range = [&](int k0, int stage, int i0, int i1) {
    const bool tail = k0 + BK > kend;
    T* st = smem + stage * D::kStage;
    if (i0 < OA::kInsts) {
      const bool second = k0 >= p.a_ksplit;
      const int krel = second ? k0 - p.a_ksplit : k0;
      rsrc_t rs;
      if constexpr (OA::kMN) {
        const int rows = min(BK, kend - k0);
        rs = make_rsrc_uniform((second ? a2 : a1) + (int64_t)krel * lda_b,
                               (uint32_t)((int64_t)(rows - 1) * lda_b + a_cols * (int64_t)sizeof(T)));
      } else {
        rs = make_rsrc_uniform((second ? a2 : a1) + (int64_t)krel * sizeof(T), a_rows - (uint32_t)(krel * sizeof(T)));
      }
#pragma unroll
      for (int i = 0; i < OA::kInsts; ++i)
        if (i >= i0 && i < i1) {
          const bool oob = !OA::kMN && tail && k0 + kca[i] >= kend;
          buf_ld16_lds(rs, oob ? kOOB : voa[i], st + (wave * OA::kInsts + i) * 1024 / (int)sizeof(T));
        }
    }
    if (i1 > OA::kInsts) {
      const bool second = k0 >= p.b_ksplit;
      const int krel = second ? k0 - p.b_ksplit : k0;
      rsrc_t rs;
      if constexpr (OB::kMN) {
        const int rows = min(BK, kend - k0);
        rs = make_rsrc_uniform((second ? b2 : b1) + (int64_t)krel * ldb_b,
                               (uint32_t)((int64_t)(rows - 1) * ldb_b + b_cols * (int64_t)sizeof(T)));
      } else {
        rs = make_rsrc_uniform((second ? b2 : b1) + (int64_t)krel * sizeof(T), b_rows - (uint32_t)(krel * sizeof(T)));
      }
#pragma unroll
      for (int i = 0; i < OB::kInsts; ++i)
        if (i + OA::kInsts >= i0 && i + OA::kInsts < i1) {
          const bool oob = !OB::kMN && tail && k0 + kcb[i] >= kend;
          buf_ld16_lds(rs, oob ? kOOB : vob[i], st + OA::kElems + (wave * OB::kInsts + i) * 1024 / (int)sizeof(T));
        }
    }
  };
  static_assert(!FAST || (!OA::kMN && !OB::kMN), "the fixed-descriptor loads take K-major operands");
  const rsrc_t rsa1 = make_rsrc_uniform(a1, a_rows), rsb1 = make_rsrc_uniform(b1, b_rows);
  const rsrc_t rsa2 = make_rsrc_uniform(a2 ? a2 : a1, a2 ? a_rows : 0u);
  const rsrc_t rsb2 = make_rsrc_uniform(b2 ? b2 : b1, b2 ? b_rows : 0u);
  auto issue = [&](int k0, int stage) {
    if constexpr (FAST) {
      // within a row: k0 + BK <= K, so a lane's offset stays inside its row
      T* st = smem + stage * D::kStage;
      const bool sa = k0 >= p.a_ksplit, sb = k0 >= p.b_ksplit;
      const uint32_t soa = __builtin_amdgcn_readfirstlane((uint32_t)((sa ? k0 - p.a_ksplit : k0) * (int)sizeof(T)));
      const uint32_t sob = __builtin_amdgcn_readfirstlane((uint32_t)((sb ? k0 - p.b_ksplit : k0) * (int)sizeof(T)));
#pragma unroll
      for (int i = 0; i < OA::kInsts; ++i)
        buf_ld16_lds_so(sa ? rsa2 : rsa1, voa[i], soa, st + (wave * OA::kInsts + i) * 1024 / (int)sizeof(T));
#pragma unroll
      for (int i = 0; i < OB::kInsts; ++i)
        buf_ld16_lds_so(sb ? rsb2 : rsb1, vob[i], sob, st + OA::kElems + (wave * OB::kInsts + i) * 1024 / (int)sizeof(T));
    } else {
      issue_range(k0, stage, 0, D::kLoads);
    }
  };

  f32x16 acc[S::kFM][S::kFN];
#pragma unroll
  for (int i = 0; i < S::kFM; ++i)
#pragma unroll
    for (int j = 0; j < S::kFN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (kend - kbeg + BK - 1) / BK;
  constexpr int kSub = BK / 16;  // MFMA k-steps per tile
  static_assert(kSub % 2 == 0, "fragment double buffer alternates over an even number of k-steps");
  const int frow = lane & 31;
  const int g = lane >> 5;
  // K-major fragment: row frow of the 32-row block at rowp, k-step st
  auto frag_k = [&](const T* rowp, int swz, int st) {
    if constexpr (sizeof(T) == 2) {
      return MM::load(rowp + (((2 * st + g) ^ swz) * 8));
    } else {
      const int c0 = 4 * st + 2 * g;
      typename MM::frag f;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(rowp + ((c0 ^ swz) * 4));
      const f32x4 hi = *reinterpret_cast<const f32x4*>(rowp + (((c0 + 1) ^ swz) * 4));
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[e] = lo[e];
        f[e + 4] = hi[e];
      }
      return f;
    }
  };
  // M/N-major fragment: column c0 .. c0+31 of the tile (this lane's column
  // c0 + frow), k = 16 st + 8 g .. +7, from two transpose reads: lane i of a
  // 16-lane group addresses row k + i / 4 at columns 4 (i % 4) .. +3 of the
  // group's 16 columns.
  const int tr_row = 8 * g + ((lane & 15) >> 2);
  const int tr_col = (lane & 16) + 4 * (lane & 3);
  auto frag_mn = [&](const T* tile, int row_elems, int c0, int st, auto op) {
    typedef decltype(op) O;
    const int col = c0 + tr_col;
    const int r0 = 16 * st + tr_row;
    const char* base = reinterpret_cast<const char*>(tile);
    const int chunk = col / kVec, half = (col / 4) & 1;
    const pf_v4i16 lo =
        lds_read_tr16(base + r0 * (row_elems * 2) + ((chunk ^ O::key(r0)) * 16) + half * 8);
    const pf_v4i16 hi =
        lds_read_tr16(base + (r0 + 4) * (row_elems * 2) + ((chunk ^ O::key(r0 + 4)) * 16) + half * 8);
    typename MM::frag f;
    const auto l = __builtin_bit_cast(bf16x4, lo);
    const auto h = __builtin_bit_cast(bf16x4, hi);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[e] = l[e];
      f[e + 4] = h[e];
    }
    return f;
  };
  typename MM::frag fa[2][S::kFM], fb[2][S::kFN];
  auto read_frags = [&](int tile, int st, int buf) {
    const T* cur = smem + (tile % NS) * D::kStage;
    if constexpr (OA::kMN) {
#pragma unroll
      for (int i = 0; i < S::kFM; ++i) fa[buf][i] = frag_mn(cur, BM, wm * S::kTM + i * 32, st, OA{});
    } else {
      const T* sa = cur + (wm * S::kTM + frow) * BK;
#pragma unroll
      for (int i = 0; i < S::kFM; ++i) fa[buf][i] = frag_k(sa + i * 32 * BK, OA::key(frow), st);
    }
    const T* curb = cur + OA::kElems;
    if constexpr (OB::kMN) {
#pragma unroll
      for (int j = 0; j < S::kFN; ++j) fb[buf][j] = frag_mn(curb, BN, wn * S::kTN + j * 32, st, OB{});
    } else {
      const T* sb = curb + (wn * S::kTN + frow) * BK;
#pragma unroll
      for (int j = 0; j < S::kFN; ++j) fb[buf][j] = frag_k(sb + j * 32 * BK, OB::key(frow), st);
    }
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < S::kFM; ++i)
#pragma unroll
      for (int j = 0; j < S::kFN; ++j) acc[i][j] = MM::mma(fa[buf][i], fb[buf][j], acc[i][j]);
  };
  // reads per k-step: one per K-major fragment, two per M/N-major one
  constexpr int kReads = S::kFM * (OA::kMN ? 2 : 1) + S::kFN * (OB::kMN ? 2 : 1);

  // Ring of NS stages, tile t in stage t % NS. The hand-off to tile kt+1
  // happens before the last k-step of tile kt, whose fragments are already
  // in registers: after the barrier the first fragments of tile kt+1 are
  // requested, the last MFMAs of tile kt are queued, and the refill of stage
  // kt % NS (tile kt+NS) is issued while they execute, so the matrix pipe
  // does not drain at tile boundaries.
  if (nk > 0) {
#pragma unroll
    for (int s0 = 0; s0 < NS; ++s0)
      if (s0 < nk) issue(kbeg + s0 * BK, s0);
    wait_stages<D::kLoads, NS - 1>(min(NS - 1, nk - 1));
    lds_barrier();
    read_frags(0, 0, 0);
  }
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int st = 0; st + 1 < kSub; ++st) {
      read_frags(kt, st + 1, (st + 1) & 1);
      mfmas(st & 1);
    }
    if constexpr (sizeof(T) == 2) pin_substeps<kReads, S::kFM * S::kFN, kSub - 1>();
    // The last k-step's fragments are in registers on every path, so the
    // compiler sees no reason to make its MFMAs wait for the younger reads
    // of tile kt+1. The scheduling fence keeps the wait behind the MFMAs
    // above.
    __builtin_amdgcn_sched_barrier(0);
    wait_lgkmcnt0();
    if (kt + 1 < nk) {
      wait_stages<D::kLoads, NS - 2>(min(NS - 2, nk - 2 - kt));
      lds_barrier();  // tile kt+1 is in LDS; every wave is done reading tile kt
      read_frags(kt + 1, 0, 0);
    }
    mfmas(1);
    if (kt + NS < nk) issue(kbeg + (kt + NS) * BK, kt % NS);  // after the hand-off above
  }
  // Every direct load has landed (the last wait_stages drained them all).
  // The stage that held tile nk-2 is free on every wave: nothing reads it
  // after the barrier that handed over tile nk-1 and no load refills it;
  // with fewer tiles an unused stage is free.
  const int free_stage = nk >= 2 ? (nk - 2) % NS : (nk == 1 ? 1 : 0);
  constexpr int kRows = D::kEpiRegion16 <= D::kStage * sizeof(T) ? 16 : 8;
  static_assert(D::kEpiRegion16 / (16 / kRows) <= D::kStage * sizeof(T), "wave epilogue regions must fit one stage");
  float* region = reinterpret_cast<float*>(smem + free_stage * D::kStage) + wave * kRows * (S::kTN + 8);
  gemm_store_wave<S, kRows>(acc, region, p, m0 + wm * S::kTM, n0 + wn * S::kTN, lane, epi);
}

// Fixed-order reduction of split-K partials ws[s][M][N], then the epilogue
// (8 consecutive columns per thread when N is a multiple of 8).
template <class Epi>
__global__ void __launch_bounds__(256) splitk_reduce_kernel(const float* __restrict__ ws, int splits, int M,
                                                            int N, const Epi epi) {
  const int64_t total = (int64_t)M * N;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if ((N & 7) == 0) {
    for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < total / 8; c += stride) {
      const int64_t idx = c * 8;
      float v[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      for (int z = 0; z < splits; ++z) {
        float t[8];
        load8(ws + (int64_t)z * total + idx, t);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += t[e];
      }
      epi.vec8((int)(idx / N), (int)(idx % N), v);
    }
    return;
  }
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
    float s = 0.0f;
    for (int z = 0; z < splits; ++z) s += ws[(int64_t)z * total + idx];
    epi((int)(idx / N), (int)(idx % N), s);
  }
}

// Epilogue writing split-K partials.
struct EpiPartial {
  float* ws;
  int N;
  int64_t slice_stride;
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    ws[(int64_t)blockIdx.z * slice_stride + (int64_t)r * N + c] = v;
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v) const {
    if ((N & 7) == 0) {
      store8(ws + (int64_t)blockIdx.z * slice_stride + (int64_t)r * N + c, v);
    } else {
      for (int e = 0; e < 8; ++e) (*this)(r, c + e, v[e]);
    }
  }
};

// ---- host side --------------------------------------------------------------

struct GemmProblem {
  const void* a;
  int64_t lda;
  const void* a2 = nullptr;
  int64_t lda2 = 0;
  int a_ksplit = 1 << 30;
  const void* b;
  int64_t ldb;
  const void* b2 = nullptr;
  int64_t ldb2 = 0;
  int b_ksplit = 1 << 30;
  int M, N, K;
  // batched problem (direct kernel only, A2/B2 unused): `batch` independent
  // products, batch z reading A at z * batch_a and B at z * batch_b
  // (elements); the epilogue finds z in blockIdx.y
  int batch = 1;
  int64_t batch_a = 0, batch_b = 0;
};

// Tile configuration chosen for a problem.
enum GemmTile { TILE_256x256 = 0, TILE_128x128 = 1, TILE_64x64 = 2 };

struct GemmPlan {
  int tile;
  int bm, bn, bk;
  int splits;
  int k_slice;
};

template <typename T>
inline GemmPlan plan_gemm(const GemmProblem& pr, int num_cu) {
  GemmPlan pl;
  const int64_t mn = (int64_t)pr.M * pr.N;
  if (sizeof(T) == 4) {
    pl.tile = TILE_128x128;
    pl.bm = pl.bn = 128;
    pl.bk = 32;
  } else if (pr.M >= 256 && pr.N >= 256 &&
             (mn >= (int64_t)256 * 256 * num_cu ||
              // long reductions: 256x256 tiles split along K still fill the chip
              (int64_t)pr.K * (((pr.M + 255) / 256) * ((pr.N + 255) / 256)) >= (int64_t)num_cu * 64 * 64)) {
    pl.tile = TILE_256x256;
    pl.bm = pl.bn = 256;
    pl.bk = 64;
  } else if (mn >= (int64_t)128 * 128 * num_cu / 2 || pr.M > 64 || pr.N > 64) {
    pl.tile = TILE_128x128;
    pl.bm = pl.bn = 128;
    pl.bk = 64;
  } else {
    pl.tile = TILE_64x64;
    pl.bm = pl.bn = 64;
    pl.bk = 64;
  }
  const int64_t tiles = (int64_t)((pr.M + pl.bm - 1) / pl.bm) * ((pr.N + pl.bn - 1) / pl.bn) * pr.batch;
  const int kblocks = (pr.K + pl.bk - 1) / pl.bk;
  int splits = 1;
  // Deterministic split-K when the tile grid cannot fill the chip and the
  // reduction is long enough for each slice to stay efficient.
  while (pr.batch == 1 && tiles * splits < num_cu && kblocks / (splits * 2) >= 8) splits *= 2;
  const int kb_per = (kblocks + splits - 1) / splits;
  pl.k_slice = kb_per * pl.bk;
  pl.splits = (kblocks + kb_per - 1) / kb_per;
  return pl;
}

template <typename T, int BM, int BN, int BK, int WM, int WN, int LA, int LB, class Epi>
inline hipError_t launch_gemm_tile(const GemmProblem& pr, const GemmPlan& pl, const Epi& epi,
                                   hipStream_t stream) {
  GemmParams p;
  p.a = pr.a;
  p.lda = pr.lda;
  p.a2 = pr.a2;
  p.lda2 = pr.lda2;
  p.a_ksplit = pr.a_ksplit;
  p.b = pr.b;
  p.ldb = pr.ldb;
  p.b2 = pr.b2;
  p.ldb2 = pr.ldb2;
  p.b_ksplit = pr.b_ksplit;
  p.M = pr.M;
  p.N = pr.N;
  p.K = pr.K;
  p.k_slice = pl.k_slice;
  p.tiles_m = (pr.M + BM - 1) / BM;
  p.tiles_n = (pr.N + BN - 1) / BN;
  // row tiles per column sweep: the sweep's A rows (group_m x BM rows of one
  // K slice) fit about 4 MiB, one XCD's L2; 2 .. 8 (long reductions such as
  // the compression take 2, K = 2048 takes 4, K = 1024 keeps 8)
  p.group_m = (int)std::min<int64_t>(
      8, std::max<int64_t>(2, ((int64_t)4 << 20) / ((int64_t)BM * std::max(pl.k_slice, BK) * (int64_t)sizeof(T))));
  p.batch_a = pr.batch_a;
  p.batch_b = pr.batch_b;
  dim3 grid(p.tiles_m * p.tiles_n, pr.batch, pl.splits);
  const bool aligned_split = (pr.a_ksplit >= pr.K || pr.a_ksplit % BK == 0) &&
                             (pr.b_ksplit >= pr.K || pr.b_ksplit % BK == 0) &&
                             (!pr.a2 || pr.lda2 == pr.lda) && (!pr.b2 || pr.ldb2 == pr.ldb);
  // 256x256 tiles run as 8 waves of 128x64: two waves per SIMD, so one
  // wave's MFMAs cover the other's load issue and barrier waits.
  constexpr int DWN = (BM == 256 && BN == 256) ? 4 : WN;
  if constexpr (LA == LAYOUT_K && LB == LAYOUT_K) {
    if (aligned_split && pl.k_slice % BK == 0) {
      if (pr.K % BK == 0)  // every slice holds whole tiles
        hipLaunchKernelGGL((gemm_direct_kernel<T, BM, BN, BK, WM, DWN, 2, Epi, LAYOUT_K, LAYOUT_K, true>), grid,
                           dim3(WM * DWN * kWave), 0, stream, p, epi);
      else
        hipLaunchKernelGGL((gemm_direct_kernel<T, BM, BN, BK, WM, DWN, 2, Epi>), grid, dim3(WM * DWN * kWave), 0,
                           stream, p, epi);
      return hipGetLastError();
    }
  } else if constexpr (sizeof(T) == 2 && BM >= 128 && BN >= 128) {
    // M/N-major operands through LDS transpose reads: rows of such an
    // operand start 16-byte aligned and hold at least one tile width
    const bool rows_ok = (LA == LAYOUT_K || (pr.lda % 8 == 0 && pr.lda >= BM)) &&
                         (LB == LAYOUT_K || (pr.ldb % 8 == 0 && pr.ldb >= BN));
    if (aligned_split && pl.k_slice % BK == 0 && rows_ok) {
      hipLaunchKernelGGL((gemm_direct_kernel<T, BM, BN, BK, WM, DWN, 2, Epi, LA, LB>), grid,
                         dim3(WM * DWN * kWave), 0, stream, p, epi);
      return hipGetLastError();
    }
  }
  if (pr.batch != 1) return hipErrorInvalidValue;  // batches run on the direct kernel only
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, BK, WM, WN, LA, LB, Epi>), grid,
                     dim3(WM * WN * kWave), 0, stream, p, epi);
  return hipGetLastError();
}

template <typename T, int LA, int LB, class Epi>
inline hipError_t launch_gemm_plan(const GemmProblem& pr, const GemmPlan& pl, const Epi& epi,
                                   hipStream_t stream) {
  if constexpr (sizeof(T) == 4) {
    return launch_gemm_tile<T, 128, 128, 32, 2, 2, LA, LB>(pr, pl, epi, stream);
  } else {
    switch (pl.tile) {
      case TILE_256x256:
        return launch_gemm_tile<T, 256, 256, 64, 2, 2, LA, LB>(pr, pl, epi, stream);
      case TILE_128x128:
        return launch_gemm_tile<T, 128, 128, 64, 2, 2, LA, LB>(pr, pl, epi, stream);
      default:
        return launch_gemm_tile<T, 64, 64, 64, 2, 2, LA, LB>(pr, pl, epi, stream);
    }
  }
}

// Bytes of fp32 workspace a problem needs for split-K partials.
template <typename T>
inline size_t gemm_workspace_bytes(const GemmProblem& pr, int num_cu) {
  const GemmPlan pl = plan_gemm<T>(pr, num_cu);
  return pl.splits > 1 ? (size_t)pl.splits * pr.M * pr.N * sizeof(float) : 0;
}

// Run C = A B^T through `epi`, splitting K through `ws` when that helps.
template <typename T, int LA, int LB, class Epi>
inline hipError_t run_gemm(const GemmProblem& pr, const Epi& epi, float* ws, int num_cu,
                           hipStream_t stream) {
  if (pr.M <= 0 || pr.N <= 0) return hipSuccess;
  GemmPlan pl = plan_gemm<T>(pr, num_cu);
  if (pl.splits <= 1 || ws == nullptr) {
    pl.splits = 1;
    pl.k_slice = ((pr.K + pl.bk - 1) / pl.bk) * pl.bk;
    if (pl.k_slice == 0) pl.k_slice = pl.bk;
    return launch_gemm_plan<T, LA, LB>(pr, pl, epi, stream);
  }
  EpiPartial part{ws, pr.N, (int64_t)pr.M * pr.N};
  hipError_t e = launch_gemm_plan<T, LA, LB>(pr, pl, part, stream);
  if (e != hipSuccess) return e;
  const int64_t total = (int64_t)pr.M * pr.N;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
  hipLaunchKernelGGL((splitk_reduce_kernel<Epi>), dim3(blocks), dim3(256), 0, stream, ws, pl.splits,
                     pr.M, pr.N, epi);
  return hipGetLastError();
}

}  // namespace pf
