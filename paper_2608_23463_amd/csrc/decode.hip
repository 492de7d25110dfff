// Proxy-KV-cache decode step and block-triggered append (Eq. 19-21, Sec. 3.8).
//
// Step (one token per sequence, the batch in lockstep), four launches:
//  1. decode_proj_kernel: u = RMSNorm(x) * gamma formed on the fly and
//     multiplied by W_q, W_k, W_v and W_alpha (one 32-column block of the
//     concatenated outputs per workgroup, MFMA over 32 batch rows): q to
//     scratch, k and v straight into slot j of the local block, alpha through
//     a sigmoid. It also stores x into block slot j.
//  2. decode_attn_kernel: the only HBM-heavy step. Cache rows of every
//     (sequence, head) are cut into slices; a workgroup streams one slice of
//     K and V with 16-byte loads (eight lanes per 64-channel row), keeps an
//     online softmax per row slot, and writes an unnormalised partial
//     (max, sum, weighted values). One extra slice per (sequence, head)
//     handles the current block's slots 0..j.
//  3. decode_combine_kernel: merges the cache slices in a fixed order (A_h),
//     normalises the local part (A_x) and forms A = A_x + alpha * A_h.
//  4. the projection kernel of step 1 in its second form:
//     y = x + A W_o^T + b_o.
// Append: compression GEMMs over whole blocks (the block is a zero-copy
// [rows, P*d] view), then the K/V proxy maps write straight into cache row n.
#include <algorithm>
#include <mutex>
#include <utility>
#include <vector>
#include <cmath>
#include <cstring>

#include "decode.hpp"
#include "epilogues.hpp"
#include "layer.hpp"
#include "runner.hpp"

namespace pf {

int decode_dims(const pf_decode_config* c, DecodeDims* d, const char** why) {
  *why = nullptr;
  if (!c) return *why = "config is NULL", PF_ERR_INVALID_ARG;
  if (c->dtype != PF_FP32 && c->dtype != PF_BF16) return *why = "dtype must be PF_FP32 or PF_BF16", PF_ERR_INVALID_ARG;
  if (c->batch < 1 || c->d_model < 1 || c->n_heads < 1 || c->head_dim < 1)
    return *why = "sizes must be >= 1", PF_ERR_INVALID_ARG;
  if ((int64_t)c->n_heads * c->head_dim != c->d_model) return *why = "n_heads * head_dim must equal d_model", PF_ERR_INVALID_ARG;
  if (c->n_levels < 1 || c->n_levels > PF_MAX_LEVELS) return *why = "n_levels must be in 1..4", PF_ERR_INVALID_ARG;
  if (!(c->rms_eps >= 0.0f)) return *why = "rms_eps must be >= 0", PF_ERR_INVALID_ARG;
  d->B = c->batch;
  d->d = c->d_model;
  d->nh = c->n_heads;
  d->dh = c->head_dim;
  d->M = c->n_levels;
  d->P = 1;
  for (int j = 0; j < d->M; ++j) {
    if (c->factors[j] < 1) return *why = "every factor k_j must be >= 1", PF_ERR_INVALID_ARG;
    d->k[j] = c->factors[j];
    d->P *= c->factors[j];
    if (d->P > (1 << 16)) return *why = "block size P too large", PF_ERR_INVALID_ARG;
  }
  d->dl[0] = d->d;
  for (int j = 1; j < d->M; ++j) d->dl[j] = c->level_dims[j - 1] > 0 ? c->level_dims[j - 1] : d->d;
  d->dl[d->M] = d->d;
  d->esize = c->dtype == PF_BF16 ? 2 : 4;
  d->eps = c->rms_eps;
  if (d->dh != 64 && d->dh != 128) return *why = "head_dim must be 64 or 128", PF_ERR_UNSUPPORTED;
  if ((int64_t)d->d * d->esize > 4096)
    return *why = "d_model * element size must be at most 4096 bytes (32 staged rows in LDS)", PF_ERR_UNSUPPORTED;
  for (int j = 0; j <= d->M; ++j)
    if (d->dl[j] % 8 != 0) return *why = "every channel width must be a multiple of 8", PF_ERR_UNSUPPORTED;
  // the append's compression GEMMs take rows of k_j * d_{j-1} elements (at
  // most 8 MiB: a GEMM tile's 256 rows share one 32-bit buffer range)
  for (int j = 0; j < d->M; ++j)
    if ((int64_t)d->k[j] * d->dl[j] * d->esize > kMaxGemmRowBytes)
      return *why = "a grouped row k_j * d_{j-1} * element size exceeds 8 MiB", PF_ERR_UNSUPPORTED;
  const int64_t lvl1_rows_per_block = d->P / d->k[0];
  d->append_rows = (int)std::max<int64_t>(1, std::min<int64_t>(4096, 65536 / lvl1_rows_per_block));
  return PF_OK;
}

// Offsets of every scratch buffer except the split-K partials: the slice
// partials of up to splits_cap cache slices per (sequence, head), and the
// append's level outputs for up to rows_cap (sequence, block) rows per chunk.
static DecodeWs decode_ws_layout(const DecodeDims& d, int splits_cap, int rows_cap) {
  DecodeWs w{};
  w.splits_cap = splits_cap;
  w.rows_cap = rows_cap;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align256(bytes);
    return o;
  };
  const size_t es = d.esize;
  w.q = take((size_t)d.B * d.d * es);
  w.alpha = take((size_t)d.B * d.nh * 4);
  w.attn = take((size_t)d.B * d.d * es);
  const size_t nparts = (size_t)d.B * d.nh * (splits_cap + 1);
  w.part_m = take(nparts * 4);
  w.part_l = take(nparts * 4);
  w.part_acc = take(nparts * d.dh * 4);
  int64_t per_block = d.P;  // rows of level j per block
  for (int j = 1; j <= d.M; ++j) {
    per_block /= d.k[j - 1];
    w.z[j] = take((size_t)rows_cap * per_block * d.dl[j] * es);
  }
  w.gemm = off;
  w.bytes = off;
  return w;
}

// ---- kernels ------------------------------------------------------------------

// ---- small-batch projections (steps 1 and 3) ------------------------------------
//
// out[b, c] for 32 rows b (blockIdx.y) and one block of 32 output columns
// (blockIdx.x) of A W^T, A = [B, d]: MFMA with the batch rows as the M side.
// The 32 rows of A are staged once in LDS (step 1: u = RMSNorm(x) * gamma,
// rounded to the activation type as a stored u would be), with 16-byte chunks
// XOR-swizzled by row so fragment reads are conflict-free. Each of the four
// waves takes a quarter of K; its weight fragments are requested eight
// k-steps ahead, and the four partial tiles are summed in LDS in a fixed order.
struct DecodeProjParams {
  const void* x;        // [B, d]: the token input (RMSNorm input; the residual of step 3)
  const void* a;        // [B, d]: step 3's A (attention output)
  const void* gamma;    // [d] RMSNorm scale (step 1)
  const void* w[4];     // step 1: W_q, W_k, W_v [d, d] and W_alpha [h, d]; step 3: W_o
  const void* bias[4];  // NULL = 0
  int width[4];         // output width of each matrix (d, d, d, h; step 3: d)
  int B, d, nh, dh;
  int64_t P;
  int j;                // local slot of the new token (lockstep)
  float eps;
  void* q;              // [B, d]
  void* k_loc;          // [B, h, P, dh]
  void* v_loc;
  float* alpha;         // [B, h]
  void* x_blk;          // [B, P, d]
  void* y;              // step 3: [B, d]
  DecodePos pos;        // per-sequence slots when pos.ragged
  __device__ __forceinline__ int slot(int b) const { return pos.ragged ? pos.j[b] : j; }
};

template <typename T>
constexpr size_t decode_small_gemm_lds(int d) {
  return (size_t)32 * d * sizeof(T) + 4 * 32 * 33 * sizeof(float) + 32 * sizeof(float);
}

template <typename T, bool PROJ, int CPL>
__global__ void __launch_bounds__(256) decode_small_gemm_kernel(const DecodeProjParams p) {
  typedef Mma<T> MM;
  constexpr int kV = 16 / sizeof(T);  // elements per 16-byte chunk
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  T* a_s = reinterpret_cast<T*>(dyn);                                     // [32][d], swizzled chunks
  float* red = reinterpret_cast<float*>(dyn + (size_t)32 * p.d * sizeof(T));  // [4][32 * 33]
  float* inv_s = red + 4 * 32 * 33;                                       // [32]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int b0 = blockIdx.y * 32;
  const int cpr = p.d / kV;  // chunks per row
  // which matrix this column block belongs to (every width but the last is
  // a multiple of 32, so a block never straddles two matrices)
  int seg = 0, cs = blockIdx.x * 32;
  if constexpr (PROJ) {
    while (seg < 3 && cs >= p.width[seg]) {
      cs -= p.width[seg];
      ++seg;
    }
  }
  const int width = p.width[seg];
  const T* x = reinterpret_cast<const T*>(p.x);
  auto a_slot = [&](int r, int c) { return a_s + (int64_t)r * p.d + ((c ^ (r & 7)) * kV); };

  // weight fragments of this wave's quarter of K, eight k-steps at a time
  const int col = cs + l32;  // B column = weight row
  const bool col_ok = col < width;
  const T* wrow = reinterpret_cast<const T*>(p.w[seg]) + (int64_t)(col_ok ? col : 0) * p.d;
  // stage the 32 rows of A: wave w takes rows 8w .. 8w+7 (CPL 16-byte
  // chunks per lane and row), every load issued before any is used
  const T* src = PROJ ? x : reinterpret_cast<const T*>(p.a);
  u32x4 raw[8][CPL];
#pragma unroll
  for (int rr = 0; rr < 8; ++rr)
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int b = min(b0 + wave * 8 + rr, p.B - 1), c = min(lane + 64 * i, cpr - 1);
      raw[rr][i] = ld16(src + (int64_t)b * p.d + c * kV);
    }
  // every other global read of the kernel goes out before the first use
  u32x4 graw[CPL];  // RMSNorm scale: the same chunks for every row
#pragma unroll
  for (int i = 0; i < CPL; ++i)
    graw[i] = PROJ ? ld16(reinterpret_cast<const T*>(p.gamma) + min(lane + 64 * i, cpr - 1) * kV)
                   : u32x4{0u, 0u, 0u, 0u};
  const int kq = p.d / 4, kbeg = wave * kq, nsteps = kq / 16;
  constexpr int kChunk = 16;  // k-steps of weight fragments requested at once
  typename MM::frag wf[kChunk];
  auto fetch_w = [&](int chunk) {  // unconditional (clamped) loads stay in flight together
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
      const int st = min(chunk * kChunk + i, nsteps - 1);
      wf[i] = MM::load(wrow + kbeg + st * 16 + g * 8);
    }
  };
  fetch_w(0);
  // the epilogue's reads (bias, residual) go out with the first requests too
  const T* bias = reinterpret_cast<const T*>(p.bias[seg]);
  float bv[4], xr[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int o = tid + u * 256, rr = o >> 5, cc = o & 31;
    const int b = min(b0 + rr, p.B - 1), c = min(cs + cc, width - 1);
    const float braw = to_f32((bias ? bias : x)[c]);  // unconditional read, no branch
    bv[u] = bias ? braw : 0.0f;
    xr[u] = PROJ ? 0.0f : to_f32(x[(int64_t)b * p.d + c]);
  }
#pragma unroll
  for (int rr = 0; rr < 8; ++rr) {
    const int r = wave * 8 + rr, b = b0 + r;
    float inv = 1.0f;
    if constexpr (PROJ) {
      float ss = 0.0f;
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        const T* v = reinterpret_cast<const T*>(&raw[rr][i]);
        if (lane + 64 * i < cpr)
#pragma unroll
          for (int e = 0; e < kV; ++e) ss += to_f32(v[e]) * to_f32(v[e]);
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ss += __shfl_xor(ss, off);
      inv = 1.0f / sqrtf(ss / (float)p.d + p.eps);
    }
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      if (c >= cpr) continue;
      u32x4 v = raw[rr][i];
      if (b >= p.B) v = u32x4{0u, 0u, 0u, 0u};
      if constexpr (PROJ) {
        if (blockIdx.x == 0 && b < p.B)  // x into block slot j
          st16(reinterpret_cast<T*>(p.x_blk) + ((int64_t)b * p.P + p.slot(b)) * p.d + c * kV, v);
        const T* xv = reinterpret_cast<const T*>(&v);
        const T* gv = reinterpret_cast<const T*>(&graw[i]);
        T uv[kV];
#pragma unroll
        for (int e = 0; e < kV; ++e) uv[e] = from_f32<T>(to_f32(xv[e]) * inv * to_f32(gv[e]));
        v = *reinterpret_cast<const u32x4*>(uv);
      }
      st16(a_slot(r, c), v);
    }
  }
  __syncthreads();

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  for (int chunk = 0; chunk * kChunk < nsteps; ++chunk) {
    if (chunk > 0) fetch_w(chunk);  // d > 1024 (bf16) only
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {  // fully unrolled: wf stays in registers
      const int st = chunk * kChunk + i;
      if (st >= nsteps) continue;
      const int k = kbeg + st * 16 + g * 8;
      typename MM::frag af;
      if constexpr (sizeof(T) == 2) {
        af = *reinterpret_cast<const typename MM::frag*>(a_slot(l32, k / kV));
      } else {
        const f32x4 lo = *reinterpret_cast<const f32x4*>(a_slot(l32, k / kV));
        const f32x4 hi = *reinterpret_cast<const f32x4*>(a_slot(l32, k / kV + 1));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          af[e] = lo[e];
          af[e + 4] = hi[e];
        }
      }
      typename MM::frag bf = wf[i];
      if (!col_ok) {
#pragma unroll
        for (int e = 0; e < 8; ++e) bf[e] = (T)0.0f;
      }
      acc = MM::mma(af, bf, acc);
    }
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) red[wave * 32 * 33 + acc_row(r, lane) * 33 + l32] = acc[r];
  __syncthreads();
  // four outputs per thread
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int o = tid + u * 256, rr = o >> 5, cc = o & 31;
    const int b = b0 + rr, c = cs + cc;
    if (b >= p.B || c >= width) continue;
    const int ri = rr * 33 + cc;
    const float v = ((red[ri] + red[32 * 33 + ri]) + red[2 * 32 * 33 + ri]) + red[3 * 32 * 33 + ri] + bv[u];
    if constexpr (PROJ) {
      if (seg == 0) {
        reinterpret_cast<T*>(p.q)[(int64_t)b * p.d + c] = from_f32<T>(v);
      } else if (seg < 3) {
        T* dst = reinterpret_cast<T*>(seg == 1 ? p.k_loc : p.v_loc);
        const int hd = c / p.dh, e = c - hd * p.dh;
        dst[(((int64_t)b * p.nh + hd) * p.P + p.slot(b)) * p.dh + e] = from_f32<T>(v);
      } else {
        p.alpha[(int64_t)b * p.nh + c] = sigmoidf(v);
      }
    } else {
      reinterpret_cast<T*>(p.y)[(int64_t)b * p.d + c] = from_f32<T>(xr[u] + v);
    }
  }
}

struct DecodeAttnParams {
  const void* q;       // [B, d]
  const void* kc;      // [B, h, n_cap, dh]
  const void* vc;
  const void* kl;      // [B, h, P, dh]
  const void* vl;
  float* part_m;       // [B*h, S+1]
  float* part_l;
  float* part_acc;     // [B*h, S+1, dh]
  const float* alpha;  // [B, h]
  void* attn;          // [B, d] output A
  int64_t n, n_cap, P;
  int j;               // local slots 0..j are valid
  int nh, splits, chunk;
  float scale_log2;
  DecodePos pos;       // per-sequence n and j when pos.ragged
};

// A[b, h, c] = A_x + alpha * A_h from the partials of one (sequence, head):
// cache slices merged in a fixed order with a running maximum (A_h, zero
// without cached rows), local slice normalised (A_x). A lane takes channels
// c0, c0 + 64, ... (kC of them); the loads of up to kBatch slices, the local
// part and alpha go out together before any is used, so a step with up to
// kBatch slices waits for memory once.
template <typename T, int DH>
__device__ __forceinline__ void combine_partials(const DecodeAttnParams& p, int bh, int b, int h, int c0) {
  constexpr int kC = DH / 64, kBatch = 32;
  const int64_t base = (int64_t)bh * (p.splits + 1);
  const float al = p.alpha[(int64_t)b * p.nh + h];
  const float lx = p.part_l[base + p.splits];
  float ax[kC];
#pragma unroll
  for (int u = 0; u < kC; ++u) ax[u] = p.part_acc[(base + p.splits) * DH + c0 + 64 * u];
  float mrun = -INFINITY, lrun = 0.0f, arun[kC];
#pragma unroll
  for (int u = 0; u < kC; ++u) arun[u] = 0.0f;
  for (int s0 = 0; s0 < p.splits; s0 += kBatch) {
    float m[kBatch], l[kBatch], a[kBatch][kC];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int s = min(s0 + i, p.splits - 1);
      m[i] = p.part_m[base + s];
      l[i] = p.part_l[base + s];
#pragma unroll
      for (int u = 0; u < kC; ++u) a[i][u] = p.part_acc[(base + s) * DH + c0 + 64 * u];
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      if (s0 + i >= p.splits || m[i] == -INFINITY) continue;
      const float mn = fmaxf(mrun, m[i]);
      const float f0 = fast_exp2(mrun - mn), f1 = fast_exp2(m[i] - mn);
      lrun = lrun * f0 + l[i] * f1;
#pragma unroll
      for (int u = 0; u < kC; ++u) arun[u] = arun[u] * f0 + a[i][u] * f1;
      mrun = mn;
    }
  }
  T* out = reinterpret_cast<T*>(p.attn) + (int64_t)b * p.nh * DH + h * DH;
#pragma unroll
  for (int u = 0; u < kC; ++u) {
    const float ah = mrun == -INFINITY ? 0.0f : arun[u] / lrun;
    out[c0 + 64 * u] = from_f32<T>(ax[u] / lx + al * ah);
  }
}

template <typename T, int DH>
__global__ void __launch_bounds__(256) decode_attn_kernel(const DecodeAttnParams p) {
  constexpr int kVec = 16 / sizeof(T);
  constexpr int LPR = DH / kVec;        // lanes per row
  constexpr int RPW = kWave / LPR;      // rows per wave per load
  constexpr int U = 4;                  // row groups in flight per lane
  const int s = blockIdx.x;
  const int bh = blockIdx.y;
  const int b = bh / p.nh, h = bh % p.nh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % LPR, rslot = lane / LPR;

  const T* base_k;
  const T* base_v;
  int64_t r0, r1;
  if (s < p.splits) {
    base_k = reinterpret_cast<const T*>(p.kc) + (int64_t)bh * p.n_cap * DH;
    base_v = reinterpret_cast<const T*>(p.vc) + (int64_t)bh * p.n_cap * DH;
    r0 = (int64_t)s * p.chunk;
    r1 = std::min<int64_t>(p.pos.ragged ? p.pos.n[b] : p.n, r0 + p.chunk);  // empty slices leave m = -inf
  } else {
    base_k = reinterpret_cast<const T*>(p.kl) + (int64_t)bh * p.P * DH;
    base_v = reinterpret_cast<const T*>(p.vl) + (int64_t)bh * p.P * DH;
    r0 = 0;
    r1 = (p.pos.ragged ? p.pos.j[b] : p.j) + 1;
  }

  float qv[kVec];
  {
    const T* qp = reinterpret_cast<const T*>(p.q) + (int64_t)b * p.nh * DH + h * DH + sub * kVec;
#pragma unroll
    for (int i = 0; i < kVec; ++i) qv[i] = to_f32(qp[i]) * p.scale_log2;
  }
  float mrun = -INFINITY, lrun = 0.0f;
  float acc[kVec];
#pragma unroll
  for (int i = 0; i < kVec; ++i) acc[i] = 0.0f;

  const int64_t step = (int64_t)4 * U * RPW;
  for (int64_t rb = r0 + (int64_t)wave * U * RPW; rb < r1; rb += step) {
    u32x4 kraw[U], vraw[U];
    bool valid[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t row = rb + u * RPW + rslot;
      valid[u] = row < r1;
      u32x4 zero = {0u, 0u, 0u, 0u};
      kraw[u] = valid[u] ? ld16(base_k + row * DH + sub * kVec) : zero;
      vraw[u] = valid[u] ? ld16(base_v + row * DH + sub * kVec) : zero;
    }
    float sc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const T* kt = reinterpret_cast<const T*>(&kraw[u]);
      float dot = 0.0f;
#pragma unroll
      for (int i = 0; i < kVec; ++i) dot += qv[i] * to_f32(kt[i]);
#pragma unroll
      for (int off = 1; off < LPR; off <<= 1) dot += __shfl_xor(dot, off);
      sc[u] = valid[u] ? dot : -INFINITY;
    }
    float mt = sc[0];
#pragma unroll
    for (int u = 1; u < U; ++u) mt = fmaxf(mt, sc[u]);
    const float mnew = fmaxf(mrun, mt);
    if (mnew == -INFINITY) continue;
    const float alpha = fast_exp2(mrun - mnew);
    mrun = mnew;
    lrun *= alpha;
#pragma unroll
    for (int i = 0; i < kVec; ++i) acc[i] *= alpha;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float pu = fast_exp2(sc[u] - mnew);
      lrun += pu;
      const T* vt = reinterpret_cast<const T*>(&vraw[u]);
#pragma unroll
      for (int i = 0; i < kVec; ++i) acc[i] += pu * to_f32(vt[i]);
    }
  }

  // merge the 4 * RPW row slots of the workgroup (fixed order)
  __shared__ float sm[4 * RPW];
  __shared__ float sl[4 * RPW];
  __shared__ float sacc[4 * RPW][DH];
  const int slot = wave * RPW + rslot;
  if (sub == 0) {
    sm[slot] = mrun;
    sl[slot] = lrun;
  }
#pragma unroll
  for (int i = 0; i < kVec; ++i) sacc[slot][sub * kVec + i] = acc[i];
  __syncthreads();
  if (tid < DH) {
    float mx = -INFINITY;
    for (int i = 0; i < 4 * RPW; ++i) mx = fmaxf(mx, sm[i]);
    float l = 0.0f, a = 0.0f;
    if (mx != -INFINITY) {
      for (int i = 0; i < 4 * RPW; ++i) {
        const float f = fast_exp2(sm[i] - mx);
        l += sl[i] * f;
        a += sacc[i][tid] * f;
      }
    }
    const int64_t pidx = (int64_t)bh * (p.splits + 1) + s;
    p.part_acc[pidx * DH + tid] = a;
    if (tid == 0) {
      p.part_m[pidx] = mx;
      p.part_l[pidx] = l;
    }
  }
}

// Merge of the partials of every (sequence, head): one wave per (sequence,
// head), DH / 64 channels per lane; see combine_partials.
template <typename T, int DH>
__global__ void __launch_bounds__(256) decode_combine_kernel(const DecodeAttnParams p, int nbh) {
  const int bh = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (bh >= nbh) return;
  const int b = bh / p.nh, h = bh % p.nh, lane = threadIdx.x & 63;
  combine_partials<T, DH>(p, bh, b, h, lane);
}

// Proxy K/V rows into the cache: row rr = r0 + r is (sequence rr / nblk,
// block rr % nblk) and lands at cache row n0 + block (per-sequence n and a
// write mask with ragged positions).
template <typename T>
struct EpiCache {
  T* cache;
  const T* bias;
  int64_t n_cap, n0, nblk, r0;
  int nh, dh;
  DecodePos pos;
  // cache row of (sequence b, block i), or -1 when the sequence is not written
  __device__ __forceinline__ int64_t row_of(int64_t b, int64_t i) const {
    if (!pos.ragged) return n0 + i;
    return ((pos.write >> b) & 1) ? pos.n[b] + i : -1;
  }
  __device__ __forceinline__ void operator()(int r, int c, float v) const {
    if (bias) v += to_f32(bias[c]);
    const int64_t rr = r0 + r;
    const int64_t b = rr / nblk, i = rr - b * nblk;
    const int64_t row = row_of(b, i);
    if (row < 0) return;
    const int hd = c / dh, e = c - hd * dh;
    cache[(((int64_t)b * nh + hd) * n_cap + row) * dh + e] = from_f32<T>(v);
  }
  __device__ __forceinline__ void vec8(int r, int c, const float* v0) const {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v0[e] + (bias ? to_f32(bias[c + e]) : 0.0f);
    const int64_t rr = r0 + r;
    const int64_t b = rr / nblk, i = rr - b * nblk;
    const int64_t row = row_of(b, i);
    if (row < 0) return;
    const int hd = c / dh, e0 = c - hd * dh;
    store8(cache + (((int64_t)b * nh + hd) * n_cap + row) * dh + e0, v);
  }
};

// ---- launch sequences ---------------------------------------------------------

template <typename T>
static void append_impl(Runner& run, const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                        const pf_decode_state& st, const DecodePos& pos, const void* x_blocks, int64_t nblk, char* ws) {
  const int64_t total = (int64_t)d.B * nblk;   // (sequence, block) rows of the [B*nblk, P*d] view
  const int64_t row_elems = d.P * d.d;
  for (int64_t r0 = 0; r0 < total; r0 += W.rows_cap) {
    const int rows = (int)std::min<int64_t>(W.rows_cap, total - r0);
    const T* zin = reinterpret_cast<const T*>(x_blocks) + r0 * row_elems;
    int64_t lvl_rows = (int64_t)rows * d.P;
    for (int j = 0; j < d.M; ++j) {  // compression C (Eq. 7, 16)
      lvl_rows /= d.k[j];
      GemmProblem pr{};
      pr.a = zin;
      pr.lda = (int64_t)d.k[j] * d.dl[j];
      pr.b = w->compress[j].w;
      pr.ldb = pr.lda;
      pr.M = (int)lvl_rows;
      pr.N = d.dl[j + 1];
      pr.K = (int)pr.lda;
      T* out = reinterpret_cast<T*>(ws + W.z[j + 1]);
      EpiLinear<T> e{out, pr.N, reinterpret_cast<const T*>(w->compress[j].b), nullptr, 0, nullptr};
      run.gemm<T, LAYOUT_K, LAYOUT_K>("append_compress_gemm", pr, e);
      zin = out;
    }
    const pf_linear* maps[2] = {&w->k_proxy, &w->v_proxy};
    void* caches[2] = {st.k_cache, st.v_cache};
    for (int i = 0; i < 2; ++i) {  // cached rows K_p, V_p (Eq. 21)
      GemmProblem pr{};
      pr.a = zin;
      pr.lda = d.d;
      pr.b = maps[i]->w;
      pr.ldb = d.d;
      pr.M = rows;
      pr.N = d.d;
      pr.K = d.d;
      EpiCache<T> e{reinterpret_cast<T*>(caches[i]), reinterpret_cast<const T*>(maps[i]->b), st.n_cap, st.n, nblk, r0,
                    d.nh, d.dh, pos};
      run.gemm<T, LAYOUT_K, LAYOUT_K>("append_kv_gemm", pr, e);
    }
  }
}

void split_plan(int64_t n, int* splits, int* chunk) {
  if (n <= 0) {
    *splits = 0;
    *chunk = kDecodeRowsPerSplit;
    return;
  }
  int64_t c = kDecodeRowsPerSplit;
  if ((n + c - 1) / c > kDecodeMaxSplits) c = (n + kDecodeMaxSplits - 1) / kDecodeMaxSplits;
  *chunk = (int)c;
  *splits = (int)((n + c - 1) / c);
}

// Lets a kernel use up to 160 KB of dynamic LDS, once per (kernel, device).
static hipError_t allow_lds(const void* kernel) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static std::vector<std::pair<const void*, int>> done;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  for (const auto& k : done)
    if (k.first == kernel && k.second == dev) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  if (e == hipSuccess && done.size() < 2 * kMaxDevices) done.emplace_back(kernel, dev);
  return e;
}

// Chunks per lane and row of the staged A: 1, 2 or 4 (d * sizeof(T) <= 4096).
template <typename T, bool PROJ>
static hipError_t launch_small_gemm(dim3 grid, const DecodeProjParams& pp, hipStream_t stream) {
  const int cpr = pp.d * (int)sizeof(T) / 16;
  const size_t lds = decode_small_gemm_lds<T>(pp.d);
  auto go = [&](auto kern) {
    hipError_t e = allow_lds(reinterpret_cast<const void*>(kern));
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, stream, pp);
    return hipGetLastError();
  };
  if (cpr <= 64) return go(decode_small_gemm_kernel<T, PROJ, 1>);
  if (cpr <= 128) return go(decode_small_gemm_kernel<T, PROJ, 2>);
  return go(decode_small_gemm_kernel<T, PROJ, 4>);
}

template <typename T>
static void step_impl(Runner& run, const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                      const pf_decode_state& st, const DecodePos& pos, const void* x_t, void* y_t, char* ws) {
  T* q = reinterpret_cast<T*>(ws + W.q);
  float* alpha = reinterpret_cast<float*>(ws + W.alpha);
  T* attn = reinterpret_cast<T*>(ws + W.attn);
  const int rblocks = (d.B + 31) / 32;

  DecodeProjParams pp{};
  pp.x = x_t;
  pp.gamma = w->rms_gamma;
  const pf_linear* lin[4] = {&w->q, &w->k, &w->v, &w->alpha};
  for (int i = 0; i < 4; ++i) {
    pp.w[i] = lin[i]->w;
    pp.bias[i] = lin[i]->b;
    pp.width[i] = i < 3 ? d.d : d.nh;
  }
  pp.B = d.B;
  pp.d = d.d;
  pp.nh = d.nh;
  pp.dh = d.dh;
  pp.P = d.P;
  pp.j = st.j;
  pp.eps = d.eps;
  pp.q = q;
  pp.k_loc = st.k_loc;
  pp.v_loc = st.v_loc;
  pp.alpha = alpha;
  pp.x_blk = st.x_blk;
  pp.pos = pos;
  static_assert(decode_small_gemm_lds<T>(2048 * 2 / sizeof(T)) <= 160 * 1024, "staged rows fit the LDS");
  run.launch("decode_proj", [&] {
    const dim3 grid(3 * d.d / 32 + (d.nh + 31) / 32, rblocks);
    return launch_small_gemm<T, true>(grid, pp, run.stream);
  });

  int64_t n_max = st.n;  // slices cover the longest cache of the batch
  if (pos.ragged) {
    n_max = 0;
    for (int b = 0; b < d.B; ++b) n_max = std::max<int64_t>(n_max, pos.n[b]);
  }
  int splits, chunk;
  split_plan(n_max, &splits, &chunk);
  DecodeAttnParams ap{};
  ap.q = q;
  ap.kc = st.k_cache;
  ap.vc = st.v_cache;
  ap.kl = st.k_loc;
  ap.vl = st.v_loc;
  ap.part_m = reinterpret_cast<float*>(ws + W.part_m);
  ap.part_l = reinterpret_cast<float*>(ws + W.part_l);
  ap.part_acc = reinterpret_cast<float*>(ws + W.part_acc);
  ap.alpha = alpha;
  ap.attn = attn;
  ap.n = st.n;
  ap.n_cap = st.n_cap;
  ap.P = d.P;
  ap.j = st.j;
  ap.nh = d.nh;
  ap.splits = splits;
  ap.chunk = chunk;
  ap.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)d.dh));
  ap.pos = pos;
  run.launch("decode_attn", [&] {
    const dim3 grid(splits + 1, d.B * d.nh);
    if (d.dh == 64)
      hipLaunchKernelGGL((decode_attn_kernel<T, 64>), grid, dim3(256), 0, run.stream, ap);
    else
      hipLaunchKernelGGL((decode_attn_kernel<T, 128>), grid, dim3(256), 0, run.stream, ap);
    return hipGetLastError();
  });
  run.launch("decode_combine", [&] {
    const int nbh = d.B * d.nh;
    const dim3 grid((nbh + 3) / 4);
    if (d.dh == 64)
      hipLaunchKernelGGL((decode_combine_kernel<T, 64>), grid, dim3(256), 0, run.stream, ap, nbh);
    else
      hipLaunchKernelGGL((decode_combine_kernel<T, 128>), grid, dim3(256), 0, run.stream, ap, nbh);
    return hipGetLastError();
  });

  DecodeProjParams op{};
  op.x = x_t;
  op.a = attn;
  op.w[0] = w->o.w;
  op.bias[0] = w->o.b;
  op.width[0] = d.d;
  op.B = d.B;
  op.d = d.d;
  op.y = y_t;
  run.launch("decode_out", [&] {
    const dim3 grid(d.d / 32, rblocks);
    return launch_small_gemm<T, false>(grid, op, run.stream);
  });
}

// Split-K need of every GEMM a step or an append can issue (any chunk size).
static size_t decode_gemm_need(const DecodeDims& d, const DecodeWs& W) {
  Runner dry(true);
  pf_decode_weights nw{};
  pf_decode_state ns{};
  ns.n_cap = 1;
  const DecodePos np{};
  for (int rows = 1; rows <= W.rows_cap; ++rows) {
    // one append of `rows` blocks of a single sequence exercises every chunk size
    DecodeDims d1 = d;
    d1.B = 1;
    if (d.esize == 2)
      append_impl<bf16>(dry, d1, W, &nw, ns, np, nullptr, rows, nullptr);
    else
      append_impl<float>(dry, d1, W, &nw, ns, np, nullptr, rows, nullptr);
  }
  if (d.esize == 2)
    step_impl<bf16>(dry, d, W, &nw, ns, np, nullptr, nullptr, nullptr);
  else
    step_impl<float>(dry, d, W, &nw, ns, np, nullptr, nullptr, nullptr);
  return dry.gemm_need;
}

DecodeWs decode_ws(const DecodeDims& d) {
  // memoised: the sizing sweep is pure arithmetic but runs on every call
  static thread_local DecodeDims last{};
  static thread_local size_t last_need = 0;
  static thread_local bool have = false;
  DecodeWs w = decode_ws_layout(d, kDecodeMaxSplits, d.append_rows);
  size_t need;
  if (have && memcmp(&last, &d, sizeof(d)) == 0) {
    need = last_need;
  } else {
    need = decode_gemm_need(d, w);
    last = d;
    last_need = need;
    have = true;
  }
  w.bytes = w.gemm + align256(need);
  return w;
}

DecodeWs decode_step_ws(const DecodeDims& d, int64_t n_max) {
  int splits, chunk;
  split_plan(n_max, &splits, &chunk);
  // the step appends at most one block per sequence: B rows
  DecodeWs w = decode_ws_layout(d, splits, (int)std::min<int64_t>(d.append_rows, d.B));
  Runner dry(true);
  pf_decode_weights nw{};
  pf_decode_state ns{};
  ns.n_cap = 1;
  ns.n = n_max;
  const DecodePos np{};
  if (d.esize == 2) {
    append_impl<bf16>(dry, d, w, &nw, ns, np, nullptr, 1, nullptr);
    step_impl<bf16>(dry, d, w, &nw, ns, np, nullptr, nullptr, nullptr);
  } else {
    append_impl<float>(dry, d, w, &nw, ns, np, nullptr, 1, nullptr);
    step_impl<float>(dry, d, w, &nw, ns, np, nullptr, nullptr, nullptr);
  }
  w.bytes = w.gemm + align256(dry.gemm_need);
  return w;
}

template <typename T>
hipError_t decode_step_run(const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                           const pf_decode_state& st, const DecodePos& pos, const void* x_t, void* y_t, char* ws,
                           hipStream_t stream) {
  Runner run(false, stream, reinterpret_cast<float*>(ws + W.gemm));
  step_impl<T>(run, d, W, w, st, pos, x_t, y_t, ws);
  return run.err;
}

template <typename T>
hipError_t cache_append_run(const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                            const pf_decode_state& st, const DecodePos& pos, const void* x_blocks, int64_t nblk,
                            char* ws, hipStream_t stream) {
  Runner run(false, stream, reinterpret_cast<float*>(ws + W.gemm));
  append_impl<T>(run, d, W, w, st, pos, x_blocks, nblk, ws);
  return run.err;
}

template hipError_t decode_step_run<bf16>(const DecodeDims&, const DecodeWs&, const pf_decode_weights*,
                                          const pf_decode_state&, const DecodePos&, const void*, void*, char*,
                                          hipStream_t);
template hipError_t decode_step_run<float>(const DecodeDims&, const DecodeWs&, const pf_decode_weights*,
                                           const pf_decode_state&, const DecodePos&, const void*, void*, char*,
                                           hipStream_t);
template hipError_t cache_append_run<bf16>(const DecodeDims&, const DecodeWs&, const pf_decode_weights*,
                                           const pf_decode_state&, const DecodePos&, const void*, int64_t, char*,
                                           hipStream_t);
template hipError_t cache_append_run<float>(const DecodeDims&, const DecodeWs&, const pf_decode_weights*,
                                            const pf_decode_state&, const DecodePos&, const void*, int64_t, char*,
                                            hipStream_t);

}  // namespace pf
