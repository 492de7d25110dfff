// Proxy-KV-cache decode (Eq. 19-21, Sec. 3.8): sizes, workspace layout and
// the launch sequences of the decode step and the cache append.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime.h>

#include "../../include/proxyformer.h"

namespace pf {

struct DecodeDims {
  int B, d, nh, dh, M;
  int k[PF_MAX_LEVELS];
  int dl[PF_MAX_LEVELS + 1];  // d_0 = d_model ... d_M = d_model
  int64_t P;
  int esize;
  float eps;
  int append_rows;            // rows (sequence, block) compressed per append GEMM chunk
};

// Per-sequence positions, passed by value in kernel arguments: sequence b
// has n[b] cached rows and j[b] filled local slots; `write` marks the
// sequences whose rows a cache write stores (bit b). With ragged = 0 every
// sequence uses the scalar n and j.
struct DecodePos {
  int32_t n[PF_MAX_RAGGED_BATCH];
  int32_t j[PF_MAX_RAGGED_BATCH];
  uint64_t write;
  int32_t ragged;
};

constexpr int kDecodeMaxSplits = 256;   // cache-row slices per (sequence, head)
constexpr int kDecodeRowsPerSplit = 1024;

struct DecodeWs {
  int splits_cap;                   // cache slices per (sequence, head) the partials hold
  int rows_cap;                     // (sequence, block) rows per append chunk
  size_t q, alpha, attn;            // [B, d], fp32 [B, h], [B, d]
  size_t part_m, part_l, part_acc;  // fp32 partial softmax states
  size_t z[PF_MAX_LEVELS];          // append: compression level outputs (j = 1..M)
  size_t gemm;
  size_t bytes;
};

int decode_dims(const pf_decode_config* c, DecodeDims* d, const char** why);
// Workspace of every decode call (steps and appends of any size).
DecodeWs decode_ws(const DecodeDims& d);
// Scratch of one decode step whose longest cache holds n_max rows: its own
// slice partials and the append of one block per sequence (smaller than
// decode_ws; the layout differs, the kernels are the same).
DecodeWs decode_step_ws(const DecodeDims& d, int64_t n_max);
// Cache slices the decode attention cuts n rows into, and their length.
void split_plan(int64_t n, int* splits, int* chunk);

// `pos` carries the per-sequence positions when st.n_seq / st.j_seq are set;
// W is the scratch layout inside ws.
template <typename T>
hipError_t decode_step_run(const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                           const pf_decode_state& st, const DecodePos& pos, const void* x_t, void* y_t, char* ws,
                           hipStream_t stream);

// Prefill (parallel form of the generation block over a chunk of T tokens):
// buffers placed after the decode workspace, which the chunk's append uses.
struct PrefillWs {
  size_t u;      // [B*T, d] RMSNorm output, later the attention output A
  size_t q, k;   // [B, h, T, dh]
  size_t vt;     // values of the chunk: bf16 [B, h, T, dh]; fp32 [B, h, dh, ld_t] (token-contiguous)
  size_t alpha;  // fp32 [B*T, h]
  size_t vct;    // fp32 only: [B, h, dh, ld_c] cached values, row-contiguous (bf16: empty)
  size_t xc;     // [B, T/P*P, d] complete blocks, gathered when T % P != 0
  size_t gemm;   // split-K partials of the chunk's GEMMs
  size_t bytes;
  int64_t ld_t, ld_c;
};

// Limits of a prefill of T tokens with cache capacity n_cap (NULL: fits).
const char* prefill_limits(const DecodeDims& d, int64_t T, int64_t n_cap);
PrefillWs prefill_ws(const DecodeDims& d, int64_t T, int64_t n_cap);

template <typename T>
hipError_t prefill_run(const DecodeDims& d, const pf_decode_weights* w, const pf_decode_state& st, const void* x,
                       int64_t n_tok, void* y, char* ws, hipStream_t stream);

template <typename T>
hipError_t cache_append_run(const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w,
                            const pf_decode_state& st, const DecodePos& pos, const void* x_blocks, int64_t nblk,
                            char* ws, hipStream_t stream);

}  // namespace pf
