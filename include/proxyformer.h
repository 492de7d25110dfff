/*
 * proxyformer.h - C ABI of the MI355X (gfx950) ProxyFormer hot-path library.
 *
 * The library computes one ProxyFormer layer (Algorithm 1 of the paper:
 * block compression, causal multi-head attention over the L/P proxies,
 * decompression and gated injection back into every token), its backward,
 * and the proxy-only KV-cache decode step with its block-triggered append
 * (Sec. 3.8, Eq. 19-21). Every step runs in hand-written HIP kernels.
 *
 * Conventions shared by every entry point
 *  - Tensor arguments are DEVICE pointers owned by the caller: contiguous,
 *    row-major, 16-byte aligned. The library never allocates or frees device
 *    memory; scratch space is the caller's `workspace` (size from the
 *    matching *_workspace_size query, alignment 256 bytes). The one
 *    exception is proxy_decode_step_static, whose scratch is a fixed array
 *    in the library's own device memory.
 *  - Activations and weights use the dtype of the config (PF_BF16: bfloat16,
 *    PF_FP32: float). Accumulation is always fp32. Weight gradients are
 *    always fp32.
 *  - Linear maps follow y = x W^T + b with W stored [out, in]; a NULL bias
 *    means zero.
 *  - `stream` is a hipStream_t passed as void* (NULL = null stream). Calls
 *    only enqueue work and return without synchronising.
 *  - Every argument is checked on the host before the first launch. A status
 *    other than PF_OK means nothing was enqueued and no buffer was touched,
 *    except PF_ERR_HIP, which reports a failed launch (text in
 *    proxy_last_error()).
 *  - Calls are re-entrant; all state lives in caller-owned structs/buffers.
 */
#ifndef PROXYFORMER_H
#define PROXYFORMER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PF_MAX_LEVELS 4

enum pf_status {
  PF_OK = 0,
  PF_ERR_INVALID_ARG = -1, /* inconsistent sizes, NULL required pointer */
  PF_ERR_UNSUPPORTED = -2, /* valid but not implemented shape/dtype */
  PF_ERR_CAPACITY = -3,    /* proxy KV cache would overflow n_cap */
  PF_ERR_WORKSPACE = -4,   /* workspace NULL or smaller than required */
  PF_ERR_HIP = -5          /* a HIP launch failed */
};

enum pf_dtype { PF_FP32 = 0, PF_BF16 = 1 };

/* Which contextualised proxy feeds each block (Algorithm 1 with Eq. 9).
 * PF_TOKEN_CAUSAL: block i receives proxy i-1 (block 0 receives zero), so
 *   output token t depends only on input tokens <= t.
 * PF_BLOCK_CAUSAL: block i receives proxy i under the causal proxy mask
 *   (the literal reading; a token sees its whole block).
 * PF_BIDIRECTIONAL: block i receives proxy i, mask M = 0 in Eq. 9. */
enum pf_mask { PF_TOKEN_CAUSAL = 0, PF_BLOCK_CAUSAL = 1, PF_BIDIRECTIONAL = 2 };

/* Local fusion of the decompressed proxy Delta into the local stream (Sec. 3.4):
 * PF_INJECT_GATED: Y = X + sigmoid([X, Delta] W_g^T + b_g) * Delta (Eq. 12);
 * PF_INJECT_ADD:   Y = X + Delta (Eq. 11); the gate weights are not read and
 *   its gradients are not written.
 * PF_INJECT_AFFINE: Y = (1 + s) * Norm(X) + t with [s | t] = Delta W_a^T + b_a
 *   per token (Eq. 13; Norm = x / sqrt(mean(x^2) + 1e-6) over d_fine, no
 *   gain); reads the affine weights instead of the gate's.
 * PF_INJECT_GATED_HEAD: Eq. 12 with one gate per head (the per-head
 *   weighting of Eq. 20): G = [X, Delta] W_g^T + b_g with the gate weight
 *   W_g [n_heads, 2 d_fine], and channel c takes the gate of head
 *   c / (d_fine / n_heads); d_fine / n_heads must be a multiple of 8. */
enum pf_injection { PF_INJECT_GATED = 0, PF_INJECT_ADD = 1, PF_INJECT_AFFINE = 2, PF_INJECT_GATED_HEAD = 3 };

/* Arithmetic of the proxy path upstream of the attention logits in bf16 mode
 * (ignored in fp32 mode). Accumulation is fp32 in both.
 * PF_PRECISION_EXTENDED (default): H, the level outputs Z_j, Q and K keep a
 *   bf16 low part next to their bf16 value (v = hi + lo, about 16 mantissa
 *   bits); the projections read [hi | lo] and the logits are
 *   Qh Kh + Ql Kh + Qh Kl. A proxy sums P * d_fine products, so with wide
 *   layers the logits are large and one bf16 rounding of Q and K moves a
 *   sharp softmax by several percent; this keeps such layers (and their
 *   backward) within the bf16 tolerance. The forward attention forms the two
 *   correction products from fp8 e5m2 copies of (Ql, Qh) and (Kh, Kl), which
 *   keeps the logits to about 2^-11 of |q||k| (one bf16 rounding: 2^-8) at
 *   1.5x the score work of plain bf16; the backward uses the bf16 parts
 *   (three products). 
 * PF_PRECISION_BF16: H, Q and K are plain bf16 values (the bf16 training the
 *   paper reports): the score product is one MFMA per tile step. */
enum pf_precision { PF_PRECISION_EXTENDED = 0, PF_PRECISION_BF16 = 1 };

/* Kernels of the level-1 decompression and the gated injection (Eq. 10 with
 * Eq. 12), bf16 layers with PF_INJECT_GATED.
 * PF_GATE_SEPARATE: the decompression GEMM writes Delta to the workspace and
 *   the gate GEMM reads [X, Delta] back (default).
 * PF_GATE_FUSED: one kernel per call forms Delta for a tile of tokens in
 *   registers and applies the gate and the residual there (the gate weight is
 *   folded into the decompression weight per block position once per call),
 *   so Delta never reaches HBM in a forward without saved activations. It
 *   moves less memory but keeps fewer matrix operations in flight per LDS
 *   byte than the two GEMMs; it applies where d_fine is a multiple of 128,
 *   d_1 a multiple of 64 and at least 128, and otherwise the separate
 *   kernels run. Results agree with PF_GATE_SEPARATE to bf16 rounding. */
enum pf_gate_fusion { PF_GATE_SEPARATE = 0, PF_GATE_FUSED = 1 };

typedef struct {
  const void* w; /* [out, in] */
  const void* b; /* [out] or NULL */
} pf_linear;

/* One layer call (Algorithm 1 inputs; factorisation of Eq. 15).
 *  batch     B >= 1 sequences, processed independently.
 *  seq_len   L >= 1 tokens per sequence. There are m = ceil(L / P) blocks
 *            (Sec. 3.1); when P does not divide L the last block is
 *            zero-padded to P tokens inside the library (its proxy sees the
 *            padding as zeros; the padding produces no output and receives
 *            no gradient). The workspace then also holds padded copies of
 *            the token tensors.
 *  d_fine    local-stream width d_0.
 *  d_proxy   proxy width d_M = n_heads * head_dim.
 *  n_levels  M in 1..4; factors[0..M-1] = k_1..k_M, P = prod k_j.
 *  level_dims[j] = d_{j+1} for j < M-1 (0 -> d_proxy); level_dims[M-1] is
 *            ignored (d_M = d_proxy). Every width is a multiple of 8, and a
 *            level's grouped row of k_j * d_{j-1} elements, 2 * d_fine and
 *            2 * d_proxy elements each span at most 8 MiB (bf16:
 *            k_j * d_{j-1} <= 4M); larger rows return PF_ERR_UNSUPPORTED (a
 *            GEMM tile addresses 256 rows through one 32-bit range).
 *  head_dim  64 or 128.
 *  dtype     pf_dtype; mask pf_mask; injection pf_injection;
 *            precision pf_precision (bf16 mode); gate_fusion pf_gate_fusion.
 *  image_width  0: the tokens are a sequence and a block is P consecutive
 *            tokens. > 0: 2-D partition of the vision instantiation
 *            (Sec. 3.9): the tokens are a raster-order image of this width
 *            and height seq_len / image_width, a block is one p x p patch
 *            (P = p * p, n_levels = 1, both sides multiples of p), tokens
 *            row by row inside a patch, blocks and proxies in raster order
 *            of the patch grid. x, x_out, dy and dx stay in raster order;
 *            the workspace then also holds patch-ordered copies of them. */
typedef struct {
  int32_t batch;
  int64_t seq_len;
  int32_t d_fine, d_proxy, n_heads, head_dim;
  int32_t n_levels;
  int32_t factors[PF_MAX_LEVELS];
  int32_t level_dims[PF_MAX_LEVELS];
  int32_t dtype, mask;
  int32_t injection;
  int32_t image_width;
  int32_t precision; /* pf_precision */
  int32_t gate_fusion; /* pf_gate_fusion */
} pf_layer_config;

/* compress[j]: W [d_{j+1}, k_{j+1} d_j]  (Eq. 7, Eq. 16)
 * q, k, v, o : W [d_proxy, d_proxy]     (Eq. 9 and its output map)
 * decompress[j]: W [k_{j+1} d_j, d_{j+1}] (Eq. 10, Eq. 17)
 * gate       : W [d_fine, 2 d_fine] acting on [X, Delta] (Eq. 12), or
 *              W [n_heads, 2 d_fine] with PF_INJECT_GATED_HEAD; not read by
 *              the other injections (may be NULL there)
 * affine     : W [2 d_fine, d_fine] acting on Delta, rows 0..d_fine-1 give
 *              s and the next d_fine rows t (Eq. 13); read only with
 *              PF_INJECT_AFFINE (may be NULL otherwise) */
typedef struct {
  pf_linear compress[PF_MAX_LEVELS];
  pf_linear q, k, v, o;
  pf_linear decompress[PF_MAX_LEVELS];
  pf_linear gate;
  pf_linear affine;
} pf_layer_weights;

typedef struct {
  void* dw; /* fp32, same shape as W, overwritten */
  void* db; /* fp32 [out], overwritten; may be NULL (not computed) */
} pf_linear_grad;

typedef struct {
  pf_linear_grad compress[PF_MAX_LEVELS];
  pf_linear_grad q, k, v, o;
  pf_linear_grad decompress[PF_MAX_LEVELS];
  pf_linear_grad gate;
  pf_linear_grad affine; /* with PF_INJECT_AFFINE */
} pf_layer_grads;

/* Bytes of scratch the forward (for_backward = 0) or backward
 * (for_backward = 1) needs; 0 for an invalid config. */
size_t proxy_layer_workspace_size(const pf_layer_config* cfg, int for_backward);

/* Bytes of the `saved` buffer the forward fills for the backward
 * (activations of every step); 0 for an invalid config. */
size_t proxy_layer_saved_size(const pf_layer_config* cfg);

/* Layer forward, Algorithm 1 (Eq. 2, 7, 8, 9, 10, 12, 15-17).
 *  x      [B, L, d_fine]  local stream X^(l-1)
 *  h_in   [B, m, d_proxy] proxy stream H^(l-1), or NULL for zero (Eq. 8
 *         then reduces to direct compression)
 *  x_out  [B, L, d_fine]  X^(l) = X + sigmoid(G) * Delta   (may not alias x)
 *  h_out  [B, m, d_proxy] H^(l) = H^(l-1) + C(X)            (returned by Alg. 1)
 *  saved  NULL, or proxy_layer_saved_size() bytes to keep activations for
 *         proxy_layer_backward.
 * Returns PF_OK or an error status (see the conventions above). */
int proxy_layer_forward(const pf_layer_config* cfg, const pf_layer_weights* w,
                        const void* x, const void* h_in, void* x_out, void* h_out,
                        void* saved, void* workspace, size_t ws_bytes, void* stream);

/* Layer backward: the chain rule through every forward step.
 *  saved   the buffer a forward with the same cfg/weights/x/h_in filled
 *  dy      [B, L, d_fine] gradient of x_out
 *  dh_out  [B, m, d_proxy] gradient of h_out, or NULL for zero
 *  dx      [B, L, d_fine] gradient of x (dtype of cfg), overwritten
 *  dh_in   [B, m, d_proxy] gradient of h_in (dtype of cfg), or NULL
 *  grads   fp32 weight/bias gradients summed over the batch, overwritten;
 *          a NULL dw skips that map's weight gradient. */
int proxy_layer_backward(const pf_layer_config* cfg, const pf_layer_weights* w,
                         const void* x, const void* h_in, const void* saved,
                         const void* dy, const void* dh_out, void* dx, void* dh_in,
                         const pf_layer_grads* grads, void* workspace, size_t ws_bytes,
                         void* stream);

/* Decode (generation block of Eq. 19-20 against the proxy cache of Eq. 21).
 *  d_model = n_heads * head_dim; head_dim 64 or 128; d_model * element size
 *  at most 4096 bytes.
 *  n_levels/factors/level_dims describe the compression C of the append
 *  (as in pf_layer_config with d_fine = d_proxy = d_model, including the
 *  8 MiB bound on a grouped row k_j * d_{j-1}). */
typedef struct {
  int32_t batch, d_model, n_heads, head_dim, n_levels;
  int32_t factors[PF_MAX_LEVELS];
  int32_t level_dims[PF_MAX_LEVELS];
  int32_t dtype;
  float rms_eps;
} pf_decode_config;

/* rms_gamma [d_model]; q,k,v,o W [d,d]; alpha W [n_heads, d] (MLP_alpha of
 * Eq. 20, followed by a sigmoid); compress as in pf_layer_weights;
 * k_proxy, v_proxy W [d,d]: the proxy-attention K/V maps whose outputs are
 * the cached rows (Eq. 21). */
typedef struct {
  const void* rms_gamma;
  pf_linear q, k, v, o, alpha;
  pf_linear compress[PF_MAX_LEVELS];
  pf_linear k_proxy, v_proxy;
} pf_decode_weights;

/* Whole inference state (caller-owned device buffers, host counters).
 *  k_cache, v_cache [B, n_heads, n_cap, head_dim]: rows 0..n-1 valid.
 *  x_blk [B, P, d]: inputs of the current block; k_loc, v_loc
 *  [B, n_heads, P, head_dim]: its keys/values; slots 0..j-1 valid.
 * With n_seq = j_seq = NULL the batch moves in lockstep (one n and one j for
 * all sequences). With both set (host arrays of B entries, batch <= 64) every
 * sequence keeps its own position: sequence b has n_seq[b] cached rows and
 * j_seq[b] filled slots, the scalar n and j are ignored, a step advances each
 * sequence by one token and appends the blocks that complete in it (Sec. 3.8
 * streams every sequence on its own; ragged batches serve sequences that
 * started at different times). */
#define PF_MAX_RAGGED_BATCH 64
typedef struct {
  void* k_cache;
  void* v_cache;
  int64_t n_cap, n;
  void* x_blk;
  void* k_loc;
  void* v_loc;
  int32_t j;
  int64_t* n_seq;  /* host [B] or NULL */
  int32_t* j_seq;  /* host [B] or NULL */
} pf_decode_state;

size_t proxy_decode_workspace_size(const pf_decode_config* cfg);

/* One decode step for the token at block position j of every sequence.
 *  x_t [B, d] layer input of the new token; y_t [B, d] output
 *  y = x + (A_x + alpha * A_h) W_o^T + b_o, where A_x attends over the
 *  current block's slots 0..j and A_h over the n cached proxies.
 * Writes x/k/v of the token into slot j; on success j += 1, and when j
 * reaches P the block is appended (as proxy_cache_append) in the same call,
 * n += 1 and j = 0. A full cache (n == n_cap when the block completes)
 * returns PF_ERR_CAPACITY before any launch. With per-sequence positions
 * (n_seq, j_seq) the same holds per sequence. */
int proxy_decode_step(const pf_decode_config* cfg, const pf_decode_weights* w,
                      pf_decode_state* st, const void* x_t, void* y_t,
                      void* workspace, size_t ws_bytes, void* stream);

/* proxy_decode_step without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). Same arguments, kernels and results as
 * proxy_decode_step; the scratch is a fixed 64 MiB array in the library's
 * device memory, one per GPU, held until the process ends. It calls no
 * allocation routine; its device address is looked up once per device on the
 * first call there (with that device current).
 *  A step needs about B * n_heads * (head_dim + 2) * 4 bytes per 1,024 cached
 *  rows of its longest sequence, plus the append of one block per sequence
 *  (about 5 MiB at 32 sequences x 16,384 rows, d_model 1024); a step needing
 *  more than 64 MiB returns PF_ERR_UNSUPPORTED before any launch.
 *  Every call on one GPU uses that GPU's one array: calls that overlap on one
 *  GPU (other streams, other threads) race and corrupt each other's results.
 *  Nothing in the array needs to start at zero; it keeps the last call's
 *  contents. */
int proxy_decode_step_static(const pf_decode_config* cfg, const pf_decode_weights* w,
                             pf_decode_state* st, const void* x_t, void* y_t, void* stream);

/* Append nblk whole blocks to the cache (prefill path and the streaming
 * update of Sec. 3.8): for each block h = C(x_block) (Eq. 7 / 16), then
 * K_p[n] = h W_kp^T + b, V_p[n] = h W_vp^T + b, n += 1 (Eq. 21).
 *  x_blocks [B, nblk * P, d]. PF_ERR_CAPACITY if n + nblk > n_cap. With
 *  per-sequence positions every sequence b appends at row n_seq[b]. */
int proxy_cache_append(const pf_decode_config* cfg, const pf_decode_weights* w,
                       pf_decode_state* st, const void* x_blocks, int64_t nblk,
                       void* workspace, size_t ws_bytes, void* stream);

/* Prefill: the parallel (training-time) form of the generation block of
 * Eq. 19-20 over the next n_tokens tokens of every sequence, with the cache
 * update of Eq. 21 for the chunk's complete blocks; the result equals
 * n_tokens calls of proxy_decode_step (up to rounding order).
 * Token t of the chunk lies in block t / P. Its output is
 * y_t = x_t + (A_x + alpha_t * A_h) W_o^T + b_o, where A_x attends over the
 * tokens of its own block up to t and A_h over the n cached proxies plus the
 * t / P blocks of the chunk before its own (appended first, each compressed
 * as proxy_cache_append does). The tokens of an unfinished last block stay
 * in the local slots.
 *  x [B, n_tokens, d]: layer inputs; y [B, n_tokens, d]: outputs (must not
 *  overlap x). Positions must be lockstep (n_seq = j_seq = NULL) with
 *  j == 0, else PF_ERR_UNSUPPORTED; PF_ERR_CAPACITY if n + n_tokens / P >
 *  n_cap. On success n += n_tokens / P and j = n_tokens % P; n_tokens = 0
 *  does nothing.
 *  workspace: proxy_prefill_workspace_size(cfg, n_tokens, st->n_cap) bytes
 *  (0 for an invalid config or sizes beyond the limits: batch * n_tokens
 *  below 2^31, head_dim * n_tokens and head_dim * n_cap elements per head
 *  below 2 GiB). */
size_t proxy_prefill_workspace_size(const pf_decode_config* cfg, int64_t n_tokens, int64_t n_cap);
int proxy_decode_prefill(const pf_decode_config* cfg, const pf_decode_weights* w,
                         pf_decode_state* st, const void* x, int64_t n_tokens, void* y,
                         void* workspace, size_t ws_bytes, void* stream);

/* Launch tracing (profiling aid). While enabled, every kernel launch of the
 * library is bracketed by two HIP events recorded on its stream and
 * attributed to a label (e.g. "gate_gemm", "attention_fwd", "decode_attn").
 *  proxy_trace_enable   1 = on, 0 = off; returns the previous setting.
 *  proxy_trace_collect  waits for every recorded event, folds it into the
 *                       per-label totals; returns the number of labels or
 *                       PF_ERR_HIP.
 *  proxy_trace_get      label i (first-seen order) into label[label_cap]
 *                       (NUL-terminated), its launch count and total
 *                       milliseconds; PF_ERR_INVALID_ARG for a bad index.
 *  proxy_trace_reset    drops all totals and pending events.
 * Tracing adds host work per launch; time throughput with it off. */
int proxy_trace_enable(int on);
int proxy_trace_collect(void);
int proxy_trace_get(int i, char* label, size_t label_cap, int64_t* launches, double* total_ms);
void proxy_trace_reset(void);

/* Matrix-core ceiling (measurement aid, not part of the layer): enqueues
 * n_workgroups workgroups of four waves on `stream`; every wave issues
 * iters x 8 independent v_mfma_f32_32x32x16_bf16 (32x32x16 multiply-adds,
 * 32,768 flops each) on register operands and touches no memory until it
 * writes one float per thread to out. out: caller-owned device buffer of
 * n_workgroups * 256 floats. Flops per call:
 * n_workgroups * 4 * iters * 8 * 32768; timing the call with events on the
 * same stream gives the achievable dense bf16 rate of the device.
 * PF_ERR_INVALID_ARG for a NULL out, n_workgroups outside [1, 2^20] or
 * iters < 1 (nothing enqueued); PF_ERR_HIP if the launch fails. */
int proxy_ceiling_mfma(void* out, int64_t n_workgroups, int32_t iters, void* stream);

/* HBM read ceiling (measurement aid, not part of the layer): enqueues
 * n_workgroups workgroups of four waves on `stream` that read the `bytes`
 * bytes at src (device memory, 16-byte aligned, bytes a multiple of 16) with
 * grid-strided 16-byte loads, four in flight per lane, and nothing else;
 * workgroup w writes the XOR of every 32-bit word it read to out[w] (a
 * caller-owned device buffer of n_workgroups uint32), so the XOR over out
 * equals the XOR of the whole buffer. Timing the call with events on the same
 * stream gives the read rate a streaming kernel can reach on the device.
 * PF_ERR_INVALID_ARG for a NULL or misaligned src, a NULL out, bytes zero or
 * not a multiple of 16, or n_workgroups outside [1, 2^20] (nothing enqueued);
 * PF_ERR_HIP if the launch fails. */
int proxy_ceiling_read(const void* src, size_t bytes, void* out, int64_t n_workgroups, void* stream);

/* Message of the last non-OK status on the calling thread. */
const char* proxy_last_error(void);

/* Library ABI version (major * 100 + minor): 101 adds pf_layer_config.precision
 * and proxy_decode_step_static; 102 adds pf_layer_config.gate_fusion; 103 adds
 * proxy_ceiling_read. */
int proxy_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PROXYFORMER_H */
