// C-ABI entry points: argument validation on the host, then dispatch to the
// dtype-specific launch sequences. Nothing is enqueued unless every check
// passes.
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "ceiling.hpp"
#include "common.hpp"
#include "decode.hpp"
#include "layer.hpp"

namespace pf {
size_t layer_gemm_ws_bytes(const LayerDims& d, bool for_backward) {
  return for_backward ? layer_backward_gemm_ws(d) : layer_forward_gemm_ws(d);
}
}  // namespace pf

using namespace pf;

static thread_local std::string g_last_error;

static int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
static int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

static int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return PF_OK;
  return fail(PF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

static bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const char* pa = reinterpret_cast<const char*>(a);
  const char* pb = reinterpret_cast<const char*>(b);
  return a && b && pa < pb + nb && pb < pa + na;
}

// NULL counts as aligned (optional pointers are checked for presence elsewhere)
static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

extern "C" {

int proxy_version(void) { return 103; }

int proxy_ceiling_mfma(void* out, int64_t n_workgroups, int32_t iters, void* stream) {
  if (!out) return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_mfma: out is NULL");
  if (n_workgroups < 1 || n_workgroups > (1 << 20))
    return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_mfma: n_workgroups must be in [1, 2^20]");
  if (iters < 1) return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_mfma: iters must be >= 1");
  return hip_status(launch_mfma_ceiling(static_cast<float*>(out), n_workgroups, iters, (hipStream_t)stream),
                    "proxy_ceiling_mfma");
}

int proxy_ceiling_read(const void* src, size_t bytes, void* out, int64_t n_workgroups, void* stream) {
  if (!src || !out) return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_read: src or out is NULL");
  if (!aligned16(src)) return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_read: src must be 16-byte aligned");
  if (bytes == 0 || bytes % 16 != 0) return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_read: bytes must be a positive multiple of 16");
  if (n_workgroups < 1 || n_workgroups > (1 << 20))
    return fail(PF_ERR_INVALID_ARG, "proxy_ceiling_read: n_workgroups must be in [1, 2^20]");
  return hip_status(launch_read_ceiling(src, bytes, static_cast<unsigned*>(out), n_workgroups, (hipStream_t)stream),
                    "proxy_ceiling_read");
}

const char* proxy_last_error(void) { return g_last_error.c_str(); }

size_t proxy_layer_workspace_size(const pf_layer_config* cfg, int for_backward) {
  LayerDims d;
  const char* why;
  if (layer_dims(cfg, &d, &why) != PF_OK) return 0;
  return layer_ws(d, for_backward != 0).bytes;
}

size_t proxy_layer_saved_size(const pf_layer_config* cfg) {
  LayerDims d;
  const char* why;
  if (layer_dims(cfg, &d, &why) != PF_OK) return 0;
  return layer_acts(d, true).bytes;
}

static int check_weights(const LayerDims& d, const pf_layer_weights* w, int injection) {
  const bool gated = injection == PF_INJECT_GATED || injection == PF_INJECT_GATED_HEAD;
  if (!w) return fail(PF_ERR_INVALID_ARG, "weights struct is NULL");
  for (int j = 0; j < d.M; ++j) {
    if (!w->compress[j].w) return fail(PF_ERR_INVALID_ARG, "compress[%d].w is NULL", j);
    if (!w->decompress[j].w) return fail(PF_ERR_INVALID_ARG, "decompress[%d].w is NULL", j);
    if (!aligned16(w->compress[j].w) || !aligned16(w->decompress[j].w) || !aligned16(w->compress[j].b) ||
        !aligned16(w->decompress[j].b))
      return fail(PF_ERR_INVALID_ARG, "level %d weights and biases must be 16-byte aligned", j);
  }
  const pf_linear* maps[5] = {&w->q, &w->k, &w->v, &w->o, &w->gate};
  const char* names[5] = {"q", "k", "v", "o", "gate"};
  for (int i = 0; i < (gated ? 5 : 4); ++i) {
    if (!maps[i]->w) return fail(PF_ERR_INVALID_ARG, "%s.w is NULL", names[i]);
    if (!aligned16(maps[i]->w) || !aligned16(maps[i]->b))
      return fail(PF_ERR_INVALID_ARG, "%s weights and bias must be 16-byte aligned", names[i]);
  }
  if (injection == PF_INJECT_AFFINE) {
    if (!w->affine.w) return fail(PF_ERR_INVALID_ARG, "affine.w is NULL");
    if (!aligned16(w->affine.w) || !aligned16(w->affine.b))
      return fail(PF_ERR_INVALID_ARG, "affine weights and bias must be 16-byte aligned");
  }
  return PF_OK;
}

int proxy_layer_forward(const pf_layer_config* cfg, const pf_layer_weights* w, const void* x, const void* h_in,
                        void* x_out, void* h_out, void* saved, void* workspace, size_t ws_bytes, void* stream) {
  LayerDims d;
  const char* why;
  int st = layer_dims(cfg, &d, &why);
  if (st != PF_OK) return fail(st, "invalid layer config: %s", why);
  if ((st = check_weights(d, w, cfg->injection)) != PF_OK) return st;
  if (!x || !x_out || !h_out) return fail(PF_ERR_INVALID_ARG, "x, x_out and h_out must be non-NULL");
  if (!aligned16(x) || !aligned16(x_out) || !aligned16(h_out) || (h_in && !aligned16(h_in)) ||
      (saved && !aligned16(saved)))
    return fail(PF_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  const size_t tok_bytes = (size_t)d.B * d.L_in * d.d_f * d.esize;
  const size_t prox_bytes = (size_t)d.B * d.m * d.d_p * d.esize;
  if (overlaps(x, tok_bytes, x_out, tok_bytes)) return fail(PF_ERR_INVALID_ARG, "x_out must not alias x");
  if (overlaps(h_out, prox_bytes, x_out, tok_bytes) || overlaps(h_out, prox_bytes, x, tok_bytes))
    return fail(PF_ERR_INVALID_ARG, "h_out must not alias x or x_out");
  const LayerWs W = layer_ws(d, false);
  if (W.bytes && (!workspace || ws_bytes < W.bytes))
    return fail(PF_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", W.bytes, workspace ? ws_bytes : 0);
  char* ws = reinterpret_cast<char*>(workspace);
  char* acts = saved ? reinterpret_cast<char*>(saved) : ws + W.acts;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // partial last block: run on a zero-padded copy; 2-D partition: on a
  // patch-ordered copy
  const int64_t row_bytes = (int64_t)d.d_f * d.esize;
  const void* xk = x;
  void* yk = x_out;
  hipError_t e = hipSuccess;
  if (d.staged()) {
    xk = ws + W.x_pad;
    yk = ws + W.y_pad;
    e = d.img_w ? permute_patches(x, ws + W.x_pad, d.B, d.L, d.img_w, d.patch, row_bytes, false, s)
                : pad_rows(x, ws + W.x_pad, d.B, d.L_in, d.L, row_bytes, s);
    if (e != hipSuccess) return hip_status(e, "proxy_layer_forward staging");
  }
  e = cfg->dtype == PF_BF16 ? layer_forward_run<bf16>(d, cfg, w, xk, h_in, yk, h_out, acts, saved != nullptr, ws, s)
                            : layer_forward_run<float>(d, cfg, w, xk, h_in, yk, h_out, acts, saved != nullptr, ws, s);
  if (e == hipSuccess && d.staged())
    e = d.img_w ? permute_patches(yk, x_out, d.B, d.L, d.img_w, d.patch, row_bytes, true, s)
                : unpad_rows(yk, x_out, d.B, d.L_in, d.L, row_bytes, s);
  return hip_status(e, "proxy_layer_forward launch");
}

int proxy_layer_backward(const pf_layer_config* cfg, const pf_layer_weights* w, const void* x, const void* h_in,
                         const void* saved, const void* dy, const void* dh_out, void* dx, void* dh_in,
                         const pf_layer_grads* grads, void* workspace, size_t ws_bytes, void* stream) {
  LayerDims d;
  const char* why;
  int st = layer_dims(cfg, &d, &why);
  if (st != PF_OK) return fail(st, "invalid layer config: %s", why);
  if ((st = check_weights(d, w, cfg->injection)) != PF_OK) return st;
  if (!x || !saved || !dy || !dx || !grads)
    return fail(PF_ERR_INVALID_ARG, "x, saved, dy, dx and grads must be non-NULL");
  if ((h_in == nullptr) != (dh_in == nullptr))
    return fail(PF_ERR_INVALID_ARG, "dh_in must be given exactly when h_in is given");
  if (!aligned16(x) || !aligned16(saved) || !aligned16(dy) || !aligned16(dx) || (dh_out && !aligned16(dh_out)) ||
      (dh_in && !aligned16(dh_in)) || (h_in && !aligned16(h_in)))
    return fail(PF_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  const size_t tok_bytes = (size_t)d.B * d.L_in * d.d_f * d.esize;
  if (overlaps(dx, tok_bytes, dy, tok_bytes)) return fail(PF_ERR_INVALID_ARG, "dx must not alias dy");
  const LayerWs W = layer_ws(d, true);
  if (W.bytes && (!workspace || ws_bytes < W.bytes))
    return fail(PF_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", W.bytes, workspace ? ws_bytes : 0);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const char* sv = reinterpret_cast<const char*>(saved);
  char* ws = reinterpret_cast<char*>(workspace);
  // partial last block: the padding has dY = 0 and its dX is dropped;
  // 2-D partition: X and dY gathered into patch order, dX scattered back
  const int64_t row_bytes = (int64_t)d.d_f * d.esize;
  const void* xk = x;
  const void* dyk = dy;
  void* dxk = dx;
  hipError_t e = hipSuccess;
  if (d.staged()) {
    xk = ws + W.x_pad;
    dyk = ws + W.dy_pad;
    dxk = ws + W.y_pad;
    if (d.img_w) {
      e = permute_patches(x, ws + W.x_pad, d.B, d.L, d.img_w, d.patch, row_bytes, false, s);
      if (e == hipSuccess) e = permute_patches(dy, ws + W.dy_pad, d.B, d.L, d.img_w, d.patch, row_bytes, false, s);
    } else {
      e = pad_rows(x, ws + W.x_pad, d.B, d.L_in, d.L, row_bytes, s);
      if (e == hipSuccess) e = pad_rows(dy, ws + W.dy_pad, d.B, d.L_in, d.L, row_bytes, s);
    }
    if (e != hipSuccess) return hip_status(e, "proxy_layer_backward staging");
  }
  e = cfg->dtype == PF_BF16
          ? layer_backward_run<bf16>(d, cfg, w, xk, h_in, sv, dyk, dh_out, dxk, dh_in, grads, ws, s)
          : layer_backward_run<float>(d, cfg, w, xk, h_in, sv, dyk, dh_out, dxk, dh_in, grads, ws, s);
  if (e == hipSuccess && d.staged())
    e = d.img_w ? permute_patches(dxk, dx, d.B, d.L, d.img_w, d.patch, row_bytes, true, s)
                : unpad_rows(dxk, dx, d.B, d.L_in, d.L, row_bytes, s);
  return hip_status(e, "proxy_layer_backward launch");
}

// ---------------------------------------------------------------- decode

size_t proxy_decode_workspace_size(const pf_decode_config* cfg) {
  DecodeDims d;
  const char* why;
  if (decode_dims(cfg, &d, &why) != PF_OK) return 0;
  return decode_ws(d).bytes;
}

// prefill_tokens >= 0: the workspace is checked against a prefill of that many tokens
// check_ws = false: the caller brings no workspace (the static-scratch step)
static int check_decode_common(const pf_decode_config* cfg, const pf_decode_weights* w, const pf_decode_state* st,
                               DecodeDims* d, void* workspace, size_t ws_bytes, int64_t prefill_tokens = -1,
                               bool check_ws = true) {
  const char* why;
  int s = decode_dims(cfg, d, &why);
  if (s != PF_OK) return fail(s, "invalid decode config: %s", why);
  if (!w || !st) return fail(PF_ERR_INVALID_ARG, "weights and state must be non-NULL");
  if (!w->rms_gamma || !w->q.w || !w->k.w || !w->v.w || !w->o.w || !w->alpha.w || !w->k_proxy.w || !w->v_proxy.w)
    return fail(PF_ERR_INVALID_ARG, "a required decode weight is NULL");
  for (int j = 0; j < d->M; ++j)
    if (!w->compress[j].w) return fail(PF_ERR_INVALID_ARG, "compress[%d].w is NULL", j);
  {
    const void* ptrs[] = {w->rms_gamma, w->q.w, w->q.b, w->k.w, w->k.b, w->v.w, w->v.b, w->o.w, w->o.b,
                          w->alpha.w, w->alpha.b, w->k_proxy.w, w->k_proxy.b, w->v_proxy.w, w->v_proxy.b,
                          w->compress[0].w, w->compress[0].b, w->compress[1].w, w->compress[1].b,
                          w->compress[2].w, w->compress[2].b, w->compress[3].w, w->compress[3].b,
                          st->k_cache, st->v_cache, st->x_blk, st->k_loc, st->v_loc};
    for (const void* p : ptrs)
      if (!aligned16(p)) return fail(PF_ERR_INVALID_ARG, "decode weights and state buffers must be 16-byte aligned");
  }
  if (!st->k_cache || !st->v_cache || !st->x_blk || !st->k_loc || !st->v_loc)
    return fail(PF_ERR_INVALID_ARG, "a decode state buffer is NULL");
  if (st->n_cap < 0) return fail(PF_ERR_INVALID_ARG, "state n_cap must be >= 0");
  if (st->n_cap > INT32_MAX) return fail(PF_ERR_UNSUPPORTED, "n_cap above 2^31 - 1");
  if ((st->n_seq == nullptr) != (st->j_seq == nullptr))
    return fail(PF_ERR_INVALID_ARG, "n_seq and j_seq must be both set or both NULL");
  if (st->n_seq) {
    if (d->B > PF_MAX_RAGGED_BATCH)
      return fail(PF_ERR_UNSUPPORTED, "per-sequence positions need batch <= %d", PF_MAX_RAGGED_BATCH);
    for (int b = 0; b < d->B; ++b) {
      if (st->n_seq[b] < 0 || st->n_seq[b] > st->n_cap)
        return fail(PF_ERR_INVALID_ARG, "n_seq[%d] must be in 0..n_cap", b);
      if (st->j_seq[b] < 0 || st->j_seq[b] >= d->P) return fail(PF_ERR_INVALID_ARG, "j_seq[%d] must be in 0..P-1", b);
    }
  } else {
    if (st->n < 0 || st->n > st->n_cap) return fail(PF_ERR_INVALID_ARG, "state n must be in 0..n_cap");
    if (st->j < 0 || st->j >= d->P) return fail(PF_ERR_INVALID_ARG, "state j must be in 0..P-1");
  }
  if (!check_ws) return PF_OK;
  size_t need;
  if (prefill_tokens >= 0) {
    if (const char* lim = prefill_limits(*d, prefill_tokens, st->n_cap))
      return fail(PF_ERR_UNSUPPORTED, "prefill: %s", lim);
    need = prefill_ws(*d, prefill_tokens, st->n_cap).bytes;
  } else {
    need = decode_ws(*d).bytes;
  }
  if (!workspace || ws_bytes < need)
    return fail(PF_ERR_WORKSPACE, "workspace too small: need %zu bytes, got %zu", need, workspace ? ws_bytes : 0);
  return PF_OK;
}

// One decode step on validated arguments with the scratch layout W inside
// ws: the step's launches, then the append of the blocks the token
// completes, then the host counters.
static int decode_step_on(const DecodeDims& d, const DecodeWs& W, const pf_decode_weights* w, pf_decode_state* st,
                          const void* x_t, void* y_t, char* ws, hipStream_t hs, const char* who) {
  DecodePos pos{};
  if (st->n_seq) {
    // per-sequence positions: the blocks that complete in this step are
    // appended together (one pass over the compression weights), each at
    // its own sequence's row
    pos.ragged = 1;
    for (int b = 0; b < d.B; ++b) {
      pos.n[b] = (int32_t)st->n_seq[b];
      pos.j[b] = st->j_seq[b];
      if (st->j_seq[b] + 1 == d.P) {
        if (st->n_seq[b] + 1 > st->n_cap)
          return fail(PF_ERR_CAPACITY, "%s: proxy cache of sequence %d full: n = %lld, n_cap = %lld", who, b,
                      (long long)st->n_seq[b], (long long)st->n_cap);
        pos.write |= (uint64_t)1 << b;
      }
    }
    hipError_t e = d.esize == 2 ? decode_step_run<bf16>(d, W, w, *st, pos, x_t, y_t, ws, hs)
                                : decode_step_run<float>(d, W, w, *st, pos, x_t, y_t, ws, hs);
    if (e != hipSuccess) return hip_status(e, who);
    if (pos.write) {
      e = d.esize == 2 ? cache_append_run<bf16>(d, W, w, *st, pos, st->x_blk, 1, ws, hs)
                       : cache_append_run<float>(d, W, w, *st, pos, st->x_blk, 1, ws, hs);
      if (e != hipSuccess) return hip_status(e, who);
    }
    for (int b = 0; b < d.B; ++b) {
      if ((pos.write >> b) & 1) {
        st->n_seq[b] += 1;
        st->j_seq[b] = 0;
      } else {
        st->j_seq[b] += 1;
      }
    }
    return PF_OK;
  }
  const bool completes = st->j + 1 == d.P;
  if (completes && st->n + 1 > st->n_cap)
    return fail(PF_ERR_CAPACITY, "%s: proxy cache full: n = %lld, n_cap = %lld", who, (long long)st->n,
                (long long)st->n_cap);
  hipError_t e = d.esize == 2 ? decode_step_run<bf16>(d, W, w, *st, pos, x_t, y_t, ws, hs)
                              : decode_step_run<float>(d, W, w, *st, pos, x_t, y_t, ws, hs);
  if (e != hipSuccess) return hip_status(e, who);
  if (completes) {
    e = d.esize == 2 ? cache_append_run<bf16>(d, W, w, *st, pos, st->x_blk, 1, ws, hs)
                     : cache_append_run<float>(d, W, w, *st, pos, st->x_blk, 1, ws, hs);
    if (e != hipSuccess) return hip_status(e, who);
    st->n += 1;
    st->j = 0;
  } else {
    st->j += 1;
  }
  return PF_OK;
}

static int check_step_io(const DecodeDims& d, const void* x_t, void* y_t) {
  if (!x_t || !y_t) return fail(PF_ERR_INVALID_ARG, "x_t and y_t must be non-NULL");
  if (!aligned16(x_t) || !aligned16(y_t)) return fail(PF_ERR_INVALID_ARG, "x_t and y_t must be 16-byte aligned");
  if (overlaps(x_t, (size_t)d.B * d.d * d.esize, y_t, (size_t)d.B * d.d * d.esize))
    return fail(PF_ERR_INVALID_ARG, "y_t must not alias x_t");
  return PF_OK;
}

int proxy_decode_step(const pf_decode_config* cfg, const pf_decode_weights* w, pf_decode_state* st, const void* x_t,
                      void* y_t, void* workspace, size_t ws_bytes, void* stream) {
  DecodeDims d;
  int s = check_decode_common(cfg, w, st, &d, workspace, ws_bytes);
  if (s != PF_OK) return s;
  if ((s = check_step_io(d, x_t, y_t)) != PF_OK) return s;
  return decode_step_on(d, decode_ws(d), w, st, x_t, y_t, reinterpret_cast<char*>(workspace),
                        reinterpret_cast<hipStream_t>(stream), "proxy_decode_step");
}

// ---------------------------------------------------------------- decode step without allocation

// Scratch of proxy_decode_step_static: one array on every device the library
// runs on, held until the process ends. In host code `scratch` only names the
// array; its device address comes from hipGetSymbolAddress, looked up once per
// device (with that device current) on the first call there.
static constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
static constexpr int kMaxDevices = 64;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

static int static_scratch(void** out) {
  static std::mutex mu;
  static void* ptr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "proxy_decode_step_static: hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PF_ERR_UNSUPPORTED, "proxy_decode_step_static: device %d beyond the %d devices it tracks", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (!ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "proxy_decode_step_static: hipGetSymbolAddress(scratch)");
    ptr[dev] = p;
  }
  *out = ptr[dev];
  return PF_OK;
}

int proxy_decode_step_static(const pf_decode_config* cfg, const pf_decode_weights* w, pf_decode_state* st,
                             const void* x_t, void* y_t, void* stream) {
  DecodeDims d;
  int s = check_decode_common(cfg, w, st, &d, nullptr, 0, -1, false);
  if (s != PF_OK) return s;
  if ((s = check_step_io(d, x_t, y_t)) != PF_OK) return s;
  int64_t n_max = st->n;  // the slices cover the longest cache of the batch
  if (st->n_seq) {
    n_max = 0;
    for (int b = 0; b < d.B; ++b) n_max = std::max<int64_t>(n_max, st->n_seq[b]);
  }
  const DecodeWs W = decode_step_ws(d, n_max);
  if (W.bytes > kStaticScratchBytes)
    return fail(PF_ERR_UNSUPPORTED,
                "proxy_decode_step_static: this step needs %zu bytes of scratch, the static scratch holds %zu "
                "(use proxy_decode_step with a workspace)", W.bytes, kStaticScratchBytes);
  void* ptr = nullptr;
  if ((s = static_scratch(&ptr)) != PF_OK) return s;
  return decode_step_on(d, W, w, st, x_t, y_t, reinterpret_cast<char*>(ptr), reinterpret_cast<hipStream_t>(stream),
                        "proxy_decode_step_static");
}

size_t proxy_prefill_workspace_size(const pf_decode_config* cfg, int64_t n_tokens, int64_t n_cap) {
  DecodeDims d;
  const char* why;
  if (decode_dims(cfg, &d, &why) != PF_OK) return 0;
  if (prefill_limits(d, n_tokens, n_cap)) return 0;
  return prefill_ws(d, n_tokens, n_cap).bytes;
}

int proxy_decode_prefill(const pf_decode_config* cfg, const pf_decode_weights* w, pf_decode_state* st, const void* x,
                         int64_t n_tokens, void* y, void* workspace, size_t ws_bytes, void* stream) {
  if (n_tokens < 0) return fail(PF_ERR_INVALID_ARG, "n_tokens must be >= 0");
  DecodeDims d;
  int s = check_decode_common(cfg, w, st, &d, workspace, ws_bytes, n_tokens);
  if (s != PF_OK) return s;
  if (st->n_seq) return fail(PF_ERR_UNSUPPORTED, "prefill needs lockstep positions (n_seq = j_seq = NULL)");
  if (st->j != 0) return fail(PF_ERR_UNSUPPORTED, "prefill starts at a block boundary (j = 0), got j = %d", st->j);
  if (n_tokens == 0) return PF_OK;
  if (!x || !y) return fail(PF_ERR_INVALID_ARG, "x and y must be non-NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(PF_ERR_INVALID_ARG, "x and y must be 16-byte aligned");
  const size_t bytes = (size_t)d.B * n_tokens * d.d * d.esize;
  if (overlaps(x, bytes, y, bytes)) return fail(PF_ERR_INVALID_ARG, "y must not alias x");
  const int64_t nblk = n_tokens / d.P;
  if (st->n + nblk > st->n_cap)
    return fail(PF_ERR_CAPACITY, "prefill of %lld blocks overflows the cache (n = %lld, n_cap = %lld)",
                (long long)nblk, (long long)st->n, (long long)st->n_cap);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);
  hipError_t e = d.esize == 2 ? prefill_run<bf16>(d, w, *st, x, n_tokens, y, ws, hs)
                              : prefill_run<float>(d, w, *st, x, n_tokens, y, ws, hs);
  if (e != hipSuccess) return hip_status(e, "proxy_decode_prefill launch");
  st->n += nblk;
  st->j = (int32_t)(n_tokens - nblk * d.P);
  return PF_OK;
}

int proxy_cache_append(const pf_decode_config* cfg, const pf_decode_weights* w, pf_decode_state* st,
                       const void* x_blocks, int64_t nblk, void* workspace, size_t ws_bytes, void* stream) {
  DecodeDims d;
  int s = check_decode_common(cfg, w, st, &d, workspace, ws_bytes);
  if (s != PF_OK) return s;
  if (nblk < 0) return fail(PF_ERR_INVALID_ARG, "nblk must be >= 0");
  if (nblk == 0) return PF_OK;
  if (!x_blocks) return fail(PF_ERR_INVALID_ARG, "x_blocks is NULL");
  if (!aligned16(x_blocks)) return fail(PF_ERR_INVALID_ARG, "x_blocks must be 16-byte aligned");
  DecodePos pos{};
  if (st->n_seq) {
    pos.ragged = 1;
    for (int b = 0; b < d.B; ++b) {
      if (st->n_seq[b] + nblk > st->n_cap)
        return fail(PF_ERR_CAPACITY, "append of %lld blocks overflows the cache of sequence %d (n = %lld, n_cap = %lld)",
                    (long long)nblk, b, (long long)st->n_seq[b], (long long)st->n_cap);
      pos.n[b] = (int32_t)st->n_seq[b];
      pos.write |= (uint64_t)1 << b;
    }
  } else if (st->n + nblk > st->n_cap) {
    return fail(PF_ERR_CAPACITY, "append of %lld blocks overflows the cache (n = %lld, n_cap = %lld)",
                (long long)nblk, (long long)st->n, (long long)st->n_cap);
  }
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  char* ws = reinterpret_cast<char*>(workspace);
  const DecodeWs W = decode_ws(d);
  hipError_t e = d.esize == 2 ? cache_append_run<bf16>(d, W, w, *st, pos, x_blocks, nblk, ws, hs)
                              : cache_append_run<float>(d, W, w, *st, pos, x_blocks, nblk, ws, hs);
  if (e != hipSuccess) return hip_status(e, "proxy_cache_append launch");
  if (st->n_seq) {
    for (int b = 0; b < d.B; ++b) st->n_seq[b] += nblk;
  } else {
    st->n += nblk;
  }
  return PF_OK;
}

}  // extern "C"
