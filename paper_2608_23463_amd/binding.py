"""ctypes binding of libproxyformer.so (the C ABI in include/proxyformer.h).

Argument marshalling only: PyTorch provides device memory (tensor.data_ptr())
and the stream; every step of the computation runs in the library's HIP
kernels. Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libproxyformer.so")
MAX_LEVELS = 4

PF_OK = 0
PF_ERR_INVALID_ARG = -1
PF_ERR_UNSUPPORTED = -2
PF_ERR_CAPACITY = -3
PF_ERR_WORKSPACE = -4
PF_ERR_HIP = -5
PF_FP32 = 0
PF_BF16 = 1
PF_INJECT_GATED = 0
PF_INJECT_ADD = 1
PF_INJECT_AFFINE = 2
PF_INJECT_GATED_HEAD = 3
PF_PRECISION_EXTENDED = 0
PF_PRECISION_BF16 = 1
PF_GATE_SEPARATE = 0
PF_GATE_FUSED = 1

EXPORTS = (
    "proxy_layer_workspace_size", "proxy_layer_saved_size", "proxy_layer_forward",
    "proxy_layer_backward", "proxy_decode_workspace_size", "proxy_decode_step",
    "proxy_cache_append", "proxy_prefill_workspace_size", "proxy_decode_prefill",
    "proxy_last_error", "proxy_version",
    "proxy_trace_enable", "proxy_trace_collect", "proxy_trace_get", "proxy_trace_reset",
    "proxy_ceiling_mfma", "proxy_decode_step_static", "proxy_ceiling_read",
)

c_void_p = ctypes.c_void_p
c_int32 = ctypes.c_int32
c_int64 = ctypes.c_int64
c_size_t = ctypes.c_size_t


class PfLinear(ctypes.Structure):
    _fields_ = [("w", c_void_p), ("b", c_void_p)]


class PfLayerConfig(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("seq_len", c_int64), ("d_fine", c_int32), ("d_proxy", c_int32),
                ("n_heads", c_int32), ("head_dim", c_int32), ("n_levels", c_int32),
                ("factors", c_int32 * MAX_LEVELS), ("level_dims", c_int32 * MAX_LEVELS),
                ("dtype", c_int32), ("mask", c_int32), ("injection", c_int32), ("image_width", c_int32),
                ("precision", c_int32), ("gate_fusion", c_int32)]


class PfLayerWeights(ctypes.Structure):
    _fields_ = [("compress", PfLinear * MAX_LEVELS), ("q", PfLinear), ("k", PfLinear), ("v", PfLinear),
                ("o", PfLinear), ("decompress", PfLinear * MAX_LEVELS), ("gate", PfLinear), ("affine", PfLinear)]


class PfLinearGrad(ctypes.Structure):
    _fields_ = [("dw", c_void_p), ("db", c_void_p)]


class PfLayerGrads(ctypes.Structure):
    _fields_ = [("compress", PfLinearGrad * MAX_LEVELS), ("q", PfLinearGrad), ("k", PfLinearGrad),
                ("v", PfLinearGrad), ("o", PfLinearGrad), ("decompress", PfLinearGrad * MAX_LEVELS),
                ("gate", PfLinearGrad), ("affine", PfLinearGrad)]


class PfDecodeConfig(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("d_model", c_int32), ("n_heads", c_int32), ("head_dim", c_int32),
                ("n_levels", c_int32), ("factors", c_int32 * MAX_LEVELS),
                ("level_dims", c_int32 * MAX_LEVELS), ("dtype", c_int32), ("rms_eps", ctypes.c_float)]


class PfDecodeWeights(ctypes.Structure):
    _fields_ = [("rms_gamma", c_void_p), ("q", PfLinear), ("k", PfLinear), ("v", PfLinear), ("o", PfLinear),
                ("alpha", PfLinear), ("compress", PfLinear * MAX_LEVELS), ("k_proxy", PfLinear),
                ("v_proxy", PfLinear)]


class PfDecodeState(ctypes.Structure):
    _fields_ = [("k_cache", c_void_p), ("v_cache", c_void_p), ("n_cap", c_int64), ("n", c_int64),
                ("x_blk", c_void_p), ("k_loc", c_void_p), ("v_loc", c_void_p), ("j", c_int32),
                ("n_seq", ctypes.POINTER(c_int64)), ("j_seq", ctypes.POINTER(c_int32))]


_lib = None

# Allocation policy of the helpers below (a test aid): when on, every buffer
# they allocate for the library to write (outputs, gradients, saved
# activations, workspace, decode state slots) starts as all-ones bytes, a NaN
# in both bf16 and fp32, and the decode and prefill workspaces are refilled
# before every call. An element the library fails to write then cannot pass
# a comparison on stale memory that happens to hold a correct value.
_poison = False


def set_poison(on: bool) -> bool:
    """Turn NaN-filled allocation on or off; returns the previous setting."""
    global _poison
    prev, _poison = _poison, bool(on)
    return prev


def _fresh(t):
    """Apply the allocation policy to a new (contiguous) buffer; returns it."""
    if _poison:
        import torch
        t.view(torch.uint8).fill_(255)
    return t


def _fresh_on(t, stream):
    """_fresh with the fill enqueued on `stream` (the stream the library call
    that reads the buffer runs on; None = the current stream)."""
    if _poison and stream is not None:
        import torch
        with torch.cuda.stream(stream):
            return _fresh(t)
    return _fresh(t)


def _empty(shape, dtype, device):
    import torch
    return _fresh(torch.empty(shape, dtype=dtype, device=device))


class ProxyFormerError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2608_23463_amd.build.build()")
    # torch first: the library then binds to the HIP runtime torch has loaded
    # (its buffers and streams are torch's). Loaded before torch, the library
    # would map the system runtime and torch its own, two runtimes in one
    # process, and the library's launches fail.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.proxy_layer_workspace_size.argtypes = [P(PfLayerConfig), c_int32]
    lib.proxy_layer_workspace_size.restype = c_size_t
    lib.proxy_layer_saved_size.argtypes = [P(PfLayerConfig)]
    lib.proxy_layer_saved_size.restype = c_size_t
    lib.proxy_layer_forward.argtypes = [P(PfLayerConfig), P(PfLayerWeights), c_void_p, c_void_p, c_void_p,
                                        c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.proxy_layer_forward.restype = c_int32
    lib.proxy_layer_backward.argtypes = [P(PfLayerConfig), P(PfLayerWeights), c_void_p, c_void_p, c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_void_p, P(PfLayerGrads), c_void_p,
                                         c_size_t, c_void_p]
    lib.proxy_layer_backward.restype = c_int32
    lib.proxy_decode_workspace_size.argtypes = [P(PfDecodeConfig)]
    lib.proxy_decode_workspace_size.restype = c_size_t
    lib.proxy_decode_step.argtypes = [P(PfDecodeConfig), P(PfDecodeWeights), P(PfDecodeState), c_void_p,
                                      c_void_p, c_void_p, c_size_t, c_void_p]
    lib.proxy_decode_step.restype = c_int32
    lib.proxy_cache_append.argtypes = [P(PfDecodeConfig), P(PfDecodeWeights), P(PfDecodeState), c_void_p,
                                       c_int64, c_void_p, c_size_t, c_void_p]
    lib.proxy_cache_append.restype = c_int32
    lib.proxy_prefill_workspace_size.argtypes = [P(PfDecodeConfig), c_int64, c_int64]
    lib.proxy_prefill_workspace_size.restype = c_size_t
    lib.proxy_decode_prefill.argtypes = [P(PfDecodeConfig), P(PfDecodeWeights), P(PfDecodeState), c_void_p,
                                         c_int64, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.proxy_decode_prefill.restype = c_int32
    lib.proxy_last_error.argtypes = []
    lib.proxy_last_error.restype = ctypes.c_char_p
    lib.proxy_version.argtypes = []
    lib.proxy_version.restype = c_int32
    lib.proxy_trace_enable.argtypes = [c_int32]
    lib.proxy_trace_enable.restype = c_int32
    lib.proxy_trace_collect.argtypes = []
    lib.proxy_trace_collect.restype = c_int32
    lib.proxy_trace_get.argtypes = [c_int32, ctypes.c_char_p, c_size_t, ctypes.POINTER(c_int64),
                                    ctypes.POINTER(ctypes.c_double)]
    lib.proxy_trace_get.restype = c_int32
    lib.proxy_trace_reset.argtypes = []
    lib.proxy_trace_reset.restype = None
    lib.proxy_ceiling_mfma.argtypes = [c_void_p, c_int64, c_int32, c_void_p]
    lib.proxy_ceiling_mfma.restype = c_int32
    lib.proxy_ceiling_read.argtypes = [c_void_p, ctypes.c_size_t, c_void_p, c_int64, c_void_p]
    lib.proxy_ceiling_read.restype = c_int32
    lib.proxy_decode_step_static.argtypes = [P(PfDecodeConfig), P(PfDecodeWeights), P(PfDecodeState), c_void_p,
                                             c_void_p, c_void_p]
    lib.proxy_decode_step_static.restype = c_int32
    _lib = lib
    return lib


def last_error() -> str:
    return load().proxy_last_error().decode()


def _check(status: int):
    if status != PF_OK:
        raise ProxyFormerError(status, last_error())


def ceiling_mfma(out, n_workgroups: int, iters: int, stream=None) -> None:
    """Enqueue the matrix-core ceiling loop (see proxy_ceiling_mfma) on
    `stream` (torch's current stream if None); out is a device float32
    tensor of n_workgroups * 256 elements."""
    if out.numel() < n_workgroups * 256 or out.dtype.itemsize != 4 or not out.is_cuda:
        raise ValueError("out must be a device float32 tensor of n_workgroups * 256 elements")
    _check(load().proxy_ceiling_mfma(c_void_p(out.data_ptr()), n_workgroups, iters, c_void_p(_stream(stream))))


def ceiling_read(src, out, n_workgroups: int, stream=None) -> None:
    """Enqueue the HBM read probe (see proxy_ceiling_read) over all bytes of
    the device tensor src on `stream` (torch's current stream if None); out is
    a device int32 tensor of at least n_workgroups elements."""
    if not src.is_cuda or not src.is_contiguous() or (src.numel() * src.element_size()) % 16 != 0:
        raise ValueError("src must be a contiguous device tensor whose size is a multiple of 16 bytes")
    if out.numel() < n_workgroups or out.element_size() != 4 or not out.is_cuda:
        raise ValueError("out must be a device 32-bit tensor of n_workgroups elements")
    _check(load().proxy_ceiling_read(c_void_p(src.data_ptr()), src.numel() * src.element_size(),
                                     c_void_p(out.data_ptr()), n_workgroups, c_void_p(_stream(stream))))


def trace_enable(on: bool) -> bool:
    return bool(load().proxy_trace_enable(int(on)))


def trace_reset() -> None:
    load().proxy_trace_reset()


def trace_collect() -> Dict[str, tuple]:
    """{label: (launches, total_ms)} of everything traced since the last reset."""
    lib = load()
    n = lib.proxy_trace_collect()
    if n < 0:
        raise ProxyFormerError(n, "trace collection failed")
    out = {}
    buf = ctypes.create_string_buffer(128)
    for i in range(n):
        cnt = c_int64()
        ms = ctypes.c_double()
        _check(lib.proxy_trace_get(i, buf, 128, ctypes.byref(cnt), ctypes.byref(ms)))
        out[buf.value.decode()] = (int(cnt.value), float(ms.value))
    return out


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# ---------------------------------------------------------------- layer

def layer_config(batch: int, seq_len: int, d_fine: int, d_proxy: int, n_heads: int, head_dim: int,
                 factors: Sequence[int], level_dims: Sequence[int] = (), dtype: str = "bf16",
                 mask: int = 0, injection: int = 0, image_width: int = 0, precision: int = 0,
                 gate_fusion: int = 0) -> PfLayerConfig:
    c = PfLayerConfig()
    c.batch = batch
    c.seq_len = seq_len
    c.d_fine = d_fine
    c.d_proxy = d_proxy
    c.n_heads = n_heads
    c.head_dim = head_dim
    c.n_levels = len(factors)
    for i, k in enumerate(factors):
        c.factors[i] = k
    for i, v in enumerate(level_dims):
        c.level_dims[i] = v
    c.dtype = PF_BF16 if dtype == "bf16" else PF_FP32
    c.mask = mask
    c.injection = injection
    c.image_width = image_width
    c.precision = precision
    c.gate_fusion = gate_fusion
    return c


def config_from_shape(shape) -> PfLayerConfig:
    """PfLayerConfig of a synth.LayerShape."""
    dims = list(shape.level_dims) if shape.level_dims else []
    return layer_config(shape.batch, shape.seq_len, shape.d_fine, shape.d_proxy, shape.n_heads,
                        shape.head_dim, shape.factors, dims, shape.dtype, shape.mask,
                        getattr(shape, "injection", 0), getattr(shape, "image_width", 0),
                        getattr(shape, "precision", 0), getattr(shape, "gate_fusion", 0))


def _lin(pair) -> PfLinear:
    if pair is None:
        return PfLinear(None, None)
    w, b = pair
    return PfLinear(_ptr(w), _ptr(b))


def layer_weights(w: Dict[str, object]) -> PfLayerWeights:
    """Weight struct from {"compress": [(W, b)...], "q": (W, b), ...} of device tensors."""
    s = PfLayerWeights()
    for i, pair in enumerate(w["compress"]):
        s.compress[i] = _lin(pair)
    for i, pair in enumerate(w["decompress"]):
        s.decompress[i] = _lin(pair)
    for name in ("q", "k", "v", "o", "gate", "affine"):
        setattr(s, name, _lin(w.get(name)))
    return s


def layer_workspace_size(cfg: PfLayerConfig, for_backward: bool = False) -> int:
    return int(load().proxy_layer_workspace_size(ctypes.byref(cfg), int(for_backward)))


def layer_saved_size(cfg: PfLayerConfig) -> int:
    return int(load().proxy_layer_saved_size(ctypes.byref(cfg)))


def _bytes(n: int, device):
    import torch
    return _fresh(torch.empty(max(n, 256), dtype=torch.uint8, device=device))


def layer_forward_raw(cfg, wstruct, x, h_in, x_out, h_out, saved, workspace, stream=None):
    """Direct call of proxy_layer_forward on preallocated tensors."""
    ws_bytes = workspace.numel() if workspace is not None else 0
    _check(load().proxy_layer_forward(ctypes.byref(cfg), ctypes.byref(wstruct), _ptr(x), _ptr(h_in),
                                      _ptr(x_out), _ptr(h_out), _ptr(saved), _ptr(workspace), ws_bytes,
                                      _stream(stream)))


def layer_forward(cfg: PfLayerConfig, weights: Dict[str, object], x, h_in=None, save: bool = False,
                  workspace=None, stream=None):
    """Allocate outputs (and workspace), run the forward; returns (x_out, h_out, saved)."""
    import torch
    m = -(-cfg.seq_len // _block(cfg))  # ceil(L / P): a partial last block has a proxy
    x_out = _empty(x.shape, x.dtype, x.device)
    h_out = _empty((cfg.batch, m, cfg.d_proxy), x.dtype, x.device)
    saved = _bytes(layer_saved_size(cfg), x.device) if save else None
    if workspace is None:
        workspace = _bytes(layer_workspace_size(cfg, False), x.device)
    layer_forward_raw(cfg, layer_weights(weights), x, h_in, x_out, h_out, saved, workspace, stream)
    return x_out, h_out, saved


def _block(cfg) -> int:
    p = 1
    for i in range(cfg.n_levels):
        p *= cfg.factors[i]
    return p


def layer_grads(g: Dict[str, object]) -> PfLayerGrads:
    s = PfLayerGrads()

    def lg(pair):
        if pair is None:
            return PfLinearGrad(None, None)
        dw, db = pair
        return PfLinearGrad(_ptr(dw), _ptr(db))

    for i, pair in enumerate(g["compress"]):
        s.compress[i] = lg(pair)
    for i, pair in enumerate(g["decompress"]):
        s.decompress[i] = lg(pair)
    for name in ("q", "k", "v", "o", "gate", "affine"):
        setattr(s, name, lg(g.get(name)))
    return s


def layer_backward(cfg: PfLayerConfig, weights: Dict[str, object], x, h_in, saved, dy, dh_out=None,
                   workspace=None, stream=None):
    """Run the backward; returns (dx, dh_in, grads) with fp32 weight gradients."""
    import torch
    dev = x.device
    dx = _empty(x.shape, x.dtype, dev)
    dh_in = _empty(h_in.shape, h_in.dtype, dev) if h_in is not None else None

    def g_like(pair):
        w, b = pair
        return (_empty(w.shape, torch.float32, dev), _empty((w.shape[0],), torch.float32, dev))

    grads = {"compress": [g_like(p) for p in weights["compress"]],
             "decompress": [g_like(p) for p in weights["decompress"]]}
    for name in ("q", "k", "v", "o"):
        grads[name] = g_like(weights[name])
    # the gate is only read (and differentiated) by gated injection
    grads["gate"] = g_like(weights["gate"]) if cfg.injection in (PF_INJECT_GATED, PF_INJECT_GATED_HEAD) else None
    grads["affine"] = g_like(weights["affine"]) if cfg.injection == PF_INJECT_AFFINE else None
    if workspace is None:
        workspace = _bytes(layer_workspace_size(cfg, True), dev)
    _check(load().proxy_layer_backward(ctypes.byref(cfg), ctypes.byref(layer_weights(weights)), _ptr(x),
                                       _ptr(h_in), _ptr(saved), _ptr(dy), _ptr(dh_out), _ptr(dx), _ptr(dh_in),
                                       ctypes.byref(layer_grads(grads)), _ptr(workspace), workspace.numel(),
                                       _stream(stream)))
    return dx, dh_in, grads


# ---------------------------------------------------------------- decode

def decode_config(batch: int, d_model: int, n_heads: int, head_dim: int, factors: Sequence[int],
                  level_dims: Sequence[int] = (), dtype: str = "bf16", rms_eps: float = 1e-6) -> PfDecodeConfig:
    c = PfDecodeConfig()
    c.batch = batch
    c.d_model = d_model
    c.n_heads = n_heads
    c.head_dim = head_dim
    c.n_levels = len(factors)
    for i, k in enumerate(factors):
        c.factors[i] = k
    for i, v in enumerate(level_dims):
        c.level_dims[i] = v
    c.dtype = PF_BF16 if dtype == "bf16" else PF_FP32
    c.rms_eps = rms_eps
    return c


def decode_weights(w: Dict[str, object]) -> PfDecodeWeights:
    s = PfDecodeWeights()
    s.rms_gamma = _ptr(w["rms_gamma"])
    for name in ("q", "k", "v", "o", "alpha", "k_proxy", "v_proxy"):
        setattr(s, name, _lin(w[name]))
    for i, pair in enumerate(w["compress"]):
        s.compress[i] = _lin(pair)
    return s


class DecodeSession:
    """Caller-owned decode state on the device plus the host counters n, j.

    With ``ragged=True`` every sequence keeps its own position: ``n_seq`` and
    ``j_seq`` (host int64 / int32 arrays of batch entries) replace n and j."""

    def __init__(self, cfg: PfDecodeConfig, weights: Dict[str, object], k_cache, v_cache, n: int = 0,
                 device="cuda", ragged: bool = False, n_seq=None, j_seq=None):
        import torch
        self.cfg = cfg
        self.weights = weights            # keeps the device tensors alive
        self.wstruct = decode_weights(weights)
        p = _block(cfg)
        dt = k_cache.dtype
        self.k_cache = k_cache
        self.v_cache = v_cache
        # slots at or past j are never read: they start as NaN under poisoning
        self.x_blk = _fresh(torch.zeros((cfg.batch, p, cfg.d_model), dtype=dt, device=device))
        self.k_loc = _fresh(torch.zeros((cfg.batch, cfg.n_heads, p, cfg.head_dim), dtype=dt, device=device))
        self.v_loc = _fresh(torch.zeros_like(self.k_loc))
        self.state = PfDecodeState(k_cache.data_ptr(), v_cache.data_ptr(), k_cache.shape[2], n,
                                   self.x_blk.data_ptr(), self.k_loc.data_ptr(), self.v_loc.data_ptr(), 0)
        self.n_seq = self.j_seq = None
        if ragged:
            import numpy as np
            # own copies: the library advances these counters in place
            self.n_seq = np.array(np.full(cfg.batch, n) if n_seq is None else n_seq, dtype=np.int64, copy=True)
            self.j_seq = np.array(np.zeros(cfg.batch) if j_seq is None else j_seq, dtype=np.int32, copy=True)
            self.state.n_seq = self.n_seq.ctypes.data_as(ctypes.POINTER(c_int64))
            self.state.j_seq = self.j_seq.ctypes.data_as(ctypes.POINTER(c_int32))
        self.workspace = _bytes(int(load().proxy_decode_workspace_size(ctypes.byref(cfg))), device)

    @property
    def n(self) -> int:
        return int(self.state.n)

    @property
    def j(self) -> int:
        return int(self.state.j)

    def step(self, x_t, y_t=None, stream=None):
        if y_t is None:
            y_t = _empty(x_t.shape, x_t.dtype, x_t.device)
        _fresh_on(self.workspace, stream)
        _check(load().proxy_decode_step(ctypes.byref(self.cfg), ctypes.byref(self.wstruct),
                                        ctypes.byref(self.state), _ptr(x_t), _ptr(y_t),
                                        _ptr(self.workspace), self.workspace.numel(), _stream(stream)))
        return y_t

    def step_static(self, x_t, y_t=None, stream=None):
        """The same step through proxy_decode_step_static (no workspace)."""
        if y_t is None:
            y_t = _empty(x_t.shape, x_t.dtype, x_t.device)
        _check(load().proxy_decode_step_static(ctypes.byref(self.cfg), ctypes.byref(self.wstruct),
                                               ctypes.byref(self.state), _ptr(x_t), _ptr(y_t), _stream(stream)))
        return y_t

    def prefill(self, x, y=None, stream=None):
        """Parallel form of the generation block over x [B, T, d] (the next T
        tokens of every sequence, from a block boundary); returns y [B, T, d].
        The prefill workspace is allocated on first use and grown as needed."""
        if y is None:
            y = _empty(x.shape, x.dtype, x.device)
        lib = load()
        need = int(lib.proxy_prefill_workspace_size(ctypes.byref(self.cfg), x.shape[1], self.state.n_cap))
        if need == 0:
            raise ProxyFormerError(-2, "prefill sizes beyond the library's limits")
        if getattr(self, "prefill_ws", None) is None or self.prefill_ws.numel() < need:
            self.prefill_ws = _bytes(need, x.device)
        _fresh_on(self.prefill_ws, stream)
        _check(lib.proxy_decode_prefill(ctypes.byref(self.cfg), ctypes.byref(self.wstruct), ctypes.byref(self.state),
                                        _ptr(x), x.shape[1], _ptr(y), _ptr(self.prefill_ws),
                                        self.prefill_ws.numel(), _stream(stream)))
        return y

    def append(self, x_blocks, nblk: int, stream=None):
        _fresh_on(self.workspace, stream)
        _check(load().proxy_cache_append(ctypes.byref(self.cfg), ctypes.byref(self.wstruct),
                                         ctypes.byref(self.state), _ptr(x_blocks), nblk,
                                         _ptr(self.workspace), self.workspace.numel(), _stream(stream)))
