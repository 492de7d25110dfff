"""Seeded synthetic inputs for the ProxyFormer layer and decode path.

This module only draws random numbers and names workload shapes. It holds
none of the method's arithmetic, so both the HIP path (through the Python
binding) and the CPU oracle can consume the same materialised arrays.

Distributions follow the workloads the paper trains and measures on
(Sec. 5.1, Table 2): local-stream activations and upstream gradients are
standard normal, every weight matrix is N(0, 0.02^2), biases are zero and
are not drawn. A bf16 workload rounds every fp32 sample to the nearest
bf16 value (round-to-nearest-even on the bit pattern) so that the device
tensor and the oracle's fp64 copy hold exactly the same numbers.

Draw order for a layer workload (one ``numpy.random.Generator(PCG64(seed))``):
X, then the weights in the order of the C-ABI weight struct (compression
levels 1..M, q, k, v, o, decompression levels 1..M, gate), then dY.
Draw order for a decode workload: the new-token stream x[steps, B, d], then
q, k, v, o, alpha, compression levels 1..M, k_proxy, v_proxy, then the
K cache and the V cache.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

TOKEN_CAUSAL = 0
BLOCK_CAUSAL = 1
BIDIRECTIONAL = 2

INJECT_GATED = 0  # Eq. 12
INJECT_ADD = 1    # Eq. 11
INJECT_AFFINE = 2  # Eq. 13
INJECT_GATED_HEAD = 3  # Eq. 12 with one gate per head (Eq. 20's per-head weighting)

# arithmetic of the GPU's proxy path in bf16 mode (pf_precision of the C ABI);
# not an input property, carried here so a shape names one complete call
PRECISION_EXTENDED = 0
PRECISION_BF16 = 1
# kernels of the level-1 decompression and the gated injection (pf_gate_fusion):
# also a property of the call, not of the inputs
GATE_SEPARATE = 0
GATE_FUSED = 1

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """Shape of one ProxyFormer layer call (Algorithm 1 inputs)."""

    batch: int
    seq_len: int
    d_fine: int
    d_proxy: int
    n_heads: int
    head_dim: int
    factors: Tuple[int, ...]          # k_1..k_M, product = P (Eq. 15)
    level_dims: Tuple[int, ...] = ()  # d_1..d_{M-1}; missing or 0 -> d_proxy
    dtype: str = "bf16"               # "bf16" or "fp32"
    mask: int = TOKEN_CAUSAL
    injection: int = INJECT_GATED
    image_width: int = 0              # > 0: raster-order image, blocks are p x p patches (Sec. 3.9)
    precision: int = PRECISION_EXTENDED
    gate_fusion: int = GATE_SEPARATE

    @property
    def block(self) -> int:
        p = 1
        for k in self.factors:
            p *= k
        return p

    @property
    def n_proxies(self) -> int:
        # m = ceil(L / P) (Sec. 3.1): a partial last block still has a proxy
        return -(-self.seq_len // self.block)

    def dims(self) -> List[int]:
        """d_0..d_M: d_0 = d_fine, d_j = level_dims[j-1] (0 or absent -> d_proxy), d_M = d_proxy."""
        m = len(self.factors)
        lv = [self.d_proxy] * m
        for j, v in enumerate(self.level_dims[:m - 1]):
            if v:
                lv[j] = v
        return [self.d_fine] + lv

    def weight_shapes(self) -> Dict[str, object]:
        d = self.dims()
        m = len(self.factors)
        comp = [(d[j + 1], self.factors[j] * d[j]) for j in range(m)]
        dec = [(self.factors[j] * d[j], d[j + 1]) for j in range(m)]
        dp = self.d_proxy
        return {
            "compress": comp,
            "q": (dp, dp), "k": (dp, dp), "v": (dp, dp), "o": (dp, dp),
            "decompress": dec,
            "gate": (self.n_heads if self.injection == INJECT_GATED_HEAD else self.d_fine, 2 * self.d_fine),
        }


@dataclasses.dataclass(frozen=True)
class DecodeShape:
    """Shape of the proxy-KV-cache decode workload (Eq. 19-21, Sec. 3.8)."""

    batch: int
    d_model: int
    n_heads: int
    head_dim: int
    factors: Tuple[int, ...]
    level_dims: Tuple[int, ...] = ()
    n0: int = 0          # cached proxy rows at the start
    steps: int = 1       # new tokens decoded per sequence
    n_cap: int = 0       # cache capacity in rows (0 -> n0 + steps // P + 1)
    dtype: str = "bf16"
    rms_eps: float = 1e-6

    @property
    def block(self) -> int:
        p = 1
        for k in self.factors:
            p *= k
        return p

    @property
    def capacity(self) -> int:
        return self.n_cap if self.n_cap else self.n0 + self.steps // self.block + 1

    def dims(self) -> List[int]:
        """d_0..d_M with d_0 = d_M = d_model and d_j = level_dims[j-1] in between."""
        m = len(self.factors)
        lv = [self.d_model] * m
        for j, v in enumerate(self.level_dims[:m - 1]):
            if v:
                lv[j] = v
        return [self.d_model] + lv


# The workloads: a small fp32 correctness layer, two bf16 layers at 64K and
# 1M tokens, a factorised forward+backward layer, the decode run, the
# language-model shape (layer and decode) and a chunked prefill.
WORKLOADS = {
    "layer_fp32_L4k_d256": LayerShape(1, 4096, 256, 256, 4, 64, (64,), dtype="fp32"),
    "layer_bf16_L64k_d1024": LayerShape(1, 65536, 1024, 1024, 16, 64, (64,)),
    "layer_bf16_L1M_d1024": LayerShape(1, 1 << 20, 1024, 1024, 16, 64, (64,)),
    "layer_bf16_L256k_d2048_f8x8": LayerShape(1, 1 << 18, 2048, 2048, 16, 128, (8, 8)),
    "decode_bf16_B32_n16k": DecodeShape(32, 1024, 16, 64, (64,), n0=16384, steps=256),
    # The paper's language-model shape (Sec. 3.2, Sec. 5.1): a 64-wide history
    # stream compressed into a 512-wide proxy stream (8 heads x 64, P = 64),
    # and the generation side decoding 512-wide tokens against that cache.
    "layer_bf16_L1M_lm_df64_dp512": LayerShape(1, 1 << 20, 64, 512, 8, 64, (64,)),
    "decode_bf16_B32_n16k_lm_d512": DecodeShape(32, 512, 8, 64, (64,), n0=16384, steps=256),
    # Chunked prefill (parallel form of the generation block, Eq. 19-20): the
    # next 4,096 tokens of 32 sequences against a 16,384-proxy cache, the
    # chunk's 64 blocks per sequence appended (Eq. 21). `steps` is the chunk.
    "prefill_bf16_B32_T4096_n16k": DecodeShape(32, 1024, 16, 64, (64,), n0=16384, steps=4096),
}
WORKLOAD_SEEDS = {name: 20260000 + i + 1 for i, name in enumerate(WORKLOADS)}


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 samples to the nearest bf16 value (ties to even).

    Returns float32 whose low 16 mantissa bits are zero.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty_like(a)
    flat_in = a.reshape(-1)
    flat_out = out.reshape(-1)
    step = 1 << 24
    for s in range(0, flat_in.size, step):
        b = flat_in[s:s + step].view(np.uint32).astype(np.uint64)
        b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
        flat_out[s:s + step] = b.astype(np.uint32).view(np.float32)
    return out


def _normal(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if dtype == "bf16":
        x = bf16_round(x)
    return x


def layer_inputs(shape: LayerShape, seed: int, with_dy: bool = False,
                 with_h_in: bool = False) -> Dict[str, object]:
    """Draw X, the layer weights (and optionally dY, H_in) for one layer call."""
    rng = np.random.Generator(np.random.PCG64(seed))
    dt = shape.dtype
    out: Dict[str, object] = {}
    out["x"] = _normal(rng, (shape.batch, shape.seq_len, shape.d_fine), 1.0, dt)
    ws = shape.weight_shapes()

    def lin(o, i):
        return (_normal(rng, (o, i), WEIGHT_STD, dt), np.zeros((o,), np.float32))

    w = {"compress": [lin(*s) for s in ws["compress"]]}
    for name in ("q", "k", "v", "o"):
        w[name] = lin(*ws[name])
    w["decompress"] = [lin(*s) for s in ws["decompress"]]
    w["gate"] = lin(*ws["gate"])
    if shape.injection == INJECT_AFFINE:   # [s | t] = Delta W_a^T + b_a (Eq. 13)
        w["affine"] = lin(2 * shape.d_fine, shape.d_fine)
    out["weights"] = w
    if with_dy:
        out["dy"] = _normal(rng, (shape.batch, shape.seq_len, shape.d_fine), 1.0, dt)
    if with_h_in:
        out["h_in"] = _normal(rng, (shape.batch, shape.n_proxies, shape.d_proxy), 1.0, dt)
    else:
        out["h_in"] = None
    return out


def decode_inputs(shape: DecodeShape, seed: int) -> Dict[str, object]:
    """Draw the new-token stream, the decode weights and the initial cache."""
    rng = np.random.Generator(np.random.PCG64(seed))
    dt = shape.dtype
    d = shape.d_model
    out: Dict[str, object] = {}
    out["x"] = _normal(rng, (shape.steps, shape.batch, d), 1.0, dt)

    def lin(o, i):
        return (_normal(rng, (o, i), WEIGHT_STD, dt), np.zeros((o,), np.float32))

    w: Dict[str, object] = {"rms_gamma": np.ones((d,), np.float32)}
    for name in ("q", "k", "v", "o"):
        w[name] = lin(d, d)
    w["alpha"] = lin(shape.n_heads, d)
    dims = shape.dims()
    w["compress"] = [lin(dims[j + 1], shape.factors[j] * dims[j])
                     for j in range(len(shape.factors))]
    w["k_proxy"] = lin(d, d)
    w["v_proxy"] = lin(d, d)
    out["weights"] = w
    cshape = (shape.batch, shape.n_heads, shape.capacity, shape.head_dim)
    kc = np.zeros(cshape, np.float32)
    vc = np.zeros(cshape, np.float32)
    n0 = shape.n0
    if n0:
        kc[:, :, :n0] = _normal(rng, (shape.batch, shape.n_heads, n0, shape.head_dim), 1.0, dt)
        vc[:, :, :n0] = _normal(rng, (shape.batch, shape.n_heads, n0, shape.head_dim), 1.0, dt)
    out["k_cache"] = kc
    out["v_cache"] = vc
    out["n0"] = n0
    return out
