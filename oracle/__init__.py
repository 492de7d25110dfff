"""CPU oracle for the ProxyFormer hot path: test infrastructure only.

This package is a plain, slow, fp64 restatement of what the paper defines:
the single-layer forward of Algorithm 1 with the reshape-linear compression
of Eq. 7, the residual proxy update of Eq. 8, causal multi-head proxy
attention (Eq. 9), reshape-linear decompression (Eq. 10) with the
factorised cascade of Eq. 15-17, gated injection (Eq. 12), the chain-rule
backward of all of it, and the proxy-KV-cache decode step with its
block-triggered append (Eq. 19-21, Sec. 3.8).

It exists to check the HIP path. Only the test suite, the smoke entry
point and the benchmark's CPU-baseline leg may import it; the product path
never calls it and shares no code with it. Matrix products and
exponentials use numpy in float64; nothing is blocked, fused or reordered
beyond processing independent rows in chunks.

Every function states the passage it follows. Readings of points the paper
leaves open are listed in the module docstrings where they apply.
"""
from .layer import (  # noqa: F401
    TOKEN_CAUSAL, BLOCK_CAUSAL, BIDIRECTIONAL, INJECT_GATED, INJECT_ADD, INJECT_AFFINE, INJECT_GATED_HEAD, rms_normalise, head_of_channel,
    sigmoid, compress, layer_forward, layer_backward, attention_rows,
    proxies_and_attention_inputs, patch_order, layer_forward_2d, layer_backward_2d,
)
from .decode import DecodeState, decode_step, cache_append, prefill, rms_norm  # noqa: F401
from .metrics import max_rel_err  # noqa: F401
