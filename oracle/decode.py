"""Oracle for the proxy-KV-cache decode step and the block-triggered append.

Test infrastructure only (see the package docstring). Follows the
generation block of the language model (Eq. 19-20) decoding one token per
sequence against the frozen proxy cache of Eq. 21, with the streaming
update of Sec. 3.8: once P new tokens have been decoded the block is
compressed, appended to the cache as one new proxy row and its local
features are dropped.

Readings of points the paper leaves open:
* The block is pre-norm: u = RMSNorm(x) (eps = 1e-6, learnable gain gamma)
  feeds q, k, v and the gate alpha. MLP_alpha of Eq. 20 is one linear map
  d -> n_heads followed by a sigmoid (the same squashing as Eq. 12).
* A_x is causal self-attention over the tokens of the current block only
  (slots 0..j): older tokens are represented by their proxies.
* A_h is attention of the same q over the cached proxy rows 0..n-1, with
  no mask; with an empty cache A_h = 0.
* A = A_x + alpha_h * A_h per head, then y = x + A W_o^T + b_o.
* The append compresses the layer inputs x of the finished block with the
  layer's compression C (Eq. 7 / Eq. 16) and projects the new proxy with the
  proxy-attention K/V maps, so each cached row is exactly the K_p / V_p row
  Eq. 9 would use for that block.
"""
from __future__ import annotations

import dataclasses
from typing import Sequence

import numpy as np

from .layer import _f64, compress, linear, sigmoid


@dataclasses.dataclass
class DecodeState:
    """Whole inference state of one layer (batch in lockstep).

    k_cache, v_cache: [B, n_heads, n_cap, d_head]; n cached rows are valid.
    x_blk: [B, P, d] inputs of the current block; k_loc, v_loc:
    [B, n_heads, P, d_head] its keys and values; j tokens are filled.
    """

    k_cache: np.ndarray
    v_cache: np.ndarray
    n: int
    x_blk: np.ndarray
    k_loc: np.ndarray
    v_loc: np.ndarray
    j: int

    @classmethod
    def empty(cls, batch, n_heads, head_dim, p_blk, n_cap, d):
        z = np.zeros
        return cls(z((batch, n_heads, n_cap, head_dim)), z((batch, n_heads, n_cap, head_dim)), 0,
                   z((batch, p_blk, d)), z((batch, n_heads, p_blk, head_dim)),
                   z((batch, n_heads, p_blk, head_dim)), 0)


def rms_norm(x, gamma, eps):
    """RMSNorm: x / sqrt(mean(x^2) + eps) * gamma, over the last axis."""
    x = _f64(x)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * _f64(gamma)


def _softmax_attend(q, keys, vals, scale):
    """softmax(q . keys / sqrt(d_head)) vals for one query vector."""
    s = (keys @ q) * scale
    mx = s.max()
    p = np.exp(s - mx)
    return (p @ vals) / p.sum()


def cache_append(state: DecodeState, weights, factors: Sequence[int], x_blocks):
    """Append whole blocks to the proxy cache (Eq. 21; streaming update, Sec. 3.8).

    x_blocks: [B, nblk*P, d]. Each block is compressed, h = C(x_block)
    (Eq. 7 / 16, no cross-layer proxy input), projected to the cached key and
    value, K_p = h W_k^T + b_k and V_p = h W_v^T + b_v, and written at row n;
    then n grows by one. Raises if the capacity would be exceeded.
    """
    x_blocks = _f64(x_blocks)
    bsz, toks, d = x_blocks.shape
    p_blk = int(np.prod(factors))
    nblk = toks // p_blk
    n_heads = state.k_cache.shape[1]
    dh = state.k_cache.shape[3]
    if state.n + nblk > state.k_cache.shape[2]:
        raise ValueError("proxy cache capacity exceeded")
    for b in range(bsz):
        h, _ = compress(x_blocks[b], factors, weights["compress"])   # [nblk, d]
        kp = linear(h, *weights["k_proxy"]).reshape(nblk, n_heads, dh)
        vp = linear(h, *weights["v_proxy"]).reshape(nblk, n_heads, dh)
        state.k_cache[b, :, state.n:state.n + nblk] = kp.transpose(1, 0, 2)
        state.v_cache[b, :, state.n:state.n + nblk] = vp.transpose(1, 0, 2)
    state.n += nblk
    return state


def decode_step(state: DecodeState, weights, factors: Sequence[int], x_t, rms_eps=1e-6):
    """Decode one token per sequence (Eq. 19-20 against the cache of Eq. 21).

    x_t: [B, d]. Returns y_t [B, d] and advances the state; when the block
    fills (j reaches P) it is appended to the cache and the local slots are
    released (Sec. 3.8).
    """
    x_t = _f64(x_t)
    bsz, d = x_t.shape
    n_heads = state.k_loc.shape[1]
    dh = state.k_loc.shape[3]
    p_blk = state.x_blk.shape[1]
    scale = 1.0 / np.sqrt(dh)
    j = state.j
    u = rms_norm(x_t, weights["rms_gamma"], rms_eps)
    q = linear(u, *weights["q"]).reshape(bsz, n_heads, dh)
    k = linear(u, *weights["k"]).reshape(bsz, n_heads, dh)
    v = linear(u, *weights["v"]).reshape(bsz, n_heads, dh)
    alpha = sigmoid(linear(u, *weights["alpha"]))                 # [B, n_heads]
    state.x_blk[:, j] = x_t
    state.k_loc[:, :, j] = k
    state.v_loc[:, :, j] = v
    attn = np.zeros((bsz, n_heads, dh))
    for b in range(bsz):
        for h in range(n_heads):
            a_x = _softmax_attend(q[b, h], state.k_loc[b, h, :j + 1], state.v_loc[b, h, :j + 1], scale)
            if state.n > 0:
                a_h = _softmax_attend(q[b, h], state.k_cache[b, h, :state.n],
                                      state.v_cache[b, h, :state.n], scale)
            else:
                a_h = np.zeros(dh)
            attn[b, h] = a_x + alpha[b, h] * a_h
    y = x_t + linear(attn.reshape(bsz, d), *weights["o"])
    state.j = j + 1
    if state.j == p_blk:
        cache_append(state, weights, factors, state.x_blk.copy())
        state.j = 0
        state.x_blk[:] = 0
        state.k_loc[:] = 0
        state.v_loc[:] = 0
    return y
