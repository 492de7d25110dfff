"""Oracle for the proxy-KV-cache decode step and the block-triggered append.

Test infrastructure only (see the package docstring). Follows the
generation block of the language model (Eq. 19-20) decoding one token per
sequence against the frozen proxy cache of Eq. 21, with the streaming
update of Sec. 3.8: once P new tokens have been decoded the block is
compressed, appended to the cache as one new proxy row and its local
features are dropped. `prefill` is the parallel form of the same block over
a whole chunk of tokens (every output at once, the chunk's complete blocks
appended), equal to that many streaming steps.

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


def prefill(state: DecodeState, weights, factors: Sequence[int], xs, rms_eps=1e-6, tokens=None):
    """Parallel form of the generation block over a chunk of tokens (Eq. 19-20).

    xs: [B, T, d], the next T tokens of every sequence, starting at a block
    boundary (state.j == 0). Token t of the chunk belongs to block t // P; it
    attends to the tokens of its own block up to itself (A_x) and to the
    cached proxies of every block completed before its own (A_h): the n0
    rows already in the cache plus one row per earlier block of the chunk
    (Eq. 21). The T // P complete blocks are appended to the cache; the
    tokens of an unfinished last block stay in the local slots, so decoding
    continues at j = T % P. The result equals T streaming decode steps.

    tokens: optional list of chunk positions; outputs are computed only
    there (the state update is always complete). Returns y [B, T, d], or
    [B, len(tokens), d] when tokens is given.
    """
    if state.j != 0:
        raise ValueError("prefill starts at a block boundary")
    xs = _f64(xs)
    bsz, T, d = xs.shape
    n_heads = state.k_loc.shape[1]
    dh = state.k_loc.shape[3]
    p_blk = state.x_blk.shape[1]
    scale = 1.0 / np.sqrt(dh)
    n0 = state.n
    nblk = T // p_blk
    if nblk:
        cache_append(state, weights, factors, xs[:, :nblk * p_blk])
    toks = list(range(T)) if tokens is None else list(tokens)
    rem = T - nblk * p_blk
    # keys and values are needed for every token some output attends to,
    # and for the unfinished block that stays in the local slots
    need = sorted({s for t in toks for s in range((t // p_blk) * p_blk, t + 1)} | set(range(nblk * p_blk, T)))
    at = {s: i for i, s in enumerate(need)}
    u_need = rms_norm(xs[:, need], weights["rms_gamma"], rms_eps)                  # [B, |need|, d]
    k = linear(u_need, *weights["k"]).reshape(bsz, len(need), n_heads, dh)
    v = linear(u_need, *weights["v"]).reshape(bsz, len(need), n_heads, dh)
    y = np.zeros((bsz, len(toks), d))
    for i, t in enumerate(toks):
        blk = t // p_blk
        local = [at[s] for s in range(blk * p_blk, t + 1)]
        n_vis = n0 + blk                  # proxies of the blocks before this one
        u = rms_norm(xs[:, t], weights["rms_gamma"], rms_eps)                       # [B, d]
        q = linear(u, *weights["q"]).reshape(bsz, n_heads, dh)
        alpha = sigmoid(linear(u, *weights["alpha"]))                              # [B, n_heads]
        attn = np.zeros((bsz, n_heads, dh))
        for b in range(bsz):
            for h in range(n_heads):
                a_x = _softmax_attend(q[b, h], k[b, local, h], v[b, local, h], scale)
                if n_vis > 0:
                    a_h = _softmax_attend(q[b, h], state.k_cache[b, h, :n_vis], state.v_cache[b, h, :n_vis], scale)
                else:
                    a_h = np.zeros(dh)
                attn[b, h] = a_x + alpha[b, h] * a_h
        y[:, i] = xs[:, t] + linear(attn.reshape(bsz, d), *weights["o"])
    state.x_blk[:] = 0
    state.k_loc[:] = 0
    state.v_loc[:] = 0
    for s in range(rem):
        state.x_blk[:, s] = xs[:, nblk * p_blk + s]
        state.k_loc[:, :, s] = k[:, at[nblk * p_blk + s]]
        state.v_loc[:, :, s] = v[:, at[nblk * p_blk + s]]
    state.j = rem
    return y
