"""Oracle for one ProxyFormer layer: forward (Algorithm 1) and backward.

Test infrastructure only (see the package docstring). All arithmetic is
float64 numpy; matrix products use ``@`` as a library primitive.

Notation: a linear map is y = x W^T + b with W stored [out, in]. d_0 is the
local-stream width d_fine, d_M the proxy width d_proxy, R_j = L/(k_1...k_j)
and m = R_M = L/P the number of proxies (Sec. 3.1, Eq. 15).

Readings of points the paper leaves open (each is also a flag or default of
the C-ABI):
* Causality of the injection. Algorithm 1 injects the contextualised proxy
  of block i into block i. Under the causal proxy mask of Eq. 9 a token
  would then see later tokens of its own block, while the language model
  only needs block causality (Sec. 3.7). TOKEN_CAUSAL (default) injects
  the proxy of block i-1 into block i and zero into block 0, so token t
  depends only on tokens <= t; BLOCK_CAUSAL is the literal reading
  (block i gets proxy i, causal proxy mask); BIDIRECTIONAL sets M = 0.
* The interaction F of Eq. 9 is multi-head attention with Q/K/V/O linear
  maps (with biases), heads taking contiguous column slices of width
  d_head, scale 1/sqrt(d_head), masked entries excluded, no positional
  encoding (NoPE, Sec. 5.1), no norm or residual inside F.
* The proxy stream returned by Algorithm 1 is H after the update of Eq. 8
  (before interaction).
* Flatten / grouping order: token-major, so grouping k consecutive rows of
  a row-major [R, d] matrix is a zero-copy reshape to [R/k, k*d].
* C and D are shared across blocks (and across groups of a level).
* The gate g of Eq. 12 is a d_fine-wide linear map of the concatenation
  [X, Delta]: G = X W_gx^T + Delta W_gd^T + b_g with W_g = [W_gx | W_gd].
* Intermediate level widths d_j default to d_proxy; there is no
  non-linearity between levels (the cascade is reshape -> project).
* The 2-D partition of the vision instantiation (Sec. 3.9) groups each
  p x p patch of a raster-order image into one block (P = p^2, one level),
  tokens row by row inside the patch, patches in raster order of the patch
  grid; the layer is otherwise unchanged (layer_forward_2d).
* The per-head gate (INJECT_GATED_HEAD) is Eq. 12 with the per-head
  weighting of Eq. 20: G = [X, Delta] W_g^T + b_g with W_g [n_heads,
  2 d_fine], and channel c takes the gate of head c // (d_fine / n_heads).
* The affine modulation of Eq. 13 leaves s, t and Norm open: s and t are
  one linear map of Delta per token, [s | t] = Delta W_a^T + b_a with W_a
  [2 d_fine, d_fine]; Norm is an RMSNorm over the d_fine channels without
  a gain (eps = 1e-6; a gain would duplicate 1 + s). As written, X is
  replaced, not added to.
* A length L that is not a multiple of P gives m = ceil(L/P) blocks
  (Sec. 3.1); the partial last block is zero-padded to P tokens, the
  padding's outputs are dropped and it receives no gradient.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

TOKEN_CAUSAL = 0
BLOCK_CAUSAL = 1
BIDIRECTIONAL = 2

# local fusion of Delta into X (Sec. 3.4)
INJECT_GATED = 0  # Eq. 12
INJECT_ADD = 1    # Eq. 11
INJECT_AFFINE = 2  # Eq. 13
INJECT_GATED_HEAD = 3  # Eq. 12 with one gate per head (the per-head weighting of Eq. 20)


def head_of_channel(d_f: int, n_heads: int):
    """Channel c of the local stream belongs to head c // (d_f / n_heads)."""
    if d_f % n_heads:
        raise ValueError("the per-head gate needs n_heads | d_fine")
    return np.arange(d_f) // (d_f // n_heads)

AFFINE_EPS = 1e-6  # RMSNorm epsilon of the affine modulation


def rms_normalise(x):
    """Norm of Eq. 13 (reading): x / sqrt(mean(x^2) + eps) per token, no gain."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + AFFINE_EPS)

_ROW_CHUNK = 512  # query rows per chunk; rows are independent (Eq. 9)


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def sigmoid(z):
    """Logistic function sigma(z) = 1 / (1 + exp(-z)), evaluated without overflow."""
    z = np.asarray(z, dtype=np.float64)
    out = np.empty_like(z)
    pos = z >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-z[pos]))
    e = np.exp(z[~pos])
    out[~pos] = e / (1.0 + e)
    return out


def linear(x, w, b):
    """y = x W^T + b (W stored [out, in]; b may be None)."""
    y = x @ _f64(w).T
    if b is not None:
        y = y + _f64(b)
    return y


def group_rows(z, k: int):
    """Partition of Eq. 2 / grouping step of Eq. 16.

    Groups k consecutive rows of z [R*k, d] and concatenates their channels:
    out[r, q*d + c] = z[r*k + q, c]. For row-major storage this index map is
    exactly a reshape.
    """
    rows, d = z.shape
    if rows % k:
        raise ValueError("row count must be a multiple of the group factor")
    return z.reshape(rows // k, k * d)


def ungroup_rows(t, k: int):
    """Unflatten of Eq. 10 / the reverse reshape of Eq. 17.

    out[r*k + q, c] = t[r, q*d + c] for t [R, k*d].
    """
    rows, kd = t.shape
    return t.reshape(rows * k, kd // k)


def compress(x, factors: Sequence[int], comp):
    """Bottom-up compression C of one sequence (Eq. 7; cascade of Eq. 16).

    x: [L, d_0]. comp: list of (W_cj [d_j, k_j d_{j-1}], b_cj) for j = 1..M.
    Level j groups k_j consecutive rows of Z_{j-1} and projects them:
    Z_j = group(Z_{j-1}, k_j) W_cj^T + b_cj. Returns c = Z_M [L/P, d_M] and the
    list of level inputs group(Z_{j-1}, k_j) (needed by the backward).
    """
    z = _f64(x)
    inputs = []
    for k, (w, b) in zip(factors, comp):
        v = group_rows(z, k)
        inputs.append(v)
        z = linear(v, w, b)
    return z, inputs


def decompress(s, factors: Sequence[int], dec):
    """Top-down decompression D = D_1 o ... o D_M of proxy rows (Eq. 10, Eq. 17).

    s: [R_M, d_M]. dec: list of (W_dj [k_j d_{j-1}, d_j], b_dj) for j = 1..M.
    Level j (applied for j = M down to 1) projects U_j up to k_j d_{j-1}
    channels and unflattens to k_j rows: U_{j-1} = ungroup(U_j W_dj^T + b_dj).
    Returns Delta = U_0 and the list of level inputs [U_M, ..., U_1].
    """
    u = _f64(s)
    inputs = []
    for j in reversed(range(len(factors))):
        w, b = dec[j]
        inputs.append(u)
        u = ungroup_rows(linear(u, w, b), factors[j])
    return u, inputs


def attention_rows(q, k, v, rows, n_heads: int, mask: int):
    """Multi-head proxy attention (Eq. 9) for selected query rows.

    q, k, v: [m, d_p], head h in columns [h*d_head, (h+1)*d_head).
    For query row i: s_ij = Q_i . K_j / sqrt(d_head); the causal mask keeps
    j <= i (both causal modes), BIDIRECTIONAL keeps every j; p_i = softmax_j(s_i)
    and O_i = sum_j p_ij V_j. Returns O [len(rows), d_p] and the natural-log
    log-sum-exp of the scores, LSE [n_heads, len(rows)].
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    m, d = q.shape
    dh = d // n_heads
    scale = 1.0 / np.sqrt(dh)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.zeros((rows.size, d))
    lse = np.zeros((n_heads, rows.size))
    for s0 in range(0, rows.size, _ROW_CHUNK):
        r = rows[s0:s0 + _ROW_CHUNK]
        kmax = m if mask == BIDIRECTIONAL else int(r.max()) + 1
        for h in range(n_heads):
            cs = slice(h * dh, (h + 1) * dh)
            sc = (q[r, cs] @ k[:kmax, cs].T) * scale
            if mask != BIDIRECTIONAL:
                sc[np.arange(kmax)[None, :] > r[:, None]] = -np.inf
            mx = sc.max(axis=1, keepdims=True)
            p = np.exp(sc - mx)
            den = p.sum(axis=1, keepdims=True)
            out[s0:s0 + r.size, cs] = (p @ v[:kmax, cs]) / den
            lse[h, s0:s0 + r.size] = (mx + np.log(den))[:, 0]
    return out, lse


def proxies_and_attention_inputs(x, weights, factors, h_in=None):
    """Steps 1-5 of Algorithm 1 up to the interaction inputs, one sequence.

    Returns c (Eq. 7/16), H = H_in + c (Eq. 8), and the projections Q, K, V of H.
    """
    c, cin = compress(x, factors, weights["compress"])
    h = c if h_in is None else _f64(h_in) + c
    q = linear(h, *weights["q"])
    k = linear(h, *weights["k"])
    v = linear(h, *weights["v"])
    return c, cin, h, q, k, v


def layer_forward(x, weights, factors: Sequence[int], n_heads: int,
                  mask: int = TOKEN_CAUSAL, h_in=None,
                  sample_blocks: Optional[Sequence[int]] = None,
                  keep: bool = False, injection: int = INJECT_GATED) -> Dict[str, object]:
    """One ProxyFormer layer (Algorithm 1) on x [B, L, d_fine].

    Steps: partition and compress every block (Eq. 2, 7, 15-16); residual
    proxy update H = H_in + c (Eq. 8); causal multi-head attention over the
    m proxies (Eq. 9) followed by the output map W_o; decompress the proxy
    each block receives (Eq. 10, 17); gated injection
    Y = X + sigmoid(G) * Delta with G = [X, Delta] W_g^T + b_g (Eq. 12),
    with INJECT_ADD the residual addition Y = X + Delta (Eq. 11), with
    INJECT_AFFINE the modulation Y = (1 + s(Delta)) * Norm(X) + t(Delta)
    (Eq. 13; [s | t] = Delta W_a^T + b_a, Norm an RMSNorm without gain).

    Returns x_out [B, L, d_fine] and h_out = H [B, m, d_proxy]. With
    ``sample_blocks`` only those blocks are decompressed and injected
    (x_out then has shape [B, len(sample_blocks), P, d_fine]); H is still
    computed for every block. With ``keep`` the intermediates needed by the
    backward are returned per sequence.
    """
    x = _f64(x)
    bsz, seq, d_f = x.shape
    p_blk = int(np.prod(factors))
    m = seq // p_blk
    if m * p_blk != seq:
        # m = ceil(L/P) blocks (Sec. 3.1): the partial last block is read as
        # zero-padded to P tokens; outputs of the padding are dropped
        # (sampled blocks keep the padded rows of the last block)
        xp = np.concatenate([x, np.zeros((bsz, (m + 1) * p_blk - seq, d_f))], axis=1)
        res = layer_forward(xp, weights, factors, n_heads, mask, h_in, sample_blocks, keep, injection)
        if sample_blocks is None:
            res["x_out"] = res["x_out"][:, :seq]
        return res
    d_p = weights["q"][0].shape[0]
    h_out = np.zeros((bsz, m, d_p))
    if sample_blocks is None:
        blocks = np.arange(m)
        x_out = np.zeros_like(x)
    else:
        blocks = np.asarray(sample_blocks, dtype=np.int64)
        x_out = np.zeros((bsz, blocks.size, p_blk, d_f))
    kept: List[Dict[str, object]] = []
    lse_all = np.zeros((bsz, n_heads, m)) if sample_blocks is None else None
    for b in range(bsz):
        hin_b = None if h_in is None else _f64(h_in)[b]
        c, cin, h, q, k, v = proxies_and_attention_inputs(x[b], weights, factors, hin_b)
        h_out[b] = h
        # which contextualised proxy feeds each block: TOKEN_CAUSAL gives
        # block i proxy i-1 (block 0 gets zero); the other modes give proxy i
        if mask == TOKEN_CAUSAL:
            src = blocks - 1
        else:
            src = blocks.copy()
        need = np.unique(src[src >= 0])
        o_need, lse = attention_rows(q, k, v, need, n_heads, mask)
        hbar_need = linear(o_need, *weights["o"])
        s = np.zeros((blocks.size, d_p))
        pos = np.searchsorted(need, src[src >= 0])
        s[src >= 0] = hbar_need[pos]
        delta, dinputs = decompress(s, factors, weights["decompress"])
        xb = x[b].reshape(m, p_blk, d_f)[blocks].reshape(-1, d_f)
        if injection == INJECT_ADD:
            g = None
            y = xb + delta
        elif injection == INJECT_GATED_HEAD:
            # Eq. 12 with one gate per head: G = [X, Delta] W_g^T + b_g, W_g [n_heads, 2 d_fine]
            wg, bg = _f64(weights["gate"][0]), _f64(weights["gate"][1])
            g = xb @ wg[:, :d_f].T + delta @ wg[:, d_f:].T + bg
            y = xb + sigmoid(g)[:, head_of_channel(d_f, n_heads)] * delta
        elif injection == INJECT_AFFINE:
            # Eq. 13: Y = (1 + s(Delta)) * Norm(X) + t(Delta), [s | t] = Delta W_a^T + b_a
            st = linear(delta, *weights["affine"])
            g = st[:, :d_f]                      # s, kept for the backward
            y = (1.0 + g) * rms_normalise(xb) + st[:, d_f:]
        else:
            wg, bg = _f64(weights["gate"][0]), _f64(weights["gate"][1])
            g = xb @ wg[:, :d_f].T + delta @ wg[:, d_f:].T + bg
            y = xb + sigmoid(g) * delta
        if sample_blocks is None:
            x_out[b] = y
            lse_full = np.zeros((n_heads, m))
            lse_full[:, need] = lse
            lse_all[b] = lse_full
        else:
            x_out[b] = y.reshape(blocks.size, p_blk, d_f)
        if keep:
            if sample_blocks is not None:
                raise ValueError("keep requires the full forward")
            hbar = np.zeros((m, d_p))
            hbar[need] = hbar_need
            o_full = np.zeros((m, d_p))
            o_full[need] = o_need
            kept.append(dict(cin=cin, h=h, q=q, k=k, v=v, o=o_full, hbar=hbar,
                             s=s, dinputs=dinputs, delta=delta, g=g, x=x[b]))
    res: Dict[str, object] = {"x_out": x_out, "h_out": h_out}
    if lse_all is not None:
        res["lse"] = lse_all
    if keep:
        res["kept"] = kept
    return res


def _attention_backward(q, k, v, o, do, n_heads, mask):
    """Chain rule through Eq. 9 for one sequence (all rows, dense per head).

    With P = softmax(S), S = Q K^T / sqrt(d_head) + M: dV = P^T dO,
    dP = dO V^T, dS = P * (dP - rowsum(dO * O)), dQ = dS K / sqrt(d_head),
    dK = dS^T Q / sqrt(d_head).

    Also returns the magnitudes of the terms that cancel in dS carried to
    dQ and dK: with |dS| := P * (|dP| + |rowsum(dO * O)|), |dQ| = |dS| |K|
    / sqrt(d_head) and |dK| = |dS|^T |Q| / sqrt(d_head) (entrywise
    absolute values; upper bounds of |dQ| and |dK|).
    """
    m, d = q.shape
    dh = d // n_heads
    scale = 1.0 / np.sqrt(dh)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dq_abs = np.zeros_like(q)
    dk_abs = np.zeros_like(k)
    for h in range(n_heads):
        cs = slice(h * dh, (h + 1) * dh)
        sc = (q[:, cs] @ k[:, cs].T) * scale
        if mask != BIDIRECTIONAL:
            sc[np.triu(np.ones((m, m), dtype=bool), 1)] = -np.inf
        mx = sc.max(axis=1, keepdims=True)
        p = np.exp(sc - mx)
        p /= p.sum(axis=1, keepdims=True)
        dv[:, cs] = p.T @ do[:, cs]
        dp = do[:, cs] @ v[:, cs].T
        rs = np.sum(do[:, cs] * o[:, cs], axis=1, keepdims=True)
        dsm = p * (dp - rs)
        dq[:, cs] = (dsm @ k[:, cs]) * scale
        dk[:, cs] = (dsm.T @ q[:, cs]) * scale
        dsm_abs = p * (np.abs(dp) + np.abs(rs))
        dq_abs[:, cs] = (dsm_abs @ np.abs(k[:, cs])) * scale
        dk_abs[:, cs] = (dsm_abs.T @ np.abs(q[:, cs])) * scale
    return dq, dk, dv, dq_abs, dk_abs


def layer_backward(x, weights, factors: Sequence[int], n_heads: int, dy,
                   mask: int = TOKEN_CAUSAL, h_in=None, dh_out=None,
                   injection: int = INJECT_GATED) -> Dict[str, object]:
    """Gradients of the layer forward (chain rule of Eq. 7-17 as read above).

    Given dY = dL/dX_out [B, L, d_fine] and optionally dH_out [B, m, d_proxy],
    returns dx, dh_in (None when h_in is None), every weight and bias gradient
    summed over the batch in the layout of the weights, the gradients of
    the projections Q, K, V per proxy ("proj_grads", [B, m, d_proxy] each),
    and for the gated injections the per-column sums over tokens of |dG|
    ("gate_abs"), the magnitude of the terms the gate bias gradient sums.
    "score_abs" holds, for the Q and K maps, entrywise bounds of their weight
    and bias gradients built from the magnitudes of the terms that cancel in
    the score gradient dS: the scale against which a gradient that cancels
    to zero (one visible key per row, where a softmax is constant) is measured.
    """
    dy = _f64(dy)
    bsz, seq, d_f = dy.shape
    p_blk = int(np.prod(factors))
    m = seq // p_blk
    if m * p_blk != seq:
        # zero-padded last block (Sec. 3.1): the padding receives no gradient
        # (dY = 0 there) and its dX is dropped
        pad = (m + 1) * p_blk - seq
        xp = np.concatenate([_f64(x), np.zeros((bsz, pad, d_f))], axis=1)
        dyp = np.concatenate([dy, np.zeros((bsz, pad, d_f))], axis=1)
        res = layer_backward(xp, weights, factors, n_heads, dyp, mask, h_in, dh_out, injection)
        res["dx"] = res["dx"][:, :seq]
        return res
    fwd = layer_forward(x, weights, factors, n_heads, mask, h_in, keep=True, injection=injection)
    nlev = len(factors)

    def zgrad(w):
        w0 = _f64(w[0])
        return [np.zeros_like(w0), np.zeros(w0.shape[0])]

    gr = {"compress": [zgrad(w) for w in weights["compress"]],
          "q": zgrad(weights["q"]), "k": zgrad(weights["k"]), "v": zgrad(weights["v"]),
          "o": zgrad(weights["o"]),
          "decompress": [zgrad(w) for w in weights["decompress"]],
          "gate": zgrad(weights["gate"]) if injection in (INJECT_GATED, INJECT_GATED_HEAD) else None,
          "affine": zgrad(weights["affine"]) if injection == INJECT_AFFINE else None}
    dx = np.zeros_like(dy)
    d_p = weights["q"][0].shape[0]
    dh_in = None if h_in is None else np.zeros((bsz, m, d_p))
    proj_grads = {name: np.zeros((bsz, m, d_p)) for name in ("q", "k", "v")}
    # entrywise bounds of the Q and K weight and bias gradients from the
    # magnitudes of the terms that cancel in dS (see _attention_backward)
    score_abs = {name: [np.zeros_like(gr[name][0]), np.zeros_like(gr[name][1])] for name in ("q", "k")}
    # per gate column, the sum over tokens of |dG|: the scale of the terms the
    # gate's bias gradient adds up (its accuracy is relative to this scale)
    gate_abs = np.zeros(_f64(weights["gate"][0]).shape[0]) if gr["gate"] is not None else None
    for b in range(bsz):
        kp = fwd["kept"][b]
        xb, delta, g = kp["x"], kp["delta"], kp["g"]
        if injection == INJECT_ADD:
            # Eq. 11: Y = X + Delta
            ddelta = dy[b]
            dxb = dy[b]
        elif injection == INJECT_GATED_HEAD:
            wg = _f64(weights["gate"][0])
            sg = sigmoid(g)                                   # [rows, n_heads]
            hc = head_of_channel(d_f, n_heads)
            gsz = d_f // n_heads
            # dG_h = sum over the head's channels of dY * Delta, times sigmoid'
            dg = (dy[b] * delta).reshape(-1, n_heads, gsz).sum(axis=2) * sg * (1.0 - sg)
            ddelta = dy[b] * sg[:, hc] + dg @ wg[:, d_f:]
            dxb = dy[b] + dg @ wg[:, :d_f]
            gr["gate"][0] += dg.T @ np.concatenate([xb, delta], axis=1)
            gr["gate"][1] += dg.sum(axis=0)
            gate_abs += np.abs(dg).sum(axis=0)
        elif injection == INJECT_AFFINE:
            # Eq. 13: Y = (1 + s) * N + t, N = X r, r = (mean(X^2) + eps)^(-1/2)
            wa = _f64(weights["affine"][0])
            r = 1.0 / np.sqrt(np.mean(xb * xb, axis=1, keepdims=True) + AFFINE_EPS)
            nx = xb * r
            dst = np.concatenate([dy[b] * nx, dy[b]], axis=1)          # [dS | dT]
            dn = dy[b] * (1.0 + g)
            dxb = r * (dn - nx * np.mean(dn * nx, axis=1, keepdims=True))
            ddelta = dst @ wa
            gr["affine"][0] += dst.T @ delta
            gr["affine"][1] += dst.sum(axis=0)
        else:
            wg = _f64(weights["gate"][0])
            sg = sigmoid(g)
            # Eq. 12: Y = X + sigmoid(G) * Delta, G = X W_gx^T + Delta W_gd^T + b_g
            dg = dy[b] * delta * sg * (1.0 - sg)
            ddelta = dy[b] * sg + dg @ wg[:, d_f:]
            dxb = dy[b] + dg @ wg[:, :d_f]
            gr["gate"][0] += dg.T @ np.concatenate([xb, delta], axis=1)
            gr["gate"][1] += dg.sum(axis=0)
            gate_abs += np.abs(dg).sum(axis=0)
        # Eq. 17 in reverse: level j = 1..M (the forward ran M..1)
        du = ddelta
        for j in range(nlev):
            u_in = kp["dinputs"][nlev - 1 - j]          # input U_j of level j
            dt = group_rows(du, factors[j])             # gradient of U_j W^T + b
            gr["decompress"][j][0] += dt.T @ u_in
            gr["decompress"][j][1] += dt.sum(axis=0)
            du = dt @ _f64(weights["decompress"][j][0])
        ds = du
        # undo the shift that chose which proxy feeds each block
        if mask == TOKEN_CAUSAL:
            dhbar = np.zeros_like(ds)
            dhbar[:-1] = ds[1:]
        else:
            dhbar = ds
        gr["o"][0] += dhbar.T @ kp["o"]
        gr["o"][1] += dhbar.sum(axis=0)
        do = dhbar @ _f64(weights["o"][0])
        dq, dk, dv, dq_abs, dk_abs = _attention_backward(kp["q"], kp["k"], kp["v"], kp["o"], do, n_heads, mask)
        dh = np.zeros_like(kp["h"]) if dh_out is None else _f64(dh_out)[b].copy()
        for name, dz in (("q", dq), ("k", dk), ("v", dv)):
            proj_grads[name][b] = dz
            gr[name][0] += dz.T @ kp["h"]
            gr[name][1] += dz.sum(axis=0)
            dh += dz @ _f64(weights[name][0])
        for name, dz_abs in (("q", dq_abs), ("k", dk_abs)):
            score_abs[name][0] += dz_abs.T @ np.abs(kp["h"])
            score_abs[name][1] += dz_abs.sum(axis=0)
        if dh_in is not None:
            dh_in[b] = dh
        # Eq. 8 passes dH to c unchanged; then Eq. 16 in reverse, level M..1
        dz = dh
        for j in reversed(range(nlev)):
            v_in = kp["cin"][j]
            gr["compress"][j][0] += dz.T @ v_in
            gr["compress"][j][1] += dz.sum(axis=0)
            dz = ungroup_rows(dz @ _f64(weights["compress"][j][0]), factors[j])
        dx[b] = dxb + dz
    return {"dx": dx, "dh_in": dh_in, "grads": gr, "proj_grads": proj_grads,
            "gate_abs": gate_abs if injection in (INJECT_GATED, INJECT_GATED_HEAD) else None,
            "score_abs": score_abs}


def patch_order(height: int, width: int, p: int):
    """Token order of the 2-D partition (Sec. 3.9): blocks are the p x p
    patches of a height x width raster-order image, taken in raster order
    of the patch grid; inside a patch the tokens go row by row. Returns
    order[j] = raster index of the j-th token of the partitioned sequence."""
    if height % p or width % p:
        raise ValueError("image sides must be multiples of the patch side")
    order = []
    for py in range(height // p):
        for px in range(width // p):
            for i in range(p):
                for j in range(p):
                    order.append((py * p + i) * width + px * p + j)
    return np.asarray(order, dtype=np.int64)


def _patch_side(factors: Sequence[int]) -> int:
    if len(factors) != 1:
        raise ValueError("the 2-D partition is single-level (P = p * p)")
    p = int(round(np.sqrt(factors[0])))
    if p * p != factors[0]:
        raise ValueError("the 2-D partition needs P = p * p")
    return p


def layer_forward_2d(x, weights, factors: Sequence[int], n_heads: int, image_width: int,
                     mask: int = BIDIRECTIONAL, h_in=None, injection: int = INJECT_GATED):
    """The layer on an image (Sec. 3.9): x [B, height * width, d_fine] in
    raster order, a block = one p x p patch (P = p^2), proxies in raster order
    of the patch grid. The tokens are gathered into patch order, the layer of
    Algorithm 1 runs on that sequence, and the output returns to raster
    order. Returns x_out (raster order) and h_out [B, (height/p)(width/p), d_proxy]."""
    x = _f64(x)
    p = _patch_side(factors)
    order = patch_order(x.shape[1] // image_width, image_width, p)
    res = layer_forward(x[:, order], weights, factors, n_heads, mask, h_in, injection=injection)
    y = np.zeros_like(x)
    y[:, order] = res["x_out"]
    return {"x_out": y, "h_out": res["h_out"]}


def layer_backward_2d(x, weights, factors: Sequence[int], n_heads: int, image_width: int, dy,
                      mask: int = BIDIRECTIONAL, h_in=None, dh_out=None, injection: int = INJECT_GATED):
    """Gradients of layer_forward_2d: the gather is a permutation, so dY is
    gathered the same way and dX scattered back to raster order."""
    x = _f64(x)
    p = _patch_side(factors)
    order = patch_order(x.shape[1] // image_width, image_width, p)
    res = layer_backward(x[:, order], weights, factors, n_heads, _f64(dy)[:, order], mask, h_in, dh_out,
                         injection)
    dx = np.zeros_like(x)
    dx[:, order] = res["dx"]
    res["dx"] = dx
    return res
