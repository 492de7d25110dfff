"""Pins for the layer oracle (CPU only).

Each test checks the oracle against something other than itself: a
hand-worked example, a closed form, an invariant, a library routine or a
brute-force loop, so that a dropped term, wrong sign, wrong index or
transposed operand anywhere in the forward fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.layer import group_rows, ungroup_rows, decompress

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand_weights(rng, d_f, d_p, factors, dims=None, bias=True, std=0.3):
    m = len(factors)
    dims = dims or [d_f] + [d_p] * m
    dims = list(dims)
    dims[-1] = d_p

    def lin(o, i):
        return (rng.standard_normal((o, i)) * std,
                rng.standard_normal(o) * 0.1 if bias else np.zeros(o))

    return {
        "compress": [lin(dims[j + 1], factors[j] * dims[j]) for j in range(m)],
        "q": lin(d_p, d_p), "k": lin(d_p, d_p), "v": lin(d_p, d_p), "o": lin(d_p, d_p),
        "decompress": [lin(factors[j] * dims[j], dims[j + 1]) for j in range(m)],
        "gate": lin(d_f, 2 * d_f),
    }


# --------------------------------------------------------------------- golden

def test_golden_hand_worked_layer():
    g = json.load(open(os.path.join(GOLDEN, "layer_tiny_worked.json")))
    masks = {"token_causal": oracle.TOKEN_CAUSAL, "block_causal": oracle.BLOCK_CAUSAL,
             "bidirectional": oracle.BIDIRECTIONAL}
    z2 = np.zeros(2)
    for case in g["cases"]:
        bg = math.log(3.0) if case["b_g"] == "ln3" else float(case["b_g"])
        w = {"compress": [(np.array(g["W_c"], float), z2)],
             "q": (np.array(g["W_q"], float), z2), "k": (np.array(g["W_k"], float), z2),
             "v": (np.array(g["W_v"], float), z2), "o": (np.array(g["W_o"], float), z2),
             "decompress": [(np.array(g["W_d"], float), np.zeros(4))],
             "gate": (np.zeros((2, 4)), np.full(2, bg))}
        x = np.array(g["x"], float)[None]
        r = oracle.layer_forward(x, w, (2,), 1, masks[case["mask"]])
        np.testing.assert_allclose(r["h_out"][0], case["h_out"], rtol=0, atol=1e-14)
        np.testing.assert_allclose(r["x_out"][0], case["x_out"], rtol=0, atol=1e-14)


# ---------------------------------------------------------------- compression

def test_group_rows_index_map():
    z = np.arange(6 * 3, dtype=float).reshape(6, 3)
    g = group_rows(z, 2)
    for r in range(3):
        for q in range(2):
            for c in range(3):
                assert g[r, q * 3 + c] == z[r * 2 + q, c]
    np.testing.assert_array_equal(ungroup_rows(g, 2), z)


def test_compress_constant_block_closed_form():
    rng = np.random.default_rng(1)
    d_f, d_p, P = 3, 5, 4
    w = rand_weights(rng, d_f, d_p, (P,))
    wc, bc = w["compress"][0]
    vals = rng.standard_normal((2, d_f))
    x = np.repeat(vals, P, axis=0)                      # block i is P copies of vals[i]
    c, _ = oracle.compress(x, (P,), w["compress"])
    wsum = sum(wc[:, p * d_f:(p + 1) * d_f] for p in range(P))
    for i in range(2):
        np.testing.assert_allclose(c[i], wsum @ vals[i] + bc, rtol=1e-13, atol=1e-13)


def _effective_two_level(w1, b1, w2, b2, k1, k2, d0, d1):
    """Single-level map equal to the two-level cascade, built from indices.

    Token p = q2*k1 + q1 of a block feeds level-1 group q2 at slot q1, so its
    channel c reaches the proxy through W2[:, q2 block] @ W1[:, q1 block].
    """
    d2 = w2.shape[0]
    weff = np.zeros((d2, k1 * k2 * d0))
    for q2 in range(k2):
        w2q = w2[:, q2 * d1:(q2 + 1) * d1]
        for q1 in range(k1):
            p = q2 * k1 + q1
            weff[:, p * d0:(p + 1) * d0] = w2q @ w1[:, q1 * d0:(q1 + 1) * d0]
    beff = b2 + sum(w2[:, q2 * d1:(q2 + 1) * d1] @ b1 for q2 in range(k2))
    return weff, beff


@pytest.mark.parametrize("k1,k2", [(2, 3), (3, 1), (1, 4)])
def test_factorised_equals_effective_single_level(k1, k2):
    rng = np.random.default_rng(2)
    d0, d1, d2 = 3, 4, 5
    w = rand_weights(rng, d0, d2, (k1, k2), dims=[d0, d1, d2])
    (w1, b1), (w2, b2) = w["compress"]
    x = rng.standard_normal((3 * k1 * k2, d0))
    c, _ = oracle.compress(x, (k1, k2), w["compress"])
    weff, beff = _effective_two_level(w1, b1, w2, b2, k1, k2, d0, d1)
    if k2 == 1:
        np.testing.assert_allclose(weff, w2 @ w1, rtol=1e-13, atol=1e-13)
    c1, _ = oracle.compress(x, (k1 * k2,), [(weff, beff)])
    np.testing.assert_allclose(c, c1, rtol=1e-12, atol=1e-12)


def test_compress_is_affine_and_update_is_residual():
    rng = np.random.default_rng(3)
    d_f, d_p, P, L = 4, 6, 4, 16
    w = rand_weights(rng, d_f, d_p, (2, 2))
    x1, x2 = rng.standard_normal((2, L, d_f))
    a = 0.3
    c1, _ = oracle.compress(x1, (2, 2), w["compress"])
    c2, _ = oracle.compress(x2, (2, 2), w["compress"])
    c12, _ = oracle.compress(a * x1 + (1 - a) * x2, (2, 2), w["compress"])
    np.testing.assert_allclose(c12, a * c1 + (1 - a) * c2, rtol=1e-12, atol=1e-12)
    h_in = rng.standard_normal((1, L // P, d_p))
    r0 = oracle.layer_forward(x1[None], w, (2, 2), 2)
    r1 = oracle.layer_forward(x1[None], w, (2, 2), 2, h_in=h_in)
    np.testing.assert_allclose(r0["h_out"][0], c1, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(r1["h_out"] - h_in, r0["h_out"], rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------ attention

def _brute_attention(q, k, v, n_heads, causal):
    m, d = q.shape
    dh = d // n_heads
    out = np.zeros((m, d))
    for h in range(n_heads):
        for i in range(m):
            js = range(i + 1) if causal else range(m)
            sc = []
            for j in js:
                s = 0.0
                for c in range(dh):
                    s += q[i, h * dh + c] * k[j, h * dh + c]
                sc.append(s / math.sqrt(dh))
            mx = max(sc)
            e = [math.exp(s - mx) for s in sc]
            tot = sum(e)
            for c in range(dh):
                out[i, h * dh + c] = sum(e[t] * v[j, h * dh + c] for t, j in enumerate(js)) / tot
    return out


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BIDIRECTIONAL])
def test_attention_brute_force(mask):
    rng = np.random.default_rng(4)
    m, d, nh = 7, 6, 2
    q, k, v = rng.standard_normal((3, m, d)) * 1.5
    o, lse = oracle.attention_rows(q, k, v, np.arange(m), nh, mask)
    ref = _brute_attention(q, k, v, nh, mask != oracle.BIDIRECTIONAL)
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)
    # log-sum-exp of row 0 (sees only key 0 when causal)
    dh = d // nh
    s00 = q[0, :dh] @ k[0, :dh] / math.sqrt(dh)
    if mask != oracle.BIDIRECTIONAL:
        assert abs(lse[0, 0] - s00) < 1e-12


def test_attention_matches_torch_sdpa():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(5)
    m, d, nh = 33, 16, 4
    q, k, v = rng.standard_normal((3, m, d))
    o, _ = oracle.attention_rows(q, k, v, np.arange(m), nh, oracle.TOKEN_CAUSAL)

    def heads(a):
        return torch.from_numpy(a).reshape(m, nh, d // nh).transpose(0, 1)

    ref = torch.nn.functional.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True)
    ref = ref.transpose(0, 1).reshape(m, d).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-11)


def test_attention_constant_values_uniform_weights_single_row():
    rng = np.random.default_rng(6)
    m, d, nh = 9, 8, 2
    q, k, v = rng.standard_normal((3, m, d)) * 3
    # constant V: any row of weights that sums to 1 returns the constant
    cv = np.tile(rng.standard_normal(d), (m, 1))
    o, _ = oracle.attention_rows(q, k, cv, np.arange(m), nh, oracle.TOKEN_CAUSAL)
    np.testing.assert_allclose(o, cv, rtol=1e-13, atol=1e-13)
    # zero queries: uniform weights, so O_i is the prefix mean of V
    o, lse = oracle.attention_rows(np.zeros_like(q), k, v, np.arange(m), nh, oracle.TOKEN_CAUSAL)
    pref = np.cumsum(v, axis=0) / np.arange(1, m + 1)[:, None]
    np.testing.assert_allclose(o, pref, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse[0], np.log(np.arange(1, m + 1)), rtol=1e-13, atol=1e-13)
    # one proxy: O = V_0
    o, _ = oracle.attention_rows(q[:1], k[:1], v[:1], [0], nh, oracle.TOKEN_CAUSAL)
    np.testing.assert_allclose(o[0], v[0], rtol=1e-14, atol=1e-14)


def test_block_size_one_is_token_attention():
    """P = 1, one level: the layer's interaction is causal attention over tokens."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(7)
    L, d, nh = 12, 8, 2
    w = rand_weights(rng, d, d, (1,))
    x = rng.standard_normal((1, L, d))
    c, _, h, q, k, v = oracle.proxies_and_attention_inputs(x[0], w, (1,))
    np.testing.assert_allclose(c, x[0] @ w["compress"][0][0].T + w["compress"][0][1], rtol=1e-13)
    o, _ = oracle.attention_rows(q, k, v, np.arange(L), nh, oracle.TOKEN_CAUSAL)

    def heads(a):
        return torch.from_numpy(a).reshape(L, nh, d // nh).transpose(0, 1)

    ref = torch.nn.functional.scaled_dot_product_attention(heads(q), heads(k), heads(v), is_causal=True)
    np.testing.assert_allclose(o, ref.transpose(0, 1).reshape(L, d).numpy(), rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------------ injection

def _constant_proxy_weights(rng, d_f, d_p, P, s0):
    """W_o = 0, b_o = s0: every contextualised proxy equals s0."""
    w = rand_weights(rng, d_f, d_p, (P,))
    w["o"] = (np.zeros((d_p, d_p)), s0.copy())
    return w


def test_zero_decompression_leaves_x_unchanged():
    rng = np.random.default_rng(8)
    d_f, d_p, P = 4, 6, 4
    w = rand_weights(rng, d_f, d_p, (2, 2))
    w["decompress"] = [(np.zeros_like(a), np.zeros_like(b)) for a, b in w["decompress"]]
    x = rng.standard_normal((2, 16, d_f))
    for mask in (0, 1, 2):
        r = oracle.layer_forward(x, w, (2, 2), 2, mask)
        assert np.array_equal(r["x_out"], x)


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BLOCK_CAUSAL])
def test_gate_closed_forms_constant_proxy(mask):
    rng = np.random.default_rng(9)
    d_f, d_p, P, L = 3, 4, 4, 12
    s0 = rng.standard_normal(d_p)
    w = _constant_proxy_weights(rng, d_f, d_p, P, s0)
    wd, bd = w["decompress"][0]
    delta_full = (wd @ s0 + bd).reshape(P, d_f)      # block receiving s0
    delta_zero = bd.reshape(P, d_f)                   # block receiving 0
    deltas = [delta_zero if (mask == oracle.TOKEN_CAUSAL and i == 0) else delta_full
              for i in range(L // P)]
    delta = np.concatenate(deltas, axis=0)
    x = rng.standard_normal((1, L, d_f))

    def run(wg, bg):
        w2 = dict(w)
        w2["gate"] = (wg, bg)
        return oracle.layer_forward(x, w2, (P,), 2, mask)["x_out"][0]

    z = np.zeros((d_f, 2 * d_f))
    np.testing.assert_allclose(run(z, np.zeros(d_f)), x[0] + 0.5 * delta, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(run(z, np.full(d_f, 40.0)), x[0] + delta, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(run(z, np.full(d_f, 2.0)), x[0] + delta / (1 + math.exp(-2.0)),
                               rtol=1e-13, atol=1e-13)
    beta = 0.7
    eye = np.eye(d_f) * beta
    # gate reads X through the first half of W_g ...
    wx = np.concatenate([eye, np.zeros((d_f, d_f))], axis=1)
    np.testing.assert_allclose(run(wx, np.zeros(d_f)),
                               x[0] + delta / (1 + np.exp(-beta * x[0])), rtol=1e-13, atol=1e-13)
    # ... and Delta through the second half
    wdl = np.concatenate([np.zeros((d_f, d_f)), eye], axis=1)
    np.testing.assert_allclose(run(wdl, np.zeros(d_f)),
                               x[0] + delta / (1 + np.exp(-beta * delta)), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BLOCK_CAUSAL])
def test_residual_add_injection_closed_form(mask):
    """Eq. 11: Y = X + Delta exactly, whatever the gate weights hold."""
    rng = np.random.default_rng(19)
    d_f, d_p, P, L = 3, 4, 4, 12
    s0 = rng.standard_normal(d_p)
    w = _constant_proxy_weights(rng, d_f, d_p, P, s0)
    wd, bd = w["decompress"][0]
    delta_full = (wd @ s0 + bd).reshape(P, d_f)
    delta_zero = bd.reshape(P, d_f)
    deltas = [delta_zero if (mask == oracle.TOKEN_CAUSAL and i == 0) else delta_full
              for i in range(L // P)]
    x = rng.standard_normal((1, L, d_f))
    w["gate"] = (rng.standard_normal((d_f, 2 * d_f)), rng.standard_normal(d_f))
    y = oracle.layer_forward(x, w, (P,), 2, mask, injection=oracle.INJECT_ADD)["x_out"][0]
    np.testing.assert_allclose(y, x[0] + np.concatenate(deltas, axis=0), rtol=1e-13, atol=1e-13)
    w.pop("gate")  # the gate is not read in this mode
    y2 = oracle.layer_forward(x, w, (P,), 2, mask, injection=oracle.INJECT_ADD)["x_out"][0]
    assert np.array_equal(y, y2)


def test_factorised_decompression_constant_proxy():
    """Two-level D of a constant proxy: reverse reshape order of Eq. 17."""
    rng = np.random.default_rng(10)
    d0, d1, d2, k1, k2 = 2, 3, 4, 2, 3
    w = rand_weights(rng, d0, d2, (k1, k2), dims=[d0, d1, d2])
    (wd1, bd1), (wd2, bd2) = w["decompress"]
    s = rng.standard_normal((2, d2))
    delta, _ = decompress(s, (k1, k2), w["decompress"])
    for i in range(2):
        t2 = wd2 @ s[i] + bd2                           # k2 groups of d1
        for q2 in range(k2):
            u1 = t2[q2 * d1:(q2 + 1) * d1]
            t1 = wd1 @ u1 + bd1                         # k1 tokens of d0
            for q1 in range(k1):
                tok = i * k1 * k2 + q2 * k1 + q1
                np.testing.assert_allclose(delta[tok], t1[q1 * d0:(q1 + 1) * d0], rtol=1e-13, atol=1e-13)


# ------------------------------------------------------------------ causality

@pytest.mark.parametrize("factors", [(4,), (2, 2)])
def test_token_causality_bit_identical(factors):
    rng = np.random.default_rng(11)
    d_f, d_p, L = 4, 6, 24
    P = int(np.prod(factors))
    w = rand_weights(rng, d_f, d_p, factors)
    x = rng.standard_normal((1, L, d_f))
    base = oracle.layer_forward(x, w, factors, 2, oracle.TOKEN_CAUSAL)
    for t in (0, 5, 11, 12, 23):
        x2 = x.copy()
        x2[0, t] += 1.0
        r = oracle.layer_forward(x2, w, factors, 2, oracle.TOKEN_CAUSAL)
        assert np.array_equal(r["x_out"][0, :t], base["x_out"][0, :t])
        assert np.array_equal(r["h_out"][0, :t // P], base["h_out"][0, :t // P])
        assert not np.array_equal(r["x_out"][0, t], base["x_out"][0, t])
        if t // P + 1 < L // P:  # a later block sees the change through its proxy
            assert not np.array_equal(r["x_out"][0, (t // P + 1) * P:], base["x_out"][0, (t // P + 1) * P:])


def test_block_causality_and_bidirectional_control():
    rng = np.random.default_rng(12)
    d_f, d_p, L, P = 4, 6, 24, 4
    w = rand_weights(rng, d_f, d_p, (P,))
    x = rng.standard_normal((1, L, d_f))
    t = 13
    x2 = x.copy()
    x2[0, t] += 1.0
    b0 = oracle.layer_forward(x, w, (P,), 2, oracle.BLOCK_CAUSAL)["x_out"][0]
    b1 = oracle.layer_forward(x2, w, (P,), 2, oracle.BLOCK_CAUSAL)["x_out"][0]
    assert np.array_equal(b0[:P * (t // P)], b1[:P * (t // P)])
    assert not np.array_equal(b0[P * (t // P):t], b1[P * (t // P):t])   # same block sees the future
    d0 = oracle.layer_forward(x, w, (P,), 2, oracle.BIDIRECTIONAL)["x_out"][0]
    d1 = oracle.layer_forward(x2, w, (P,), 2, oracle.BIDIRECTIONAL)["x_out"][0]
    assert not np.array_equal(d0[:P], d1[:P])


def test_sampled_forward_matches_full():
    rng = np.random.default_rng(13)
    d_f, d_p, L = 4, 6, 32
    w = rand_weights(rng, d_f, d_p, (2, 2))
    x = rng.standard_normal((2, L, d_f))
    for mask in (0, 1, 2):
        full = oracle.layer_forward(x, w, (2, 2), 2, mask)
        blocks = [0, 3, 7]
        s = oracle.layer_forward(x, w, (2, 2), 2, mask, sample_blocks=blocks)
        ref = full["x_out"].reshape(2, 8, 4, d_f)[:, blocks]
        np.testing.assert_allclose(s["x_out"], ref, rtol=1e-13, atol=1e-13)
        np.testing.assert_array_equal(s["h_out"], full["h_out"])


# ------------------------------------------------------ partial last block

@pytest.mark.parametrize("factors", [(4,), (2, 2)])
def test_partial_last_block_prefix_and_last_proxy(factors):
    """m = ceil(L / P) blocks (Sec. 3.1), the last one partial: with token
    causality the complete blocks' outputs and proxies equal those of the
    layer run on the complete blocks alone, and the last proxy is the
    compression of the partial block with zero padding, i.e. its weight
    columns for the missing tokens drop out."""
    rng = np.random.default_rng(90 + len(factors))
    d_f, d_p, nh, B = 4, 6, 2, 2
    P = int(np.prod(factors))
    full, rem = 3, 3                      # three complete blocks and 3 tokens
    L = full * P + rem
    w = rand_weights(rng, d_f, d_p, factors)
    x = rng.standard_normal((B, L, d_f))
    res = oracle.layer_forward(x, w, factors, nh, oracle.TOKEN_CAUSAL)
    assert res["x_out"].shape == (B, L, d_f) and res["h_out"].shape == (B, full + 1, d_p)
    head = oracle.layer_forward(x[:, :full * P], w, factors, nh, oracle.TOKEN_CAUSAL)
    np.testing.assert_array_equal(res["x_out"][:, :full * P], head["x_out"])
    np.testing.assert_array_equal(res["h_out"][:, :full], head["h_out"])
    if len(factors) == 1:
        wc, bc = w["compress"][0]
        for b in range(B):
            tail = x[b, full * P:].reshape(-1)
            np.testing.assert_allclose(res["h_out"][b, -1], wc[:, :rem * d_f] @ tail + bc, rtol=1e-12, atol=1e-12)


def test_partial_last_block_outputs_ignore_padding_content():
    """Under token causality the partial block receives the proxy of the block
    before it, so its outputs do not depend on what fills the missing tokens;
    under block causality they do (its own proxy includes the padding)."""
    rng = np.random.default_rng(93)
    d_f, d_p, nh, B, P = 4, 6, 2, 1, 4
    L = 2 * P + 1
    w = rand_weights(rng, d_f, d_p, (P,))
    x = rng.standard_normal((B, L, d_f))
    junk = np.concatenate([x, rng.standard_normal((B, 3 * P - L, d_f))], axis=1)
    for mask, same in ((oracle.TOKEN_CAUSAL, True), (oracle.BLOCK_CAUSAL, False)):
        a = oracle.layer_forward(x, w, (P,), nh, mask)["x_out"]
        b = oracle.layer_forward(junk, w, (P,), nh, mask)["x_out"][:, :L]
        assert np.array_equal(a, b) == same, mask


# ------------------------------------------------------------ 2-D partition

def test_patch_proxies_closed_form():
    """Sec. 3.9: a block is a p x p patch. Without H_in each proxy is the
    compression of its patch's pixels (row by row), patches in raster order."""
    rng = np.random.default_rng(101)
    d_f, d_p, nh, B, p, hgt, wid = 3, 4, 2, 2, 2, 4, 6
    w = rand_weights(rng, d_f, d_p, (p * p,))
    x = rng.standard_normal((B, hgt * wid, d_f))
    res = oracle.layer_forward_2d(x, w, (p * p,), nh, wid)
    wc, bc = w["compress"][0]
    img = x.reshape(B, hgt, wid, d_f)
    for b in range(B):
        k = 0
        for py in range(hgt // p):
            for px in range(wid // p):
                patch = img[b, py * p:(py + 1) * p, px * p:(px + 1) * p].reshape(-1)
                np.testing.assert_allclose(res["h_out"][b, k], wc @ patch + bc, rtol=1e-12, atol=1e-12)
                k += 1


def test_patch_order_is_a_permutation_and_one_column_is_1d():
    order = oracle.patch_order(6, 4, 2)
    assert sorted(order.tolist()) == list(range(24))
    # a single column of patches: patch order = raster order, same layer as 1-D
    rng = np.random.default_rng(102)
    w = rand_weights(rng, 3, 4, (4,))
    x = rng.standard_normal((1, 8 * 2, 3))
    np.testing.assert_array_equal(oracle.patch_order(8, 2, 2), np.arange(16))
    a = oracle.layer_forward_2d(x, w, (4,), 2, 2, mask=oracle.BLOCK_CAUSAL)
    b = oracle.layer_forward(x, w, (4,), 2, oracle.BLOCK_CAUSAL)
    np.testing.assert_array_equal(a["x_out"], b["x_out"])


def test_patch_block_causality():
    """Block-causal over the patch grid: changing one pixel changes the outputs
    of its own patch and of later patches only (raster order of patches)."""
    rng = np.random.default_rng(103)
    d_f, d_p, nh, p, hgt, wid = 3, 4, 2, 2, 4, 4
    w = rand_weights(rng, d_f, d_p, (p * p,))
    x = rng.standard_normal((1, hgt * wid, d_f))
    y0 = oracle.layer_forward_2d(x, w, (p * p,), nh, wid, mask=oracle.BLOCK_CAUSAL)["x_out"]
    x2 = x.copy()
    x2[0, 2 * wid + 1] += 1.0            # pixel (2, 1): patch (1, 0), the third patch
    y1 = oracle.layer_forward_2d(x2, w, (p * p,), nh, wid, mask=oracle.BLOCK_CAUSAL)["x_out"]
    patch_of = lambda t: (t // wid // p) * (wid // p) + (t % wid) // p
    for t in range(hgt * wid):
        changed = not np.array_equal(y0[0, t], y1[0, t])
        assert changed == (patch_of(t) >= 2), t


# ------------------------------------------------------- affine modulation

def _affine_weights(rng, d_f, scale=0.3):
    return (rng.standard_normal((2 * d_f, d_f)) * scale, rng.standard_normal(2 * d_f) * 0.1)


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BIDIRECTIONAL])
def test_affine_modulation_constant_terms(mask):
    """Eq. 13 with s and t independent of Delta (W_a = 0): every output row
    minus t, divided by 1 + s, is a positive multiple of its input row with
    mean square mean(x^2) / (mean(x^2) + eps) (the RMSNorm reading)."""
    rng = np.random.default_rng(111)
    d_f, d_p, nh, B, P, L = 4, 6, 2, 2, 4, 12
    w = rand_weights(rng, d_f, d_p, (P,))
    s0 = rng.uniform(-0.5, 0.5, d_f)
    t0 = rng.standard_normal(d_f)
    w["affine"] = (np.zeros((2 * d_f, d_f)), np.concatenate([s0, t0]))
    x = rng.standard_normal((B, L, d_f))
    y = oracle.layer_forward(x, w, (P,), nh, mask, injection=oracle.INJECT_AFFINE)["x_out"]
    n = (y - t0) / (1.0 + s0)
    ratio = n / x
    np.testing.assert_allclose(ratio, ratio[..., :1] * np.ones_like(ratio), rtol=1e-12)
    assert np.all(ratio > 0)
    ms = np.mean(x * x, axis=-1)
    np.testing.assert_allclose(np.mean(n * n, axis=-1), ms / (ms + oracle.layer.AFFINE_EPS), rtol=1e-12)


def test_affine_modulation_is_affine_in_the_decompressed_signal():
    """With X fixed, Y depends on Delta through one linear map per token: Y is
    affine in the decompression biases (doubling their offset from the
    baseline doubles Y's change), unlike the gate of Eq. 12."""
    rng = np.random.default_rng(112)
    d_f, d_p, nh, B, P, L = 4, 6, 2, 1, 4, 8
    w = rand_weights(rng, d_f, d_p, (P,))
    w["affine"] = _affine_weights(rng, d_f)
    x = rng.standard_normal((B, L, d_f))
    wd, bd = w["decompress"][0]
    outs = []
    for k in (0.0, 1.0, 2.0):
        w2 = dict(w)
        w2["decompress"] = [(wd, bd + k * 0.7)]
        outs.append(oracle.layer_forward(x, w2, (P,), nh, oracle.BIDIRECTIONAL,
                                         injection=oracle.INJECT_AFFINE)["x_out"])
    np.testing.assert_allclose(outs[2] - outs[0], 2 * (outs[1] - outs[0]), rtol=1e-10, atol=1e-12)
    assert np.max(np.abs(outs[1] - outs[0])) > 1e-3


# ----------------------------------------------------------- per-head gate

@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BIDIRECTIONAL])
def test_per_head_gate_equals_channel_gate_with_tied_rows(mask):
    """The per-head gate is the channel gate of Eq. 12 whose rows (and biases)
    are tied within each head's channel group."""
    rng = np.random.default_rng(121)
    d_f, d_p, nh, B, P, L = 6, 6, 3, 2, 4, 12
    w = rand_weights(rng, d_f, d_p, (P,))
    wh = (rng.standard_normal((nh, 2 * d_f)) * 0.3, rng.standard_normal(nh) * 0.2)
    x = rng.standard_normal((B, L, d_f))
    w_head = dict(w)
    w_head["gate"] = wh
    hc = oracle.head_of_channel(d_f, nh)
    np.testing.assert_array_equal(hc, [0, 0, 1, 1, 2, 2])
    w_chan = dict(w)
    w_chan["gate"] = (wh[0][hc], wh[1][hc])
    a = oracle.layer_forward(x, w_head, (P,), nh, mask, injection=oracle.INJECT_GATED_HEAD)["x_out"]
    b = oracle.layer_forward(x, w_chan, (P,), nh, mask, injection=oracle.INJECT_GATED)["x_out"]
    np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-13)
