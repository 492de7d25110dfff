"""Pins for the decode and append oracle (CPU only).

The streaming decode is checked against a parallel-form computation written
independently here (every token's output from its visible local tokens and
the proxies of all blocks completed before it), the append against the
layer's own proxy keys and values, and a few closed forms.
"""
import math

import numpy as np
import pytest

import oracle
from oracle import DecodeState


def decode_weights(rng, d, nh, factors, std=0.3):
    p_blk = int(np.prod(factors))
    dims = [d] * (len(factors) + 1)

    def lin(o, i):
        return (rng.standard_normal((o, i)) * std, rng.standard_normal(o) * 0.1)

    return {"rms_gamma": 1.0 + 0.1 * rng.standard_normal(d),
            "q": lin(d, d), "k": lin(d, d), "v": lin(d, d), "o": lin(d, d),
            "alpha": lin(nh, d),
            "compress": [lin(dims[j + 1], factors[j] * dims[j]) for j in range(len(factors))],
            "k_proxy": lin(d, d), "v_proxy": lin(d, d)}


def _parallel_form(xs, w, nh, P, k0, v0, j0, x_prev_blk, eps):
    """Every output of a streaming run, computed without any running state.

    Token t (0-based in the new stream) sits at block position (j0 + t) % P.
    It attends to the tokens of its block up to itself (some may predate the
    stream: x_prev_blk), and to the initial cache plus one proxy per block
    completed before its own (single-level compression written out).
    """
    steps, bsz, d = xs.shape
    dh = d // nh
    wc, bc = w["compress"][0]
    out = np.zeros((steps, bsz, d))
    allx = np.concatenate([x_prev_blk.transpose(1, 0, 2), xs], axis=0)   # [j0+steps, B, d]
    for t in range(steps):
        g = j0 + t                       # index in allx
        blk = g // P
        start = blk * P
        for b in range(bsz):
            def norm(v):
                return v / math.sqrt(float(np.mean(v * v)) + eps) * w["rms_gamma"]
            u = norm(allx[g, b])
            q = w["q"][0] @ u + w["q"][1]
            keys = np.stack([w["k"][0] @ norm(allx[s, b]) + w["k"][1] for s in range(start, g + 1)])
            vals = np.stack([w["v"][0] @ norm(allx[s, b]) + w["v"][1] for s in range(start, g + 1)])
            ck, cv = [k0[b]], [v0[b]]
            for pb in range(blk):
                h = wc @ allx[pb * P:(pb + 1) * P, b].reshape(-1) + bc
                ck.append((w["k_proxy"][0] @ h + w["k_proxy"][1]).reshape(nh, 1, dh))
                cv.append((w["v_proxy"][0] @ h + w["v_proxy"][1]).reshape(nh, 1, dh))
            ck = np.concatenate(ck, axis=1)
            cv = np.concatenate(cv, axis=1)
            alpha = 1 / (1 + np.exp(-(w["alpha"][0] @ u + w["alpha"][1])))
            att = np.zeros(d)
            for h_ in range(nh):
                cs = slice(h_ * dh, (h_ + 1) * dh)
                s = keys[:, cs] @ q[cs] / math.sqrt(dh)
                p = np.exp(s - s.max())
                ax = p @ vals[:, cs] / p.sum()
                if ck.shape[1]:
                    s = ck[h_] @ q[cs] / math.sqrt(dh)
                    p = np.exp(s - s.max())
                    ah = p @ cv[h_] / p.sum()
                else:
                    ah = 0.0
                att[cs] = ax + alpha[h_] * ah
            out[t, b] = allx[g, b] + w["o"][0] @ att + w["o"][1]
    return out


@pytest.mark.parametrize("n0,j0", [(0, 0), (5, 0), (3, 2)])
def test_streaming_equals_parallel_form(n0, j0):
    rng = np.random.default_rng(40 + n0 + j0)
    bsz, d, nh, P = 2, 8, 2, 4
    dh = d // nh
    w = decode_weights(rng, d, nh, (P,))
    steps = 11
    cap = n0 + (j0 + steps) // P + 1
    st = DecodeState.empty(bsz, nh, dh, P, cap, d)
    st.k_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
    st.v_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
    st.n = n0
    k0 = st.k_cache[:, :, :n0].copy()
    v0 = st.v_cache[:, :, :n0].copy()
    x_prev = rng.standard_normal((bsz, j0, d))
    for t in range(j0):    # tokens of the current block decoded before the stream starts
        oracle.decode_step(st, w, (P,), x_prev[:, t])
    assert st.n == n0 and st.j == j0
    xs = rng.standard_normal((steps, bsz, d))
    ys = np.stack([oracle.decode_step(st, w, (P,), xs[t]) for t in range(steps)])
    ref = _parallel_form(xs, w, nh, P, k0, v0, j0, x_prev, 1e-6)
    np.testing.assert_allclose(ys, ref, rtol=1e-12, atol=1e-12)
    # Eq. 21: one proxy row per completed block
    assert st.n == n0 + (j0 + steps) // P
    assert st.j == (j0 + steps) % P


def test_append_equals_layer_proxy_keys_values():
    rng = np.random.default_rng(50)
    bsz, d, nh, factors = 2, 6, 2, (2, 3)
    P = 6
    w = decode_weights(rng, d, nh, factors)
    x = rng.standard_normal((bsz, 3 * P, d))
    st = DecodeState.empty(bsz, nh, d // nh, P, 4, d)
    oracle.cache_append(st, w, factors, x)
    assert st.n == 3
    lw = {"compress": w["compress"], "q": w["q"], "k": w["k_proxy"], "v": w["v_proxy"]}
    for b in range(bsz):
        _, _, _, _, k, v = oracle.proxies_and_attention_inputs(x[b], lw, factors)
        np.testing.assert_allclose(st.k_cache[b, :, :3].transpose(1, 0, 2).reshape(3, d), k, rtol=1e-13)
        np.testing.assert_allclose(st.v_cache[b, :, :3].transpose(1, 0, 2).reshape(3, d), v, rtol=1e-13)
    with pytest.raises(ValueError):
        oracle.cache_append(st, w, factors, x[:, :2 * P])


def test_alpha_off_and_constant_proxy_values():
    rng = np.random.default_rng(51)
    bsz, d, nh, P = 2, 8, 2, 4
    dh = d // nh
    w = decode_weights(rng, d, nh, (P,))
    x = rng.standard_normal((bsz, d))

    def fresh(n0, const=None):
        st = DecodeState.empty(bsz, nh, dh, P, n0 + 1, d)
        if const is None:
            st.k_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
            st.v_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
        else:
            st.k_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
            st.v_cache[:, :, :n0] = const[:, :, None, :]
        st.n = n0
        return st

    # alpha -> 0: the cache does not matter
    w_off = dict(w)
    w_off["alpha"] = (np.zeros_like(w["alpha"][0]), np.full(nh, -40.0))
    y_a = oracle.decode_step(fresh(7), w_off, (P,), x)
    y_b = oracle.decode_step(fresh(0), w_off, (P,), x)
    np.testing.assert_allclose(y_a, y_b, rtol=0, atol=1e-12)
    # constant cached values: A_h equals the constant whatever the keys
    const = rng.standard_normal((bsz, nh, dh))
    y1 = oracle.decode_step(fresh(9, const), w, (P,), x)
    y2 = oracle.decode_step(fresh(1, const), w, (P,), x)
    np.testing.assert_allclose(y1, y2, rtol=0, atol=1e-12)


def test_first_token_empty_cache_closed_form():
    """j = 0, n = 0: A_x = v of the token itself, A_h = 0."""
    rng = np.random.default_rng(52)
    bsz, d, nh, P = 3, 8, 4, 4
    w = decode_weights(rng, d, nh, (P,))
    x = rng.standard_normal((bsz, d))
    st = DecodeState.empty(bsz, nh, d // nh, P, 2, d)
    y = oracle.decode_step(st, w, (P,), x)
    u = x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + 1e-6) * w["rms_gamma"]
    v = u @ w["v"][0].T + w["v"][1]
    np.testing.assert_allclose(y, x + v @ w["o"][0].T + w["o"][1], rtol=1e-12, atol=1e-12)


def test_cache_is_one_over_p_of_full_kv():
    """Eq. 21: proxy rows per layer are L/P of the token rows a full cache keeps."""
    rng = np.random.default_rng(53)
    bsz, d, nh, P = 1, 4, 1, 8
    w = decode_weights(rng, d, nh, (2, 4))
    L = 5 * P
    st = DecodeState.empty(bsz, nh, d, P, 8, d)
    oracle.cache_append(st, w, (2, 4), rng.standard_normal((bsz, L, d)))
    assert st.n * P == L


def _stream_state(bsz, nh, dh, P, cap, d, n0, rng):
    st = DecodeState.empty(bsz, nh, dh, P, cap, d)
    st.k_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
    st.v_cache[:, :, :n0] = rng.standard_normal((bsz, nh, n0, dh))
    st.n = n0
    return st


def _copy_state(st):
    return DecodeState(st.k_cache.copy(), st.v_cache.copy(), st.n, st.x_blk.copy(), st.k_loc.copy(),
                       st.v_loc.copy(), st.j)


@pytest.mark.parametrize("n0,T,factors", [(0, 11, (4,)), (5, 12, (4,)), (3, 3, (4,)), (2, 17, (2, 2)),
                                          (0, 1, (4,))])
def test_prefill_equals_streaming_steps(n0, T, factors):
    """The parallel form over a chunk gives every output and the whole state
    that T streaming decode steps give (Eq. 19-21, Sec. 3.8)."""
    rng = np.random.default_rng(70 + n0 + T)
    bsz, d, nh = 2, 8, 2
    dh = d // nh
    P = int(np.prod(factors))
    w = decode_weights(rng, d, nh, factors)
    cap = n0 + T // P + 1
    a = _stream_state(bsz, nh, dh, P, cap, d, n0, rng)
    b = _copy_state(a)
    xs = rng.standard_normal((bsz, T, d))
    y_par = oracle.prefill(a, w, factors, xs)
    y_seq = np.stack([oracle.decode_step(b, w, factors, xs[:, t]) for t in range(T)], axis=1)
    np.testing.assert_allclose(y_par, y_seq, rtol=1e-12, atol=1e-12)
    assert (a.n, a.j) == (b.n, b.j) == (n0 + T // P, T % P)
    for name in ("k_cache", "v_cache", "x_blk", "k_loc", "v_loc"):
        np.testing.assert_allclose(getattr(a, name), getattr(b, name), rtol=1e-12, atol=1e-12, err_msg=name)
    # decoding continues from the prefilled state exactly as from the streamed one
    x_next = rng.standard_normal((bsz, d))
    np.testing.assert_allclose(oracle.decode_step(a, w, factors, x_next), oracle.decode_step(b, w, factors, x_next),
                               rtol=1e-12, atol=1e-12)


def test_prefill_equals_independent_parallel_form():
    rng = np.random.default_rng(81)
    bsz, d, nh, P, n0, T = 2, 8, 2, 4, 3, 14
    dh = d // nh
    w = decode_weights(rng, d, nh, (P,))
    st = _stream_state(bsz, nh, dh, P, n0 + T // P + 1, d, n0, rng)
    k0 = st.k_cache[:, :, :n0].copy()
    v0 = st.v_cache[:, :, :n0].copy()
    xs = rng.standard_normal((bsz, T, d))
    y = oracle.prefill(st, w, (P,), xs)
    ref = _parallel_form(xs.transpose(1, 0, 2), w, nh, P, k0, v0, 0, np.zeros((bsz, 0, d)), 1e-6)
    np.testing.assert_allclose(y, ref.transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_prefill_token_subset_matches_full():
    rng = np.random.default_rng(82)
    bsz, d, nh, P, n0, T = 2, 8, 2, 4, 2, 13
    dh = d // nh
    w = decode_weights(rng, d, nh, (P,))
    a = _stream_state(bsz, nh, dh, P, n0 + T // P + 1, d, n0, rng)
    b = _copy_state(a)
    xs = rng.standard_normal((bsz, T, d))
    toks = [0, 5, 7, 12]
    full = oracle.prefill(a, w, (P,), xs)
    part = oracle.prefill(b, w, (P,), xs, tokens=toks)
    np.testing.assert_allclose(part, full[:, toks], rtol=1e-12, atol=1e-12)
    for name in ("k_cache", "v_cache", "x_blk", "k_loc", "v_loc"):
        np.testing.assert_array_equal(getattr(a, name), getattr(b, name), err_msg=name)


def test_prefill_requires_block_boundary():
    rng = np.random.default_rng(83)
    w = decode_weights(rng, 8, 2, (4,))
    st = _stream_state(1, 2, 4, 4, 4, 8, 0, rng)
    oracle.decode_step(st, w, (4,), rng.standard_normal((1, 8)))
    with pytest.raises(ValueError):
        oracle.prefill(st, w, (4,), rng.standard_normal((1, 3, 8)))
