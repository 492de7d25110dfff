"""Pins for the oracle's layer backward (CPU only).

Central finite differences in float64 check every gradient the backward
returns, in every mask mode and with a factorised cascade; the dual
causality test checks that the gradient respects the forward's causal
structure.
"""
import numpy as np
import pytest

import oracle
from test_oracle_layer import rand_weights


def _loss(x, w, factors, nh, mask, h_in, dy, dh, injection=oracle.INJECT_GATED):
    r = oracle.layer_forward(x, w, factors, nh, mask, h_in, injection=injection)
    val = float(np.sum(r["x_out"] * dy))
    if dh is not None:
        val += float(np.sum(r["h_out"] * dh))
    return val


def _param_paths(w):
    paths = []
    for name in ("q", "k", "v", "o", "gate"):
        if name not in w:
            continue
        paths += [((name, 0),), ((name, 1),)]
    for lvl in range(len(w["compress"])):
        paths += [("compress", (lvl, 0)), ("compress", (lvl, 1))]
        paths += [("decompress", (lvl, 0)), ("decompress", (lvl, 1))]
    return paths


def _get(w, path):
    if len(path) == 1:
        name, idx = path[0]
        return w[name][idx]
    name, (lvl, idx) = path
    return w[name][lvl][idx]


def _set(w, path, val):
    import copy
    w2 = copy.deepcopy(w)
    if len(path) == 1:
        name, idx = path[0]
        t = list(w2[name])
        t[idx] = val
        w2[name] = tuple(t)
    else:
        name, (lvl, idx) = path
        t = list(w2[name][lvl])
        t[idx] = val
        w2[name][lvl] = tuple(t)
    return w2


def _grad_of(gr, path):
    if len(path) == 1:
        name, idx = path[0]
        return gr[name][idx]
    name, (lvl, idx) = path
    return gr[name][lvl][idx]


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BLOCK_CAUSAL, oracle.BIDIRECTIONAL])
@pytest.mark.parametrize("factors", [(4,), (2, 4), (4, 2)])
def test_backward_finite_differences(mask, factors):
    rng = np.random.default_rng(20 + mask)
    d_f, d_p, nh, L, B = 4, 6, 2, 16, 2
    dims = [d_f] + [5] * (len(factors) - 1) + [d_p]   # d_1 differs from d_0 and d_M
    w = rand_weights(rng, d_f, d_p, factors, dims=dims, std=0.4)
    x = rng.standard_normal((B, L, d_f))
    m = L // int(np.prod(factors))
    h_in = rng.standard_normal((B, m, d_p))
    dy = rng.standard_normal((B, L, d_f))
    dh = rng.standard_normal((B, m, d_p))
    res = oracle.layer_backward(x, w, factors, nh, dy, mask, h_in, dh)
    eps = 1e-5

    def fd(fplus, fminus):
        return (fplus - fminus) / (2 * eps)

    # input gradients along random directions
    for _ in range(3):
        vx = rng.standard_normal(x.shape)
        num = fd(_loss(x + eps * vx, w, factors, nh, mask, h_in, dy, dh),
                 _loss(x - eps * vx, w, factors, nh, mask, h_in, dy, dh))
        ana = float(np.sum(res["dx"] * vx))
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (num, ana)
        vh = rng.standard_normal(h_in.shape)
        num = fd(_loss(x, w, factors, nh, mask, h_in + eps * vh, dy, dh),
                 _loss(x, w, factors, nh, mask, h_in - eps * vh, dy, dh))
        ana = float(np.sum(res["dh_in"] * vh))
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (num, ana)
    # every weight and bias
    for path in _param_paths(w):
        p0 = _get(w, path)
        v = rng.standard_normal(p0.shape)
        num = fd(_loss(x, _set(w, path, p0 + eps * v), factors, nh, mask, h_in, dy, dh),
                 _loss(x, _set(w, path, p0 - eps * v), factors, nh, mask, h_in, dy, dh))
        ana = float(np.sum(_grad_of(res["grads"], path) * v))
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (path, num, ana)


@pytest.mark.parametrize("factors", [(4,), (2, 4)])
def test_backward_finite_differences_residual_add(factors):
    """Eq. 11 injection: every gradient against central differences (no gate)."""
    rng = np.random.default_rng(31)
    d_f, d_p, nh, L, B = 4, 6, 2, 16, 2
    dims = [d_f] + [5] * (len(factors) - 1) + [d_p]
    w = rand_weights(rng, d_f, d_p, factors, dims=dims, std=0.4)
    w.pop("gate")
    x = rng.standard_normal((B, L, d_f))
    m = L // int(np.prod(factors))
    h_in = rng.standard_normal((B, m, d_p))
    dy = rng.standard_normal((B, L, d_f))
    dh = rng.standard_normal((B, m, d_p))
    inj = oracle.INJECT_ADD
    res = oracle.layer_backward(x, w, factors, nh, dy, oracle.TOKEN_CAUSAL, h_in, dh, injection=inj)
    assert res["grads"]["gate"] is None
    eps = 1e-5
    vx = rng.standard_normal(x.shape)
    num = (_loss(x + eps * vx, w, factors, nh, 0, h_in, dy, dh, inj) -
           _loss(x - eps * vx, w, factors, nh, 0, h_in, dy, dh, inj)) / (2 * eps)
    ana = float(np.sum(res["dx"] * vx))
    assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (num, ana)
    vh = rng.standard_normal(h_in.shape)
    num = (_loss(x, w, factors, nh, 0, h_in + eps * vh, dy, dh, inj) -
           _loss(x, w, factors, nh, 0, h_in - eps * vh, dy, dh, inj)) / (2 * eps)
    ana = float(np.sum(res["dh_in"] * vh))
    assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (num, ana)
    for path in _param_paths(w):
        p0 = _get(w, path)
        v = rng.standard_normal(p0.shape)
        num = (_loss(x, _set(w, path, p0 + eps * v), factors, nh, 0, h_in, dy, dh, inj) -
               _loss(x, _set(w, path, p0 - eps * v), factors, nh, 0, h_in, dy, dh, inj)) / (2 * eps)
        ana = float(np.sum(_grad_of(res["grads"], path) * v))
        assert abs(num - ana) <= 1e-6 * max(1.0, abs(ana)), (path, num, ana)


def test_backward_without_h_in_and_dh_out():
    rng = np.random.default_rng(30)
    d_f, d_p, nh, L = 3, 4, 2, 12
    w = rand_weights(rng, d_f, d_p, (3,))
    x = rng.standard_normal((1, L, d_f))
    dy = rng.standard_normal((1, L, d_f))
    res = oracle.layer_backward(x, w, (3,), nh, dy)
    assert res["dh_in"] is None
    eps = 1e-5
    vx = rng.standard_normal(x.shape)
    num = (_loss(x + eps * vx, w, (3,), nh, 0, None, dy, None)
           - _loss(x - eps * vx, w, (3,), nh, 0, None, dy, None)) / (2 * eps)
    assert abs(num - float(np.sum(res["dx"] * vx))) < 1e-6 * max(1.0, abs(num))


def test_backward_dual_causality():
    """Token-causal forward: dY[t] can only reach dX[s] for s <= t."""
    rng = np.random.default_rng(31)
    d_f, d_p, nh, L = 4, 6, 2, 24
    w = rand_weights(rng, d_f, d_p, (2, 2))
    x = rng.standard_normal((1, L, d_f))
    dy = rng.standard_normal((1, L, d_f))
    base = oracle.layer_backward(x, w, (2, 2), nh, dy)["dx"]
    for t in (3, 10, 17):
        dy2 = dy.copy()
        dy2[0, t] += 1.0
        r = oracle.layer_backward(x, w, (2, 2), nh, dy2)["dx"]
        assert np.array_equal(r[0, t + 1:], base[0, t + 1:])
        assert not np.array_equal(r[0, t], base[0, t])


def test_key_bias_gradient_vanishes():
    """Softmax is invariant to one constant added to every key (Eq. 9), so
    dL/db_k = sum of dK over proxies is zero up to rounding in every mode."""
    rng = np.random.default_rng(32)
    d_f, d_p, nh, L = 4, 6, 2, 24
    w = rand_weights(rng, d_f, d_p, (4,), std=0.5)
    x = rng.standard_normal((2, L, d_f))
    dy = rng.standard_normal((2, L, d_f))
    for mask in (0, 1, 2):
        res = oracle.layer_backward(x, w, (4,), nh, dy, mask)
        scale = np.max(np.sum(np.abs(res["proj_grads"]["k"]), axis=(0, 1)))
        assert scale > 1e-3
        assert np.max(np.abs(res["grads"]["k"][1])) < 1e-12 * scale
        np.testing.assert_allclose(res["grads"]["k"][1], res["proj_grads"]["k"].sum(axis=(0, 1)), atol=1e-14)



def test_score_gradient_bounds():
    """score_abs bounds the Q and K weight and bias gradients entrywise (the
    triangle inequality over the terms of dS and of the products after it),
    in every mask, and is of the gradients' own order where they do not
    cancel (the weight gradients here)."""
    rng = np.random.default_rng(33)
    d_f, d_p, nh, L = 4, 6, 2, 24
    w = rand_weights(rng, d_f, d_p, (4,), std=0.5)
    x = rng.standard_normal((2, L, d_f))
    dy = rng.standard_normal((2, L, d_f))
    for mask in (0, 1, 2):
        res = oracle.layer_backward(x, w, (4,), nh, dy, mask)
        for name in ("q", "k"):
            for i in (0, 1):
                g, bound = np.abs(res["grads"][name][i]), res["score_abs"][name][i]
                assert np.all(g <= bound * (1 + 1e-12) + 1e-15), (mask, name, i)
            assert np.max(np.abs(res["grads"][name][0])) > 1e-2 * np.max(res["score_abs"][name][0]), (mask, name)


@pytest.mark.parametrize("mask", [oracle.BLOCK_CAUSAL, oracle.BIDIRECTIONAL])
@pytest.mark.parametrize("L", [8, 5])
def test_single_proxy_score_gradients_vanish(mask, L):
    """One proxy (L <= P = 8): every attention row sees one key, and a
    softmax over one key is constant (Eq. 9), so the loss does not depend on
    W_q, b_q, W_k, b_k. Central differences in those weights are zero; the
    oracle's gradients are zero up to rounding, against a score_abs that is
    not (in these masks the proxy feeds its own block, so dO != 0)."""
    rng = np.random.default_rng(34 + L + mask)
    d_f, d_p, nh = 4, 6, 2
    w = rand_weights(rng, d_f, d_p, (8,), std=0.5)
    x = rng.standard_normal((1, L, d_f))
    dy = rng.standard_normal((1, L, d_f))
    res = oracle.layer_backward(x, w, (8,), nh, dy, mask)
    eps = 1e-4
    for name in ("q", "k"):
        for i in (0, 1):
            path = ((name, i),)
            v = rng.standard_normal(np.shape(_get(w, path)))
            num = (_loss(x, _set(w, path, _get(w, path) + eps * v), (8,), nh, mask, None, dy, None)
                   - _loss(x, _set(w, path, _get(w, path) - eps * v), (8,), nh, mask, None, dy, None)) / (2 * eps)
            assert abs(num) < 1e-9, (name, i, num)
            scale = np.max(res["score_abs"][name][i])
            assert scale > 1e-3, (name, i)
            assert np.max(np.abs(res["grads"][name][i])) < 1e-12 * scale, (name, i)

@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BIDIRECTIONAL])
def test_backward_finite_differences_partial_last_block(mask):
    """L % P != 0: the zero-padded last block (Sec. 3.1) in the backward."""
    rng = np.random.default_rng(95 + mask)
    factors = (2, 2)
    d_f, d_p, nh, L, B = 4, 6, 2, 14, 2
    w = rand_weights(rng, d_f, d_p, factors, std=0.4)
    x = rng.standard_normal((B, L, d_f))
    m = -(-L // 4)
    h_in = rng.standard_normal((B, m, d_p))
    dy = rng.standard_normal((B, L, d_f))
    dh = rng.standard_normal((B, m, d_p))
    res = oracle.layer_backward(x, w, factors, nh, dy, mask, h_in, dh)
    assert res["dx"].shape == x.shape
    eps = 1e-5
    for idx in [(0, 0, 1), (1, 12, 2), (0, 13, 0), (1, 13, 3)]:   # incl. the partial block's tokens
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (_loss(xp, w, factors, nh, mask, h_in, dy, dh) - _loss(xm, w, factors, nh, mask, h_in, dy, dh)) / (2 * eps)
        assert abs(fd - res["dx"][idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, res["dx"][idx])
    for path in _param_paths(w):
        wt = _get(w, path)
        flat = np.unravel_index(rng.integers(wt.size), wt.shape)
        wp, wm = wt.copy(), wt.copy()
        wp[flat] += eps
        wm[flat] -= eps
        fd = (_loss(x, _set(w, path, wp), factors, nh, mask, h_in, dy, dh)
              - _loss(x, _set(w, path, wm), factors, nh, mask, h_in, dy, dh)) / (2 * eps)
        g = _grad_of(res["grads"], path)[flat]
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(fd)), (path, flat, fd, g)


def test_backward_finite_differences_2d_partition():
    rng = np.random.default_rng(104)
    d_f, d_p, nh, B, p, hgt, wid = 3, 4, 2, 1, 2, 4, 4
    w = rand_weights(rng, d_f, d_p, (p * p,), std=0.4)
    x = rng.standard_normal((B, hgt * wid, d_f))
    dy = rng.standard_normal((B, hgt * wid, d_f))
    res = oracle.layer_backward_2d(x, w, (p * p,), nh, wid, dy)

    def loss(xx, ww):
        return float(np.sum(oracle.layer_forward_2d(xx, ww, (p * p,), nh, wid)["x_out"] * dy))

    eps = 1e-5
    for idx in [(0, 0, 0), (0, 5, 1), (0, 10, 2), (0, 15, 0)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (loss(xp, w) - loss(xm, w)) / (2 * eps)
        assert abs(fd - res["dx"][idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, res["dx"][idx])
    for path in _param_paths(w):
        wt = _get(w, path)
        flat = np.unravel_index(rng.integers(wt.size), wt.shape)
        wp, wm = wt.copy(), wt.copy()
        wp[flat] += eps
        wm[flat] -= eps
        fd = (loss(x, _set(w, path, wp)) - loss(x, _set(w, path, wm))) / (2 * eps)
        g = _grad_of(res["grads"], path)[flat]
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(fd)), (path, flat, fd, g)


@pytest.mark.parametrize("mask,factors", [(oracle.TOKEN_CAUSAL, (4,)), (oracle.BIDIRECTIONAL, (2, 2))])
def test_backward_finite_differences_affine_modulation(mask, factors):
    """Eq. 13 injection: dX through the RMSNorm, dDelta and dW_a / db_a."""
    rng = np.random.default_rng(97 + mask)
    d_f, d_p, nh, L, B = 4, 6, 2, 16, 2
    w = rand_weights(rng, d_f, d_p, factors, std=0.4)
    del w["gate"]
    w["affine"] = (rng.standard_normal((2 * d_f, d_f)) * 0.4, rng.standard_normal(2 * d_f) * 0.1)
    x = rng.standard_normal((B, L, d_f))
    m = L // int(np.prod(factors))
    h_in = rng.standard_normal((B, m, d_p))
    dy = rng.standard_normal((B, L, d_f))
    dh = rng.standard_normal((B, m, d_p))
    inj = oracle.INJECT_AFFINE
    res = oracle.layer_backward(x, w, factors, nh, dy, mask, h_in, dh, injection=inj)
    assert res["grads"]["gate"] is None
    eps = 1e-5
    for idx in [(0, 0, 0), (1, 7, 2), (0, 15, 3)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (_loss(xp, w, factors, nh, mask, h_in, dy, dh, inj) - _loss(xm, w, factors, nh, mask, h_in, dy, dh, inj)) / (2 * eps)
        assert abs(fd - res["dx"][idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, res["dx"][idx])
    for path in _param_paths(w) + [(("affine", 0),), (("affine", 1),)]:
        wt = _get(w, path)
        flat = np.unravel_index(rng.integers(wt.size), wt.shape)
        wp, wm = wt.copy(), wt.copy()
        wp[flat] += eps
        wm[flat] -= eps
        fd = (_loss(x, _set(w, path, wp), factors, nh, mask, h_in, dy, dh, inj)
              - _loss(x, _set(w, path, wm), factors, nh, mask, h_in, dy, dh, inj)) / (2 * eps)
        g = _grad_of(res["grads"], path)[flat]
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(fd)), (path, flat, fd, g)


@pytest.mark.parametrize("mask", [oracle.TOKEN_CAUSAL, oracle.BLOCK_CAUSAL])
def test_backward_finite_differences_per_head_gate(mask):
    rng = np.random.default_rng(131 + mask)
    factors = (2, 2)
    d_f, d_p, nh, L, B = 6, 6, 3, 16, 2
    w = rand_weights(rng, d_f, d_p, factors, std=0.4)
    w["gate"] = (rng.standard_normal((nh, 2 * d_f)) * 0.4, rng.standard_normal(nh) * 0.1)
    x = rng.standard_normal((B, L, d_f))
    m = L // 4
    h_in = rng.standard_normal((B, m, d_p))
    dy = rng.standard_normal((B, L, d_f))
    dh = rng.standard_normal((B, m, d_p))
    inj = oracle.INJECT_GATED_HEAD
    res = oracle.layer_backward(x, w, factors, nh, dy, mask, h_in, dh, injection=inj)
    eps = 1e-5
    for idx in [(0, 0, 0), (1, 9, 4), (0, 15, 5)]:
        xp, xm = x.copy(), x.copy()
        xp[idx] += eps
        xm[idx] -= eps
        fd = (_loss(xp, w, factors, nh, mask, h_in, dy, dh, inj) - _loss(xm, w, factors, nh, mask, h_in, dy, dh, inj)) / (2 * eps)
        assert abs(fd - res["dx"][idx]) <= 1e-6 * max(1.0, abs(fd)), (idx, fd, res["dx"][idx])
    for path in _param_paths(w):
        wt = _get(w, path)
        flat = np.unravel_index(rng.integers(wt.size), wt.shape)
        wp, wm = wt.copy(), wt.copy()
        wp[flat] += eps
        wm[flat] -= eps
        fd = (_loss(x, _set(w, path, wp), factors, nh, mask, h_in, dy, dh, inj)
              - _loss(x, _set(w, path, wm), factors, nh, mask, h_in, dy, dh, inj)) / (2 * eps)
        g = _grad_of(res["grads"], path)[flat]
        assert abs(fd - g) <= 1e-6 * max(1.0, abs(fd)), (path, flat, fd, g)
