"""GPU parity of decode steps and prefill over seeded random shapes.

A fixed seed draws combinations the hand-picked cases leave out: 1-40
sequences, 1-4 heads of 64 or 128 channels (d_model * element size up to the
4 KB limit), one or two levels with factors in {1, 2, 3, 4, 8} (P <= 64) and
free middle widths, empty, short and long caches, and step counts that
cross block boundaries (so appends happen mid-run), in bf16 and fp32. Decode
outputs of every step, appended cache rows and the counters are compared with
the oracle; prefill of the same stream in one call, its state, and three
decode steps after it likewise; batches with per-sequence positions
(random cache lengths and block fill), each sequence against the oracle
run on it alone; appends of many blocks at once; and a stream prefilled in
random chunks against one prefill, bit for bit.
"""
import dataclasses
import math

import numpy as np
import pytest

import oracle
from cache_cases import oracle_state
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape
from helpers import assert_close, dev, dev_weights, host
from test_gpu_decode import make_session, run_and_compare
from test_gpu_prefill import chunk, compare_state

pytestmark = pytest.mark.gpu

N_DECODE = 16
N_PREFILL = 12


def draw_shapes(n: int, seed: int):
    rng = np.random.default_rng(seed)
    shapes = []
    while len(shapes) < n:
        dtype = "fp32" if rng.random() < 0.3 else "bf16"
        dh = int(rng.choice([64, 128]))
        nh = int(rng.integers(1, 5))
        if nh * dh * (4 if dtype == "fp32" else 2) > 4096:
            continue
        levels = int(rng.integers(1, 3))
        factors = tuple(int(rng.choice([1, 2, 3, 4, 8])) for _ in range(levels))
        block = math.prod(factors)
        if block > 64:
            continue
        level_dims = tuple(8 * int(rng.integers(2, 33)) for _ in range(levels - 1))
        r = rng.random()
        n0 = 0 if r < 0.2 else int(rng.integers(1, 100)) if r < 0.6 else int(rng.integers(100, 2000))
        steps = int(rng.integers(1, 2 * block + 6))
        shapes.append(DecodeShape(int(rng.integers(1, 41)), nh * dh, nh, dh, factors, level_dims, n0=n0,
                                  steps=steps, dtype=dtype))
    return shapes


DECODE = draw_shapes(N_DECODE, 20261204)
# room for the three decode steps after the prefill (each may complete a block)
PREFILL = [dataclasses.replace(s, n_cap=s.n0 + (s.steps + 3) // s.block + 1)
           for s in draw_shapes(N_PREFILL, 20261205)]


@pytest.mark.parametrize("i", range(N_DECODE))
def test_decode_parity_random_shape(gpu, i):
    shape = DECODE[i]
    print(f"[random decode {i}] {shape}", flush=True)
    inp = synth.decode_inputs(shape, 3000 + i)
    run_and_compare(shape, inp, label=f"random decode {i}")


@pytest.mark.parametrize("i", range(N_PREFILL))
def test_prefill_parity_random_shape(gpu, i):
    import torch
    shape = PREFILL[i]
    print(f"[random prefill {i}] {shape}", flush=True)
    inp = synth.decode_inputs(shape, 4000 + i)
    xs = chunk(inp)
    sess = make_session(shape, inp)
    y = sess.prefill(dev(xs, shape.dtype))
    torch.cuda.synchronize()
    seqs = list(range(shape.batch))
    st = oracle_state(shape, inp, seqs)
    ref = oracle.prefill(st, inp["weights"], shape.factors, xs, shape.rms_eps)
    assert_close(host(y), ref, shape.dtype, f"random prefill {i} y")
    compare_state(sess, st, shape, seqs, inp["n0"], f"random prefill {i}")
    rng = np.random.default_rng(i)
    more = rng.standard_normal((3, shape.batch, shape.d_model)).astype(np.float32)
    if shape.dtype == "bf16":
        more = synth.bf16_round(more)
    got = [host(sess.step(dev(more[t], shape.dtype))) for t in range(3)]
    want = [oracle.decode_step(st, inp["weights"], shape.factors, more[t], shape.rms_eps) for t in range(3)]
    assert_close(np.stack(got), np.stack(want), shape.dtype, f"random prefill {i} decode after prefill")


N_RAGGED = 6


def draw_ragged(i: int):
    """A random batch with per-sequence positions: cache lengths 0..300,
    local-block fill 0..P-1, 1-64 sequences (the per-sequence limit)."""
    rng = np.random.default_rng(20261206 + i)
    while True:
        dtype = "fp32" if rng.random() < 0.3 else "bf16"
        dh = int(rng.choice([64, 128]))
        nh = int(rng.integers(1, 4))
        factors = tuple(int(rng.choice([1, 2, 3, 4, 8])) for _ in range(int(rng.integers(1, 3))))
        if math.prod(factors) <= 32:
            break
    P = math.prod(factors)
    b = int(rng.integers(1, 65))
    steps = int(rng.integers(1, 2 * P + 6))
    n0 = rng.integers(0, 300, size=b).astype(np.int64)
    n0[rng.random(b) < 0.2] = 0
    j0 = rng.integers(0, P, size=b).astype(np.int32)
    cap = int(n0.max()) + (steps + P) // P + 1
    shape = DecodeShape(b, nh * dh, nh, dh, factors, n0=0, steps=steps, n_cap=cap, dtype=dtype)
    return shape, n0, j0, rng


@pytest.mark.parametrize("i", range(N_RAGGED))
def test_ragged_decode_parity_random(gpu, i):
    """Per-sequence positions drawn at random; each sequence must match the
    oracle decoding that sequence alone, with its own appends."""
    import torch
    from paper_2608_23463_amd import binding as B
    shape, n0, j0, rng = draw_ragged(i)
    print(f"[random ragged {i}] {shape} n0={n0.tolist()} j0={j0.tolist()}", flush=True)
    P, h, dh, d, b = shape.block, shape.n_heads, shape.head_dim, shape.d_model, shape.batch
    inp = synth.decode_inputs(shape, 5000 + i)
    rnd = (lambda a: synth.bf16_round(a)) if shape.dtype == "bf16" else (lambda a: a)
    kc = rnd(rng.standard_normal((b, h, shape.capacity, dh)).astype(np.float32))
    vc = rnd(rng.standard_normal((b, h, shape.capacity, dh)).astype(np.float32))
    x_blk = rnd(rng.standard_normal((b, P, d)).astype(np.float32))
    k_loc = rnd(rng.standard_normal((b, h, P, dh)).astype(np.float32))
    v_loc = rnd(rng.standard_normal((b, h, P, dh)).astype(np.float32))
    cfg = B.decode_config(b, d, h, dh, shape.factors, (), shape.dtype, shape.rms_eps)
    sess = B.DecodeSession(cfg, dev_weights(inp["weights"], shape.dtype), dev(kc, shape.dtype),
                           dev(vc, shape.dtype), ragged=True, n_seq=n0, j_seq=j0)
    sess.x_blk.copy_(dev(x_blk, shape.dtype))
    sess.k_loc.copy_(dev(k_loc, shape.dtype))
    sess.v_loc.copy_(dev(v_loc, shape.dtype))
    got = np.stack([host(sess.step(dev(inp["x"][t], shape.dtype))) for t in range(shape.steps)])
    torch.cuda.synchronize()
    kc_after, vc_after = host(sess.k_cache), host(sess.v_cache)
    for s in range(b):
        st = oracle.DecodeState(kc[s:s + 1].astype(np.float64), vc[s:s + 1].astype(np.float64), int(n0[s]),
                                x_blk[s:s + 1].astype(np.float64), k_loc[s:s + 1].astype(np.float64),
                                v_loc[s:s + 1].astype(np.float64), int(j0[s]))
        ref = np.stack([oracle.decode_step(st, inp["weights"], shape.factors, inp["x"][t][s:s + 1], shape.rms_eps)
                        for t in range(shape.steps)])
        assert_close(got[:, s:s + 1], ref, shape.dtype, f"random ragged {i} sequence {s} y")
        assert sess.n_seq[s] == st.n and sess.j_seq[s] == st.j, (s, sess.n_seq[s], sess.j_seq[s], st.n, st.j)
        new = slice(int(n0[s]), st.n)
        assert_close(kc_after[s:s + 1, :, new], st.k_cache[:, :, new], shape.dtype, f"ragged {i}/{s} K rows")
        assert_close(vc_after[s:s + 1, :, new], st.v_cache[:, :, new], shape.dtype, f"ragged {i}/{s} V rows")
        assert np.array_equal(kc_after[s, :, st.n:], kc[s, :, st.n:])


N_APPEND = 6


@pytest.mark.parametrize("i", range(N_APPEND))
def test_append_parity_random(gpu, i):
    """proxy_cache_append of 1-80 whole blocks per sequence at once (the
    prefill of a history), random factorisation, widths and dtype."""
    import torch
    rng = np.random.default_rng(20261209 + i)
    while True:
        levels = int(rng.integers(1, 4))
        factors = tuple(int(rng.choice([1, 2, 3, 4, 8])) for _ in range(levels))
        if math.prod(factors) <= 64:
            break
    dtype = "fp32" if rng.random() < 0.3 else "bf16"
    dh = int(rng.choice([64, 128]))
    nh = int(rng.integers(1, 4))
    nblk = int(rng.integers(1, 81))
    n0 = int(rng.integers(0, 50))
    shape = DecodeShape(int(rng.integers(1, 20)), nh * dh, nh, dh, factors,
                        tuple(8 * int(rng.integers(2, 33)) for _ in range(levels - 1)),
                        n0=n0, steps=0, n_cap=n0 + nblk + 1, dtype=dtype)
    print(f"[random append {i}] {shape} nblk={nblk}", flush=True)
    inp = synth.decode_inputs(shape, 8000 + i)
    sess = make_session(shape, inp)
    xb = rng.standard_normal((shape.batch, nblk * shape.block, shape.d_model)).astype(np.float32)
    if dtype == "bf16":
        xb = synth.bf16_round(xb)
    sess.append(dev(xb, dtype), nblk)
    torch.cuda.synchronize()
    st = oracle_state(shape, inp, range(shape.batch))
    oracle.cache_append(st, inp["weights"], shape.factors, xb)
    assert sess.n == st.n == n0 + nblk
    assert_close(host(sess.k_cache)[:, :, :st.n], st.k_cache[:, :, :st.n], dtype, f"random append {i} K")
    assert_close(host(sess.v_cache)[:, :, :st.n], st.v_cache[:, :, :st.n], dtype, f"random append {i} V")


N_CHUNKED = 4


@pytest.mark.parametrize("i", range(N_CHUNKED))
def test_chunked_prefill_random(gpu, i):
    """A token stream prefilled in random chunks (whole blocks, then a ragged
    tail) gives the same outputs and state as one prefill, bit for bit."""
    import torch
    rng = np.random.default_rng(20261210 + i)
    factors = tuple(int(rng.choice([2, 4, 8])) for _ in range(int(rng.integers(1, 3))))
    P = math.prod(factors)
    nblocks = int(rng.integers(2, 12))
    tail = int(rng.integers(0, P))
    shape = DecodeShape(int(rng.integers(1, 6)), 128, 2, 64, factors, n0=int(rng.integers(0, 100)),
                        steps=nblocks * P + tail)
    print(f"[random chunked prefill {i}] {shape}", flush=True)
    inp = synth.decode_inputs(shape, 9000 + i)
    xs = dev(chunk(inp), shape.dtype)
    a = make_session(shape, inp)
    ya = a.prefill(xs)
    b = make_session(shape, inp)
    cuts = sorted(rng.choice(np.arange(1, nblocks), size=int(rng.integers(1, nblocks)), replace=False).tolist())
    edges = [0] + [c * P for c in cuts] + [shape.steps]
    parts = [b.prefill(xs[:, lo:hi].contiguous()) for lo, hi in zip(edges[:-1], edges[1:])]
    torch.cuda.synchronize()
    assert torch.equal(ya, torch.cat(parts, dim=1)), edges
    assert (a.n, a.j) == (b.n, b.j)
    n, j = a.n, a.j
    assert torch.equal(a.k_cache[:, :, :n], b.k_cache[:, :, :n]) and torch.equal(a.v_cache[:, :, :n], b.v_cache[:, :, :n])
    if j:
        assert torch.equal(a.x_blk[:, :j], b.x_blk[:, :j])
        assert torch.equal(a.k_loc[:, :, :j], b.k_loc[:, :, :j]) and torch.equal(a.v_loc[:, :, :j], b.v_loc[:, :, :j])
