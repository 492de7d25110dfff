"""GPU parity of the prefill (parallel form of the generation block, Eq. 19-20,
with the chunk's complete blocks appended, Eq. 21).

The HIP path and the oracle prefill the same seeded chunk from the same
initial cache: every output, the appended cache rows, the local slots of an
unfinished last block and the counters n, j are compared (infinity-norm
relative error, 1e-4 fp32, 2e-2 bf16); then both decode a few more tokens
from the prefilled state. At the full 32 x 4,096-token chunk the oracle
follows two sequences at sampled tokens (sequences are independent).
Cache rows past n start as NaN and must stay untouched.

The cache-sensitive cases (`cache_cases`: 16,500 cached rows, 258 key tiles
per head) also compare y - x; planted mistakes in the oracle (the cached
read dropped, one slice or one 64-key tile of cached rows left out) move it
by at least five times the tolerance (`test_parity_sensitivity.py`).
"""
import numpy as np
import pytest

import cache_cases as cc
import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape
from helpers import assert_close, dev, host
from cache_cases import oracle_state
from test_gpu_decode import assert_rows_untouched, make_session

pytestmark = pytest.mark.gpu

# `steps` is the chunk length T
CASES = {
    "bf16_small_ragged_tail": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=23),
    "fp32_small_ragged_tail": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=23, dtype="fp32"),
    "bf16_empty_cache_short_chunk": DecodeShape(2, 128, 2, 64, (8,), n0=0, steps=5),
    "bf16_empty_cache_whole_blocks": DecodeShape(2, 128, 2, 64, (8,), n0=0, steps=40),
    "bf16_dh128_factorised": DecodeShape(2, 256, 2, 128, (2, 4), level_dims=(192,), n0=300, steps=200),
    "bf16_lm_shape": DecodeShape(2, 512, 8, 64, (64,), n0=1100, steps=640),
    "bf16_small_blocks_many_tiles": DecodeShape(2, 256, 4, 64, (16,), n0=777, steps=300),
    "bf16_large_blocks": DecodeShape(2, 256, 4, 64, (16, 16), n0=130, steps=700),
    "fp32_dh128": DecodeShape(2, 256, 2, 128, (8,), n0=70, steps=150, dtype="fp32"),
    "bf16_batch_over_32": DecodeShape(35, 128, 2, 64, (4,), n0=6, steps=9),
    "bf16_max_width": DecodeShape(2, 2048, 16, 128, (4,), n0=20, steps=14),
}


def chunk(inp):
    """[steps, B, d] token stream -> [B, T, d] chunk."""
    return np.ascontiguousarray(inp["x"].transpose(1, 0, 2))


def compare_state(sess, st, shape, seqs, n0, label):
    assert sess.n == st.n and sess.j == st.j, (sess.n, sess.j, st.n, st.j)
    if st.n > n0:
        assert_close(host(sess.k_cache)[seqs][:, :, n0:st.n], st.k_cache[:, :, n0:st.n], shape.dtype,
                     f"{label} appended K rows")
        assert_close(host(sess.v_cache)[seqs][:, :, n0:st.n], st.v_cache[:, :, n0:st.n], shape.dtype,
                     f"{label} appended V rows")
    if st.j:
        j = st.j
        assert_close(host(sess.x_blk)[seqs][:, :j], st.x_blk[:, :j], shape.dtype, f"{label} x_blk")
        assert_close(host(sess.k_loc)[seqs][:, :, :j], st.k_loc[:, :, :j], shape.dtype, f"{label} k_loc")
        assert_close(host(sess.v_loc)[seqs][:, :, :j], st.v_loc[:, :, :j], shape.dtype, f"{label} v_loc")
    assert_rows_untouched(sess, seqs, st.n)


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_parity_small(gpu, name):
    import torch
    shape = CASES[name]
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.decode_inputs(shape, seed=sum(map(ord, name)) + 7)
    xs = chunk(inp)
    sess = make_session(shape, inp)
    y = sess.prefill(dev(xs, shape.dtype))
    torch.cuda.synchronize()
    seqs = list(range(shape.batch))
    st = oracle_state(shape, inp, seqs)
    ref = oracle.prefill(st, inp["weights"], shape.factors, xs, shape.rms_eps)
    assert_close(host(y), ref, shape.dtype, f"{name} y")
    compare_state(sess, st, shape, seqs, inp["n0"], name)
    # decoding continues from the prefilled state
    rng = np.random.default_rng(5)
    more = synth.bf16_round(rng.standard_normal((3, shape.batch, shape.d_model)).astype(np.float32))
    got = [host(sess.step(dev(more[t], shape.dtype))) for t in range(3)]
    want = [oracle.decode_step(st, inp["weights"], shape.factors, more[t], shape.rms_eps) for t in range(3)]
    assert_close(np.stack(got), np.stack(want), shape.dtype, f"{name} decode after prefill")
    assert sess.n == st.n and sess.j == st.j


def test_prefill_in_whole_block_chunks_equals_one_chunk(gpu):
    """Two chunks of whole blocks reproduce one chunk of both, bit for bit
    (every output depends only on its own block and the cache rows)."""
    import torch
    shape = DecodeShape(2, 256, 4, 64, (16,), n0=40, steps=96)
    inp = synth.decode_inputs(shape, 31)
    xs = dev(chunk(inp), shape.dtype)
    a = make_session(shape, inp)
    ya = a.prefill(xs)
    b = make_session(shape, inp)
    y1 = b.prefill(xs[:, :64].contiguous())
    y2 = b.prefill(xs[:, 64:].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(ya, torch.cat([y1, y2], dim=1))
    assert (a.n, a.j) == (b.n, b.j) == (40 + 6, 0)
    n = a.n  # rows past n start as NaN and are not state
    assert torch.equal(a.k_cache[:, :, :n], b.k_cache[:, :, :n]) and torch.equal(a.v_cache[:, :, :n], b.v_cache[:, :, :n])


@pytest.mark.parametrize("name", ["prefill_bf16_B32_T4096_n16k"])
def test_prefill_parity_full_workload_sampled(gpu, name):
    import torch
    shape = synth.WORKLOADS[name]
    print(f"[workload {name}] generating inputs", flush=True)
    inp = synth.decode_inputs(shape, synth.WORKLOAD_SEEDS[name])
    xs = chunk(inp)
    sess = make_session(shape, inp)
    print(f"[workload {name}] prefill", flush=True)
    y = sess.prefill(dev(xs, shape.dtype))
    torch.cuda.synchronize()
    seqs = [0, 31]
    T, P = shape.steps, shape.block
    rng = np.random.default_rng(11)
    toks = sorted({0, 1, P - 1, P, P + 1, 2047, 2048 + 37, T - 2, T - 1} | set(rng.integers(0, T, 7).tolist()))
    got = host(y[seqs][:, toks])
    st = oracle_state(shape, inp, seqs)
    print(f"[workload {name}] oracle on sequences {seqs}, tokens {toks}", flush=True)
    ref = oracle.prefill(st, inp["weights"], shape.factors, xs[seqs], shape.rms_eps, tokens=toks)
    assert_close(got, ref, shape.dtype, f"{name} y (sampled)")
    compare_state(sess, st, shape, seqs, inp["n0"], name)


@pytest.mark.parametrize("name", list(cc.PREFILL_CASES))
def test_prefill_parity_cache_sensitive(gpu, name):
    """Every output (y and y - x), appended rows, local slots and counters."""
    import torch
    shape = cc.PREFILL_CASES[name]
    print(f"[cache-sensitive prefill {name}] {shape}", flush=True)
    inp = cc.build(shape, name, cc.prefill_seed(name))
    xs = cc.chunk(inp)
    sess = make_session(shape, inp)
    y = sess.prefill(dev(xs, shape.dtype))
    torch.cuda.synchronize()
    seqs = list(range(shape.batch))
    ref, st = cc.oracle_prefill(shape, inp)
    got = host(y)
    assert_close(got, ref, shape.dtype, f"{name} y")
    assert_close(got - xs, ref - xs, shape.dtype, f"{name} y - x")
    compare_state(sess, st, shape, seqs, inp["n0"], name)
