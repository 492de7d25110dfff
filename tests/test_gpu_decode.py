"""GPU parity of the proxy-KV-cache decode step and the cache append.

The HIP path and the oracle decode the same seeded token stream from the same
initial cache; outputs of every step, the appended cache rows and the
counters n, j are compared (infinity-norm relative error, 1e-4 fp32, 2e-2
bf16). At the full 32 x 16,384-row workload the oracle follows a sample of
the sequences (sequences are independent).
"""
import numpy as np
import pytest

import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape
from helpers import assert_close, dev, dev_weights, host

pytestmark = pytest.mark.gpu


def make_session(shape, inp):
    from paper_2608_23463_amd import binding as B
    cfg = B.decode_config(shape.batch, shape.d_model, shape.n_heads, shape.head_dim, shape.factors,
                          shape.level_dims, shape.dtype, shape.rms_eps)
    w = dev_weights(inp["weights"], shape.dtype)
    kc = dev(inp["k_cache"], shape.dtype)
    vc = dev(inp["v_cache"], shape.dtype)
    return B.DecodeSession(cfg, w, kc, vc, n=inp["n0"])


def oracle_state(shape, inp, seqs):
    st = oracle.DecodeState.empty(len(seqs), shape.n_heads, shape.head_dim, shape.block, shape.capacity,
                                  shape.d_model)
    st.k_cache[:] = inp["k_cache"][seqs]
    st.v_cache[:] = inp["v_cache"][seqs]
    st.n = inp["n0"]
    return st


def run_and_compare(shape, inp, seqs=None, label=""):
    import torch
    seqs = list(range(shape.batch)) if seqs is None else list(seqs)
    sess = make_session(shape, inp)
    ys = []
    for t in range(shape.steps):
        ys.append(sess.step(dev(inp["x"][t], shape.dtype)))
    torch.cuda.synchronize()
    got = np.stack([host(y) for y in ys])[:, seqs]
    st = oracle_state(shape, inp, seqs)
    ref = np.stack([oracle.decode_step(st, inp["weights"], shape.factors, inp["x"][t][seqs], shape.rms_eps)
                    for t in range(shape.steps)])
    assert sess.n == st.n and sess.j == st.j
    assert_close(got, ref, shape.dtype, f"{label} y (all steps)")
    n0 = inp["n0"]
    if st.n > n0:
        kc = host(sess.k_cache)[seqs][:, :, n0:st.n]
        vc = host(sess.v_cache)[seqs][:, :, n0:st.n]
        assert_close(kc, st.k_cache[:, :, n0:st.n], shape.dtype, f"{label} appended K rows")
        assert_close(vc, st.v_cache[:, :, n0:st.n], shape.dtype, f"{label} appended V rows")
    return sess


CASES = {
    "bf16_small": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=11),
    "fp32_small": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=11, dtype="fp32"),
    "bf16_empty_cache": DecodeShape(2, 128, 2, 64, (8,), n0=0, steps=20),
    "bf16_dh128_factorised": DecodeShape(2, 256, 2, 128, (2, 4), level_dims=(192,), n0=3000, steps=17),
    "bf16_many_splits": DecodeShape(4, 512, 8, 64, (16,), n0=5000, steps=33),
    "bf16_lm_shape": DecodeShape(3, 512, 8, 64, (64,), n0=1100, steps=70),
}


@pytest.mark.parametrize("name", list(CASES))
def test_decode_parity_small(gpu, name):
    shape = CASES[name]
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.decode_inputs(shape, seed=sum(map(ord, name)))
    run_and_compare(shape, inp, label=name)


@pytest.mark.parametrize("name", ["decode_bf16_B32_n16k", "decode_bf16_B32_n16k_lm_d512"])
def test_decode_parity_full_workload_sampled(gpu, name):
    shape = synth.WORKLOADS[name]
    print(f"[workload {name}] generating inputs", flush=True)
    inp = synth.decode_inputs(shape, synth.WORKLOAD_SEEDS[name])
    run_and_compare(shape, inp, seqs=[0, 17, 31], label=name)


def test_append_matches_oracle(gpu):
    import torch
    shape = DecodeShape(4, 256, 4, 64, (8, 8), n0=2, steps=0, n_cap=40)
    inp = synth.decode_inputs(shape, 99)
    sess = make_session(shape, inp)
    rng = np.random.default_rng(1)
    nblk = 33
    xb = synth.bf16_round(rng.standard_normal((shape.batch, nblk * shape.block, shape.d_model)).astype(np.float32))
    sess.append(dev(xb, shape.dtype), nblk)
    torch.cuda.synchronize()
    st = oracle_state(shape, inp, range(shape.batch))
    oracle.cache_append(st, inp["weights"], shape.factors, xb)
    assert sess.n == st.n == 2 + nblk
    assert_close(host(sess.k_cache)[:, :, :st.n], st.k_cache[:, :, :st.n], "bf16", "append K")
    assert_close(host(sess.v_cache)[:, :, :st.n], st.v_cache[:, :, :st.n], "bf16", "append V")


def test_snapshot_restore_bitwise(gpu):
    """The caller-owned state is the whole inference state."""
    import torch
    from paper_2608_23463_amd import binding as B
    shape = DecodeShape(2, 128, 2, 64, (4,), n0=7, steps=10)
    inp = synth.decode_inputs(shape, 5)
    a = make_session(shape, inp)
    for t in range(6):
        a.step(dev(inp["x"][t], shape.dtype))
    b = make_session(shape, inp)
    for name in ("k_cache", "v_cache", "x_blk", "k_loc", "v_loc"):
        getattr(b, name).copy_(getattr(a, name))
    b.state.n, b.state.j = a.state.n, a.state.j
    for t in range(6, 10):
        ya = a.step(dev(inp["x"][t], shape.dtype))
        yb = b.step(dev(inp["x"][t], shape.dtype))
        torch.cuda.synchronize()
        assert torch.equal(ya, yb)


def test_ragged_positions_match_per_sequence_oracle(gpu):
    """Per-sequence positions: four sequences with different cache lengths and
    different fill of their current block decode together; each must match the
    oracle run on that sequence alone (blocks complete at different steps)."""
    import torch
    from paper_2608_23463_amd import binding as B
    shape = DecodeShape(4, 128, 2, 64, (8,), n0=0, steps=21, n_cap=24)
    P, h, dh, d = shape.block, shape.n_heads, shape.head_dim, shape.d_model
    inp = synth.decode_inputs(shape, 77)
    rng = np.random.default_rng(78)
    n0 = np.array([0, 5, 13, 2], dtype=np.int64)
    j0 = np.array([0, 3, 7, 5], dtype=np.int32)
    bf = synth.bf16_round
    kc = bf(rng.standard_normal((4, h, shape.capacity, dh)).astype(np.float32))
    vc = bf(rng.standard_normal((4, h, shape.capacity, dh)).astype(np.float32))
    x_blk = bf(rng.standard_normal((4, P, d)).astype(np.float32))
    k_loc = bf(rng.standard_normal((4, h, P, dh)).astype(np.float32))
    v_loc = bf(rng.standard_normal((4, h, P, dh)).astype(np.float32))
    cfg = B.decode_config(4, d, h, dh, shape.factors, (), "bf16", shape.rms_eps)
    sess = B.DecodeSession(cfg, dev_weights(inp["weights"], "bf16"), dev(kc, "bf16"), dev(vc, "bf16"),
                           ragged=True, n_seq=n0, j_seq=j0)
    sess.x_blk.copy_(dev(x_blk, "bf16"))
    sess.k_loc.copy_(dev(k_loc, "bf16"))
    sess.v_loc.copy_(dev(v_loc, "bf16"))
    ys = [host(sess.step(dev(inp["x"][t], "bf16"))) for t in range(shape.steps)]
    torch.cuda.synchronize()
    got = np.stack(ys)
    for b in range(4):
        st = oracle.DecodeState(kc[b:b + 1].astype(np.float64), vc[b:b + 1].astype(np.float64), int(n0[b]),
                                x_blk[b:b + 1].astype(np.float64), k_loc[b:b + 1].astype(np.float64),
                                v_loc[b:b + 1].astype(np.float64), int(j0[b]))
        ref = np.stack([oracle.decode_step(st, inp["weights"], shape.factors, inp["x"][t][b:b + 1], shape.rms_eps)
                        for t in range(shape.steps)])
        assert_close(got[:, b:b + 1], ref, "bf16", f"ragged sequence {b} y")
        assert sess.n_seq[b] == st.n and sess.j_seq[b] == st.j, (b, sess.n_seq[b], sess.j_seq[b], st.n, st.j)
        new = slice(int(n0[b]), st.n)
        assert_close(host(sess.k_cache)[b:b + 1, :, new], st.k_cache[:, :, new], "bf16", f"ragged {b} K rows")
        assert_close(host(sess.v_cache)[b:b + 1, :, new], st.v_cache[:, :, new], "bf16", f"ragged {b} V rows")
        # rows past the sequence's own length are untouched
        assert np.array_equal(host(sess.k_cache)[b, :, st.n:], kc[b, :, st.n:])


def test_ragged_mode_with_equal_positions_is_lockstep_bitwise(gpu):
    import torch
    shape = CASES["bf16_small"]
    inp = synth.decode_inputs(shape, 5)
    a = make_session(shape, inp)
    from paper_2608_23463_amd import binding as B
    cfg = B.decode_config(shape.batch, shape.d_model, shape.n_heads, shape.head_dim, shape.factors,
                          shape.level_dims, shape.dtype, shape.rms_eps)
    b = B.DecodeSession(cfg, dev_weights(inp["weights"], shape.dtype), dev(inp["k_cache"], shape.dtype),
                        dev(inp["v_cache"], shape.dtype), n=inp["n0"], ragged=True)
    for t in range(shape.steps):
        ya = a.step(dev(inp["x"][t], shape.dtype))
        yb = b.step(dev(inp["x"][t], shape.dtype))
        torch.cuda.synchronize()
        assert torch.equal(ya, yb), t
    assert all(b.n_seq == a.n) and all(b.j_seq == a.j)
    assert torch.equal(a.k_cache, b.k_cache) and torch.equal(a.v_cache, b.v_cache)
