"""GPU parity of the proxy-KV-cache decode step and the cache append.

The HIP path and the oracle decode the same seeded token stream from the same
initial cache; outputs of every step, the appended cache rows and the
counters n, j are compared (infinity-norm relative error, 1e-4 fp32, 2e-2
bf16). At the full 32 x 16,384-row workload the oracle follows a sample of
the sequences (sequences are independent). Cache rows past n start as NaN
and must stay untouched (the outputs, workspace and local slots start as NaN
too: the gpu fixture turns on the binding's NaN-filled allocation).

The cache-sensitive cases (`cache_cases`) make the cached read alpha * A_h
of Eq. 19-20 carry the output and also compare the sublayer output y - x;
planted mistakes in the oracle (the cached read dropped, one slice of 1,024
cached rows left out) move y - x by at least five times the tolerance
(`test_parity_sensitivity.py`). With the workload's own weights y - x is
small next to x and its bf16 rounding alone would exceed the tolerance, so
the other cases compare y.
"""
import numpy as np
import pytest

import cache_cases as cc
from cache_cases import oracle_state
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
    # capacity past the valid rows is never read: it starts as NaN
    kc[:, :, inp["n0"]:] = float("nan")
    vc[:, :, inp["n0"]:] = float("nan")
    return B.DecodeSession(cfg, w, kc, vc, n=inp["n0"])


def assert_rows_untouched(sess, seqs, n):
    """Cache rows at or past n were not written (they still hold NaN)."""
    import torch
    for c in (sess.k_cache, sess.v_cache):
        assert bool(torch.isnan(c[seqs][:, :, n:].float()).all()), "a cache row past n was written"


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
    assert_rows_untouched(sess, seqs, st.n)
    return sess


CASES = {
    "bf16_small": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=11),
    "fp32_small": DecodeShape(3, 128, 2, 64, (4,), n0=5, steps=11, dtype="fp32"),
    "bf16_empty_cache": DecodeShape(2, 128, 2, 64, (8,), n0=0, steps=20),
    "bf16_dh128_factorised": DecodeShape(2, 256, 2, 128, (2, 4), level_dims=(192,), n0=3000, steps=17),
    "bf16_many_splits": DecodeShape(4, 512, 8, 64, (16,), n0=5000, steps=33),
    "bf16_lm_shape": DecodeShape(3, 512, 8, 64, (64,), n0=1100, steps=70),
    # 37 sequences: the projection kernel's second 32-row block holds 5 rows
    "bf16_batch_over_32": DecodeShape(37, 128, 2, 64, (4,), n0=9, steps=6),
    # the widest rows a step takes (d_model * element size = 4 KB): four 16-byte chunks per
    # lane when the projection kernel stages x, and (bf16) a second chunk of weight fragments
    "bf16_max_width": DecodeShape(2, 2048, 16, 128, (4,), n0=40, steps=9),
    "fp32_max_width": DecodeShape(2, 1024, 8, 128, (4,), n0=40, steps=9, dtype="fp32"),
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
    n = a.n  # rows past n are not state (a's start as NaN)
    assert torch.equal(a.k_cache[:, :, :n], b.k_cache[:, :, :n]) and torch.equal(a.v_cache[:, :, :n], b.v_cache[:, :, :n])



@pytest.mark.parametrize("name,cut", [("bf16_batch_over_32", 32), ("bf16_batch_over_32", 17), ("fp32_small", 1),
                                      ("bf16_lm_shape", 2)])
def test_batch_split_is_bitwise_invariant(gpu, name, cut):
    """Sequences are independent (Eq. 19-21 act per sequence): decoding the
    batch as two sessions of cut and B - cut sequences, each on its own
    stream and running concurrently, gives the one-session outputs and cache
    rows bit for bit (appends included); a row of one sequence read or
    written for another, or the 32-row blocks of the projections mixing
    rows, would show here."""
    import torch
    from paper_2608_23463_amd import binding as B
    shape = CASES[name]
    inp = synth.decode_inputs(shape, 11)
    full = make_session(shape, inp)
    w = dev_weights(inp["weights"], shape.dtype)
    kc, vc = full.k_cache.clone(), full.v_cache.clone()
    halves = []
    for lo, hi in ((0, cut), (cut, shape.batch)):
        cfg = B.decode_config(hi - lo, shape.d_model, shape.n_heads, shape.head_dim, shape.factors,
                              shape.level_dims, shape.dtype, shape.rms_eps)
        halves.append((B.DecodeSession(cfg, w, kc[lo:hi], vc[lo:hi], n=inp["n0"]), lo, hi, torch.cuda.Stream()))
    main = torch.cuda.current_stream()
    for t in range(shape.steps):
        x = dev(inp["x"][t], shape.dtype)
        y_full = full.step(x)
        y_split = torch.full_like(x, float("nan"))
        start = torch.cuda.Event()
        start.record(main)
        for sess, lo, hi, stream in halves:
            stream.wait_event(start)
            with torch.cuda.stream(stream):
                sess.step(x[lo:hi], y_split[lo:hi], stream=stream)
        for _, _, _, stream in halves:
            done = torch.cuda.Event()
            done.record(stream)
            main.wait_event(done)
        torch.cuda.synchronize()
        assert torch.equal(y_full, y_split), f"{name} cut {cut}: step {t}"
    n = full.n
    assert all(sess.n == n and sess.j == full.j for sess, _, _, _ in halves)
    assert torch.equal(full.k_cache[:, :, :n], kc[:, :, :n]) and torch.equal(full.v_cache[:, :, :n], vc[:, :, :n])


def run_gpu_steps(shape, inp):
    import torch
    sess = make_session(shape, inp)
    ys = [sess.step(dev(inp["x"][t], shape.dtype)) for t in range(shape.steps)]
    torch.cuda.synchronize()
    return sess, np.stack([host(y) for y in ys])


@pytest.mark.parametrize("name", list(cc.DECODE_CASES))
def test_decode_parity_cache_sensitive(gpu, name):
    """17 cache slices; y and y - x against the oracle, appended rows, counters."""
    shape = cc.DECODE_CASES[name]
    print(f"[cache-sensitive decode {name}] {shape}", flush=True)
    inp = cc.build(shape, name, cc.decode_seed(name))
    sess, got = run_gpu_steps(shape, inp)
    ref, st = cc.oracle_decode(shape, inp)
    x = inp["x"].astype(np.float64)
    assert_close(got, ref, shape.dtype, f"{name} y")
    assert_close(got - x, ref - x, shape.dtype, f"{name} y - x")
    assert sess.n == st.n and sess.j == st.j
    n0 = inp["n0"]
    assert st.n > n0
    assert_close(host(sess.k_cache)[:, :, n0:st.n], st.k_cache[:, :, n0:st.n], shape.dtype, f"{name} appended K")
    assert_close(host(sess.v_cache)[:, :, n0:st.n], st.v_cache[:, :, n0:st.n], shape.dtype, f"{name} appended V")
    assert_rows_untouched(sess, list(range(shape.batch)), st.n)


def test_decode_alpha_off_ignores_the_cache(gpu):
    """b_alpha = -40 gives alpha < 1e-16 (Eq. 20): the output must equal the
    oracle decoding from an EMPTY initial cache, whatever the 16,500 cached
    rows hold (the block appended on the way is compared as well)."""
    shape = cc.DECODE_CASES["sharp"]
    inp = cc.build(shape, "sharp", cc.decode_seed("sharp") + 1)
    inp["weights"]["alpha"] = (inp["weights"]["alpha"][0], np.full(shape.n_heads, -40.0, np.float32))
    sess, got = run_gpu_steps(shape, inp)
    empty = dict(inp)
    empty["k_cache"] = np.zeros_like(inp["k_cache"])
    empty["v_cache"] = np.zeros_like(inp["v_cache"])
    empty["n0"] = 0
    ref, st = cc.oracle_decode(shape, empty)
    x = inp["x"].astype(np.float64)
    assert_close(got, ref, shape.dtype, "alpha off: y")
    assert_close(got - x, ref - x, shape.dtype, "alpha off: y - x")
    assert sess.n == inp["n0"] + st.n and sess.j == st.j
    n0 = inp["n0"]
    assert_close(host(sess.k_cache)[:, :, n0:n0 + st.n], st.k_cache[:, :, :st.n], shape.dtype, "alpha off: appended K")


def test_decode_constant_cached_values_closed_form(gpu):
    """Every cached value row of (sequence, head) equal to one vector c gives
    A_h = c whatever the attention weights (softmax rows sum to 1), so
    y = y_without_cache + (alpha * c) W_o^T over all 17 slices; alpha is
    sigmoid(RMSNorm(x) W_alpha^T + b_alpha) (Eq. 20). No block completes."""
    base = cc.DECODE_CASES["sharp"]
    shape = DecodeShape(base.batch, base.d_model, base.n_heads, base.head_dim, base.factors, n0=base.n0,
                        steps=base.block - 1)
    inp = cc.build(shape, "sharp", cc.decode_seed("sharp") + 2)
    rng = np.random.default_rng(3)
    c = synth.bf16_round(rng.standard_normal((shape.batch, shape.n_heads, 1, shape.head_dim)).astype(np.float32))
    inp["v_cache"][:, :, :shape.n0] = c
    sess, got = run_gpu_steps(shape, inp)
    empty = dict(inp)
    empty["n0"] = 0
    y0, _ = cc.oracle_decode(shape, empty)
    w = {k: v for k, v in inp["weights"].items()}
    wa, ba = (np.asarray(a, np.float64) for a in w["alpha"])
    wo = np.asarray(w["o"][0], np.float64)
    ref = np.zeros_like(y0)
    for t in range(shape.steps):
        u = oracle.rms_norm(inp["x"][t], w["rms_gamma"], shape.rms_eps)
        alpha = oracle.sigmoid(u @ wa.T + ba)                                   # [B, h]
        ah = (alpha[:, :, None] * c[:, :, 0, :]).reshape(shape.batch, shape.d_model)
        ref[t] = y0[t] + ah @ wo.T
    x = inp["x"].astype(np.float64)
    assert_close(got, ref, shape.dtype, "constant V: y")
    assert_close(got - x, ref - x, shape.dtype, "constant V: y - x")
    assert sess.n == shape.n0 and sess.j == shape.steps
