"""GPU parity of decode steps and prefill over seeded random shapes.

A fixed seed draws combinations the hand-picked cases leave out: 1-40
sequences, 1-4 heads of 64 or 128 channels (d_model * element size up to the
4 KB limit), one or two levels with factors in {1, 2, 3, 4, 8} (P <= 64) and
free middle widths, empty, short and long caches, and step counts that
cross block boundaries (so appends happen mid-run), in bf16 and fp32. Decode
outputs of every step, appended cache rows and the counters are compared with
the oracle; prefill of the same stream in one call, its state, and three
decode steps after it likewise.
"""
import dataclasses
import math

import numpy as np
import pytest

import oracle
from cache_cases import oracle_state
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape
from helpers import assert_close, dev, host
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
