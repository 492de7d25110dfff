"""proxy_decode_step_static, the decode step that allocates nothing, against
proxy_decode_step with a caller workspace (through the C ABI).

Two sessions decode the same tokens from the same state, one through each
entry point; outputs, counters and caches must be bit-identical (the two
share every kernel). Two calls in a row, the second on a smaller shape
(fewer sequences, narrower model, shorter cache), each starting two tokens
before the end of a block, so a step appends a block through the static
scratch too. The static scratch keeps the previous call's contents, so the
second call also shows that nothing in it needs clearing.
"""
import numpy as np
import pytest

from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape
from helpers import dev
from test_gpu_decode import make_session

pytestmark = pytest.mark.gpu

CALLS = [
    ("32 x 1024, 16,384 rows", DecodeShape(32, 1024, 16, 64, (64,), n0=16384, steps=3)),
    ("3 x 256, 2,000 rows", DecodeShape(3, 256, 4, 64, (16,), n0=2000, steps=3)),
]


def test_static_scratch_step_matches_workspace_step(gpu):
    import torch
    for label, shape in CALLS:
        print(f"[no-alloc decode] {label}", flush=True)
        inp = synth.decode_inputs(shape, 9000 + shape.batch)
        a = make_session(shape, inp)
        b = make_session(shape, inp)
        j0 = shape.block - 2
        rng = np.random.default_rng(shape.batch)
        for name in ("x_blk", "k_loc", "v_loc"):
            slots = getattr(a, name)
            full = synth.bf16_round(rng.standard_normal(tuple(slots.shape)).astype(np.float32))
            val = dev(full, shape.dtype)
            getattr(a, name).copy_(val)
            getattr(b, name).copy_(val)
        a.state.j = b.state.j = j0
        for t in range(shape.steps):
            x_t = dev(inp["x"][t], shape.dtype)
            ya = a.step(x_t)
            yb = b.step_static(x_t)
            torch.cuda.synchronize()
            assert torch.equal(ya, yb), (label, t)
        assert (a.n, a.j) == (b.n, b.j) == (shape.n0 + 1, (j0 + shape.steps) % shape.block)
        n = a.n
        assert torch.equal(a.k_cache[:, :, :n], b.k_cache[:, :, :n]), label
        assert torch.equal(a.v_cache[:, :, :n], b.v_cache[:, :, :n]), label
