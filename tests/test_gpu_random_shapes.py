"""GPU parity of the layer over seeded random shapes (through the C ABI).

The hand-picked cases elsewhere cover each feature on its own; here a fixed
seed draws combinations of them: dtype, 1-3 levels with factors in
{1, 2, 3, 4, 8} (P <= 64), widths that are multiples of 8 but mostly not of
the tiles, 1-3 heads of 64 or 128 channels, partial last blocks, all three
masks, all four injections, both precisions and both gate kernels, one or two
sequences, with and without H_in. Every shape is within the library's
documented limits; forward outputs and (for a subset) every gradient are
compared with the oracle at the usual tolerances. Random image layers (p x p
patches, Sec. 3.9) are checked forward and backward as well.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import LayerShape
from helpers import assert_close, dev, dev_weights, host
from test_gpu_backward import compare, run_gpu_backward

pytestmark = pytest.mark.gpu

N_FORWARD = 40
N_BACKWARD = 24


def draw_shapes(n: int, seed: int):
    rng = np.random.default_rng(seed)
    shapes = []
    while len(shapes) < n:
        dtype = "fp32" if rng.random() < 0.3 else "bf16"
        dh = int(rng.choice([64, 128]))
        nh = int(rng.integers(1, 4))
        d_f = 8 * int(rng.integers(1, 40))
        levels = int(rng.integers(1, 4))
        factors = tuple(int(rng.choice([1, 2, 3, 4, 8])) for _ in range(levels))
        block = math.prod(factors)
        if block > 64:
            continue
        level_dims = tuple(8 * int(rng.integers(2, 33)) for _ in range(levels - 1))
        # proxies: often a single attention tile, often several with a ragged last one
        m = int(rng.integers(1, 20)) if rng.random() < 0.5 else int(rng.integers(20, 300))
        tail = int(rng.integers(1, block)) if block > 1 and rng.random() < 0.4 else 0
        seq_len = (m - 1) * block + tail if tail else m * block
        injection = int(rng.integers(0, 4))
        if injection == synth.INJECT_GATED_HEAD and (d_f % nh or (d_f // nh) % 8):
            continue
        shapes.append(LayerShape(
            int(rng.integers(1, 3)), seq_len, d_f, nh * dh, nh, dh, factors, level_dims, dtype,
            mask=int(rng.integers(0, 3)), injection=injection,
            precision=int(rng.integers(0, 2)) if dtype == "bf16" else synth.PRECISION_EXTENDED,
            gate_fusion=int(rng.integers(0, 2)) if dtype == "bf16" and injection == synth.INJECT_GATED
            else synth.GATE_SEPARATE))
    return shapes


FORWARD = draw_shapes(N_FORWARD, 20261202)
BACKWARD = draw_shapes(N_BACKWARD, 20261203)


def sharpen(shape, inp):
    """Q/K weights x4 so that attention is far from uniform, except in plain
    bf16 precision, whose one rounding of Q and K moves a sharp softmax by
    about the tolerance itself (a documented property of that precision)."""
    if shape.dtype == "bf16" and shape.precision == synth.PRECISION_BF16:
        return
    for key in ("q", "k"):
        w, b = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(w * 4) if shape.dtype == "bf16" else w * 4, b)


def test_random_shapes_are_accepted():
    from paper_2608_23463_amd import binding as B
    B.load()
    for shape in FORWARD + BACKWARD:
        assert B.layer_workspace_size(B.config_from_shape(shape)) > 0, shape


@pytest.mark.parametrize("i", range(N_FORWARD))
def test_forward_parity_random_shape(gpu, i):
    from paper_2608_23463_amd import binding as B
    import torch
    shape = FORWARD[i]
    with_h = i % 2 == 0
    print(f"[random forward {i}] {shape} h_in={with_h}", flush=True)
    inp = synth.layer_inputs(shape, 1000 + i, with_h_in=with_h)
    sharpen(shape, inp)
    x_out, h_out, _ = B.layer_forward(B.config_from_shape(shape), dev_weights(inp["weights"], shape.dtype),
                                      dev(inp["x"], shape.dtype), dev(inp["h_in"], shape.dtype))
    torch.cuda.synchronize()
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask, inp["h_in"],
                               injection=shape.injection)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"random {i} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"random {i} x_out")


@pytest.mark.parametrize("i", range(N_BACKWARD))
def test_backward_parity_random_shape(gpu, i):
    shape = BACKWARD[i]
    with_h = i % 2 == 1
    print(f"[random backward {i}] {shape} h_in={with_h}", flush=True)
    inp = synth.layer_inputs(shape, 2000 + i, with_dy=True, with_h_in=with_h)
    sharpen(shape, inp)
    dh_out = None
    if with_h:
        rng = np.random.default_rng(i)
        dh_out = rng.standard_normal((shape.batch, shape.n_proxies, shape.d_proxy)).astype(np.float32)
        if shape.dtype == "bf16":
            dh_out = synth.bf16_round(dh_out)
    res = run_gpu_backward(shape, inp, dh_out)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask,
                                inp["h_in"], dh_out, injection=shape.injection)
    compare(shape, inp, res, ref, f"random {i}")


N_IMAGES = 8


def draw_image(i: int):
    """A random image layer (Sec. 3.9): p x p patches (p in 1..8), a grid of
    1..12 x 1..12 patches, random widths, heads, mask, injection and dtype."""
    rng = np.random.default_rng(20261207 + i)
    while True:
        dtype = "fp32" if rng.random() < 0.3 else "bf16"
        p = int(rng.integers(1, 9))
        gw, gh = int(rng.integers(1, 13)), int(rng.integers(1, 13))
        dh = int(rng.choice([64, 128]))
        nh = int(rng.integers(1, 4))
        d_f = 8 * int(rng.integers(1, 40))
        injection = int(rng.integers(0, 4))
        if injection == synth.INJECT_GATED_HEAD and (d_f % nh or (d_f // nh) % 8):
            continue
        return LayerShape(int(rng.integers(1, 3)), gw * p * gh * p, d_f, nh * dh, nh, dh, (p * p,), (), dtype,
                          mask=int(rng.integers(0, 3)), injection=injection, image_width=gw * p,
                          precision=int(rng.integers(0, 2)) if dtype == "bf16" else synth.PRECISION_EXTENDED)


@pytest.mark.parametrize("i", range(N_IMAGES))
def test_image_partition_parity_random(gpu, i):
    """Forward and backward of a random image layer against the oracle's
    gather -> layer -> scatter form."""
    from paper_2608_23463_amd import binding as B
    import torch
    shape = draw_image(i)
    print(f"[random image {i}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, 6000 + i, with_dy=True, with_h_in=True)
    sharpen(shape, inp)
    x_out, h_out, _ = B.layer_forward(B.config_from_shape(shape), dev_weights(inp["weights"], shape.dtype),
                                      dev(inp["x"], shape.dtype), dev(inp["h_in"], shape.dtype))
    torch.cuda.synchronize()
    ref = oracle.layer_forward_2d(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.image_width,
                                  shape.mask, inp["h_in"], injection=shape.injection)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"random image {i} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"random image {i} x_out")
    res = run_gpu_backward(shape, inp)
    refb = oracle.layer_backward_2d(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.image_width,
                                    inp["dy"], shape.mask, inp["h_in"], None, injection=shape.injection)
    compare(shape, inp, res, refb, f"random image {i}")


N_FUSED = 8


def draw_fused(i: int):
    """A random layer that takes the fused decompression + gate kernel (bf16,
    gated, d_fine a multiple of 128, level-1 input width a multiple of 64 and
    at least 128): 1-2 levels, partial blocks, all masks, both precisions."""
    rng = np.random.default_rng(20261208 + i)
    while True:
        levels = int(rng.integers(1, 3))
        factors = tuple(int(rng.choice([1, 2, 3, 4, 8])) for _ in range(levels))
        block = math.prod(factors)
        if block <= 64:
            break
    dh = int(rng.choice([64, 128]))
    nh = int(rng.integers(1, 4))
    level_dims = tuple(64 * int(rng.integers(2, 6)) for _ in range(levels - 1))
    m = int(rng.integers(1, 200))
    tail = int(rng.integers(1, block)) if block > 1 and rng.random() < 0.4 else 0
    return LayerShape(int(rng.integers(1, 3)), (m - 1) * block + tail if tail else m * block,
                      128 * int(rng.integers(1, 5)), nh * dh, nh, dh, factors, level_dims, "bf16",
                      mask=int(rng.integers(0, 3)), precision=int(rng.integers(0, 2)),
                      gate_fusion=synth.GATE_FUSED)


@pytest.mark.parametrize("i", range(N_FUSED))
def test_fused_gate_parity_random(gpu, i):
    """Forward and backward through the fused decompression + gate kernel
    (the forward saves Delta and G for the backward)."""
    from paper_2608_23463_amd import binding as B
    import torch
    shape = draw_fused(i)
    print(f"[random fused {i}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, 7000 + i, with_dy=True, with_h_in=i % 2 == 0)
    sharpen(shape, inp)
    x_out, h_out, _ = B.layer_forward(B.config_from_shape(shape), dev_weights(inp["weights"], shape.dtype),
                                      dev(inp["x"], shape.dtype), dev(inp["h_in"], shape.dtype))
    torch.cuda.synchronize()
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask, inp["h_in"])
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"random fused {i} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"random fused {i} x_out")
    res = run_gpu_backward(shape, inp)
    refb = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask,
                                 inp["h_in"], None)
    compare(shape, inp, res, refb, f"random fused {i}")
