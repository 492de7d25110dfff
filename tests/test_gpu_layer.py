"""GPU parity of the layer forward against the CPU oracle (through the C ABI).

Every case runs the HIP path and the oracle on the same seeded inputs and
compares whole output tensors with the infinity-norm relative error
(1e-4 for fp32, 2e-2 for bf16, fp32 accumulation), plus bit-exact
invariants (causality, zero decompression, run-to-run determinism).
"""
import zlib

import numpy as np
import pytest

import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import LayerShape
from helpers import assert_close, dev, dev_weights, host

pytestmark = pytest.mark.gpu

SMALL = {
    # ragged: m = 37 proxies (not a multiple of any tile), d = 192 (3 heads)
    "bf16_ragged_tc": (LayerShape(2, 37 * 16, 192, 192, 3, 64, (16,)), True),
    "bf16_ragged_bc": (LayerShape(1, 37 * 16, 192, 192, 3, 64, (16,), mask=synth.BLOCK_CAUSAL), False),
    "bf16_ragged_bi": (LayerShape(1, 37 * 16, 192, 192, 3, 64, (16,), mask=synth.BIDIRECTIONAL), True),
    "fp32_ragged_tc": (LayerShape(2, 37 * 16, 192, 192, 3, 64, (16,), dtype="fp32"), True),
    "bf16_factorised": (LayerShape(1, 64 * 70, 128, 256, 2, 128, (4, 2, 8), level_dims=(96, 160)), True),
    "fp32_factorised": (LayerShape(1, 8 * 40, 64, 128, 1, 128, (2, 4), level_dims=(48,), dtype="fp32"), False),
    "bf16_dfine_ne_dproxy": (LayerShape(1, 64 * 300, 64, 512, 8, 64, (64,)), False),
    "bf16_single_block": (LayerShape(1, 64, 128, 128, 2, 64, (64,)), False),
    "bf16_block1": (LayerShape(1, 200, 64, 128, 2, 64, (1,)), False),
    # residual-add injection (Eq. 11): the decompression epilogue writes Y = X + Delta
    "bf16_inject_add": (LayerShape(2, 37 * 16, 192, 192, 3, 64, (16,), injection=synth.INJECT_ADD), True),
    "fp32_inject_add_factorised": (LayerShape(1, 8 * 40, 64, 128, 1, 128, (2, 4), level_dims=(48,), dtype="fp32",
                                              injection=synth.INJECT_ADD), False),
    # affine modulation (Eq. 13): [S | T] from Delta, Y = (1 + S) Norm(X) + T in the GEMM epilogue
    "bf16_inject_affine": (LayerShape(2, 37 * 16, 192, 192, 3, 64, (16,), injection=synth.INJECT_AFFINE), True),
    "fp32_inject_affine_factorised_bi": (LayerShape(1, 8 * 40, 64, 128, 1, 128, (2, 4), level_dims=(48,),
                                                    dtype="fp32", mask=synth.BIDIRECTIONAL,
                                                    injection=synth.INJECT_AFFINE), False),
    # per-head gate (Eq. 12 with the per-head weighting of Eq. 20): N = n_heads gate GEMM + combine
    "bf16_inject_gated_head": (LayerShape(2, 37 * 16, 192, 192, 3, 64, (16,), injection=synth.INJECT_GATED_HEAD),
                               True),
    "fp32_gated_head_factorised": (LayerShape(1, 8 * 40, 64, 128, 2, 64, (2, 4), level_dims=(48,), dtype="fp32",
                                              injection=synth.INJECT_GATED_HEAD), False),
    "bf16_gated_head_lm_shape": (LayerShape(1, 64 * 300, 64, 512, 8, 64, (64,), injection=synth.INJECT_GATED_HEAD),
                                 False),
    # d_fine = 3072: a row is 384 runs of 8, more than one combine block covers at a time
    "bf16_gated_head_wide": (LayerShape(1, 16 * 24, 3072, 256, 4, 64, (16,), injection=synth.INJECT_GATED_HEAD),
                             False),
    # partial last block (L % P != 0, m = ceil(L / P), zero-padded, Sec. 3.1)
    "bf16_partial_block_tc": (LayerShape(2, 37 * 16 + 5, 192, 192, 3, 64, (16,)), True),
    "fp32_partial_block_factorised_bi": (LayerShape(1, 8 * 40 + 3, 64, 128, 1, 128, (2, 4), level_dims=(48,),
                                                    dtype="fp32", mask=synth.BIDIRECTIONAL), False),
    "bf16_shorter_than_one_block": (LayerShape(1, 40, 128, 128, 2, 64, (64,), mask=synth.BLOCK_CAUSAL), True),
    # the fused decompression + gate kernel (bf16, gated, d_fine a multiple of 128, level-1
    # input width a multiple of 64): 74 ragged rows of 16 positions; a factorised cascade
    # whose level 1 (k_1 = 4, d_1 = 128) runs fused after two unfused levels
    "bf16_fused_gate_ragged_tc": (LayerShape(2, 37 * 16, 256, 192, 3, 64, (16,), gate_fusion=synth.GATE_FUSED),
                                  True),
    "bf16_fused_gate_factorised_bi": (LayerShape(1, 64 * 70, 128, 256, 2, 128, (4, 2, 8), level_dims=(128, 192),
                                                 mask=synth.BIDIRECTIONAL, gate_fusion=synth.GATE_FUSED), True),
    # d_fine a multiple of 8 but not of the K tile (72 bf16, 40 fp32): the gate's [X | Delta]
    # split falls inside a K tile, and the gate GEMM (N = d_fine) has a partial column tile
    "bf16_odd_width": (LayerShape(2, 37 * 16, 72, 128, 2, 64, (16,)), True),
    "fp32_odd_width": (LayerShape(1, 37 * 16, 40, 128, 2, 64, (16,), dtype="fp32"), True),
}


def run_gpu(shape, inp, save=False):
    from paper_2608_23463_amd import binding as B
    cfg = B.config_from_shape(shape)
    x = dev(inp["x"], shape.dtype)
    h_in = dev(inp["h_in"], shape.dtype)
    w = dev_weights(inp["weights"], shape.dtype)
    x_out, h_out, saved = B.layer_forward(cfg, w, x, h_in, save=save)
    import torch
    torch.cuda.synchronize()
    return x_out, h_out


@pytest.mark.parametrize("name", list(SMALL))
def test_forward_parity_small(gpu, name):
    shape, with_h = SMALL[name]
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, seed=zlib.crc32(name.encode()) % 1000, with_h_in=with_h)
    # larger weights than the workload's 0.02 so that attention is not uniform
    rng = np.random.default_rng(7)
    for key in ("q", "k"):
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 4) if shape.dtype == "bf16" else wq * 4, bq)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask, inp["h_in"],
                               injection=shape.injection)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")


BIASED = {
    # fused gate (d_fine 256) and unfused (d_fine 192; fp32) with every bias drawn
    "bf16_fused_gate": LayerShape(2, 29 * 16, 256, 128, 2, 64, (16,), gate_fusion=synth.GATE_FUSED),
    "bf16_fused_gate_factorised": LayerShape(1, 40 * 8, 128, 128, 2, 64, (2, 4), level_dims=(128,),
                                             gate_fusion=synth.GATE_FUSED),
    "bf16_separate_gate": LayerShape(2, 29 * 16, 256, 128, 2, 64, (16,)),
    "bf16_unfused": LayerShape(2, 29 * 16, 192, 128, 2, 64, (16,)),
    "fp32_unfused": LayerShape(1, 29 * 16, 128, 128, 2, 64, (16,), dtype="fp32"),
}


def draw_biases(shape, inp, seed):
    """Non-zero biases (std 0.5) in every linear map (the workloads' are zero)
    and W_o scaled by 8 (exact in bf16), so the injected signal X_out - X is
    as large as X and a dropped decompression or gate bias moves it by a few
    percent."""
    rng = np.random.default_rng(seed)
    w = inp["weights"]
    w["o"] = (w["o"][0] * np.float32(8), w["o"][1])

    def b(n):
        v = (rng.standard_normal(n) * 0.5).astype(np.float32)
        return synth.bf16_round(v) if shape.dtype == "bf16" else v
    for key in ("compress", "decompress"):
        w[key] = [(wm, b(wm.shape[0])) for wm, _ in w[key]]
    for key in ("q", "k", "v", "o", "gate"):
        w[key] = (w[key][0], b(w[key][0].shape[0]))


@pytest.mark.parametrize("name", list(BIASED))
def test_forward_parity_with_biases(gpu, name):
    shape = BIASED[name]
    print(f"[case {name}, biases drawn] {shape}", flush=True)
    inp = synth.layer_inputs(shape, zlib.crc32(name.encode()) % 1000, with_h_in=True)
    draw_biases(shape, inp, 17)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask, inp["h_in"])
    x = inp["x"].astype(np.float64)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")
    assert_close(host(x_out) - x, ref["x_out"] - x, shape.dtype, f"{name} x_out - x")


# Four sequences x 16 heads over 1,000-1,024 proxies (a grid of 512
# attention workgroups, more than the chip holds at once); m = 1000 leaves a
# ragged last query tile and a partial last key tile.
INJECTED = {
    "bf16_many_heads_tc": LayerShape(4, 16 * 1000, 64, 1024, 16, 64, (16,)),
    "bf16_many_heads_bc": LayerShape(4, 16 * 1024, 64, 1024, 16, 64, (16,), mask=synth.BLOCK_CAUSAL),
    "bf16_many_heads_bi": LayerShape(4, 16 * 1000, 64, 1024, 16, 64, (16,), mask=synth.BIDIRECTIONAL),
    # the factorised 256K-token workload's heads (16 x 128, d_proxy = 2048, P = 8 x 8) over
    # 1,000 proxies: eight 128-query workgroups per head, the last one ragged
    "bf16_dh128_heads_tc": LayerShape(2, 64 * 1000, 64, 2048, 16, 128, (8, 8)),
    "bf16_dh128_heads_bc": LayerShape(2, 64 * 1000, 64, 2048, 16, 128, (8, 8), mask=synth.BLOCK_CAUSAL),
    "bf16_dh128_heads_bi": LayerShape(2, 64 * 1000, 64, 2048, 16, 128, (8, 8), mask=synth.BIDIRECTIONAL),
}


@pytest.mark.parametrize("name", list(INJECTED))
def test_forward_parity_injected_signal(gpu, name):
    """The injected signal X_out - X (which carries the attention output
    through W_o and the decompression) is compared as well as X_out, so an
    attention error cannot hide behind the residual. W_o is scaled by 8 (exact
    in bf16) so that signal is as large as X: otherwise the bf16 rounding of
    X_out alone (half a unit in the last place of |X_out| ~ 5) is a few
    percent of it."""
    shape = INJECTED[name]
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, seed=zlib.crc32(name.encode()) % 1000, with_h_in=True)
    for key in ("q", "k"):  # logits with std of a few units: attention neither uniform nor one-hot
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 2), bq)
    wo, bo = inp["weights"]["o"]
    inp["weights"]["o"] = (wo * 8, bo)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask, inp["h_in"])
    x = inp["x"].astype(np.float64)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")
    assert_close(host(x_out) - x, ref["x_out"] - x, shape.dtype, f"{name} x_out - x")


@pytest.mark.parametrize("name", ["layer_fp32_L4k_d256", "layer_bf16_L64k_d1024"])
def test_forward_parity_workload(gpu, name):
    shape = synth.WORKLOADS[name]
    print(f"[workload {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")


@pytest.mark.parametrize("name", ["layer_bf16_L1M_d1024", "layer_bf16_L1M_lm_df64_dp512",
                                  "layer_bf16_L256k_d2048_f8x8"])
def test_forward_parity_L1M_sampled(gpu, name):
    """Full-size layers (1M tokens; the factorised 256K-token workload with
    4,096 proxies over 16 heads of 128): every proxy, and 64 sampled blocks
    of X_out."""
    shape = synth.WORKLOADS[name]
    print(f"[workload {name}] generating inputs", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    x_out, h_out = run_gpu(shape, inp)
    m = shape.n_proxies
    rng = np.random.default_rng(123)
    blocks = sorted(set([0, 1, m - 2, m - 1] + list(rng.choice(np.arange(2, m - 2), 60, replace=False))))
    print(f"[workload {name}] oracle on {len(blocks)} sampled blocks", flush=True)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask,
                               sample_blocks=blocks)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out (all proxies)")
    got = host(x_out.reshape(1, m, shape.block, shape.d_fine)[:, blocks])
    assert_close(got, ref["x_out"], shape.dtype, f"{name} x_out (sampled blocks)")


@pytest.mark.parametrize("name", ["layer_bf16_L64k_d1024", "layer_bf16_L1M_d1024", "layer_bf16_L1M_lm_df64_dp512"])
def test_forward_parity_plain_bf16_precision(gpu, name):
    """PF_PRECISION_BF16: H, Q and K as plain bf16 values (one score MFMA per
    tile step). The 64K-token layer in full; the 1M-token layers on every
    proxy and 64 sampled blocks."""
    import dataclasses
    shape = dataclasses.replace(synth.WORKLOADS[name], precision=synth.PRECISION_BF16)
    print(f"[workload {name}, plain bf16] generating inputs", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    x_out, h_out = run_gpu(shape, inp)
    m = shape.n_proxies
    blocks = None
    if shape.seq_len > 65536:
        rng = np.random.default_rng(321)
        blocks = sorted(set([0, 1, m - 2, m - 1] + list(rng.choice(np.arange(2, m - 2), 60, replace=False))))
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask,
                               sample_blocks=blocks)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} plain bf16 h_out")
    got = host(x_out) if blocks is None else host(x_out.reshape(1, m, shape.block, shape.d_fine)[:, blocks])
    assert_close(got, ref["x_out"], shape.dtype, f"{name} plain bf16 x_out")


def test_extended_precision_beats_plain_bf16(gpu):
    """The correction products of PF_PRECISION_EXTENDED are applied: on the
    64K-token layer (logit std ~11, where one bf16 rounding of Q and K moves
    the softmax by percents) the extended output is at least twice as close
    to the fp64 oracle as the plain-bf16 output of the same inputs. Both
    pass 2e-2, so a correction that silently dropped out would pass every
    tolerance check but not this one."""
    import dataclasses
    name = "layer_bf16_L64k_d1024"
    shape = synth.WORKLOADS[name]
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask)
    errs = {}
    for prec in (synth.PRECISION_EXTENDED, synth.PRECISION_BF16):
        x_out, _ = run_gpu(dataclasses.replace(shape, precision=prec), inp)
        errs[prec] = assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} precision {prec} x_out")
    assert errs[synth.PRECISION_EXTENDED] <= 0.5 * errs[synth.PRECISION_BF16], errs


def test_extended_precision_with_large_keys_and_small_queries(gpu):
    """The correction rows cover the magnitudes Q and K take: with W_k scaled
    by 256 and W_q by 1/256 (powers of two, so the bf16 weights stay exact)
    every logit is the same as on the plain 64K-token layer, but the keys
    reach ~1e3 and the scaled queries ~1e-3. Extended precision must still be
    at least twice as close to the oracle as plain bf16 (an fp8 format of too
    little range would saturate the keys or flush the queries and lose the
    correction)."""
    import dataclasses
    name = "layer_bf16_L64k_d1024"
    shape = synth.WORKLOADS[name]
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    wq, bq = inp["weights"]["q"]
    wk, bk = inp["weights"]["k"]
    inp["weights"]["q"] = (wq / 256.0, bq / 256.0)
    inp["weights"]["k"] = (wk * 256.0, bk * 256.0)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask)
    errs = {}
    for prec in (synth.PRECISION_EXTENDED, synth.PRECISION_BF16):
        x_out, _ = run_gpu(dataclasses.replace(shape, precision=prec), inp)
        errs[prec] = assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} K*256 Q/256 precision {prec} x_out")
    assert errs[synth.PRECISION_EXTENDED] <= 0.5 * errs[synth.PRECISION_BF16], errs


@pytest.mark.parametrize("name", ["layer_bf16_L64k_d1024", "layer_bf16_L1M_d1024"])
def test_forward_parity_fused_gate(gpu, name):
    """PF_GATE_FUSED at the workload widths (d_fine 1024, P = 64): the 64K-token
    layer in full, the 1M-token layer on every proxy and 64 sampled blocks."""
    import dataclasses
    shape = dataclasses.replace(synth.WORKLOADS[name], gate_fusion=synth.GATE_FUSED)
    print(f"[workload {name}, fused gate] generating inputs", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[name])
    x_out, h_out = run_gpu(shape, inp)
    m = shape.n_proxies
    blocks = None
    if shape.seq_len > 65536:
        rng = np.random.default_rng(654)
        blocks = sorted(set([0, 1, m - 2, m - 1] + list(rng.choice(np.arange(2, m - 2), 60, replace=False))))
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask,
                               sample_blocks=blocks)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} fused gate h_out")
    got = host(x_out) if blocks is None else host(x_out.reshape(1, m, shape.block, shape.d_fine)[:, blocks])
    assert_close(got, ref["x_out"], shape.dtype, f"{name} fused gate x_out")


def test_zero_decompression_is_identity_bitwise(gpu):
    shape = synth.WORKLOADS["layer_bf16_L64k_d1024"]
    inp = synth.layer_inputs(shape, 5)
    inp["weights"]["decompress"] = [(np.zeros_like(a), b) for a, b in inp["weights"]["decompress"]]
    x_out, _ = run_gpu(shape, inp)
    import torch
    assert torch.equal(x_out, dev(inp["x"], shape.dtype))


@pytest.mark.parametrize("factors", [(64,), (8, 8)])
def test_token_causality_bit_identical(gpu, factors):
    import torch
    shape = LayerShape(1, 64 * 96, 256, 256, 4, 64, factors)
    inp = synth.layer_inputs(shape, 11)
    x0, h0 = run_gpu(shape, inp)
    for t in (0, 1000, 64 * 50 + 7, 64 * 96 - 1):
        inp2 = dict(inp)
        x = inp["x"].copy()
        x[0, t] += 1.0
        inp2["x"] = x
        x1, h1 = run_gpu(shape, inp2)
        assert torch.equal(x1[0, :t], x0[0, :t]), t
        assert torch.equal(h1[0, :t // 64], h0[0, :t // 64]), t
        assert not torch.equal(x1[0, t], x0[0, t])


def test_run_twice_bitwise(gpu):
    import torch
    shape = LayerShape(1, 64 * 200, 512, 512, 8, 64, (64,))
    inp = synth.layer_inputs(shape, 12)
    a = run_gpu(shape, inp)
    b = run_gpu(shape, inp)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_layer_stack_with_cross_layer_proxies_and_dynamic_p(gpu):
    """Three stacked layers (Sec. 3.1, Sec. 3.6): layer 2 takes layer 1's proxy
    stream as H_in (Eq. 8); layer 3 uses another block size, so its proxy
    state is re-extracted from the local stream (H_in absent). The chain of
    HIP calls matches the chained oracle."""
    from paper_2608_23463_amd import binding as B
    L, d = 64 * 24, 256
    shapes = [LayerShape(1, L, d, d, 4, 64, (16,)), LayerShape(1, L, d, d, 4, 64, (16,)),
              LayerShape(1, L, d, d, 4, 64, (8, 8))]
    ws = [synth.layer_inputs(s, 40 + i)["weights"] for i, s in enumerate(shapes)]
    x0 = synth.layer_inputs(shapes[0], 39)["x"]
    # GPU chain
    x = dev(x0, "bf16")
    h = None
    for i, s in enumerate(shapes):
        h_in = h if i == 1 else None
        x, h, _ = B.layer_forward(B.config_from_shape(s), dev_weights(ws[i], "bf16"), x, h_in)
    import torch
    torch.cuda.synchronize()
    # oracle chain on the same (bf16-valued) inputs; intermediate activations stay fp64
    rx, rh = x0, None
    for i, s in enumerate(shapes):
        r = oracle.layer_forward(rx, ws[i], s.factors, s.n_heads, s.mask, rh if i == 1 else None)
        rx, rh = r["x_out"], r["h_out"]
    assert_close(host(h), rh, "bf16", "stack layer 3 h_out")
    assert_close(host(x), rx, "bf16", "stack layer 3 x_out")


IMAGES = {
    # 2-D partition (Sec. 3.9): a 32 x 48 image in 4 x 4 patches (P = 16), and 16 x 16 in 8 x 8 patches
    "bf16_image_32x48_p4_bi": LayerShape(2, 32 * 48, 192, 192, 3, 64, (16,), mask=synth.BIDIRECTIONAL,
                                         image_width=48),
    "fp32_image_16x16_p8_bc": LayerShape(1, 16 * 16, 64, 128, 2, 64, (64,), dtype="fp32",
                                         mask=synth.BLOCK_CAUSAL, image_width=16),
}


@pytest.mark.parametrize("name", list(IMAGES))
def test_forward_parity_2d_partition(gpu, name):
    shape = IMAGES[name]
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, seed=zlib.crc32(name.encode()) % 1000, with_h_in=True)
    for key in ("q", "k"):
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 4) if shape.dtype == "bf16" else wq * 4, bq)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward_2d(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.image_width,
                                  shape.mask, inp["h_in"])
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")


@pytest.mark.parametrize("name,shape", [
    ("bf16_affine_L16k_d1024", LayerShape(1, 16384, 1024, 1024, 16, 64, (64,), injection=synth.INJECT_AFFINE)),
    ("bf16_gated_head_L16k_d1024", LayerShape(1, 16384, 1024, 1024, 16, 64, (64,),
                                              injection=synth.INJECT_GATED_HEAD)),
    ("bf16_partial_block_L16k_d1024", LayerShape(1, 16384 - 23, 1024, 1024, 16, 64, (64,))),
])
def test_forward_parity_variants_at_width_1024(gpu, name, shape):
    """Injection variants and a partial last block at the workloads' width
    (d = 1024, 16 heads, P = 64) over 16K tokens: every output compared."""
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, zlib.crc32(name.encode()) % 1000)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.mask,
                               injection=shape.injection)
    assert_close(host(h_out), ref["h_out"], shape.dtype, f"{name} h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, f"{name} x_out")


def test_forward_parity_2d_partition_image_128x128(gpu):
    """A 128 x 128 image in 8 x 8 patches (P = 64, 256 proxies) at d = 1024."""
    shape = LayerShape(1, 128 * 128, 1024, 1024, 16, 64, (64,), mask=synth.BIDIRECTIONAL, image_width=128)
    inp = synth.layer_inputs(shape, 77)
    x_out, h_out = run_gpu(shape, inp)
    ref = oracle.layer_forward_2d(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.image_width,
                                  shape.mask)
    assert_close(host(h_out), ref["h_out"], shape.dtype, "image 128x128 h_out")
    assert_close(host(x_out), ref["x_out"], shape.dtype, "image 128x128 x_out")
