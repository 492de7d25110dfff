"""GPU parity of the layer backward against the CPU oracle (through the C ABI).

The HIP forward (saving activations) and backward run on seeded inputs; dX,
dH_in and every weight and bias gradient are compared with the oracle's
chain rule (itself pinned by finite differences) with the infinity-norm
relative error (1e-4 fp32, 2e-2 bf16), plus bit-exact dual causality and
run-to-run determinism.
"""
import zlib

import numpy as np
import pytest

import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import LayerShape
from helpers import dev, dev_weights, host

pytestmark = pytest.mark.gpu

# Layers with few attention rows (one or two proxies, or at most FEW_ROWS
# rows over all sequences and heads): bound on the error of the Q and K
# gradients relative to the terms that cancel in dS (bf16: four units in the
# last place, the bf16 rounding of dO, V and plain bf16 logits that the
# cancellation magnifies; fp32: a tenth of its tolerance)
TERM_TOL = {"bf16": 2.0 ** -7, "fp32": 1e-5}
FEW_ROWS = 16


def run_gpu_backward(shape, inp, dh_out=None):
    import torch
    from paper_2608_23463_amd import binding as B
    cfg = B.config_from_shape(shape)
    x = dev(inp["x"], shape.dtype)
    h_in = dev(inp["h_in"], shape.dtype)
    w = dev_weights(inp["weights"], shape.dtype)
    _, _, saved = B.layer_forward(cfg, w, x, h_in, save=True)
    dx, dh_in, grads = B.layer_backward(cfg, w, x, h_in, saved, dev(inp["dy"], shape.dtype),
                                       dev(dh_out, shape.dtype))
    torch.cuda.synchronize()
    return dx, dh_in, grads


def compare(shape, inp, res, ref, label):
    """Every gradient against the oracle; all are reported before asserting.

    The key bias gradient is zero in exact arithmetic (softmax is invariant
    to adding one constant to every key, so each row of dS sums to zero).
    Its error is measured against the scale of its summands,
    max_c sum_rows |dK[row, c]| (oracle), instead of its own ~0 magnitude.
    The per-head gate's bias gradient (n_heads columns, each a sum of
    cancelling terms over every token) is measured the same way, against
    max_c sum_rows |dG[row, c]|. The Q and K weight and bias gradients come
    from dS = P * (dP - rowsum(dO * O)), a difference of terms that cancel;
    with many keys and rows the rounding averages out and the measure above
    applies, but with one or two proxies every row sees one or two keys (one
    key: the gradients are zero, a softmax over one key being constant), and
    with a handful of attention rows in all nothing averages, so there they
    may instead be within TERM_TOL of those terms (the oracle's "score_abs"
    bounds).
    """
    from helpers import TOL
    dx, dh_in, grads = res
    dt = shape.dtype
    errs = {}

    def chk(got, want, what, scale=None):
        if scale is None:
            e = oracle.max_rel_err(got, want)
        else:
            diff = float(np.max(np.abs(np.asarray(got, np.float64) - want)))
            # a zero scale (every summand zero, e.g. one proxy: no key gradient) asks for an exact zero
            e = diff / scale if scale > 0 else diff
        errs[what] = e
        print(f"  {label} {what}: max rel err {e:.3e} (tol {TOL[dt]:g})", flush=True)

    def chk_score(got, want, terms, what, scale=None):
        # within the tolerance of the result (or of `scale`); with one or two proxies (one or two
        # keys per row) or few attention rows in all, where nothing averages the rounding of the
        # terms that cancel in dS, alternatively within TERM_TOL of those terms
        got = np.asarray(got, np.float64)
        diff = float(np.max(np.abs(got - want)))
        if scale is None:
            e = oracle.max_rel_err(got, want)
        else:
            e = diff / scale if scale > 0 else diff
        tmax = float(np.max(terms))
        e_terms = diff / tmax if tmax > 0 else diff
        few = shape.n_proxies <= 2 or shape.batch * shape.n_heads * shape.n_proxies <= FEW_ROWS
        errs[what] = 0.0 if few and e_terms <= TERM_TOL[dt] else e
        print(f"  {label} {what}: max rel err {e:.3e} (tol {TOL[dt]:g}), against the cancelling terms "
              f"{e_terms:.3e}" + (f" (bound {TERM_TOL[dt]:.2e}, few attention rows)" if few else ""),
              flush=True)

    chk(host(dx), ref["dx"], "dx")
    if ref["dh_in"] is not None:
        chk(host(dh_in), ref["dh_in"], "dh_in")
    rg = ref["grads"]
    for name in ("q", "k", "v", "o", "gate", "affine"):
        if rg.get(name) is None:  # the gate (or the affine map) only with its injection mode
            assert grads.get(name) is None
            continue
        if name in ("q", "k"):
            sa = ref["score_abs"][name]
            chk_score(host(grads[name][0]), rg[name][0], sa[0], f"dW_{name}")
            key_scale = float(np.max(np.sum(np.abs(ref["proj_grads"]["k"]), axis=(0, 1)))) if name == "k" else None
            chk_score(host(grads[name][1]), rg[name][1], sa[1], f"db_{name}", key_scale)
            continue
        chk(host(grads[name][0]), rg[name][0], f"dW_{name}")
        if name == "gate" and shape.injection == synth.INJECT_GATED_HEAD:
            # n_heads columns, each a sum over every token of a head's summed dY * Delta: the
            # terms cancel (a sum ~1e-3 of their magnitude is common), so the bias gradient is
            # measured against the magnitude of its summands, as the key bias above
            chk(host(grads[name][1]), rg[name][1], "db_gate", float(np.max(ref["gate_abs"])))
        else:
            chk(host(grads[name][1]), rg[name][1], f"db_{name}")
    for kind in ("compress", "decompress"):
        for j in range(len(shape.factors)):
            chk(host(grads[kind][j][0]), rg[kind][j][0], f"dW_{kind}[{j}]")
            chk(host(grads[kind][j][1]), rg[kind][j][1], f"db_{kind}[{j}]")
    bad = {k: v for k, v in errs.items() if not v <= TOL[dt]}
    assert not bad, f"{label}: gradients above tolerance: {bad}"


CASES = {
    "fp32_tc_factorised": (LayerShape(2, 8 * 37, 64, 128, 2, 64, (2, 4), level_dims=(96,), dtype="fp32"), True),
    "fp32_bc": (LayerShape(1, 16 * 40, 64, 128, 1, 128, (16,), mask=synth.BLOCK_CAUSAL, dtype="fp32"), False),
    "fp32_bi": (LayerShape(1, 16 * 40, 128, 128, 2, 64, (16,), mask=synth.BIDIRECTIONAL, dtype="fp32"), True),
    "bf16_tc_ragged": (LayerShape(2, 16 * 37, 192, 192, 3, 64, (16,)), True),
    "bf16_tc_factorised": (LayerShape(1, 64 * 70, 128, 256, 2, 128, (8, 8), level_dims=(160,)), True),
    "bf16_bi": (LayerShape(1, 16 * 130, 128, 256, 4, 64, (16,), mask=synth.BIDIRECTIONAL), False),
    # the language-model shape (64-wide local stream, 512-wide proxies, 8 x 64, P = 64) over
    # 10,240 tokens: 160 proxies, and enough token rows for the transposed weight-gradient path
    "bf16_lm_shape": (LayerShape(1, 64 * 160, 64, 512, 8, 64, (64,)), True),
    # the same with plain bf16 H, Q, K (PF_PRECISION_BF16) and the drawn Q/K weights (with 4x
    # sharpened logits plain bf16 puts dW_q at 2.2e-2: the extended precision is the default)
    "bf16_lm_shape_plain": (LayerShape(1, 64 * 160, 64, 512, 8, 64, (64,), precision=synth.PRECISION_BF16), True,
                            False),
    # residual-add injection (Eq. 11); level 1 groups pairs of 16,384 tokens, so its weight
    # gradients (8,192 rows) take the transposed path with column sums from the transpose
    "bf16_inject_add": (LayerShape(1, 16384, 128, 256, 4, 64, (2, 8), injection=synth.INJECT_ADD), True),
    "fp32_inject_add_factorised": (LayerShape(2, 8 * 37, 64, 128, 2, 64, (2, 4), level_dims=(96,), dtype="fp32",
                                              injection=synth.INJECT_ADD), False),
    # affine modulation (Eq. 13); 16,384 token rows take the transposed weight-gradient path
    "bf16_inject_affine": (LayerShape(1, 16384, 128, 256, 4, 64, (2, 8), injection=synth.INJECT_AFFINE), True),
    "fp32_inject_affine": (LayerShape(2, 8 * 37, 64, 128, 2, 64, (2, 4), level_dims=(96,), dtype="fp32",
                                      injection=synth.INJECT_AFFINE), False),
    # per-head gate; 16,384 token rows take the transposed weight-gradient path
    "bf16_inject_gated_head": (LayerShape(1, 16384, 128, 256, 4, 64, (2, 8), injection=synth.INJECT_GATED_HEAD),
                               True),
    "fp32_inject_gated_head": (LayerShape(2, 8 * 37, 64, 128, 2, 64, (2, 4), level_dims=(96,), dtype="fp32",
                                          injection=synth.INJECT_GATED_HEAD), False),
    # d_fine = 3072 (768 channels per head): head sums over 96 runs of 8 per head. fp32 with the
    # sharpened attention checks the kernels at 1e-4; bf16 keeps the drawn Q/K weights, since at
    # this width a sharp softmax leaves the compression-bias gradient (a sum over 24 proxies
    # with cancellation) at the 2e-2 edge of bf16 itself (the fp32 run of it: 1e-5)
    "fp32_gated_head_wide": (LayerShape(1, 16 * 24, 3072, 256, 4, 64, (16,), dtype="fp32",
                                        injection=synth.INJECT_GATED_HEAD), False),
    "bf16_gated_head_wide": (LayerShape(1, 16 * 24, 3072, 256, 4, 64, (16,), injection=synth.INJECT_GATED_HEAD),
                             False, False),
    # the fused decompression + gate forward (d_fine 256) writes the saved Delta and G
    "bf16_fused_gate": (LayerShape(1, 16 * 130, 256, 256, 4, 64, (16,), gate_fusion=synth.GATE_FUSED), True),
    # partial last block (L % P != 0): zero-padded inside the library, dY = 0 on the padding
    "bf16_tc_partial_block": (LayerShape(2, 16 * 37 + 9, 192, 192, 3, 64, (16,)), True),
    "fp32_bi_partial_block_factorised": (LayerShape(1, 8 * 37 + 5, 64, 128, 2, 64, (2, 4), level_dims=(96,),
                                                    dtype="fp32", mask=synth.BIDIRECTIONAL), True),
    # d_fine a multiple of 8 but not of the K tile: the [X | Delta] split inside a K tile
    "bf16_odd_width": (LayerShape(2, 16 * 37, 72, 128, 2, 64, (16,)), True),
    "fp32_odd_width": (LayerShape(1, 16 * 37, 40, 128, 2, 64, (16,), dtype="fp32"), True),
    # one proxy (a full block, and a partial one) in the masks where it feeds its own block: the
    # Q and K maps get no gradient
    "bf16_single_proxy_bidirectional": (LayerShape(2, 5, 80, 192, 3, 64, (8,), mask=synth.BIDIRECTIONAL), True),
    "fp32_single_proxy_block_causal": (LayerShape(1, 8, 64, 128, 1, 128, (2, 4), level_dims=(96,),
                                                  mask=synth.BLOCK_CAUSAL, dtype="fp32"), True),
    # two proxies, token-causal: proxy 0 (one key) feeds block 1, proxy 1 feeds nothing, so the
    # Q and K maps again get no gradient
    "bf16_two_proxies_token_causal": (LayerShape(2, 27, 208, 128, 2, 64, (2, 8), level_dims=(240,)), True),
    # two proxies, block-causal, plain bf16: the second row's two-key softmax gradient is a few
    # percent of the terms that form it, with nothing to average its bf16 rounding
    "bf16_plain_two_proxies_block_causal": (LayerShape(1, 128, 176, 256, 2, 128, (4, 8, 2), level_dims=(72, 152),
                                                       mask=synth.BLOCK_CAUSAL, injection=synth.INJECT_AFFINE,
                                                       precision=synth.PRECISION_BF16), True, False),
    # fp32 over 16,384 token rows and 8,192 level-1 rows: the weight gradients run on
    # transposed (K-contiguous) copies of their operands
    "fp32_transposed_wgrad": (LayerShape(1, 16384, 64, 128, 2, 64, (2, 8), level_dims=(96,), dtype="fp32"), True),
}


@pytest.mark.parametrize("name", list(CASES))
def test_backward_parity_small(gpu, name):
    shape, with_h, *opt = CASES[name]
    sharpen = opt[0] if opt else True
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, zlib.crc32(name.encode()) % 1000, with_dy=True, with_h_in=with_h)
    # attention that is far from uniform, so the attention backward matters
    for key in ("q", "k") if sharpen else ():
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 4) if shape.dtype == "bf16" else wq * 4, bq)
    dh_out = None
    if with_h:
        rng = np.random.default_rng(3)
        dh_out = rng.standard_normal((shape.batch, shape.n_proxies, shape.d_proxy)).astype(np.float32)
        if shape.dtype == "bf16":
            dh_out = synth.bf16_round(dh_out)
    res = run_gpu_backward(shape, inp, dh_out)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask,
                                inp["h_in"], dh_out, injection=shape.injection)
    compare(shape, inp, res, ref, name)


@pytest.mark.timeout(300)
def test_backward_parity_fp32_token_rows_past_the_transposes(gpu):
    """fp32 over 2 x 1,050,624 tokens: the gate's weight and bias gradients
    reduce over 2,101,248 token rows, whose transposed rows would pass the
    8 MiB operand-row limit, so they read the token-major operands as they
    are (K of two million rows); the level rows (8,208) still take the
    transposed copies. Every gradient compared; the oracle takes seconds."""
    shape = LayerShape(2, 1050624, 8, 64, 1, 64, (256,), dtype="fp32")
    print(f"[fp32 2.1M token rows] {shape}", flush=True)
    inp = synth.layer_inputs(shape, 77, with_dy=True, with_h_in=True)
    for key in ("q", "k"):
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (wq * 4, bq)
    res = run_gpu_backward(shape, inp)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask,
                                inp["h_in"], None)
    compare(shape, inp, res, ref, "fp32_2.1M_rows")


def test_backward_parity_factorised_workload_reduced_L(gpu):
    """The 256K-token factorised workload's widths, heads and factors at L = 8192."""
    full = synth.WORKLOADS["layer_bf16_L256k_d2048_f8x8"]
    shape = LayerShape(1, 8192, full.d_fine, full.d_proxy, full.n_heads, full.head_dim, full.factors)
    print(f"[workload reduced] {shape}", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS["layer_bf16_L256k_d2048_f8x8"], with_dy=True)
    res = run_gpu_backward(shape, inp)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask)
    compare(shape, inp, res, ref, "L8192_d2048_f8x8")


@pytest.mark.timeout(400)
def test_backward_parity_factorised_workload_widths_many_tiles(gpu):
    """The 256K-token factorised workload's widths, heads and factors (d = 2048,
    16 x 128, P = 8 x 8) over 650 proxies: six 128-row query and key
    workgroups per head in the attention backward (the last one ragged) and
    full-size level GEMMs, every gradient compared. The oracle takes about a
    minute here."""
    full = synth.WORKLOADS["layer_bf16_L256k_d2048_f8x8"]
    shape = LayerShape(1, 64 * 650, full.d_fine, full.d_proxy, full.n_heads, full.head_dim, full.factors)
    print(f"[workload widths, m = 650] {shape}: generating inputs", flush=True)
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS["layer_bf16_L256k_d2048_f8x8"] + 1, with_dy=True)
    res = run_gpu_backward(shape, inp)
    print("[workload widths, m = 650] oracle backward", flush=True)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask)
    compare(shape, inp, res, ref, "L41600_d2048_f8x8")


@pytest.mark.parametrize("mask", [synth.TOKEN_CAUSAL, synth.BLOCK_CAUSAL, synth.BIDIRECTIONAL])
def test_backward_parity_dh128_many_tiles(gpu, mask):
    """16 heads of 128 over 1,000 proxies (eight query and key workgroups per
    head, the last ragged) with a narrow local stream, attention sharpened,
    every gradient compared."""
    shape = LayerShape(1, 64 * 1000, 64, 2048, 16, 128, (8, 8), mask=mask)
    print(f"[case dh128 m = 1000 mask {mask}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, 600 + mask, with_dy=True, with_h_in=True)
    for key in ("q", "k"):
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 2), bq)
    rng = np.random.default_rng(5)
    dh_out = synth.bf16_round(rng.standard_normal((1, shape.n_proxies, shape.d_proxy)).astype(np.float32))
    res = run_gpu_backward(shape, inp, dh_out)
    ref = oracle.layer_backward(inp["x"], inp["weights"], shape.factors, shape.n_heads, inp["dy"], shape.mask,
                                inp["h_in"], dh_out)
    compare(shape, inp, res, ref, f"dh128_m1000_mask{mask}")


def test_backward_dual_causality_bitwise(gpu):
    """Token-causal layer: dY[t] cannot reach dX[s] for s > t."""
    import torch
    shape = LayerShape(1, 64 * 40, 256, 256, 4, 64, (8, 8))
    inp = synth.layer_inputs(shape, 21, with_dy=True)
    base = run_gpu_backward(shape, inp)[0]
    for t in (5, 64 * 17 + 3, 64 * 40 - 2):
        inp2 = dict(inp)
        dy = inp["dy"].copy()
        dy[0, t] += 1.0
        inp2["dy"] = dy
        got = run_gpu_backward(shape, inp2)[0]
        assert torch.equal(got[0, t + 1:], base[0, t + 1:]), t
        assert not torch.equal(got[0, t], base[0, t])


def test_backward_run_twice_bitwise(gpu):
    import torch
    shape = LayerShape(1, 64 * 50, 256, 256, 4, 64, (64,))
    inp = synth.layer_inputs(shape, 22, with_dy=True)
    a = run_gpu_backward(shape, inp)
    b = run_gpu_backward(shape, inp)
    assert torch.equal(a[0], b[0])
    for name in ("q", "k", "v", "o", "gate"):
        assert torch.equal(a[2][name][0], b[2][name][0]) and torch.equal(a[2][name][1], b[2][name][1])
    assert torch.equal(a[2]["compress"][0][0], b[2]["compress"][0][0])


@pytest.mark.parametrize("name,shape", [
    ("bf16_image_32x32_p4_bi", LayerShape(1, 32 * 32, 128, 256, 4, 64, (16,), mask=synth.BIDIRECTIONAL,
                                          image_width=32)),
    ("fp32_image_16x24_p4_bc", LayerShape(1, 16 * 24, 64, 128, 2, 64, (16,), dtype="fp32",
                                          mask=synth.BLOCK_CAUSAL, image_width=24)),
])
def test_backward_parity_2d_partition(gpu, name, shape):
    print(f"[case {name}] {shape}", flush=True)
    inp = synth.layer_inputs(shape, zlib.crc32(name.encode()) % 1000, with_dy=True, with_h_in=True)
    for key in ("q", "k"):
        wq, bq = inp["weights"][key]
        inp["weights"][key] = (synth.bf16_round(wq * 4) if shape.dtype == "bf16" else wq * 4, bq)
    rng = np.random.default_rng(4)
    dh_out = rng.standard_normal((shape.batch, shape.n_proxies, shape.d_proxy)).astype(np.float32)
    if shape.dtype == "bf16":
        dh_out = synth.bf16_round(dh_out)
    res = run_gpu_backward(shape, inp, dh_out)
    ref = oracle.layer_backward_2d(inp["x"], inp["weights"], shape.factors, shape.n_heads, shape.image_width,
                                   inp["dy"], shape.mask, inp["h_in"], dh_out)
    compare(shape, inp, res, ref, name)
