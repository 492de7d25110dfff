"""The decode and prefill parity checks can see the proxy-cache read (CPU only).

For every case in `cache_cases`, mistakes planted in the oracle's inputs (the
cached read dropped; one 1,024-row slice or one 64-key tile of cached rows
left out) must move the sublayer output y - x by at least five times the
bf16 tolerance (infinity-norm relative error), so a GPU result within
tolerance of the unmodified oracle cannot have made that mistake. The GPU
tests compare exactly these outputs on exactly these inputs. The bf16
rounding of the oracle's own y, the GPU's last step, must leave y - x within
a quarter of the tolerance, so the comparison is one the GPU can pass.
"""
import numpy as np
import pytest

import oracle
import cache_cases as cc
from helpers import TOL
from paper_2608_23463_amd import synth

MARGIN = 5 * TOL["bf16"]


def assert_output_rounding_fits(ref, x, label):
    err = oracle.max_rel_err(synth.bf16_round(ref.astype(np.float32)) - x, ref - x)
    print(f"  {label}: bf16 rounding of y moves y - x by {err:.3e}")
    assert err <= TOL["bf16"] / 4, f"{label}: output rounding alone moves y - x by {err:.3e}"


@pytest.mark.parametrize("name", list(cc.DECODE_CASES))
def test_decode_planted_mistakes_are_visible(name):
    shape = cc.DECODE_CASES[name]
    inp = cc.build(shape, name, cc.decode_seed(name))
    ref, _ = cc.oracle_decode(shape, inp)
    x = inp["x"].astype(np.float64)
    assert_output_rounding_fits(ref, x, name)
    for label, mut in cc.mutations(shape, name, inp, prefill=False):
        got, _ = cc.oracle_decode(shape, mut)
        err = oracle.max_rel_err(got - x, ref - x)
        print(f"  {name}: {label}: y - x moves by {err:.3e} (y alone {oracle.max_rel_err(got, ref):.3e})")
        assert err >= MARGIN, f"{name}: planted mistake '{label}' moves y - x by only {err:.3e}"


@pytest.mark.parametrize("name", list(cc.PREFILL_CASES))
def test_prefill_planted_mistakes_are_visible(name):
    shape = cc.PREFILL_CASES[name]
    inp = cc.build(shape, name, cc.prefill_seed(name))
    toks = cc.prefill_tokens(shape)
    ref, _ = cc.oracle_prefill(shape, inp, tokens=toks)
    x = cc.chunk(inp)[:, toks].astype(np.float64)
    assert_output_rounding_fits(ref, x, name)
    for label, mut in cc.mutations(shape, name, inp, prefill=True):
        got, _ = cc.oracle_prefill(shape, mut, tokens=toks)
        err = oracle.max_rel_err(got - x, ref - x)
        print(f"  {name}: {label}: y - x moves by {err:.3e} (y alone {oracle.max_rel_err(got, ref):.3e})")
        assert err >= MARGIN, f"{name}: planted mistake '{label}' moves y - x by only {err:.3e}"


def test_alpha_off_and_constant_value_pins_are_checkable():
    """The inputs of the GPU pins in test_gpu_decode.py (alpha off, constant
    cached values): the output rounding leaves y - x within a quarter of the
    tolerance there too."""
    shape = cc.DECODE_CASES["sharp"]
    inp = cc.build(shape, "sharp", cc.decode_seed("sharp") + 1)
    ref, _ = cc.oracle_decode(shape, cc.alpha_off(inp))
    assert_output_rounding_fits(ref, inp["x"].astype(np.float64), "alpha off")
    inp = cc.build(shape, "sharp", cc.decode_seed("sharp") + 2)
    inp["v_cache"][:, :, :shape.n0] = inp["v_cache"][:, :, :1]
    ref, _ = cc.oracle_decode(shape, inp)
    assert_output_rounding_fits(ref, inp["x"].astype(np.float64), "constant V")


def test_cases_span_many_slices_and_tiles():
    for shape in list(cc.DECODE_CASES.values()) + list(cc.PREFILL_CASES.values()):
        assert -(-shape.n0 // cc.SLICE_ROWS) >= 16
        assert -(-shape.n0 // cc.TILE_ROWS) >= 200
