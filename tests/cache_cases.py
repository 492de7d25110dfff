"""Seeded decode and prefill inputs whose outputs depend strongly on the proxy
cache read of Eq. 19-21, and the planted mistakes each must expose.

With the workload's own weights (std 0.02) attention over thousands of
random cached rows is close to uniform, so the cached part alpha * A_h of
y = x + (A_x + alpha * A_h) W_o^T + b_o is small next to x, and a check of y
alone hardly sees it. The inputs here change only the weights and the cache
contents (input construction, none of the method's arithmetic):

* "sharp": W_q scaled by a power of two so the logits against the N(0, 1)
  cached keys have a standard deviation of about 4; the softmax over the
  cache is then carried by a few rows and A_h is of the order of one cached
  value, larger than A_x.
* "uniform": W_q = 0 and b_q = 0, so every visible key has the same weight
  and A_h is the mean of the visible cached values. The values carry offsets
  that alternate in sign from one 64-row tile to the next (amplitude 256) and
  from one 1,024-row slice to the next (amplitude 16), so their mean nearly
  cancels and leaving out any tile or slice moves A_h by about one unit.

In both, W_o is scaled by 16 (exact in bf16) so the sublayer output y - x
is as large as x: otherwise the bf16 rounding of y alone (half a unit in the
last place of |y| ~ 4) would be a few percent of y - x.

The GPU decode streams the cache in slices of 1,024 rows and the prefill
attention in tiles of 64 keys; n0 = 16,500 rows gives 17 slices (the last
one partial) and 258 tiles. A check compares y - x (the attention sublayer
output) as well as y.

Mistakes are planted in the oracle's inputs on the CPU: alpha forced to 0
(b_alpha = -1e9, the cached read dropped) and one slice or tile of cached rows
removed (the rows behind it move up). `tests/test_parity_sensitivity.py`
checks that each planted mistake moves y - x by at least five times the bf16
tolerance, so a GPU result within tolerance cannot have made it.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2608_23463_amd import synth
from paper_2608_23463_amd.synth import DecodeShape

SLICE_ROWS = 1024   # cache rows per slice of the decode attention
TILE_ROWS = 64      # keys per tile of the prefill attention
N0 = 16500          # 17 slices (16 full + 116 rows), 258 tiles

# `steps` is the number of decode steps (decode) or the chunk length (prefill)
DECODE_CASES = {
    "sharp": DecodeShape(2, 128, 2, 64, (16,), n0=N0, steps=20),
    "uniform": DecodeShape(2, 128, 2, 64, (16,), n0=N0, steps=20),
    "sharp_dh128_factorised": DecodeShape(2, 256, 2, 128, (4, 4), n0=N0, steps=18),
}
PREFILL_CASES = {
    "sharp": DecodeShape(2, 128, 2, 64, (16,), n0=N0, steps=100),
    "uniform": DecodeShape(2, 128, 2, 64, (16,), n0=N0, steps=100),
}
LOGIT_STD = 4.0
WO_SCALE = 16.0


def _kind(name: str) -> str:
    return "uniform" if name.startswith("uniform") else "sharp"


def build(shape: DecodeShape, name: str, seed: int):
    """Draw the case's inputs (synth draw order), then reshape the weights and
    cache as described in the module docstring."""
    inp = synth.decode_inputs(shape, seed)
    w = inp["weights"]
    d, dh, n0 = shape.d_model, shape.head_dim, shape.n0
    w["o"] = (w["o"][0] * np.float32(WO_SCALE), w["o"][1])
    if _kind(name) == "sharp":
        # q = u W_q^T with u of unit RMS: per-channel std 0.02 sqrt(d); a logit
        # q.k / sqrt(dh) against N(0, 1) keys then has std 0.02 sqrt(d) too
        f = 2.0 ** round(np.log2(LOGIT_STD / (synth.WEIGHT_STD * np.sqrt(d))))
        w["q"] = (w["q"][0] * np.float32(f), w["q"][1])   # a power of two keeps bf16 values exact
    else:
        w["q"] = (np.zeros_like(w["q"][0]), np.zeros_like(w["q"][1]))
        rng = np.random.default_rng(seed + 1)
        sign = rng.choice([-1.0, 1.0], size=(shape.batch, shape.n_heads, 1, dh))
        rows = np.arange(n0)
        tile = np.where((rows // TILE_ROWS) % 2 == 0, 1.0, -1.0)[None, None, :, None]
        slc = np.where((rows // SLICE_ROWS) % 2 == 0, 1.0, -1.0)[None, None, :, None]
        vc = inp["v_cache"]
        vc[:, :, :n0] = synth.bf16_round((vc[:, :, :n0] + sign * (256.0 * tile + 16.0 * slc)).astype(np.float32))
    return inp


def alpha_off(inp):
    """Planted mistake: the cached read is dropped (alpha = sigmoid(-1e9) = 0)."""
    out = dict(inp)
    w = dict(inp["weights"])
    w["alpha"] = (w["alpha"][0], np.full_like(w["alpha"][1], -1e9))
    out["weights"] = w
    return out


def drop_rows(inp, lo: int, hi: int):
    """Planted mistake: cached rows [lo, hi) are left out of every attention."""
    out = dict(inp)
    for key in ("k_cache", "v_cache"):
        c = inp[key]
        kept = np.concatenate([c[:, :, :lo], c[:, :, hi:]], axis=2)
        pad = np.zeros(c.shape[:2] + (hi - lo,) + c.shape[3:], c.dtype)
        out[key] = np.concatenate([kept, pad], axis=2)
    out["n0"] = inp["n0"] - (hi - lo)
    return out


def oracle_state(shape: DecodeShape, inp, seqs):
    st = oracle.DecodeState.empty(len(seqs), shape.n_heads, shape.head_dim, shape.block, shape.capacity,
                                  shape.d_model)
    st.k_cache[:] = inp["k_cache"][seqs]
    st.v_cache[:] = inp["v_cache"][seqs]
    st.n = inp["n0"]
    return st


def oracle_decode(shape: DecodeShape, inp, seqs=None):
    """Outputs of every decode step [steps, len(seqs), d] and the final state."""
    seqs = list(range(shape.batch)) if seqs is None else list(seqs)
    st = oracle_state(shape, inp, seqs)
    ys = np.stack([oracle.decode_step(st, inp["weights"], shape.factors, inp["x"][t][seqs], shape.rms_eps)
                   for t in range(shape.steps)])
    return ys, st


def chunk(inp):
    """[steps, B, d] token stream -> [B, T, d] prefill chunk."""
    return np.ascontiguousarray(inp["x"].transpose(1, 0, 2))


def oracle_prefill(shape: DecodeShape, inp, seqs=None, tokens=None):
    """Prefill outputs [len(seqs), T or len(tokens), d] and the final state."""
    seqs = list(range(shape.batch)) if seqs is None else list(seqs)
    st = oracle_state(shape, inp, seqs)
    y = oracle.prefill(st, inp["weights"], shape.factors, chunk(inp)[seqs], shape.rms_eps, tokens=tokens)
    return y, st


def dominant_slice(shape: DecodeShape, inp) -> int:
    """Slice holding the largest attention weight of the first token's query
    (sequence 0, head 0) over the initial cache: the slice whose loss a sharp
    case must expose."""
    w = inp["weights"]
    x = np.asarray(inp["x"][0][0], np.float64)
    u = oracle.rms_norm(x, w["rms_gamma"], shape.rms_eps)
    dh = shape.head_dim
    q = (np.asarray(w["q"][0], np.float64) @ u)[:dh]
    s = inp["k_cache"][0, 0, :inp["n0"]].astype(np.float64) @ q
    return int(np.argmax(s)) // SLICE_ROWS


def mutations(shape: DecodeShape, name: str, inp, prefill: bool):
    """(label, mutated inputs) pairs: planted mistakes the case must expose."""
    n0 = inp["n0"]
    out = [("cached read dropped (alpha = 0)", alpha_off(inp))]
    if _kind(name) == "sharp":
        s = dominant_slice(shape, inp)
        out.append((f"dominant slice {s} dropped", drop_rows(inp, s * SLICE_ROWS, min(n0, (s + 1) * SLICE_ROWS))))
        return out
    last = (n0 - 1) // SLICE_ROWS
    for s in (0, 7, last - 1, last):
        out.append((f"slice {s} dropped", drop_rows(inp, s * SLICE_ROWS, min(n0, (s + 1) * SLICE_ROWS))))
    if prefill:
        lt = (n0 - 1) // TILE_ROWS
        for t in (0, 129, lt - 1):
            out.append((f"tile {t} dropped", drop_rows(inp, t * TILE_ROWS, (t + 1) * TILE_ROWS)))
    return out


def decode_seed(name: str) -> int:
    return 4242 + sum(map(ord, name))


def prefill_seed(name: str) -> int:
    return 5353 + sum(map(ord, name))


# Prefill outputs the sensitivity checks compare: the first and last tokens of
# the chunk, both sides of block boundaries, and the unfinished tail block.
def prefill_tokens(shape: DecodeShape):
    P, T = shape.block, shape.steps
    return sorted({0, 1, P - 1, P, 2 * P + 3, T // 2, T - P - 1, T - 2, T - 1})
