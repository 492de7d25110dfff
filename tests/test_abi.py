"""Host-only checks of the C ABI: the library loads, exports every function
the header declares, and rejects invalid arguments before any launch.
No test here touches a GPU (every call fails validation or is a size query).
"""
import ctypes
import os
import re

import pytest

from paper_2608_23463_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "proxyformer.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(proxy_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libproxyformer.so is not built (run __graft_entry__.build())")
    return B.load()


def test_exports_every_declared_function(lib):
    names = header_functions()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.proxy_version() == 103


def _cfg(**kw):
    base = dict(batch=1, seq_len=4096, d_fine=256, d_proxy=256, n_heads=4, head_dim=64, factors=(64,),
                dtype="bf16", mask=0)
    base.update(kw)
    return B.layer_config(**base)


def test_size_queries(lib):
    cfg = _cfg()
    ws = B.layer_workspace_size(cfg)
    saved = B.layer_saved_size(cfg)
    assert ws > 0 and saved > 0 and ws % 256 == 0 and saved % 256 == 0
    # saved activations include at least Delta and G for every token
    assert saved >= 2 * 4096 * 256 * 2
    assert B.layer_workspace_size(cfg, True) > 0
    for bad in (dict(seq_len=0), dict(n_heads=3), dict(factors=()), dict(head_dim=32, n_heads=8),
                dict(d_fine=100), dict(batch=0), dict(dtype="fp16")):
        c = _cfg(**bad) if "dtype" not in bad else _cfg()
        if "dtype" in bad:
            c.dtype = 7
        assert B.layer_workspace_size(c) == 0, bad
        assert B.layer_saved_size(c) == 0, bad


def _weights_struct(nlev=1, null=None):
    w = B.PfLayerWeights()
    fake = 0x10000  # never dereferenced: every call below fails validation first
    for i in range(nlev):
        w.compress[i] = B.PfLinear(fake, None)
        w.decompress[i] = B.PfLinear(fake, None)
    for name in ("q", "k", "v", "o", "gate"):
        setattr(w, name, B.PfLinear(fake, None))
    if null:
        setattr(w, null, B.PfLinear(None, None))
    return w


def _fwd(lib, cfg, w, x=2 << 32, xo=3 << 32, ho=4 << 32, ws=5 << 32, ws_bytes=1 << 40):
    return lib.proxy_layer_forward(ctypes.byref(cfg), ctypes.byref(w), x, None, xo, ho, None, ws, ws_bytes, None)


@pytest.mark.parametrize("bad,status", [
    (dict(seq_len=0), B.PF_ERR_INVALID_ARG),
    (dict(n_heads=8), B.PF_ERR_INVALID_ARG),
    (dict(mask=5), B.PF_ERR_INVALID_ARG),
    (dict(injection=4), B.PF_ERR_INVALID_ARG),
    (dict(precision=2), B.PF_ERR_INVALID_ARG),
    (dict(gate_fusion=2), B.PF_ERR_INVALID_ARG),
    (dict(head_dim=32, n_heads=8), B.PF_ERR_UNSUPPORTED),
    (dict(d_fine=100), B.PF_ERR_UNSUPPORTED),
])
def test_forward_rejects_bad_config(lib, bad, status):
    cfg = _cfg(**bad)
    assert _fwd(lib, cfg, _weights_struct()) == status
    assert B.last_error()


def test_forward_rejects_oversize_head_before_any_launch(lib):
    # P = 1 and 2^23 tokens: one head of 128 bf16 channels over 2^23 proxies is
    # 2 GiB, beyond the attention kernels' 32-bit buffer offsets. The forward
    # and backward refuse it on the host (pointers are never dereferenced)
    cfg = _cfg(seq_len=1 << 23, d_fine=8, d_proxy=128, n_heads=1, head_dim=128, factors=(1,))
    assert _fwd(lib, cfg, _weights_struct()) == B.PF_ERR_UNSUPPORTED
    assert "2 GiB" in B.last_error()
    assert B.layer_workspace_size(cfg) == 0 and B.layer_saved_size(cfg) == 0
    g = B.PfLayerGrads()
    st = lib.proxy_layer_backward(ctypes.byref(cfg), ctypes.byref(_weights_struct()), 0x20000, None, 0x70000,
                                  0x30000, None, 0x40000, None, ctypes.byref(g), 0x50000, 1 << 40, None)
    assert st == B.PF_ERR_UNSUPPORTED
    # one proxy fewer (2^23 - 64 tokens) fits
    ok = _cfg(seq_len=(1 << 23) - 64, d_fine=8, d_proxy=128, n_heads=1, head_dim=128, factors=(1,))
    assert B.layer_workspace_size(ok) > 0


def test_grouped_rows_beyond_the_gemm_range_are_rejected(lib):
    """A GEMM tile addresses 256 operand rows through one 32-bit range below
    the 2^31 out-of-range offset: a level's grouped row (k_j * d_{j-1}
    elements) may span at most 8 MiB. P * d_fine = 4M bf16 elements (8 MiB)
    fits; 4M + 256 does not, nor 2M fp32 + 64, nor a second level's row."""
    ok = _cfg(seq_len=4096 * 2, d_fine=1024, d_proxy=256, factors=(4096,))
    assert B.layer_workspace_size(ok) > 0
    for bad in (dict(seq_len=4096 * 2, d_fine=1024 + 8, d_proxy=256, factors=(4096,)),
                dict(seq_len=2048 * 2, d_fine=1024 + 8, d_proxy=256, factors=(2048,), dtype="fp32"),
                dict(seq_len=64 * 8192, d_fine=64, d_proxy=256, factors=(64, 8192), level_dims=(1032,))):
        cfg = _cfg(**bad)
        assert _fwd(lib, cfg, _weights_struct(len(bad["factors"]))) == B.PF_ERR_UNSUPPORTED, bad
        assert "8 MiB" in B.last_error(), bad
        assert B.layer_workspace_size(cfg) == 0 and B.layer_saved_size(cfg) == 0


def test_proxy_rows_beyond_the_gemm_range_are_rejected(lib):
    """The projections read H with its low part beside it, rows of
    2 * d_proxy elements, under the same 8 MiB row limit: 8,192 heads of 128
    in fp32 (exactly 8 MiB) fit; one more head does not, nor 16,385 heads of
    128 in bf16."""
    ok = _cfg(seq_len=64, d_proxy=8192 * 128, n_heads=8192, head_dim=128, dtype="fp32")
    assert B.layer_workspace_size(ok) > 0
    for bad in (dict(seq_len=64, d_proxy=8193 * 128, n_heads=8193, head_dim=128, dtype="fp32"),
                dict(seq_len=64, d_proxy=16385 * 128, n_heads=16385, head_dim=128)):
        cfg = _cfg(**bad)
        assert _fwd(lib, cfg, _weights_struct(1)) == B.PF_ERR_UNSUPPORTED, bad
        assert "d_proxy" in B.last_error() and "8 MiB" in B.last_error(), bad
        assert B.layer_workspace_size(cfg) == 0 and B.layer_saved_size(cfg) == 0


def test_plain_bf16_precision_drops_the_low_parts(lib):
    # the low parts of H, Q and K (and the doubled K of the Q/K GEMMs) exist
    # only with PF_PRECISION_EXTENDED in bf16 mode
    ext, plain = _cfg(), _cfg(precision=B.PF_PRECISION_BF16)
    m, dp = 4096 // 64, 256
    assert B.layer_saved_size(ext) - B.layer_saved_size(plain) >= 3 * m * dp * 2
    f32 = _cfg(dtype="fp32")
    f32p = _cfg(dtype="fp32", precision=B.PF_PRECISION_BF16)
    assert B.layer_saved_size(f32) == B.layer_saved_size(f32p)


def test_gate_fusion_workspace(lib):
    # fused (bf16, gated, d_fine a multiple of 128): the forward workspace
    # holds the folded weight C[p] and bias b'[p] per block position instead
    # of Delta; where the fused kernel does not apply the option changes nothing
    L, P, df, d1 = 1 << 16, 64, 256, 256
    sep, fus = _cfg(seq_len=L), _cfg(seq_len=L, gate_fusion=B.PF_GATE_FUSED)
    delta, fold = L * df * 2, P * df * d1 * 2 + P * df * 4
    assert B.layer_workspace_size(sep) - B.layer_workspace_size(fus) >= delta - fold - 4096
    assert B.layer_workspace_size(sep) - B.layer_workspace_size(fus) <= delta - fold + 4096
    for kw in (dict(dtype="fp32"), dict(d_fine=192), dict(injection=B.PF_INJECT_ADD)):
        assert B.layer_workspace_size(_cfg(seq_len=L, **kw)) == \
            B.layer_workspace_size(_cfg(seq_len=L, gate_fusion=B.PF_GATE_FUSED, **kw)), kw


def test_partial_last_block_sizes(lib):
    # L = 4000 with P = 64: m = 63 blocks, the last zero-padded (Sec. 3.1)
    ragged, whole = _cfg(seq_len=4000), _cfg(seq_len=63 * 64)
    assert B.layer_saved_size(ragged) == B.layer_saved_size(whole)
    tok = 4000 * 256 * 2
    pad = 63 * 64 * 256 * 2
    assert B.layer_workspace_size(ragged) >= B.layer_workspace_size(whole) + 2 * pad
    assert B.layer_workspace_size(ragged, True) >= B.layer_workspace_size(whole, True) + 3 * pad
    assert tok < pad


def test_forward_rejects_bad_pointers(lib):
    cfg = _cfg()
    assert _fwd(lib, cfg, _weights_struct(null="gate")) == B.PF_ERR_INVALID_ARG
    assert "gate" in B.last_error()
    assert _fwd(lib, cfg, _weights_struct(), x=None) == B.PF_ERR_INVALID_ARG
    assert _fwd(lib, cfg, _weights_struct(), xo=(2 << 32) + 4096) == B.PF_ERR_INVALID_ARG  # x_out aliases x
    assert "alias" in B.last_error()
    assert _fwd(lib, cfg, _weights_struct(), x=(2 << 32) + 8) == B.PF_ERR_INVALID_ARG  # misaligned
    assert _fwd(lib, cfg, _weights_struct(), ws_bytes=1024) == B.PF_ERR_WORKSPACE
    assert _fwd(lib, cfg, _weights_struct(), ws=None) == B.PF_ERR_WORKSPACE


def test_gate_weights_only_required_by_gated_injection(lib):
    w = _weights_struct(null="gate")
    assert _fwd(lib, _cfg(), w) == B.PF_ERR_INVALID_ARG
    assert "gate" in B.last_error()
    # with residual-add injection a NULL gate passes validation; the call then
    # stops at the next check (a NULL x), so nothing is launched
    assert _fwd(lib, _cfg(injection=B.PF_INJECT_ADD), w, x=None) == B.PF_ERR_INVALID_ARG
    assert "gate" not in B.last_error()


def test_backward_rejects_bad_arguments(lib):
    cfg = _cfg()
    g = B.PfLayerGrads()
    w = _weights_struct()
    st = lib.proxy_layer_backward(ctypes.byref(cfg), ctypes.byref(w), 0x20000, None, None, 0x30000, None,
                                  0x40000, None, ctypes.byref(g), 0x50000, 1 << 40, None)
    assert st == B.PF_ERR_INVALID_ARG  # saved is NULL
    st = lib.proxy_layer_backward(ctypes.byref(cfg), ctypes.byref(w), 0x20000, 0x60000, 0x70000, 0x30000, None,
                                  0x40000, None, ctypes.byref(g), 0x50000, 1 << 40, None)
    assert st == B.PF_ERR_INVALID_ARG  # h_in given without dh_in


def _dcfg(**kw):
    base = dict(batch=2, d_model=128, n_heads=2, head_dim=64, factors=(4,), dtype="bf16")
    base.update(kw)
    return B.decode_config(**base)


def _dweights():
    w = B.PfDecodeWeights()
    fake = 0x10000
    w.rms_gamma = fake
    for name in ("q", "k", "v", "o", "alpha", "k_proxy", "v_proxy"):
        setattr(w, name, B.PfLinear(fake, None))
    w.compress[0] = B.PfLinear(fake, None)
    return w


def _dstate(n=0, n_cap=4, j=0):
    return B.PfDecodeState(0x20000, 0x30000, n_cap, n, 0x40000, 0x50000, 0x60000, j)


def test_decode_rejects_grouped_rows_beyond_the_gemm_range(lib):
    """The append's compression GEMMs take rows of k_j * d_{j-1} elements:
    at most 8 MiB (P = 4096 at d_model 1024 in bf16 fits, P = 8192 does not)."""
    ok = _dcfg(d_model=1024, n_heads=16, factors=(4096,))
    assert int(lib.proxy_decode_workspace_size(ctypes.byref(ok))) > 0
    bad = _dcfg(d_model=1024, n_heads=16, factors=(8192,))
    assert int(lib.proxy_decode_workspace_size(ctypes.byref(bad))) == 0
    st = _dstate()
    assert lib.proxy_decode_step(ctypes.byref(bad), ctypes.byref(_dweights()), ctypes.byref(st), 0x70000, 0x80000,
                                 0x90000, 1 << 40, None) == B.PF_ERR_UNSUPPORTED
    assert "8 MiB" in B.last_error()


def test_decode_validation(lib):
    cfg = _dcfg()
    ws = int(lib.proxy_decode_workspace_size(ctypes.byref(cfg)))
    assert ws > 0
    w = _dweights()
    # j out of range
    st = _dstate(j=4)
    assert lib.proxy_decode_step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), 0x70000, 0x80000,
                                 0x90000, ws, None) == B.PF_ERR_INVALID_ARG
    # block completes with a full cache
    st = _dstate(n=4, n_cap=4, j=3)
    assert lib.proxy_decode_step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), 0x70000, 0x80000,
                                 0x90000, ws, None) == B.PF_ERR_CAPACITY
    assert st.n == 4 and st.j == 3  # untouched
    # append past capacity
    st = _dstate(n=2, n_cap=4)
    assert lib.proxy_cache_append(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), 0x70000, 3, 0x90000, ws,
                                  None) == B.PF_ERR_CAPACITY
    assert st.n == 2
    # nothing to append is a no-op
    assert lib.proxy_cache_append(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), None, 0, 0x90000, ws,
                                  None) == B.PF_OK
    # workspace too small
    assert lib.proxy_decode_step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(_dstate()), 0x70000, 0x80000,
                                 0x90000, 16, None) == B.PF_ERR_WORKSPACE
    # bad config
    bad = _dcfg(n_heads=3)
    assert lib.proxy_decode_step(ctypes.byref(bad), ctypes.byref(w), ctypes.byref(_dstate()), 0x70000, 0x80000,
                                 0x90000, ws, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_decode_workspace_size(ctypes.byref(bad)) == 0


def test_prefill_validation(lib):
    cfg = _dcfg()
    pws = int(lib.proxy_prefill_workspace_size(ctypes.byref(cfg), 10, 4))
    assert pws > int(lib.proxy_decode_workspace_size(ctypes.byref(cfg))) and pws % 256 == 0
    assert lib.proxy_prefill_workspace_size(ctypes.byref(cfg), -1, 4) == 0
    assert lib.proxy_prefill_workspace_size(ctypes.byref(_dcfg(n_heads=3)), 10, 4) == 0
    w = _dweights()

    def call(st, x=0x70000, n_tok=10, y=0x80000, ws=0x90000, nbytes=pws):
        return lib.proxy_decode_prefill(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), x, n_tok, y, ws,
                                        nbytes, None)

    # not at a block boundary
    st = _dstate(j=1)
    assert call(st) == B.PF_ERR_UNSUPPORTED
    # per-sequence positions
    import numpy as np
    st = _dstate()
    n_seq = np.zeros(2, np.int64)
    j_seq = np.zeros(2, np.int32)
    st.n_seq = n_seq.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    st.j_seq = j_seq.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert call(st) == B.PF_ERR_UNSUPPORTED
    # 10 tokens = 2 complete blocks of 4 into a cache with room for 1
    st = _dstate(n=3, n_cap=4)
    assert call(st) == B.PF_ERR_CAPACITY
    assert st.n == 3 and st.j == 0
    # workspace too small, negative count, aliasing, NULL input
    assert call(_dstate(), nbytes=pws - 256) == B.PF_ERR_WORKSPACE
    assert call(_dstate(), n_tok=-1) == B.PF_ERR_INVALID_ARG
    assert call(_dstate(), y=0x70000 + 256) == B.PF_ERR_INVALID_ARG
    assert call(_dstate(), x=None) == B.PF_ERR_INVALID_ARG
    # nothing to prefill is a no-op
    st = _dstate(n=1)
    assert call(st, n_tok=0, x=None, y=None) == B.PF_OK
    assert st.n == 1 and st.j == 0


def test_2d_partition_validation(lib):
    ok = _cfg(seq_len=64 * 64, factors=(64,))
    ok.image_width = 64
    assert B.layer_workspace_size(ok) > B.layer_workspace_size(_cfg(seq_len=64 * 64, factors=(64,)))
    for bad_w, fac, status in ((60, (64,), B.PF_ERR_INVALID_ARG),    # width not a multiple of p = 8
                               (48, (64,), B.PF_ERR_INVALID_ARG),    # 4096 / 48 is not whole
                               (64, (32,), B.PF_ERR_INVALID_ARG),    # P not a square
                               (64, (4, 16), B.PF_ERR_UNSUPPORTED),  # one level only
                               (-1, (64,), B.PF_ERR_INVALID_ARG)):
        c = _cfg(seq_len=64 * 64, factors=fac)
        c.image_width = bad_w
        assert _fwd(lib, c, _weights_struct(nlev=len(fac))) == status, (bad_w, fac)
        assert B.layer_workspace_size(c) == 0


def test_affine_weights_required_by_affine_injection(lib):
    cfg = _cfg(injection=2)
    assert B.layer_workspace_size(cfg) > 0 and B.layer_saved_size(cfg) > B.layer_saved_size(_cfg())
    w = _weights_struct(null="gate")   # the gate is not read with Eq. 13
    assert _fwd(lib, cfg, w) == B.PF_ERR_INVALID_ARG and "affine" in B.last_error()
    w.affine = B.PfLinear(0x10000, 0x10008)  # misaligned bias
    assert _fwd(lib, cfg, w) == B.PF_ERR_INVALID_ARG


def test_per_head_gate_shape_limits(lib):
    # d_fine = 256, 4 heads: 64 channels per head
    assert B.layer_workspace_size(_cfg(injection=3)) > 0
    # 256 / 8 heads = 32 channels: fine; d_fine = 24 over 4 heads = 6 channels: not a multiple of 8
    for kw, status in ((dict(d_fine=24), B.PF_ERR_UNSUPPORTED),
                       (dict(d_fine=4096 + 256, injection=3), B.PF_ERR_UNSUPPORTED)):
        c = _cfg(**kw)
        c.injection = 3
        assert _fwd(lib, c, _weights_struct()) == status, kw


def test_mfma_ceiling_rejects_bad_arguments(lib):
    """The ceiling probe validates on the host before it launches anything."""
    assert lib.proxy_ceiling_mfma(None, 16, 10, None) == B.PF_ERR_INVALID_ARG
    assert "out is NULL" in lib.proxy_last_error().decode()
    assert lib.proxy_ceiling_mfma(ctypes.c_void_p(0x90000), 0, 10, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_ceiling_mfma(ctypes.c_void_p(0x90000), (1 << 20) + 1, 10, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_ceiling_mfma(ctypes.c_void_p(0x90000), 16, 0, None) == B.PF_ERR_INVALID_ARG


def test_read_ceiling_rejects_bad_arguments(lib):
    """The read probe validates on the host before it launches anything
    (the pointers are never dereferenced)."""
    p = ctypes.c_void_p(0x90000)
    assert lib.proxy_ceiling_read(None, 1024, p, 16, None) == B.PF_ERR_INVALID_ARG
    assert "NULL" in lib.proxy_last_error().decode()
    assert lib.proxy_ceiling_read(p, 1024, None, 16, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_ceiling_read(ctypes.c_void_p(0x90008), 1024, p, 16, None) == B.PF_ERR_INVALID_ARG
    assert "aligned" in lib.proxy_last_error().decode()
    assert lib.proxy_ceiling_read(p, 0, p, 16, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_ceiling_read(p, 1000, p, 16, None) == B.PF_ERR_INVALID_ARG
    assert "multiple of 16" in lib.proxy_last_error().decode()
    assert lib.proxy_ceiling_read(p, 1024, p, 0, None) == B.PF_ERR_INVALID_ARG
    assert lib.proxy_ceiling_read(p, 1024, p, (1 << 20) + 1, None) == B.PF_ERR_INVALID_ARG


def test_static_decode_step_rejects_before_any_launch(lib):
    """proxy_decode_step_static validates on the host: bad arguments, and a
    step whose scratch would exceed the fixed 64 MiB array (64 sequences of
    16 x 128 channels over 2^20 cached rows: 256 slices of partials)."""
    cfg = B.decode_config(64, 2048, 16, 128, (64,))
    w = B.PfDecodeWeights()
    fake = 0x10000
    w.rms_gamma = fake
    for name in ("q", "k", "v", "o", "alpha", "k_proxy", "v_proxy"):
        setattr(w, name, B.PfLinear(fake, None))
    w.compress[0] = B.PfLinear(fake, None)
    st = B.PfDecodeState(fake, fake, 1 << 20, 1 << 20, fake, fake, fake, 0)
    step = lib.proxy_decode_step_static
    assert step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), 1 << 40, 2 << 40, None) == B.PF_ERR_UNSUPPORTED
    assert "static scratch" in B.last_error()
    assert st.n == 1 << 20 and st.j == 0  # nothing advanced
    assert step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), None, 2 << 40, None) == B.PF_ERR_INVALID_ARG
    st.j = 64  # j must be below P
    assert step(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(st), 1 << 40, 2 << 40, None) == B.PF_ERR_INVALID_ARG
