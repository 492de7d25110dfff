#!/usr/bin/env python3
"""Throughput of the ProxyFormer hot path on one MI355X; prints one JSON line.

value: layer-forward tokens/s on the 1M-token workload (batch 1, L = 1,048,576,
d = 1024, 16 heads x 64, P = 64, bf16 with fp32 accumulation), inputs resident
in HBM, W untimed warmup calls then K timed calls bracketed by
torch.cuda.synchronize() and HIP events on the launch stream.

Extra objects on the same line:
  kernels      per-kernel average duration from the library's event tracing
               (a second pass over K calls) and achieved TFLOP/s or GB/s
  variants     the same forward with residual-add injection (Eq. 11), affine
               modulation (Eq. 13) and the per-head gate
  ceilings     a 1 GiB device copy and a 2 GiB read-only stream (achievable HBM
               rates) and an MFMA-only loop (achievable dense bf16 rate) beside
               the vendor peaks
  roofline     the dominant kernel against the MI355X peak of its bound, with
               its matrix-core busy fraction and clock from the committed
               counter summary (while the kernel sources are unchanged) and
               the socket power under sustained forwards (amd-smi, if present)
  decode       proxy-KV decode tokens/s: 32 sequences, 16,384 cached proxy
               rows each, 256 new tokens per sequence including the 4
               block-triggered appends
  train        forward (saving activations) + backward tokens/s on the
               factorised workload (L = 262,144, d = 2048, 16 x 128, P = 8 x 8)
  lm           the paper's language-model shape: layer forward tokens/s at
               L = 1M with a 64-wide local stream and a 512-wide proxy stream
               (8 x 64, P = 64), and decode tokens/s at d_model = 512
  prefill      parallel form of the generation block: the next 4,096 tokens
               of 32 sequences against 16,384 cached proxies (d = 1024,
               16 x 64, P = 64), the chunk's 64 blocks per sequence appended
  cpu_baseline the CPU oracle timed on a bounded sample of the same workload
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ProxyFormer layer fwd tokens/sec at L=1M, P=64; proxy-KV decode tokens/sec"
LAYER_WORKLOAD = "layer_bf16_L1M_d1024"
DECODE_WORKLOAD = "decode_bf16_B32_n16k"
TRAIN_WORKLOAD = "layer_bf16_L256k_d2048_f8x8"
LM_LAYER_WORKLOAD = "layer_bf16_L1M_lm_df64_dp512"
LM_DECODE_WORKLOAD = "decode_bf16_B32_n16k_lm_d512"
PREFILL_WORKLOAD = "prefill_bf16_B32_T4096_n16k"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0
CPU_SAMPLE_TOKENS = 393216
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_layer_bf16_L1M_d1024_decode_bf16_B32_n16k.txt")
MFMA_FILE = os.path.join(ROOT, "profiles", "mfma_counters_layer_bf16_L1M_d1024_decode_bf16_B32_n16k.txt")
KERNEL_SOURCES = ["paper_2608_23463_amd/csrc/gemm.hpp", "paper_2608_23463_amd/csrc/epilogues.hpp",
                  "paper_2608_23463_amd/csrc/common.hpp", "paper_2608_23463_amd/csrc/attention.hpp",
                  "paper_2608_23463_amd/csrc/attention_fwd.hip", "paper_2608_23463_amd/csrc/layer_fwd.hip",
                  "paper_2608_23463_amd/csrc/decode.hip", "paper_2608_23463_amd/csrc/decode.hpp"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def counter_value(path: str, key: str):
    """Value of `key` in a committed counter summary, or None when the summary
    is missing or the kernel sources changed since the counters were taken."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return None
    v = vals.get(key)
    return float(v) if v else None


def measured_traffic(label: str):
    """HBM bytes per launch of `label` (FETCH_SIZE and WRITE_SIZE passes)."""
    return counter_value(TRAFFIC_FILE, f"{label}_bytes_per_launch")


def measured_mfma(label: str):
    """Matrix-core busy fraction of `label` at the clock it ran at, and that
    clock in GHz (SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE pass)."""
    util = counter_value(MFMA_FILE, f"{label}_mfma_util")
    clk = counter_value(MFMA_FILE, f"{label}_clock_ghz")
    return (util, clk) if util is not None and clk is not None else None


def layer_flops(shape):
    """Algorithmic flops per launch of each forward kernel (multiply-add = 2)."""
    B, L, df, dp = shape.batch, shape.seq_len, shape.d_fine, shape.d_proxy
    P = shape.block
    m = L // P
    dims = shape.dims()
    comp = 0
    rows = B * L
    for j, k in enumerate(shape.factors):
        rows //= k
        comp += 2 * rows * (k * dims[j]) * dims[j + 1]
    return {
        "compress_gemm": comp / len(shape.factors),
        "qkv_gemm": 2 * B * m * dp * dp,
        "attention_fwd": 2.0 * B * dp * m * (m + 1),   # QK^T and PV over the causal triangle
        "o_gemm": 2 * B * m * dp * dp,
        "decompress_gemm": comp / len(shape.factors),
        "gate_gemm": 2 * B * L * df * 2 * df,
        # PF_GATE_FUSED: D = S W_d[p]^T and G = S C[p]^T + X_p W_gx^T per token,
        # after the fold C[p] = W_gd W_d[p] for the k_1 positions
        "fused_gate": 2 * B * L * df * (2 * dims[1] + df),
        "gate_fold_gemm": 2 * shape.factors[0] * df * df * dims[1],
    }


def to_dev(a, dt):
    import numpy as np
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")
    return t.to(torch.bfloat16 if dt == "bf16" else torch.float32)


def dev_weights(w, dt):
    out = {}
    for k, v in w.items():
        if isinstance(v, list):
            out[k] = [(to_dev(a, dt), to_dev(b, dt)) for a, b in v]
        elif isinstance(v, tuple):
            out[k] = (to_dev(v[0], dt), to_dev(v[1], dt))
        else:
            out[k] = to_dev(v, dt)
    return out


def time_calls(call, steps, warmup):
    """Average milliseconds of `call` over `steps` timed calls after `warmup`
    untimed ones (HIP events on torch's current stream, which the library's
    launches use)."""
    import torch
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        call()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def trace_calls(call, steps):
    """{label: (launches, total_ms)} of the library's launches over `steps` calls."""
    import torch
    from paper_2608_23463_amd import binding as B
    B.trace_reset()
    B.trace_enable(True)
    for _ in range(steps):
        call()
    torch.cuda.synchronize()
    tr = B.trace_collect()
    B.trace_enable(False)
    return tr


def attention_roofline(tr, flops, steps):
    """The proxy attention's algorithmic TFLOP/s from a trace."""
    cnt, tot = tr["attention_fwd"]
    avg = tot / cnt
    tf = flops["attention_fwd"] / (avg * 1e-3) / 1e12
    return {"kernel": "attention_fwd", "bound": "mfma", "achieved": round(tf, 1), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4), "avg_ms": round(avg, 4),
            "work_per_launch": flops["attention_fwd"]}


def kernel_table(tr, flops, steps, counters: bool):
    """Per-kernel entries of a trace: launches per call, average duration,
    algorithmic TFLOP/s, and (for the headline workload, while the kernel
    sources match the committed summaries) counter HBM rate and matrix-core
    busy fraction."""
    kernels = {}
    for label, (cnt, tot) in tr.items():
        avg = tot / cnt
        ent = {"launches_per_step": cnt / steps, "avg_ms": round(avg, 4)}
        if label in flops:
            ent["tflops"] = round(flops[label] / (avg * 1e-3) / 1e12, 1)
        hbm = measured_traffic(label) if counters else None
        if hbm:  # measured HBM bytes per launch over this run's duration
            ent["hbm_gbs"] = round(hbm / (avg * 1e-3) / 1e9, 1)
        mf = measured_mfma(label) if counters else None
        if mf:  # counters: matrix cores busy at the clock the kernel ran at
            ent["mfma_util_counters"], ent["clock_ghz_counters"] = mf
        kernels[label] = ent
    return kernels


def socket_power(call, seconds=2.5):
    """Socket power of GPU 0 (W, from `amd-smi metric -p -g 0`) while `call`
    runs back to back for about `seconds`: one reading before the load and
    the median and maximum of the readings taken after the first 0.75 s of
    load (the tool's figure lags by a few hundred milliseconds). None where
    amd-smi is not available or prints no socket power."""
    import re
    import shutil
    import subprocess
    import threading
    import torch
    exe = shutil.which("amd-smi")
    if exe is None:
        return None

    def read():
        try:
            r = subprocess.run([exe, "metric", "-p", "-g", "0"], capture_output=True, text=True, timeout=10)
        except (OSError, subprocess.SubprocessError):
            return None
        m = re.search(r"SOCKET_POWER:\s*([0-9.]+)\s*W", r.stdout)
        return float(m.group(1)) if m else None

    idle = read()
    samples = []
    stop = threading.Event()
    t0 = time.time()

    def sampler():
        while not stop.is_set():
            v = read()
            if v is not None and time.time() - t0 > 0.75:
                samples.append(v)
            time.sleep(0.2)

    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    while time.time() - t0 < seconds:
        for _ in range(10):
            call()
        torch.cuda.synchronize()
    stop.set()
    th.join(timeout=15)
    if not samples:
        return None
    samples.sort()
    return {"gpu": 0, "before_load_w": idle, "under_load_median_w": samples[len(samples) // 2],
            "under_load_max_w": samples[-1], "readings": len(samples), "load": "layer forwards back to back"}


def bench_layer(steps, warmup, workload=LAYER_WORKLOAD):
    import torch
    from paper_2608_23463_amd import binding as B
    from paper_2608_23463_amd import synth
    shape = synth.WORKLOADS[workload]
    headline = workload == LAYER_WORKLOAD
    log(f"generating {workload} inputs")
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[workload])
    sample = None
    if headline:
        sample = {"x": inp["x"][:, :CPU_SAMPLE_TOKENS].copy(), "weights": inp["weights"]}
    x = to_dev(inp["x"], shape.dtype)
    del inp["x"]
    w = dev_weights(inp["weights"], shape.dtype)
    cfg = B.config_from_shape(shape)
    ws = torch.empty(B.layer_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    m = shape.n_proxies
    x_out = torch.empty_like(x)
    h_out = torch.empty((1, m, shape.d_proxy), dtype=x.dtype, device="cuda")
    wst = B.layer_weights(w)
    tokens = shape.seq_len * shape.batch

    def forward(c, weights=wst, workspace=ws):
        return lambda: B.layer_forward_raw(c, weights, x, None, x_out, h_out, None, workspace)

    log(f"timing {steps} forward calls after {warmup} warmup calls")
    ms = time_calls(forward(cfg), steps, warmup)
    log("tracing per-kernel durations")
    tr = trace_calls(forward(cfg), steps)
    flops = layer_flops(shape)
    kernels = kernel_table(tr, flops, steps, headline)
    dom = max((k for k in tr if k in flops), key=lambda k: tr[k][1])
    dom_ms = tr[dom][1] / tr[dom][0]
    achieved = flops[dom] / (dom_ms * 1e-3) / 1e12
    # the committed counter summary covers the headline workload only
    traffic = measured_traffic(dom) if headline else None
    roof = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic, "work_per_launch": flops[dom], "avg_ms": round(dom_ms, 4)}
    mf = measured_mfma(dom) if headline else None
    if mf:
        roof["mfma_util_counters"], roof["clock_ghz_counters"] = mf
    if headline:
        log("sampling socket power under sustained forwards")
        roof["socket_power"] = socket_power(forward(cfg))

    def entry(ms_v, **extra):
        return {"ms_per_step": round(ms_v, 4), "value": round(tokens / (ms_v * 1e-3), 1), "unit": "tokens/s",
                **extra}

    variants = {"attention_extended": attention_roofline(tr, flops, steps)}
    # plain bf16 H, Q, K (PF_PRECISION_BF16): one score MFMA per tile step
    cfg_p = B.config_from_shape(shape)
    cfg_p.precision = B.PF_PRECISION_BF16
    ws_p = torch.empty(B.layer_workspace_size(cfg_p), dtype=torch.uint8, device="cuda")
    ms_p = time_calls(forward(cfg_p, workspace=ws_p), steps, warmup)
    tr_p = trace_calls(forward(cfg_p, workspace=ws_p), steps)
    variants["precision_bf16"] = entry(ms_p, attention=attention_roofline(tr_p, flops, steps),
                                       kernels=kernel_table(tr_p, flops, steps, False))
    del ws_p
    if headline:
        # PF_GATE_FUSED: level-1 decompression, gate and residual in one kernel
        # (Delta stays in registers) after the per-position weight fold
        cfg_f = B.config_from_shape(shape)
        cfg_f.gate_fusion = B.PF_GATE_FUSED
        ws_f = torch.empty(B.layer_workspace_size(cfg_f), dtype=torch.uint8, device="cuda")
        ms_f = time_calls(forward(cfg_f, workspace=ws_f), steps, warmup)
        tr_f = trace_calls(forward(cfg_f, workspace=ws_f), steps)
        variants["gate_fused"] = entry(ms_f, kernels=kernel_table(tr_f, flops, steps, False))
        del ws_f
        # the same inputs with residual-add injection (Eq. 11): no gate GEMM
        cfg_add = B.config_from_shape(shape)
        cfg_add.injection = B.PF_INJECT_ADD
        ws_add = torch.empty(B.layer_workspace_size(cfg_add), dtype=torch.uint8, device="cuda")
        variants["inject_add"] = entry(time_calls(forward(cfg_add, workspace=ws_add), steps, warmup))
        del ws_add
        # affine modulation (Eq. 13): [S | T] GEMM (N = 2 d_fine, K = d_fine) instead of the gate
        cfg_aff = B.config_from_shape(shape)
        cfg_aff.injection = B.PF_INJECT_AFFINE
        gen = torch.Generator(device="cuda")
        gen.manual_seed(13)
        w_aff = dict(w)
        w_aff["affine"] = ((torch.randn(2 * shape.d_fine, shape.d_fine, generator=gen, device="cuda") * 0.02)
                           .to(x.dtype), torch.zeros(2 * shape.d_fine, dtype=x.dtype, device="cuda"))
        ws_aff = torch.empty(B.layer_workspace_size(cfg_aff), dtype=torch.uint8, device="cuda")
        variants["inject_affine"] = entry(time_calls(forward(cfg_aff, B.layer_weights(w_aff), ws_aff), steps,
                                                     warmup))
        del ws_aff, w_aff
        # per-head gate (Eq. 12 with one gate per head): N = n_heads gate GEMM and a combine pass
        cfg_gh = B.config_from_shape(shape)
        cfg_gh.injection = B.PF_INJECT_GATED_HEAD
        w_gh = dict(w)
        w_gh["gate"] = ((torch.randn(shape.n_heads, 2 * shape.d_fine, generator=gen, device="cuda") * 0.02)
                        .to(x.dtype), torch.zeros(shape.n_heads, dtype=x.dtype, device="cuda"))
        ws_gh = torch.empty(B.layer_workspace_size(cfg_gh), dtype=torch.uint8, device="cuda")
        variants["inject_gated_head"] = entry(time_calls(forward(cfg_gh, B.layer_weights(w_gh), ws_gh), steps,
                                                         warmup))
        del ws_gh, w_gh
    del x, x_out, h_out, ws, w
    torch.cuda.empty_cache()
    return shape, ms, kernels, roof, sample, variants


def hbm_copy_ceiling():
    """Achievable HBM rate on this device: a 1 GiB device-to-device copy
    (reads and writes 1 GiB), best of five."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    b.copy_(a)
    torch.cuda.synchronize()
    best = None
    for _ in range(5):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        b.copy_(a)
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop)
        best = ms if best is None else min(best, ms)
    del a, b
    torch.cuda.empty_cache()
    return round(2 * n / (best * 1e-3) / 1e9, 1)


def hbm_read_ceiling():
    """Achievable HBM read rate on this device: the library's read probe
    (grid-strided 16-byte loads, nothing else) over a 2 GiB buffer, 4,096
    workgroups, ten calls back to back, best of three."""
    import torch
    from paper_2608_23463_amd import binding as B
    n, n_wg, calls = 2 << 30, 4096, 10
    src = torch.zeros(n, dtype=torch.uint8, device="cuda")
    out = torch.empty(n_wg, dtype=torch.int32, device="cuda")
    B.ceiling_read(src, out, n_wg)
    torch.cuda.synchronize()
    best = None
    for _ in range(3):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(calls):
            B.ceiling_read(src, out, n_wg)
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop) / calls
        best = ms if best is None else min(best, ms)
    del src, out
    torch.cuda.empty_cache()
    return round(n / (best * 1e-3) / 1e9, 1)


def mfma_ceiling():
    """Achievable dense bf16 MFMA rate on this device: the library's MFMA-only
    loop (1,024 workgroups of four waves, no memory traffic), best of three."""
    import torch
    from paper_2608_23463_amd import binding as B
    n_wg, iters = 1024, 20000
    out = torch.empty(n_wg * 256, dtype=torch.float32, device="cuda")
    B.ceiling_mfma(out, n_wg, 100)
    torch.cuda.synchronize()
    best = None
    for _ in range(3):
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        B.ceiling_mfma(out, n_wg, iters)
        stop.record()
        torch.cuda.synchronize()
        ms = start.elapsed_time(stop)
        best = ms if best is None else min(best, ms)
    flops = n_wg * 4 * iters * 8 * 32768
    return round(flops / (best * 1e-3) / 1e12, 1)


def bench_decode(workload=DECODE_WORKLOAD):
    import numpy as np
    import torch
    from paper_2608_23463_amd import binding as B
    from paper_2608_23463_amd import synth
    shape = synth.WORKLOADS[workload]
    log(f"generating {workload} inputs")
    inp = synth.decode_inputs(shape, synth.WORKLOAD_SEEDS[workload])
    cfg = B.decode_config(shape.batch, shape.d_model, shape.n_heads, shape.head_dim, shape.factors,
                          shape.level_dims, shape.dtype, shape.rms_eps)
    kc = to_dev(inp.pop("k_cache"), shape.dtype)
    vc = to_dev(inp.pop("v_cache"), shape.dtype)
    xs = to_dev(inp["x"], shape.dtype)
    sess = B.DecodeSession(cfg, dev_weights(inp["weights"], shape.dtype), kc, vc, n=shape.n0)
    ys = torch.empty_like(xs)

    def run_all():
        sess.state.n = shape.n0
        sess.state.j = 0
        for t in range(shape.steps):
            sess.step(xs[t], ys[t])

    log("decode warmup")
    run_all()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {shape.steps} decode steps")
    start.record()
    run_all()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop)
    B.trace_reset()
    B.trace_enable(True)
    run_all()
    torch.cuda.synchronize()
    tr = B.trace_collect()
    B.trace_enable(False)
    attn = tr.get("decode_attn")
    out = {"metric": "proxy-KV decode tokens/s", "value": round(shape.batch * shape.steps / (ms * 1e-3), 1),
           "unit": "tokens/s", "ms_total": round(ms, 3), "ms_per_step": round(ms / shape.steps, 4),
           "workload": workload, "batch": shape.batch, "cached_rows": shape.n0, "steps": shape.steps,
           "appends": shape.steps // shape.block}
    if attn:
        avg = attn[1] / attn[0]
        # K and V rows read per step: every cached row once (n grows by one per block)
        n_mean = shape.n0 + (shape.steps // shape.block) / 2.0
        nbytes = 2 * shape.batch * shape.n_heads * n_mean * shape.head_dim * 2
        gbs = nbytes / (avg * 1e-3) / 1e9
        out["roofline"] = {"kernel": "decode_attn", "bound": "hbm", "achieved": round(gbs, 1),
                           "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                           "traffic": measured_traffic("decode_attn") if workload == DECODE_WORKLOAD else None,
                           "avg_ms": round(avg, 4),
                           "work_per_launch": nbytes}
        # the whole step (projections, merge and output map included) against HBM
        step_gbs = nbytes / (ms / shape.steps * 1e-3) / 1e9
        out["step_hbm"] = {"achieved": round(step_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                           "frac": round(step_gbs / PEAK_HBM_GBS, 4)}
    out["kernels"] = {k: {"launches": c, "avg_ms": round(t / c, 4)} for k, (c, t) in tr.items()}
    del kc, vc, xs, ys, sess
    torch.cuda.empty_cache()
    return out


def prefill_attn_flops(shape):
    """Algorithmic MFMA flops of the prefill attention: 4 * d_head per visible
    (token, key) pair and head; token t sees t % P + 1 tokens of its block and
    n0 + t // P cached proxies."""
    P, T = shape.block, shape.steps
    pairs = 0
    for t in range(T):
        pairs += t % P + 1 + shape.n0 + t // P
    return 4.0 * shape.head_dim * shape.batch * shape.n_heads * pairs


def bench_prefill(workload=PREFILL_WORKLOAD, calls=3):
    import numpy as np
    import torch
    from paper_2608_23463_amd import binding as B
    from paper_2608_23463_amd import synth
    shape = synth.WORKLOADS[workload]
    log(f"generating {workload} inputs")
    inp = synth.decode_inputs(shape, synth.WORKLOAD_SEEDS[workload])
    cfg = B.decode_config(shape.batch, shape.d_model, shape.n_heads, shape.head_dim, shape.factors,
                          shape.level_dims, shape.dtype, shape.rms_eps)
    kc = to_dev(inp.pop("k_cache"), shape.dtype)
    vc = to_dev(inp.pop("v_cache"), shape.dtype)
    x = to_dev(np.ascontiguousarray(inp.pop("x").transpose(1, 0, 2)), shape.dtype)   # [B, T, d]
    sess = B.DecodeSession(cfg, dev_weights(inp["weights"], shape.dtype), kc, vc, n=shape.n0)
    y = torch.empty_like(x)

    def one():
        sess.state.n = shape.n0   # every call prefills the same chunk onto the same cache
        sess.state.j = 0
        sess.prefill(x, y)

    log("prefill warmup")
    one()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {calls} prefill calls")
    start.record()
    for _ in range(calls):
        one()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / calls
    B.trace_reset()
    B.trace_enable(True)
    for _ in range(calls):
        one()
    torch.cuda.synchronize()
    tr = B.trace_collect()
    B.trace_enable(False)
    toks = shape.batch * shape.steps
    out = {"metric": "prefill tokens/s (parallel generation block)", "value": round(toks / (ms * 1e-3), 1),
           "unit": "tokens/s", "ms_per_call": round(ms, 3), "workload": workload, "batch": shape.batch,
           "chunk_tokens": shape.steps, "cached_rows": shape.n0, "appended_blocks": shape.steps // shape.block}
    attn = tr.get("prefill_attn")
    if attn:
        avg = attn[1] / attn[0]
        fl = prefill_attn_flops(shape)
        tf = fl / (avg * 1e-3) / 1e12
        out["roofline"] = {"kernel": "prefill_attn", "bound": "mfma", "achieved": round(tf, 1),
                           "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(tf / PEAK_BF16_TFLOPS, 4),
                           "traffic": None, "avg_ms": round(avg, 4), "work_per_launch": fl}
    out["kernels"] = {k: {"launches": c, "avg_ms": round(t / c, 4)} for k, (c, t) in tr.items()}
    del kc, vc, x, y, sess
    torch.cuda.empty_cache()
    return out


def bench_train(steps):
    import torch
    from paper_2608_23463_amd import binding as B
    from paper_2608_23463_amd import synth
    shape = synth.WORKLOADS[TRAIN_WORKLOAD]
    log(f"generating {TRAIN_WORKLOAD} inputs")
    inp = synth.layer_inputs(shape, synth.WORKLOAD_SEEDS[TRAIN_WORKLOAD], with_dy=True)
    x = to_dev(inp.pop("x"), shape.dtype)
    dy = to_dev(inp.pop("dy"), shape.dtype)
    w = dev_weights(inp["weights"], shape.dtype)
    cfg = B.config_from_shape(shape)
    ws_f = torch.empty(B.layer_workspace_size(cfg, False), dtype=torch.uint8, device="cuda")
    ws_b = torch.empty(B.layer_workspace_size(cfg, True), dtype=torch.uint8, device="cuda")
    saved = torch.empty(B.layer_saved_size(cfg), dtype=torch.uint8, device="cuda")
    x_out = torch.empty_like(x)
    h_out = torch.empty((1, shape.n_proxies, shape.d_proxy), dtype=x.dtype, device="cuda")
    wst = B.layer_weights(w)

    def step():
        B.layer_forward_raw(cfg, wst, x, None, x_out, h_out, saved, ws_f)
        B.layer_backward(cfg, w, x, None, saved, dy, workspace=ws_b)

    log("train warmup")
    step()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"timing {steps} forward+backward steps")
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / steps
    B.trace_reset()
    B.trace_enable(True)
    step()
    torch.cuda.synchronize()
    tr = B.trace_collect()
    B.trace_enable(False)
    out = {"metric": "layer forward+backward tokens/s", "value": round(shape.seq_len / (ms * 1e-3), 1),
           "unit": "tokens/s", "ms_per_step": round(ms, 3), "workload": TRAIN_WORKLOAD,
           "seq_len": shape.seq_len, "d": shape.d_fine, "levels": list(shape.factors),
           "kernels": {k: {"launches": c, "avg_ms": round(t / c, 4)} for k, (c, t) in tr.items()}}
    del x, dy, w, ws_f, ws_b, saved, x_out, h_out
    torch.cuda.empty_cache()
    return out


def cpu_model() -> str:
    """Model name of the host CPU (first entry of /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(shape, sample):
    import oracle
    nproc = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    try:  # the threads numpy's BLAS runs the oracle's matrix products on
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = nproc
    log(f"oracle on {CPU_SAMPLE_TOKENS} tokens")
    t0 = time.perf_counter()
    oracle.layer_forward(sample["x"], sample["weights"], shape.factors, shape.n_heads, shape.mask)
    dt = time.perf_counter() - t0
    return {"value": round(CPU_SAMPLE_TOKENS / dt, 1), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "nproc": nproc, "cpu_count": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"full layer forward (fp64) over the first {CPU_SAMPLE_TOKENS} tokens "
                      f"({CPU_SAMPLE_TOKENS // shape.block} blocks) of the 1M-token workload; cores = BLAS "
                      f"threads of the oracle's matrix products, nproc = CPUs this process may run on",
            "seconds": round(dt, 2)}


def pmc_pass():
    """Minimal dispatch sequence for hardware-counter runs: two layer forwards
    on the 1M-token shape, one more with the fused decompression + gate kernel,
    and two decode steps at the decode workload's shape
    (random device data; traffic does not depend on the values), then one
    plain 1 GiB device-to-device copy whose FETCH_SIZE and WRITE_SIZE
    calibrate the counters (it must read and write 1 GiB)."""
    import torch
    from paper_2608_23463_amd import binding as B
    from paper_2608_23463_amd import synth
    B.load()
    shape = synth.WORKLOADS[LAYER_WORKLOAD]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(0)
    dt = torch.bfloat16

    def rn(*sz, std=1.0):
        return (torch.randn(*sz, generator=gen, device="cuda") * std).to(dt)

    wsh = shape.weight_shapes()
    w = {"compress": [(rn(*z, std=0.02), None) for z in wsh["compress"]],
         "decompress": [(rn(*z, std=0.02), None) for z in wsh["decompress"]]}
    for k in ("q", "k", "v", "o", "gate"):
        w[k] = (rn(*wsh[k], std=0.02), None)
    x = rn(shape.batch, shape.seq_len, shape.d_fine)
    cfg = B.config_from_shape(shape)
    ws = torch.empty(B.layer_workspace_size(cfg), dtype=torch.uint8, device="cuda")
    x_out = torch.empty_like(x)
    h_out = torch.empty((1, shape.n_proxies, shape.d_proxy), dtype=dt, device="cuda")
    wst = B.layer_weights(w)
    for _ in range(2):
        B.layer_forward_raw(cfg, wst, x, None, x_out, h_out, None, ws)
        torch.cuda.synchronize()
    del ws
    # one forward through the fused decompression + gate kernel
    cfg_f = B.config_from_shape(shape)
    cfg_f.gate_fusion = B.PF_GATE_FUSED
    ws = torch.empty(B.layer_workspace_size(cfg_f), dtype=torch.uint8, device="cuda")
    B.layer_forward_raw(cfg_f, wst, x, None, x_out, h_out, None, ws)
    torch.cuda.synchronize()
    del x, x_out, h_out, ws, w, wst
    torch.cuda.empty_cache()
    # two decode steps at the decode workload's shape (random device data)
    ds = synth.WORKLOADS[DECODE_WORKLOAD]
    dcfg = B.decode_config(ds.batch, ds.d_model, ds.n_heads, ds.head_dim, ds.factors, ds.level_dims, ds.dtype,
                           ds.rms_eps)
    cache_shape = (ds.batch, ds.n_heads, ds.n0 + ds.steps // ds.block + 1, ds.head_dim)
    kc = rn(*cache_shape)
    vc = rn(*cache_shape)
    dw = {"rms_gamma": torch.ones(ds.d_model, dtype=dt, device="cuda")}
    for k, (o, i) in {"q": (ds.d_model, ds.d_model), "k": (ds.d_model, ds.d_model), "v": (ds.d_model, ds.d_model),
                      "o": (ds.d_model, ds.d_model), "alpha": (ds.n_heads, ds.d_model),
                      "k_proxy": (ds.d_model, ds.d_model), "v_proxy": (ds.d_model, ds.d_model)}.items():
        dw[k] = (rn(o, i, std=0.02), None)
    dd = ds.dims()
    dw["compress"] = [(rn(dd[j + 1], ds.factors[j] * dd[j], std=0.02), None) for j in range(len(ds.factors))]
    sess = B.DecodeSession(dcfg, dw, kc, vc, n=ds.n0)
    xs = rn(2, ds.batch, ds.d_model)
    ys = torch.empty_like(xs)
    for t in range(2):
        sess.step(xs[t], ys[t])
        torch.cuda.synchronize()
    del sess, kc, vc
    torch.cuda.empty_cache()
    a = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    print("pmc pass done: 2 forwards, 1 fused-gate forward, 2 decode steps, 1 GiB copy", flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-train", action="store_true")
    ap.add_argument("--no-lm", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="only the short dispatch sequence used for counter runs (prints no JSON)")
    args = ap.parse_args()
    if args.pmc_pass:
        pmc_pass()
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library runs the hot path on a single MI355X and has no "
              "multi-GPU path; run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2608_23463_amd import binding as B
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.load()
    shape, ms, kernels, roof, sample, variants = bench_layer(args.steps, args.warmup)
    result = {
        "metric": METRIC,
        "value": round(shape.seq_len * shape.batch / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": LAYER_WORKLOAD, "batch": shape.batch, "seq_len": shape.seq_len,
                   "d_fine": shape.d_fine, "d_proxy": shape.d_proxy, "n_heads": shape.n_heads,
                   "head_dim": shape.head_dim, "P": shape.block, "levels": list(shape.factors),
                   "proxy_precision": "extended (bf16 hi/lo parts of H, Q, K)",
                   "parallelism": "single GPU"},
        "roofline": roof,
        "kernels": kernels,
        "variants": variants,
        "ceilings": {"hbm_copy_gbs": hbm_copy_ceiling(), "hbm_read_gbs": hbm_read_ceiling(),
                     "hbm_peak_gbs": PEAK_HBM_GBS,
                     "mfma_loop_bf16_tflops": mfma_ceiling(),
                     "mfma_bf16_peak_tflops": PEAK_BF16_TFLOPS},
    }
    if not args.no_decode:
        result["decode"] = bench_decode()
    if not args.no_train:
        result["train"] = bench_train(max(1, min(args.steps, 5)))
    if not args.no_prefill:
        result["prefill"] = bench_prefill()
    if not args.no_lm:
        lshape, lms, lkernels, lroof, _, lvariants = bench_layer(args.steps, args.warmup, LM_LAYER_WORKLOAD)
        result["lm"] = {"metric": "layer fwd tokens/s (language-model shape)",
                        "value": round(lshape.seq_len * lshape.batch / (lms * 1e-3), 1), "unit": "tokens/s",
                        "ms_per_step": round(lms, 4), "workload": LM_LAYER_WORKLOAD, "d_fine": lshape.d_fine,
                        "d_proxy": lshape.d_proxy, "n_heads": lshape.n_heads, "roofline": lroof,
                        "kernels": lkernels, "variants": lvariants}
        if not args.no_decode:
            result["lm"]["decode"] = bench_decode(LM_DECODE_WORKLOAD)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(shape, sample)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
