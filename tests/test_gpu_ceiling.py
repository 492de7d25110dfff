"""The ceiling probes (proxy_ceiling_mfma, proxy_ceiling_read) through the C ABI.

Read probe: the XOR over its per-workgroup outputs equals the XOR of every
32-bit word of the buffer, which shows each word was read exactly once (a
word read twice or skipped changes the XOR for almost every pattern).

Matrix-core probe:

Every thread's output is predictable on the CPU: each wave multiplies the
same 32x16 by 16x32 bf16 tiles (lane l supplies row / column l % 32 and
k = 8 (l / 32) .. +7) into eight accumulators, iters times, and writes the
sum of its 8 x 16 accumulator registers; register r of lane l holds row
8 (r / 4) + 4 (l / 32) + r % 4 of column l % 32. A match shows the probe ran
exactly iters x 8 MFMAs per wave, which is what its flop count assumes.
"""
import numpy as np
import pytest

from paper_2608_23463_amd import synth

pytestmark = pytest.mark.gpu


def expected_outputs(n_workgroups: int, iters: int) -> np.ndarray:
    # operands formed as the kernel forms them: an fp32 product, rounded to bf16
    a = np.zeros((32, 16), dtype=np.float32)
    bt = np.zeros((32, 16), dtype=np.float32)  # B transposed: [column, k]
    for lane in range(64):
        g = lane // 32
        for e in range(8):
            a[lane % 32, 8 * g + e] = np.float32(0.001) * np.float32((lane + e) & 7)
            bt[lane % 32, 8 * g + e] = np.float32(0.002) * np.float32((lane * 3 + e) & 7)
    a = synth.bf16_round(a).astype(np.float64)
    bt = synth.bf16_round(bt).astype(np.float64)
    c = a @ bt.T  # [row, column]
    per_lane = np.zeros(64)
    for lane in range(64):
        rows = [8 * (r // 4) + 4 * (lane // 32) + r % 4 for r in range(16)]
        per_lane[lane] = 8 * iters * c[rows, lane % 32].sum()
    return np.tile(per_lane, 4 * n_workgroups)


def test_mfma_ceiling_matches_the_predicted_sums(gpu):
    import torch
    from paper_2608_23463_amd import binding as B
    n_wg, iters = 6, 37
    out = torch.full((n_wg * 256,), float("nan"), dtype=torch.float32, device="cuda")
    B.ceiling_mfma(out, n_wg, iters)
    again = torch.empty_like(out)
    B.ceiling_mfma(again, n_wg, iters)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = expected_outputs(n_wg, iters)
    assert np.isfinite(got).all()
    assert np.abs(got - ref).max() <= 1e-5 * np.abs(ref).max(), np.abs(got - ref).max()
    assert torch.equal(out, again)


@pytest.mark.parametrize("words,n_wg", [(4 * 1000, 3), (4 * 256 * 4 * 7 + 12, 5), (1 << 20, 64)])
def test_read_ceiling_reads_every_word_once(gpu, words, n_wg):
    import torch
    from paper_2608_23463_amd import binding as B
    rng = np.random.default_rng(words + n_wg)
    host = rng.integers(-(1 << 31), (1 << 31) - 1, size=words, dtype=np.int64).astype(np.int32)
    src = torch.from_numpy(host).to("cuda")
    out = torch.zeros(n_wg, dtype=torch.int32, device="cuda")
    B.ceiling_read(src, out, n_wg)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host.view(np.uint32))
