"""Host-side checks of the seeded workload generator."""
import numpy as np
import torch

from paper_2607_17733_amd import workloads as W


def test_width_counts_match_configs():
    assert W.width_counts(128, 0.10, 0.10) == (102, 13, 13)
    assert W.width_counts(128, 0.15, 0.15) == (90, 19, 19)
    assert W.width_counts(448, 0.15, 0.15) == (314, 67, 67)
    assert W.width_counts(256, 0.10, 0.05) == (217, 26, 13)
    assert W.width_counts(896, 0.10, 0.05) == (761, 90, 45)
    assert W.width_counts(256, 0.10, 0.30) == (153, 26, 77)
    assert W.width_counts(896, 0.10, 0.30) == (537, 90, 269)


def test_bf16_conversion_is_round_to_nearest_even():
    g = np.random.default_rng(0)
    x = (g.standard_normal(100000) * np.exp2(g.integers(-60, 60, 100000))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.to_bf16_bits(x), ref)


def test_tiny_case_structure():
    c = W.tiny()
    assert (c.M, c.K, c.N) == (16, 256, 256)
    assert sorted(c.perm.tolist()) == list(range(256))
    assert c.widths.tolist() == [4] * 6 + [6, 8]
    a = W.bf16_bits_to_f32(c.a_bits)
    big = np.where(np.abs(a).max(axis=0) > 20)[0]
    assert len(big) == 2
    assert set(big.tolist()) <= set(c.perm[224:].tolist())   # in the 8-bit block
    c2 = W.tiny()
    assert np.array_equal(c.a_bits, c2.a_bits) and np.array_equal(c.w_bits, c2.w_bits)


def test_outlier_channels_fill_high_precision_blocks():
    c = W.make_linear(2, "t", 8, 4096, 16, 0.10, 0.10)
    scales = W.channel_scales(2, 4096)
    n8 = c.meta["n8"]
    eight = c.perm[-32 * n8:]
    assert np.all(scales[eight].min() >= scales[c.perm[: -32 * n8]].max())
    assert (scales > 1).sum() == 41 + 205
