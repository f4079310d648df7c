"""Pins of the fused-producer oracle (RMS normalisation before the
quantizer) against things other than itself: exact rationals, closed forms,
power-of-two scale invariance, torch's float32 RMS normalisation."""
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import fused


def _bf16(a):
    return fused.f32_to_bf16(np.asarray(a, dtype=np.float32))


def test_f32_to_bf16_round_to_nearest_even():
    # 1 + 2^-8 is the halfway point between 1 and 1 + 2^-7: ties go to even (1)
    vals = np.array([1.0, 1 + 2**-8, 1 + 3 * 2**-8, -1 - 2**-8, 2.0**127 * 1.999999], np.float32)
    got = fused.bf16_to_f32(fused.f32_to_bf16(vals))
    assert got.tolist() == [1.0, 1.0, 1 + 2**-6, -1.0, float(np.float32(np.inf))]
    assert torch.equal(torch.from_numpy(vals).to(torch.bfloat16).float(),
                       torch.from_numpy(got))


def test_mean_square_is_exact_rational_for_small_rows():
    g = np.random.Generator(np.random.PCG64(31))
    x = _bf16(g.normal(size=(4, 64)))
    r = fused.row_inv_rms(x, 1e-5)
    for i in range(4):
        ms = sum(Fraction(float(v)) ** 2 for v in fused.bf16_to_f32(x[i])) / 64
        exact = 1.0 / np.sqrt(float(ms) + float(np.float32(1e-5)))
        assert r[i] == np.float32(exact)


def test_constant_row_closed_form():
    x = _bf16(np.full((1, 128), 3.0))
    g = _bf16(np.ones(128))
    y = fused.bf16_to_f32(fused.rmsnorm_bf16(x, g, 0.0))
    assert np.all(y == 1.0)                                    # 3 / sqrt(9) = 1


def test_zero_row_gives_zero():
    y = fused.rmsnorm_bf16(np.zeros((2, 64), np.uint16), _bf16(np.ones(64)), 1e-6)
    assert not fused.bf16_to_f32(y).any()


def test_power_of_two_scale_invariance():
    g = np.random.Generator(np.random.PCG64(32))
    x = g.normal(size=(8, 256)) * g.uniform(0.1, 50, size=256)
    gain = _bf16(g.uniform(0.5, 2.0, size=256))
    y1 = fused.rmsnorm_bf16(_bf16(x), gain, 0.0)
    y2 = fused.rmsnorm_bf16(_bf16(x * 2.0**-9), gain, 0.0)
    assert np.array_equal(y1, y2)


def test_matches_torch_float32_rmsnorm_to_rounding():
    g = np.random.Generator(np.random.PCG64(33))
    x = _bf16(g.normal(size=(16, 4096)) * g.uniform(0.5, 30, size=4096))
    gain = _bf16(g.uniform(0.5, 1.5, size=4096))
    y = fused.bf16_to_f32(fused.rmsnorm_bf16(x, gain, 1e-5))
    xt = torch.from_numpy(fused.bf16_to_f32(x))
    ref = xt * torch.rsqrt(xt.pow(2).mean(-1, keepdim=True) + 1e-5)
    ref = ref.to(torch.bfloat16).float() * torch.from_numpy(fused.bf16_to_f32(gain))
    np.testing.assert_allclose(y, ref.numpy(), rtol=2**-7, atol=0)


def test_exp32_accuracy_and_exact_points():
    t = np.linspace(-100, 88, 200001, dtype=np.float32)
    e = fused.exp32(t).astype(np.float64)
    ref = np.exp(t.astype(np.float64))
    ok = ref > 1e-37                                            # normal float32 results
    assert np.max(np.abs(e[ok] - ref[ok]) / ref[ok]) < 3 * 2.0**-24
    assert fused.exp32(np.float32(0.0)) == 1.0
    assert fused.exp32(np.float32(200.0)) == np.inf
    assert fused.exp32(np.float32(-200.0)) == 0.0


def test_silu_against_float64_and_identities():
    g = np.random.Generator(np.random.PCG64(41))
    x = (g.normal(size=100000) * 8).astype(np.float32)
    s = fused.silu32(x).astype(np.float64)
    x64 = x.astype(np.float64)
    ref = x64 / (1 + np.exp(-x64))
    big = np.abs(ref) > 1e-30
    assert np.max(np.abs(s[big] - ref[big]) / np.abs(ref[big])) < 4 * 2.0**-24
    assert fused.silu32(np.float32(0.0)) == 0.0
    assert np.isnan(fused.silu32(np.float32(np.nan)))
    assert fused.silu32(np.float32(-1000.0)) == 0.0               # g / inf


def test_swiglu_matches_torch_bf16_to_rounding():
    g = np.random.Generator(np.random.PCG64(42))
    gate = _bf16(g.normal(size=(64, 512)) * 3)
    up = _bf16(g.normal(size=(64, 512)))
    y = fused.bf16_to_f32(fused.swiglu_bf16(gate, up))
    gt = torch.from_numpy(fused.bf16_to_f32(gate)).to(torch.bfloat16)
    ut = torch.from_numpy(fused.bf16_to_f32(up)).to(torch.bfloat16)
    ref = (torch.nn.functional.silu(gt) * ut).float().numpy()
    np.testing.assert_allclose(y, ref, rtol=2**-7, atol=1e-30)
    # the two differ at most in the last bf16 bit, and rarely
    assert np.mean(y != ref) < 0.01
