"""Pins of the MXINT-KV decode attention oracle against things other than
itself: closed forms (equal scores average V; a dominant key selects its
V row), token-order invariance, and torch's float64 scaled dot-product
attention on the dequantized cache."""
import numpy as np
import torch

from oracle import attn


def _case(seed, B, Hq, Hkv, T, D=128):
    g = np.random.Generator(np.random.PCG64(seed))
    kd = g.normal(size=(B * T * Hkv, D))
    vd = g.normal(size=(B * T * Hkv, D))
    q = g.normal(size=(B, Hq, D))
    return q, kd, vd


def test_zero_query_averages_values():
    q, kd, vd = _case(1, 2, 8, 2, 37)
    o = attn.attention(np.zeros_like(q), kd, vd, 2, 8, 2, 37, 0.1)
    v = vd.reshape(2, 37, 2, 128)
    for b in range(2):
        for h in range(8):
            np.testing.assert_allclose(o[b, h], v[b, :, h // 4].mean(0), rtol=1e-13)


def test_dominant_key_selects_its_value():
    q, kd, vd = _case(2, 1, 4, 1, 50)
    kd = kd * 1e-3
    kd[17] = q[0, 0] * 50                                # row 17 = token 17 of head 0
    o = attn.attention(q, kd, vd, 1, 4, 1, 50, 1.0)
    np.testing.assert_allclose(o[0, 0], vd[17], rtol=1e-9, atol=1e-9)


def test_token_order_invariance():
    q, kd, vd = _case(3, 1, 8, 8, 64)
    perm = np.random.Generator(np.random.PCG64(4)).permutation(64)
    k2 = kd.reshape(64, 8, 128)[perm].reshape(-1, 128)
    v2 = vd.reshape(64, 8, 128)[perm].reshape(-1, 128)
    a = attn.attention(q, kd, vd, 1, 8, 8, 64, 0.088)
    b = attn.attention(q, k2, v2, 1, 8, 8, 64, 0.088)
    np.testing.assert_allclose(a, b, rtol=1e-12)


def test_matches_torch_sdpa_float64():
    B, Hq, Hkv, T = 2, 16, 4, 33
    q, kd, vd = _case(5, B, Hq, Hkv, T)
    o = attn.attention(q, kd, vd, B, Hq, Hkv, T, 1 / np.sqrt(128))
    G = Hq // Hkv
    k = torch.from_numpy(kd.reshape(B, T, Hkv, 128)).permute(0, 2, 1, 3)
    v = torch.from_numpy(vd.reshape(B, T, Hkv, 128)).permute(0, 2, 1, 3)
    k = k.repeat_interleave(G, dim=1)
    v = v.repeat_interleave(G, dim=1)
    qt = torch.from_numpy(q).unsqueeze(2)                 # [B, Hq, 1, D]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, k, v).squeeze(2).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-10, atol=1e-12)


def test_dequantized_cache_matches_exact_rationals():
    from oracle import exact
    g = np.random.Generator(np.random.PCG64(6))
    bits = (g.normal(size=(12, 128)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    widths = [4, 4, 6, 8]
    d = attn.dequantize_cache(bits, widths)
    for r in range(12):
        for blk, m in enumerate(widths):
            q, E = exact.quantize_block([int(b) for b in bits[r, 32 * blk:32 * blk + 32]], m)
            ref = exact.dequantize_block(q, E, m)
            assert [float(v) for v in ref] == d[r, 32 * blk:32 * blk + 32].tolist()
