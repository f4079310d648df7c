"""GPU parity of decode attention over the MXINT KV cache (C ABI
mxq_attn_decode) against the float64 oracle in oracle/attn.py.

The caches are quantized on the GPU by mxq_quantize_rows (whose bit-exact
parity with the oracle's quantizer the quantizer tests establish) and by the
oracle's quantizer for the reference; the test also checks that the two
agree on the packed rows it reads, so the comparison is of the attention
alone.  Tolerance: float32 arithmetic against float64.  A score carries a
rounding error of a few units of 2^-24 times the sum of |q_d k_d| over the
128 products; the softmax turns an absolute score error into the same
relative error of its weight, and the output is a convex combination of V
rows, so the per-head error relative to the largest |V| of the head stays
near 1e-6 for these inputs: the test asks for 1e-5 (the GEMM's bar).
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import attn as oattn
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from parity_util import say, to_dev_bf16

pytestmark = pytest.mark.gpu

D = 128
TOL = 1e-5
MIXES = [(n4, n6, 4 - n4 - n6) for n4 in range(4, -1, -1) for n6 in range(4 - n4, -1, -1)]


def _widths(mix):
    n4, n6, n8 = mix
    return [4] * n4 + [6] * n6 + [8] * n8


def _run(seed, B, Hq, Hkv, T, widths, seqs=None):
    say("attn seed=%d B=%d Hq=%d Hkv=%d T=%d widths=%s" % (seed, B, Hq, Hkv, T, widths))
    qb, kb, vb = W.attn_inputs(seed, B, Hq, Hkv, T)
    fmt = mxq.Format(D, widths)
    kc = mxq.quantize_rows(to_dev_bf16(kb), fmt)
    vc = mxq.quantize_rows(to_dev_bf16(vb), fmt)
    scale = 1.0 / np.sqrt(D)
    o = mxq.attn_decode(to_dev_bf16(qb.reshape(-1, D)).reshape(B, Hq, D), kc, vc, fmt,
                        B, Hq, Hkv, T, scale)
    torch.cuda.synchronize()
    o = o.cpu().numpy().astype(np.float64)
    seqs = range(B) if seqs is None else seqs
    rows = T * Hkv
    qf = W.bf16_bits_to_f32(qb).astype(np.float64)
    for b in seqs:
        sl = slice(b * rows, (b + 1) * rows)
        kd = oattn.dequantize_cache(kb[sl], widths)
        vd = oattn.dequantize_cache(vb[sl], widths)
        ref = oattn.attention(qf[b:b + 1], kd, vd, 1, Hq, Hkv, T, scale)[0]
        vmax = np.abs(vd.reshape(T, Hkv, D)).max(axis=(0, 2))          # per KV head
        err = np.abs(o[b] - ref).max(axis=1) / vmax[np.arange(Hq) // (Hq // Hkv)]
        assert np.all(np.isfinite(o[b]))
        assert err.max() <= TOL, (b, int(err.argmax()), err.max())
    return o


def test_cache_rows_match_oracle_quantizer():
    widths = [4, 6, 8, 8]
    _, kb, _ = W.attn_inputs(1, 1, 4, 2, 70)
    fmt = mxq.Format(D, widths)
    mant, exp = mxq.quantize_rows(to_dev_bf16(kb), fmt)
    q, e = mxq.unpack_act(mant, exp, fmt, kb.shape[0])
    qo, eo = oracle.quantize(kb, widths=widths)
    assert np.array_equal(q.cpu().numpy(), qo) and np.array_equal(e.cpu().numpy(), eo)


@pytest.mark.parametrize("mix", MIXES)
def test_every_width_mix(mix):
    _run(10 + MIXES.index(mix), 2, 8, 2, 70, _widths(mix))


@pytest.mark.parametrize("T", [1, 2, 63, 64, 65, 255, 256, 257, 1000])
def test_ragged_lengths(T):
    _run(40 + T, 1, 8, 4, T, [4, 4, 4, 4])


@pytest.mark.parametrize("Hq,Hkv", [(4, 4), (8, 1), (16, 1), (64, 8), (6, 2), (12, 4)])
def test_head_groupings(Hq, Hkv):
    _run(60 + Hq + Hkv, 2, Hq, Hkv, 130, [4, 4, 6, 8])


def test_single_token_returns_its_value_row():
    # softmax over one token is 1: the output is that token's V row exactly
    widths = [4, 4, 6, 8]
    qb, kb, vb = W.attn_inputs(5, 3, 8, 2, 1)
    o = _run(5, 3, 8, 2, 1, widths)
    vd = oattn.dequantize_cache(vb, widths).reshape(3, 2, D)
    for b in range(3):
        for h in range(8):
            assert np.array_equal(o[b, h], vd[b, h // 4].astype(np.float32).astype(np.float64))


def test_llama70b_cache_4k_batch1():
    # 64 query heads, 8 KV heads, 4096 cached tokens, all-4-bit K and V
    _run(7, 1, 64, 8, 4096, [4, 4, 4, 4])


def test_llama70b_cache_4k_batch16_sampled():
    # the benchmark's shape; the oracle checks the first and last sequences
    _run(8, 16, 64, 8, 4096, [4, 4, 4, 4], seqs=[0, 15])


def test_hundreds_of_token_splits():
    # one sequence and one KV head over a 40000-token cache: about 300 splits
    # merged by the combine step
    fmt = mxq.Format(D, [4, 4, 4, 4])
    assert mxq.attn_work_bytes(fmt, 1, 8, 1, 40000) // (8 * 130 * 4) > 256
    _run(11, 1, 8, 1, 40000, [4, 4, 4, 4])


def test_mixed_widths_long_cache():
    _run(9, 2, 64, 8, 2048, [4, 4, 4, 8])


def test_repeat_calls_identical():
    B, Hq, Hkv, T, widths = 2, 16, 2, 900, [4, 6, 6, 8]
    qb, kb, vb = W.attn_inputs(3, B, Hq, Hkv, T)
    fmt = mxq.Format(D, widths)
    kc = mxq.quantize_rows(to_dev_bf16(kb), fmt)
    vc = mxq.quantize_rows(to_dev_bf16(vb), fmt)
    q = to_dev_bf16(qb.reshape(-1, D)).reshape(B, Hq, D)
    a = mxq.attn_decode(q, kc, vc, fmt, B, Hq, Hkv, T, 0.1)
    b = mxq.attn_decode(q, kc, vc, fmt, B, Hq, Hkv, T, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_rejects_bad_arguments():
    fmt = mxq.Format(D, [4, 4, 4, 4])
    q = torch.zeros((1, 8, D), dtype=torch.bfloat16, device="cuda")
    kc = mxq.quantize_rows(torch.zeros((4 * 2, D), dtype=torch.bfloat16, device="cuda"), fmt)
    with pytest.raises(mxq.MxqError):                      # Hq not a multiple of Hkv
        mxq.attn_decode(q, kc, kc, fmt, 1, 8, 3, 4, 0.1)
    with pytest.raises(mxq.MxqError):                      # a cache shorter than its rows
        mxq.attn_decode(q, kc, kc, fmt, 1, 8, 2, 400, 0.1)
    with pytest.raises(mxq.MxqError):                      # a head dimension other than 128
        mxq.attn_decode(q, kc, kc, mxq.Format(256, [4] * 8), 1, 8, 2, 4, 0.1)
    with pytest.raises(mxq.MxqError):                      # a short work buffer
        mxq.attn_decode(q, kc, kc, fmt, 1, 8, 2, 4, 0.1,
                        work=torch.empty(16, dtype=torch.uint8, device="cuda"))
