"""Pins of the oracle's 3-bit blocks (the 3-6-8 template of the paper's
average-bitwidth study, Section 5): a hand-worked block, a brute-force
nearest-grid-point check, the GEMM against float64 products of the
dequantized values, and the packed layout (2q in the 4-bit nibble plane)."""
import numpy as np

import oracle
from paper_2607_17733_amd import workloads as W

RNE, RNA = 0, 1
SYM, FULL = 0, 1


def _bits(x):
    return W.to_bf16_bits(np.asarray(x, np.float32))


def test_hand_worked_block():
    # max |x| = 1.9 -> e = 0, LSB 2^-1: x * 2 rounded to nearest even, |q| <= 3
    x = np.zeros(32, np.float32)
    x[:7] = [1.0, 0.75, 0.25, -1.0, 0.3, 1.9, -1.25]
    q, e = oracle.quantize(_bits(x)[None, :], widths=[3])
    assert e[0, 0] == 127
    assert list(q[0, :7]) == [2, 2, 0, -2, 1, 3, -2]
    x2 = x.copy()
    x2[5] = -1.9                                     # -3.8 clamps to -4 in the full range
    qf, _ = oracle.quantize(_bits(x2)[None, :], widths=[3], clamp_mode=FULL)
    qs, _ = oracle.quantize(_bits(x2)[None, :], widths=[3], clamp_mode=SYM)
    assert qf[0, 5] == -4 and qs[0, 5] == -3


def _floor_log2(a):
    e = 0
    while 2.0 ** e > a:
        e -= 1
    while 2.0 ** (e + 1) <= a:
        e += 1
    return e


def test_brute_force_nearest_grid_point():
    g = np.random.Generator(np.random.PCG64(31))
    for mode in (RNE, RNA):
        for clamp in (SYM, FULL):
            x = (g.standard_normal((40, 32)) * np.exp(g.uniform(-4, 4, (40, 1)))).astype(np.float32)
            bits = _bits(x)
            xv = W.bf16_bits_to_f32(bits).astype(np.float64)
            q, e = oracle.quantize(bits, widths=[3], round_mode=mode, clamp_mode=clamp)
            for r in range(40):
                ee = _floor_log2(np.abs(xv[r]).max())
                assert e[r, 0] == ee + 127
                lsb = 2.0 ** (ee - 1)
                ks = np.arange(-4 if clamp == FULL else -3, 4)
                for t in range(32):
                    d = np.abs(xv[r, t] - ks * lsb)
                    best = ks[d == d.min()]
                    if len(best) == 2:                 # a tie
                        best = [best[np.argmax(np.abs(best))]] if mode == RNA else \
                               [b for b in best if b % 2 == 0]
                    assert q[r, t] == best[0], (r, t, xv[r, t], q[r, t], best)


def test_gemm_with_three_bit_blocks():
    g = np.random.Generator(np.random.PCG64(32))
    widths = [3, 3, 6, 8]
    a = _bits(g.standard_normal((5, 128)))
    w = _bits(g.standard_normal((7, 128)) * 0.02)
    qa, ea = oracle.quantize(a, widths=widths)
    qw, ew = oracle.quantize(w, widths=widths)
    y = oracle.gemm(qa, ea, qw, ew, widths)
    ref = oracle.dequantize(qa, ea, widths) @ oracle.dequantize(qw, ew, widths).T
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-300)


def test_three_bit_blocks_pack_as_doubled_four_bit():
    g = np.random.Generator(np.random.PCG64(33))
    x = _bits(g.standard_normal((3, 96)))
    q, _ = oracle.quantize(x, widths=[3, 3, 8])
    assert oracle.act_row_bytes([3, 3, 8]) == 16 + 16 + 32
    p = oracle.pack_act(q, [3, 3, 8])
    for blk in range(2):
        nib = p[:, 16 * blk:16 * blk + 16]
        lo = (nib & 15).astype(np.int8)
        hi = (nib >> 4).astype(np.int8)
        v = np.stack([lo, hi], axis=-1).reshape(3, 32)
        v = np.where(v >= 8, v - 16, v)
        assert np.array_equal(v, 2 * q[:, 32 * blk:32 * blk + 32])
