"""Pins of the oracle's 3-bit blocks (the 3-6-8 template of the paper's
average-bitwidth study, Section 5): a hand-worked block, a brute-force
nearest-grid-point check, the GEMM against float64 products of the
dequantized values, and the packed layout (12 bytes per block, element t's
3-bit two's complement field at bits 3t .. 3t + 2)."""
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


def test_three_bit_blocks_pack_at_twelve_bytes():
    # 3 bits per element: a block of 32 takes 12 bytes; the row pads to 16
    assert oracle.act_row_bytes([3]) == 16
    assert oracle.act_row_bytes([3, 3, 8]) == 12 + 12 + 32 + 8
    assert oracle.act_row_bytes([3, 3, 3, 3]) == 48
    g = np.random.Generator(np.random.PCG64(33))
    x = _bits(g.standard_normal((3, 96)))
    q, _ = oracle.quantize(x, widths=[3, 3, 8])
    p = oracle.pack_act(q, [3, 3, 8])
    assert p.shape == (3, 64)
    for blk in range(2):
        # read the 96-bit little-endian integer field by field
        v = [int.from_bytes(bytes(p[r, 12 * blk:12 * blk + 12]), "little") for r in range(3)]
        for r in range(3):
            for t in range(32):
                f = (v[r] >> (3 * t)) & 7
                assert (f - 8 if f >= 4 else f) == q[r, 32 * blk + t]
    assert np.array_equal(p[:, 24:56].view(np.int8), q[:, 64:96])
    assert not p[:, 56:].any()


def test_three_bit_packing_hand_worked():
    # elements 0..2 = 1, -1, -3 and the rest 0: fields 001, 111, 101 at bits
    # 0, 3, 6; LSB first, bits 0-8 read 1 0 0 1 1 1 1 0 | 1: bytes 0x79, 0x01
    # (the third field straddles the byte boundary)
    q = np.zeros((1, 32), np.int8)
    q[0, :3] = [1, -1, -3]
    p = oracle.pack_act(q, [3])
    assert list(p[0, :3]) == [0x79, 0x01, 0x00]
    q[0, :] = 0
    q[0, 31] = -4                                    # field 100 at bits 93..95
    p = oracle.pack_act(q, [3])
    assert list(p[0, :12]) == [0] * 11 + [0x80]
