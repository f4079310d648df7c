"""Pins of the calibration oracle (Algorithm 1, Theorem A.1, Algorithm 2)
against things other than itself: brute force on small inputs, a library
matrix product, the theorem's closed form checked by counting bits, and a
plain Python sort."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import calib


def _bf16(a):
    return (np.asarray(a, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def test_sensitivity_is_diag_of_xtx_brute_force():
    g = np.random.Generator(np.random.PCG64(11))
    samples = [_bf16(g.normal(size=(5, 64)) * g.uniform(0.5, 40, size=64)) for _ in range(3)]
    s = calib.column_sensitivity(samples)
    # exact rationals: every bf16 value and its square is a dyadic rational
    for k in range(64):
        exact = Fraction(0)
        for x in samples:
            for r in range(x.shape[0]):
                v = Fraction(float(calib._as_f64(x[r:r + 1, k:k + 1])[0, 0]))
                exact += v * v
        # at most 15 roundings of at most half an ulp each
        assert abs(Fraction(s[k]) - exact) <= exact * Fraction(16, 2**53)


def test_sensitivity_matches_matmul_diagonal():
    g = np.random.Generator(np.random.PCG64(12))
    x = _bf16(g.normal(size=(300, 96)))
    xs = calib._as_f64(x)
    ref = np.diag(xs.T @ xs)
    np.testing.assert_allclose(calib.sample_sensitivity(x), ref, rtol=1e-12)


def test_sample_order_matters_only_through_rounding():
    g = np.random.Generator(np.random.PCG64(13))
    samples = [_bf16(g.normal(size=(7, 32))) for _ in range(4)]
    a = calib.column_sensitivity(samples)
    b = calib.column_sensitivity(samples[::-1])
    np.testing.assert_allclose(a, b, rtol=1e-14)


def test_theorem_a1_closed_form_gives_budget():
    # with fractional 6-bit counts R * S_i * (d_i - 32), the average is B
    d = [4096, 4096, 14336, 1024]
    S = [0.3, 1.0, 0.7, 0.05]
    for B in (4.03, 4.1, 4.25, 4.5):
        R = calib.ratio(d, S, B)
        bits = sum(8 * 32 + 6 * R * s * (di - 32) + 4 * (1 - R * s) * (di - 32)
                   for di, s in zip(d, S))
        assert bits / sum(d) == pytest.approx(B, abs=1e-12)


def test_floored_allocation_stays_within_budget():
    d = [4096, 4096, 14336, 1024, 8192]
    S = [0.3, 1.0, 0.7, 0.05, 0.5]
    for B in (4.03, 4.1, 4.25, 4.5, 5.0):
        R = calib.ratio(d, S, B)
        layers = [calib.counts(di, R, s) for di, s in zip(d, S)]
        avg = calib.average_bits(layers)
        assert avg <= B + 1e-12
        # rounding down to whole blocks loses under 32 columns of 2 bits per layer
        assert avg >= B - 2 * 32 * len(d) / sum(d) - 1e-12
        for (n4, n6, n8), di in zip(layers, d):
            assert n8 == 1 and n4 >= 0 and n6 >= 0 and 32 * (n4 + n6 + n8) == di


def _check_average_bits(avg_fn):
    """average_bits against things other than itself: hand-counted layers,
    the bits of the C oracle's packed rows (written by independent code from
    the storage layout), and the paper's operating point (Section 5: one
    8-bit block of 32 columns per layer gives 4.02-4.03 bits over
    LLaMA-2-7B's seven linears, six with d_in 4096 and one with 11008)."""
    import oracle
    assert avg_fn([(127, 0, 1)]) == Fraction(127 * 4 + 8, 128)
    assert avg_fn([(0, 3, 0)]) == 6.0 and avg_fn([(1, 1, 1)]) == 6.0
    assert avg_fn([(2, 0, 0), (0, 0, 2)]) == 6.0
    assert avg_fn([(3, 1, 0), (0, 0, 4)]) == Fraction(4 * 3 + 6 + 8 * 4, 8)
    # (even 6-bit counts, so the packed rows carry no 16-byte padding)
    for layers in ([(102, 14, 12)], [(90, 20, 18), (314, 66, 68)], [(6, 0, 2), (0, 2, 6)]):
        bits = sum(8 * oracle.act_row_bytes([4] * a + [6] * b + [8] * c) for a, b, c in layers)
        cols = sum(32 * (a + b + c) for a, b, c in layers)
        assert abs(avg_fn(layers) - bits / cols) < 1e-12
    d_in = [4096] * 6 + [11008]
    avg = avg_fn([(d // 32 - 1, 0, 1) for d in d_in])
    assert 4.02 <= avg <= 4.03


def test_average_bits_pinned(oracle_lib):
    _check_average_bits(calib.average_bits)


@pytest.mark.parametrize("mutant", [
    lambda L: sum(32 * (4 * a + 8 * b + 8 * c) for a, b, c in L) / sum(32 * (a + b + c) for a, b, c in L),
    lambda L: sum(32 * (4 * a + 6 * b) for a, b, c in L) / sum(32 * (a + b + c) for a, b, c in L),
    lambda L: sum(32 * (4 * a + 6 * b + 8 * c) for a, b, c in L) / sum(32 * (a + b) for a, b, c in L),
    lambda L: sum(32 * (4 * a + 6 * b + 8 * c) + 8 * (a + b + c) for a, b, c in L)
    / sum(32 * (a + b + c) for a, b, c in L),
    lambda L: float(np.mean([(4 * a + 6 * b + 8 * c) / (a + b + c) for a, b, c in L])),
], ids=["6-bit as 8", "8-bit dropped", "8-bit columns dropped", "exponent bits added",
        "unweighted layer mean"])
def test_average_bits_pin_catches_mutants(oracle_lib, mutant):
    with pytest.raises(AssertionError):
        _check_average_bits(mutant)


def test_counts_clamp():
    assert calib.counts(256, 100.0, 1.0) == (0, 7, 1)       # all but the 8-bit block
    assert calib.counts(256, -3.0, 1.0) == (7, 0, 1)
    assert calib.counts(256, 0.5, 1.0) == (4, 3, 1)         # floor(0.5 * 224) = 112 -> 3 blocks


def test_sort_matches_python_sorted_with_ties():
    g = np.random.Generator(np.random.PCG64(14))
    s = g.integers(0, 20, size=500).astype(np.float64)      # many ties
    s[[3, 77]] = np.nan
    ref = sorted(range(500), key=lambda k: (-(np.inf if np.isnan(s[k]) else s[k]), k))
    assert calib.sort_desc(s).tolist() == ref


def test_allocate_structure():
    g = np.random.Generator(np.random.PCG64(15))
    s = g.exponential(size=256)
    perm, widths = calib.allocate(s, n6=2, n8=1)
    assert sorted(perm.tolist()) == list(range(256))
    assert widths.tolist() == [4] * 5 + [6] * 2 + [8]
    order = sorted(range(256), key=lambda k: (-s[k], k))
    assert perm[-32:].tolist() == order[:32]                 # the 32 most sensitive: 8-bit
    assert perm[160:224].tolist() == order[32:96]            # the next 64: 6-bit
    assert perm[:160].tolist() == order[96:]                 # the rest, in sorted order
