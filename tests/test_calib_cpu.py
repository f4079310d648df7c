"""Host-only calibration entry points against the oracle: Theorem A.1's R and
Algorithm 2's block counts, bit for bit, and argument validation before any
launch (no device work here)."""
import ctypes

import numpy as np
import pytest

from oracle import calib
from paper_2607_17733_amd import mxq


def test_ratio_and_counts_match_oracle():
    g = np.random.Generator(np.random.PCG64(21))
    for _ in range(300):
        n = int(g.integers(1, 12))
        d = [int(32 * g.integers(1, 900)) for _ in range(n)]
        S = [float(v) for v in g.uniform(0, 1, size=n)]
        B = float(g.uniform(4.0, 6.0))
        if sum(2 * s * (di - 32) for s, di in zip(S, d)) == 0:
            continue
        R = mxq.calib_ratio(d, S, B)
        assert R == calib.ratio(d, S, B)                       # same sums, same order
        for di, s in zip(d, S):
            n8b = int(g.integers(0, 3))
            assert mxq.calib_counts(di, R, s, n8b) == calib.counts(di, R, s, n8b)


def test_counts_clamp_and_floor():
    assert mxq.calib_counts(256, 100.0, 1.0) == calib.counts(256, 100.0, 1.0) == (0, 7, 1)
    assert mxq.calib_counts(256, -3.0, 1.0) == (7, 0, 1)
    assert mxq.calib_counts(256, 0.5, 1.0) == (4, 3, 1)
    assert mxq.calib_counts(32, 0.5, 1.0) == (0, 0, 1)


def test_calibration_validation():
    lib = mxq.lib()
    fake = ctypes.c_void_p(16)
    R = ctypes.c_double(0)
    d = (ctypes.c_int64 * 2)(64, 100)                          # 100 is not a multiple of 32
    s = (ctypes.c_double * 2)(0.5, 0.5)
    assert lib.mxq_calib_ratio(2, d, s, 4.5, ctypes.byref(R)) == 2
    d0 = (ctypes.c_int64 * 1)(32)
    assert lib.mxq_calib_ratio(1, d0, s, 4.5, ctypes.byref(R)) == 2   # zero denominator
    assert lib.mxq_calib_ratio(0, d0, s, 4.5, ctypes.byref(R)) == 2
    assert lib.mxq_calib_colsq(None, 4, 64, 64, fake, 0, None) == 1
    assert lib.mxq_calib_colsq(fake, 4, 63, 64, fake, 0, None) == 2
    assert lib.mxq_calib_colsq(fake, -1, 64, 64, fake, 0, None) == 2
    assert lib.mxq_calib_perm(fake, 96, 2, 2, fake, None) == 2        # 4 blocks > 3
    assert lib.mxq_calib_perm(fake, 100, 0, 1, fake, None) == 2
    assert lib.mxq_calib_perm(None, 96, 0, 1, fake, None) == 1
