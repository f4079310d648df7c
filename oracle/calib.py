"""Calibration oracle: the offline step that produces the path's inputs (the
column permutation and the per-block width map).

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the product
library; it shares no code with the GPU path.  Plain numpy in float64, with
the steps in the paper's order.

Paper: MXSens (arXiv 2607.17733), Section 3 (Algorithm 1: a column's
sensitivity is the diagonal of the accumulated Hessian approximation
X^T X over the calibration samples), Section 4.2 and Algorithm 2 (top 32
columns 8-bit, the next N6 = floor(R * S_layer * (d_in - 32)) columns
6-bit, the rest 4-bit), Appendix A, Theorem A.1 (the control parameter R
for an average bitwidth B).

Readings (where the paper is silent): sensitivities are summed in float64,
each sample's rows in row order and the samples in sample order; the sort is
descending and stable (equal sensitivities keep column order; a NaN counts
as +inf); N6 is rounded down to whole 32-column blocks and clamped to
[0, d_in - 32]; the permutation lists the 4-bit columns, then the 6-bit,
then the 8-bit, each in sorted order, so that the width map is non-decreasing.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32


def _as_f64(x) -> np.ndarray:
    """bf16 bit patterns (uint16 / int16) or floats -> float64 (exact)."""
    x = np.asarray(x)
    if x.dtype in (np.uint16, np.int16):
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def sample_sensitivity(x) -> np.ndarray:
    """diag(X^T X) of one calibration sample X [rows, K]: per column, the sum
    over rows (in row order, starting from zero) of x^2, in float64."""
    x = _as_f64(x)
    part = np.zeros(x.shape[1], dtype=np.float64)
    for r in range(x.shape[0]):
        part += x[r] * x[r]
    return part


def column_sensitivity(samples) -> np.ndarray:
    """Algorithm 1 for one linear layer: H accumulates X_i^T X_i sample by
    sample; the sensitivity is diag(H)."""
    s = None
    for x in samples:
        part = sample_sensitivity(x)
        s = part if s is None else s + part
    return s


def ratio(d_in, s_layer, B: float) -> float:
    """Theorem A.1: R = ((B - 4) * sum d_i - 4 * 32 * n) /
    sum(2 * S_i * (d_i - 32)) for n layers of input widths d_i and layer
    sensitivities S_i, so that 32 8-bit columns per layer plus R * S_i *
    (d_i - 32) 6-bit columns average B bits."""
    # plain sums in layer order (the allocation floors R * S * (d - 32), so
    # the rounding order is part of the definition)
    total, den = 0.0, 0.0
    for d, S in zip(d_in, s_layer):
        total += float(d)
        den += 2.0 * float(S) * float(d - BLOCK)
    return ((B - 4.0) * total - 4.0 * BLOCK * len(d_in)) / den


def counts(d_in: int, R: float, s_layer: float, n8_blocks: int = 1):
    """Algorithm 2's split of one layer, in 32-column blocks: n8_blocks
    8-bit blocks (the paper: one, the top 32 columns), N6 = floor(R * S *
    (d_in - 32)) columns rounded down to whole blocks and clamped to the
    columns left, the rest 4-bit.  Returns (n4, n6, n8)."""
    nb = d_in // BLOCK
    n8 = min(n8_blocks, nb)
    n6_cols = int(np.floor(R * s_layer * (d_in - BLOCK)))
    n6 = max(0, min(n6_cols // BLOCK, nb - n8))
    return nb - n6 - n8, n6, n8


def sort_desc(s) -> np.ndarray:
    """Column indices by descending sensitivity, ties in column order (NaN
    as +inf)."""
    s = np.asarray(s, dtype=np.float64)
    key = np.where(np.isnan(s), np.inf, s)
    return np.lexsort((np.arange(len(s)), -key))


def allocate(s, n6: int, n8: int):
    """Algorithm 2 for one layer: the 8-bit set is the first 32 * n8 sorted
    columns, the 6-bit set the next 32 * n6, the 4-bit set the rest.
    Returns (perm, widths): perm lists the 4-bit, 6-bit and 8-bit columns
    (each in sorted order) and widths is the matching per-block map."""
    I = sort_desc(s)
    K = len(I)
    nb = K // BLOCK
    n4 = nb - n6 - n8
    i8 = I[:BLOCK * n8]
    i6 = I[BLOCK * n8:BLOCK * (n8 + n6)]
    i4 = I[BLOCK * (n8 + n6):]
    perm = np.concatenate([i4, i6, i8]).astype(np.int32)
    widths = np.array([4] * n4 + [6] * n6 + [8] * n8, dtype=np.uint8)
    return perm, widths


def average_bits(layers) -> float:
    """Average mantissa bits over layers given as (n4, n6, n8) block counts."""
    bits = sum(32 * (4 * a + 6 * b + 8 * c) for a, b, c in layers)
    cols = sum(32 * (a + b + c) for a, b, c in layers)
    return bits / cols
