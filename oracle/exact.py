"""Exact rational-arithmetic mini-oracle for tiny inputs (test infrastructure).

A second, independent statement of the MXINT definition: bf16 values are
decoded field by field into ``fractions.Fraction``, the shared exponent is
found by comparing against powers of two, and rounding inspects the exact
fractional part.  No floating point is involved anywhere, so this pins the C
oracle (which uses frexp/ldexp/nearbyint in double) from a different
direction.  Pure Python loops: use only for a few blocks.

Paper: MXSens (arXiv 2607.17733), Section 2 (shared power-of-two scale per
32-element block, fixed-point integer elements), Section 4.1 (one width per
block), Section 5.1 (8-bit exponent).
"""
from __future__ import annotations

import math
from fractions import Fraction

BLOCK = 32


def bf16_fraction(bits: int):
    """Exact value of a bf16 bit pattern, or None for NaN / infinity."""
    sign = -1 if (bits >> 15) & 1 else 1
    field = (bits >> 7) & 0xFF
    frac = bits & 0x7F
    if field == 0xFF:
        return None
    if field == 0:
        mag = Fraction(frac, 1) * Fraction(2) ** (-126 - 7)
    else:
        mag = Fraction(128 + frac, 1) * Fraction(2) ** (field - 127 - 7)
    return sign * mag


def floor_log2(a: Fraction) -> int:
    """Largest integer e with 2**e <= a (a > 0), by comparison only."""
    e = 0
    two = Fraction(2)
    while two ** e > a:
        e -= 1
    while two ** (e + 1) <= a:
        e += 1
    return e


def round_half(v: Fraction, ties_away: bool) -> int:
    fl = math.floor(v)
    rest = v - fl
    half = Fraction(1, 2)
    if rest > half:
        return fl + 1
    if rest < half:
        return fl
    if ties_away:
        return fl + 1 if v > 0 else fl
    return fl if fl % 2 == 0 else fl + 1


def quantize_block(bits_block, m: int, ties_away: bool = False,
                   full_clamp: bool = False):
    """Return (mantissas, E) for one block of 32 bf16 bit patterns."""
    xs = [bf16_fraction(b) for b in bits_block]
    if any(x is None for x in xs):
        return [0] * len(xs), 255
    amax = max(abs(x) for x in xs)
    if amax == 0:
        return [0] * len(xs), 0
    e = min(max(floor_log2(amax), -127), 127)
    s = e - (m - 2)
    qmax = 2 ** (m - 1) - 1
    qmin = -(2 ** (m - 1)) if full_clamp else -qmax
    out = []
    for x in xs:
        r = round_half(x / Fraction(2) ** s, ties_away)
        out.append(min(max(r, qmin), qmax))
    return out, e + 127


def dequantize_block(q, E: int, m: int):
    if E == 255:
        return None
    s = E - 127 - (m - 2)
    return [Fraction(v) * Fraction(2) ** s for v in q]


def gemm_exact(qa, ea, qw, ew, widths):
    """Exact Y[i][j] = sum_b P_b * 2^(sa+sw) as Fractions (None = NaN)."""
    M, N = len(qa), len(qw)
    K = len(qa[0])
    nb = K // BLOCK
    Y = [[Fraction(0)] * N for _ in range(M)]
    for i in range(M):
        for j in range(N):
            acc = Fraction(0)
            nan = False
            for b in range(nb):
                if ea[i][b] == 255 or ew[j][b] == 255:
                    nan = True
                    continue
                p = sum(int(qa[i][b * BLOCK + t]) * int(qw[j][b * BLOCK + t])
                        for t in range(BLOCK))
                m = int(widths[b])
                s = (int(ea[i][b]) - 127 - (m - 2)) + (int(ew[j][b]) - 127 - (m - 2))
                acc += Fraction(p) * Fraction(2) ** s
            Y[i][j] = None if nan else acc
    return Y


def absbound_exact(qa, ea, qw, ew, widths):
    """Exact S[i][j] = sum_b |P_b| * 2^(sa+sw) as Fractions: the sum of the
    magnitudes of the per-block terms of Y (blocks touching an E = 255
    exponent are left out)."""
    M, N = len(qa), len(qw)
    nb = len(qa[0]) // BLOCK
    S = [[Fraction(0)] * N for _ in range(M)]
    for i in range(M):
        for j in range(N):
            acc = Fraction(0)
            for b in range(nb):
                if ea[i][b] == 255 or ew[j][b] == 255:
                    continue
                dq_a = dequantize_block(qa[i][b * BLOCK:(b + 1) * BLOCK], int(ea[i][b]),
                                        int(widths[b]))
                dq_w = dequantize_block(qw[j][b * BLOCK:(b + 1) * BLOCK], int(ew[j][b]),
                                        int(widths[b]))
                acc += abs(sum(x * y for x, y in zip(dq_a, dq_w)))
            S[i][j] = acc
    return S
