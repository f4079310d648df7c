"""Host-side decoders of the GEMM buffers (test infrastructure).

Written from the layouts that include/mxq.h states, independently of the HIP
sources: the FP6 (e3m2, e2m3) and FP8 (e4m3) codes are decoded from the OCP
microscaling element definitions, the folded weight words are unfolded by
evaluating the header's fold formulas on single payload bits (so a fold that
loses or merges a bit is detected, not assumed away), and every mantissa is
rebuilt from its digits.  A test can then compare the buffers element by
element with the oracle's mantissas and exponents.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32
LANES = 64
GROUP_STEPS = 4
TILE_ROWS = 16
SUPER_COLS = 128
SLABS = 8


def _fp_table(ebits, mbits, bias, nan_code=None):
    n = 1 << (1 + ebits + mbits)
    t = np.zeros(n)
    for c in range(n):
        s, e, m = c >> (ebits + mbits), (c >> mbits) & ((1 << ebits) - 1), c & ((1 << mbits) - 1)
        if nan_code is not None and (c & (n // 2 - 1)) == nan_code:
            t[c] = np.nan
            continue
        if e == 0:
            v = m / (1 << mbits) * 2.0 ** (1 - bias)
        else:
            v = (1 + m / (1 << mbits)) * 2.0 ** (e - bias)
        t[c] = -v if s else v
    return t


E3M2 = _fp_table(3, 2, 3)
E2M3 = _fp_table(2, 3, 1)
E4M3 = _fp_table(4, 3, 7, nan_code=0x7F)


def fp6_codes(b: np.ndarray) -> np.ndarray:
    """[..., 24] bytes -> [..., 32] 6-bit codes (element t at bits 6t)."""
    bits = np.unpackbits(np.ascontiguousarray(b, np.uint8), axis=-1, bitorder="little")
    bits = bits.reshape(bits.shape[:-1] + (32, 6)).astype(np.int64)
    return (bits << np.arange(6)).sum(axis=-1)


def _int_of(v, what):
    r = np.rint(v)
    assert np.all(np.isfinite(v)) and np.all(r == v), "%s: digit is not an integer" % what
    return r.astype(np.int64)


class Geo:
    """Segments, steps and scale groups of a width map (header: "Steps and
    lanes")."""

    def __init__(self, widths):
        w = np.asarray(widths)
        self.nb_total = len(w)
        self.nb = [int((w == m).sum()) for m in (3, 4, 6, 8)]
        self.per = [4, 4, 2, 2]
        self.S = [-(-n // p) for n, p in zip(self.nb, self.per)]
        self.b0 = list(np.cumsum([0] + self.nb[:3]))
        self.st0 = list(np.cumsum([0] + self.S[:3]))
        groups = [-(-S // GROUP_STEPS) for S in self.S]
        self.G0 = list(np.cumsum([0] + groups[:3]))
        self.ngroups = int(sum(groups))
        self.nsteps = int(sum(self.S))

    def steps(self):
        """(segment, global step, step within the segment)."""
        for seg in range(4):
            for sl in range(self.S[seg]):
                yield seg, self.st0[seg] + sl, sl

    def block(self, seg, sl, j):
        """Global block index of block j of step sl of a segment, or None
        for a zero block."""
        i = self.per[seg] * sl + j
        return self.b0[seg] + i if i < self.nb[seg] else None

    def group_byte(self, seg, sl):
        return self.G0[seg] + sl // GROUP_STEPS, sl % GROUP_STEPS


# --------------------------------------------------------------------------
# (A) the activation operand image
# --------------------------------------------------------------------------

def act_lane_bytes(seg):
    return 32 if seg == 3 else 24


def act_tile_bytes(g: Geo):
    return sum(g.S[s] * LANES * act_lane_bytes(s) for s in range(4))


def decode_act(img: np.ndarray, sc: np.ndarray, widths, M: int):
    """Activation image -> (q [M, K], E [M, nb], pad_ok): mantissas rebuilt
    from their digits, exponents from the lanes' scale bytes; pad_ok is True
    when rows past M, zero blocks and unused scale bytes are all zero."""
    g = Geo(widths)
    K = g.nb_total * BLOCK
    tiles = -(-M // TILE_ROWS)
    Mp = tiles * TILE_ROWS
    tb, tsc = act_tile_bytes(g), g.ngroups * LANES * 4
    assert img.size == tiles * tb and sc.size == tiles * tsc, "image sizes"
    img = img.reshape(tiles, tb)
    sc = sc.reshape(tiles, g.ngroups, LANES, 4)
    q = np.zeros((Mp, K), np.int64)
    E = np.zeros((Mp, g.nb_total), np.int64)
    pad_ok = True
    used = np.zeros(sc.shape, bool)
    off = 0
    for seg, st, sl in g.steps():
        L = act_lane_bytes(seg)
        lanes = img[:, off:off + LANES * L].reshape(tiles, 4, 16, L)   # [tile, g, r, bytes]
        off += LANES * L
        G, k = g.group_byte(seg, sl)
        sbytes = sc[:, G, :, k].reshape(tiles, 4, 16).astype(np.int64)
        used[:, G, :, k] = True
        rows = (np.arange(tiles)[:, None] * TILE_ROWS + np.arange(16)[None, :]).reshape(-1)
        if seg <= 1:
            v = E3M2[fp6_codes(lanes)]                        # [tile, g, r, 32]
            for j in range(4):
                b = g.block(seg, sl, j)
                vals = v[:, j].reshape(-1, 32)
                e = sbytes[:, j].reshape(-1)
                if b is None:
                    pad_ok &= not vals.any() and not e.any()
                    continue
                qq = _int_of(vals / 2 if seg == 0 else vals, "3/4-bit activation")
                q[rows, b * BLOCK:(b + 1) * BLOCK] = qq
                E[rows, b] = e
        elif seg == 2:
            v = E3M2[fp6_codes(lanes)]
            for j in range(2):
                b = g.block(seg, sl, j)
                vh = v[:, 2 * j].reshape(-1, 32)
                vl = v[:, 2 * j + 1].reshape(-1, 32)
                eh = sbytes[:, 2 * j].reshape(-1)
                el = sbytes[:, 2 * j + 1].reshape(-1)
                if b is None:
                    pad_ok &= not vh.any() and not vl.any() and not eh.any() and not el.any()
                    continue
                h = _int_of(2 * vh, "6-bit high digit")
                l = _int_of(16 * vl, "6-bit low digit")
                assert np.all((l >= 0) & (l <= 7)), "6-bit low digit out of range"
                q[rows, b * BLOCK:(b + 1) * BLOCK] = 8 * h + l
                assert np.array_equal(eh, el), "6-bit scale bytes of the two planes differ"
                E[rows, b] = eh
        else:
            for j in range(2):
                b = g.block(seg, sl, j)
                hi = np.concatenate([lanes[:, e, :, 16 * j:16 * j + 16] for e in (0, 1)], axis=-1)
                lo = np.concatenate([lanes[:, 2 + e, :, 16 * j:16 * j + 16] for e in (0, 1)],
                                    axis=-1)
                vh = E4M3[hi.reshape(-1, 32).astype(np.int64)]
                vl = E4M3[lo.reshape(-1, 32).astype(np.int64)]
                eh = sbytes[:, 2 * j].reshape(-1)
                el = sbytes[:, 2 * j + 1].reshape(-1)
                if b is None:
                    pad_ok &= not hi.any() and not lo.any() and not eh.any() and not el.any()
                    continue
                h = _int_of(vh / 2, "8-bit high digit")
                l = _int_of(8 * vl, "8-bit low digit")
                assert np.all((l >= 0) & (l <= 15)), "8-bit low digit out of range"
                q[rows, b * BLOCK:(b + 1) * BLOCK] = 16 * h + l
                assert np.array_equal(eh, el), "8-bit scale bytes of the two planes differ"
                E[rows, b] = eh
    assert off == tb
    pad_ok &= not q[M:].any() and not E[M:].any()
    pad_ok &= not sc[~used].any()
    return q[:M], E[:M], bool(pad_ok)


# --------------------------------------------------------------------------
# (B) the weights
# --------------------------------------------------------------------------

M32 = 0xFFFFFFFF
F4Z0, F4Z2 = 0x18618618, 0x61861861


def fold4(d):
    return [d[0] | (d[1] & F4Z0), d[2] | (d[1] & F4Z2),
            d[3] | (d[4] & F4Z0), d[5] | (d[4] & F4Z2)]


def fold3(d):
    return [d[0] | (d[1] >> 1), d[3] | (d[4] >> 1),
            (d[2] | (d[5] << 3) | (d[5] >> 31)) & M32]


def fold2(d):
    return [d[0] | d[1] | d[2], d[3] | d[4] | d[5]]


def _payload_bits(field_bits):
    """Bit positions (of the 192-bit word sequence D0..D5) that a code with
    the given set bits per 6-bit field may use."""
    return [6 * t + f for t in range(32) for f in field_bits]


def _fold_map(fold, field_bits):
    """Evaluate a fold on each payload bit alone: the stored bit it lands on.
    Fails if a payload bit is lost, lands on two bits, or two payload bits
    share one stored bit."""
    mp = {}
    for p in _payload_bits(field_bits):
        d = [0] * 6
        d[p // 32] = 1 << (p % 32)
        out = fold(d)
        hits = [(w, b) for w, x in enumerate(out) for b in range(32) if (x >> b) & 1]
        assert len(hits) == 1, "fold loses or duplicates payload bit %d" % p
        mp[p] = hits[0][0] * 32 + hits[0][1]
    assert len(set(mp.values())) == len(mp), "fold merges payload bits"
    return mp


# payload of the symmetric-clamp codes: s|k with k <= 7 (4-bit) or k <= 3
# (3-bit, e2m3 s|k: k in the mantissa bits), and the sign-free 2-bit high
# digits of 6-bit blocks
_MAP4 = _fold_map(fold4, (0, 1, 2, 5))
_MAP3 = _fold_map(fold3, (0, 1, 5))
_MAP2 = _fold_map(fold2, (0, 1))


def _unfold(words: np.ndarray, mp) -> np.ndarray:
    """[..., n] uint32 stored words -> [..., 32] 6-bit codes."""
    words = words.astype(np.uint64)
    codes = np.zeros(words.shape[:-1] + (32,), np.int64)
    for p, s in mp.items():
        bit = (words[..., s // 32] >> np.uint64(s % 32)) & np.uint64(1)
        codes[..., p // 6] |= bit.astype(np.int64) << (p % 6)
    return codes


def _raw_codes(words: np.ndarray) -> np.ndarray:
    b = words.astype("<u4").view(np.uint8).reshape(words.shape[:-1] + (24,))
    return fp6_codes(b)


def w_chunk_bytes(seg, full):
    return [(768, 1024), (1024, 1536), (768, 1024), (1024, 1024)][seg][int(full)]


def w_super_bytes(g: Geo, full):
    return sum(g.S[s] * SLABS * w_chunk_bytes(s, full) for s in range(4))


def _words(b: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(b).view("<u4")


def decode_weights(wm: np.ndarray, we: np.ndarray, widths, N: int, full: bool):
    """Weight buffers -> (q [Np, K], E [Np, nb], ok) for Np = N rounded up to
    128; ok is False if a layout rule is broken (a zero block or padding
    column that is not zero, a code outside its documented range, unused
    scale bytes that are not zero)."""
    g = Geo(widths)
    K = g.nb_total * BLOCK
    sup = -(-N // SUPER_COLS)
    Np = sup * SUPER_COLS
    sb, ssc = w_super_bytes(g, full), g.ngroups * 2048
    assert wm.size == sup * sb and we.size == sup * ssc, "weight buffer sizes"
    wm = wm.reshape(sup, sb)
    sc = we.reshape(sup, g.ngroups, LANES, GROUP_STEPS, SLABS)     # [.., lane, k, slab]
    q = np.zeros((Np, K), np.int64)
    E = np.zeros((Np, g.nb_total), np.int64)
    ok = True
    used = np.zeros(sc.shape, bool)
    off = 0
    cols = (np.arange(sup)[:, None, None] * SUPER_COLS + 16 * np.arange(SLABS)[None, :, None]
            + np.arange(16)[None, None, :])                          # [sup, slab, c]
    for seg, st, sl in g.steps():
        C = w_chunk_bytes(seg, full)
        ch = wm[:, off:off + SLABS * C].reshape(sup, SLABS, C)
        off += SLABS * C
        G, k = g.group_byte(seg, sl)
        sbytes = sc[:, G, :, k, :].astype(np.int64)                   # [sup, lane, slab]
        used[:, G, :, k, :] = True
        if seg <= 1:
            if seg == 0 and not full:
                xy = _words(ch[:, :, :512]).reshape(sup, SLABS, LANES, 2)
                z = _words(ch[:, :, 512:768]).reshape(sup, SLABS, LANES, 1)
                codes = _unfold(np.concatenate([xy, z], axis=-1), _MAP3)
            elif seg == 1 and full:
                a = _words(ch[:, :, :1024]).reshape(sup, SLABS, LANES, 4)
                b = _words(ch[:, :, 1024:1536]).reshape(sup, SLABS, LANES, 2)
                codes = _raw_codes(np.concatenate([a, b], axis=-1))
            else:
                codes = _unfold(_words(ch).reshape(sup, SLABS, LANES, 4), _MAP4)
            tab = E2M3 if seg == 0 else E3M2
            mult = 8 if seg == 0 else 16
            qall = _int_of(tab[codes] * mult, "3/4-bit weight")        # [sup, slab, lane, 32]
            for j in range(4):
                b = g.block(seg, sl, j)
                qq = qall[:, :, 16 * j:16 * j + 16]                    # [sup, slab, c, 32]
                e = sbytes[:, 16 * j:16 * j + 16, :].transpose(0, 2, 1)  # [sup, slab, c]
                if b is None:
                    ok &= not qq.any() and not e.any()
                    continue
                q[cols.reshape(-1), b * BLOCK:(b + 1) * BLOCK] = qq.reshape(-1, 32)
                E[cols.reshape(-1), b] = e.reshape(-1)
        elif seg == 2:
            lo = _unfold(_words(ch[:, :, :512]).reshape(sup, SLABS, 32, 4), _MAP4)
            vl = E3M2[lo]
            if full:
                hi = _unfold(_words(ch[:, :, 512:1024]).reshape(sup, SLABS, 32, 4), _MAP4)
                vh = E3M2[hi]
                ok &= bool(np.all((hi >> 5) == (lo >> 5)) or not full)
            else:
                hm = _unfold(_words(ch[:, :, 512:768]).reshape(sup, SLABS, 32, 2), _MAP2)
                vh = np.where(lo >> 5, -1.0, 1.0) * E3M2[hm]
            l = _int_of(np.abs(vl) * 16, "6-bit low weight digit")
            h = _int_of(np.abs(vh) * 16, "6-bit high weight digit")
            ok &= bool(np.all(l <= 7) and np.all(h <= (4 if full else 3)))
            sign = np.where(lo >> 5, -1, 1)
            qall = sign * (8 * h + l)                                  # [sup, slab, u, 32]
            for j in range(2):
                b = g.block(seg, sl, j)
                qq = qall[:, :, 16 * j:16 * j + 16]
                e0 = sbytes[:, 32 * j:32 * j + 16, :].transpose(0, 2, 1)
                e1 = sbytes[:, 32 * j + 16:32 * j + 32, :].transpose(0, 2, 1)
                ok &= bool(np.array_equal(e0, e1))
                if b is None:
                    ok &= not qq.any() and not e0.any()
                    continue
                q[cols.reshape(-1), b * BLOCK:(b + 1) * BLOCK] = qq.reshape(-1, 32)
                E[cols.reshape(-1), b] = e0.reshape(-1)
        else:
            by = ch.reshape(sup, SLABS, 32, 32).astype(np.int64)       # [sup, slab, u, 32]
            if full:
                qall = np.where(by >= 128, by - 256, by)
            else:
                qall = np.where(by & 128, -(by & 127), by & 127)
                ok &= not np.any(by == 128)                             # no -0 byte
            for j in range(2):
                b = g.block(seg, sl, j)
                qq = qall[:, :, 16 * j:16 * j + 16]
                e0 = sbytes[:, 32 * j:32 * j + 16, :].transpose(0, 2, 1)
                e1 = sbytes[:, 32 * j + 16:32 * j + 32, :].transpose(0, 2, 1)
                ok &= bool(np.array_equal(e0, e1))
                if b is None:
                    ok &= not qq.any() and not e0.any()
                    continue
                q[cols.reshape(-1), b * BLOCK:(b + 1) * BLOCK] = qq.reshape(-1, 32)
                E[cols.reshape(-1), b] = e0.reshape(-1)
    assert off == sb
    ok &= not q[N:].any() and not E[N:].any()
    ok &= not sc[~used].any()
    return q, E, bool(ok)
