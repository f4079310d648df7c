"""Host-side decoder of the matrix-core operand images (test infrastructure).

Written from the layout that include/mxq.h documents, independently of the
HIP sources: FP6 e3m2 and FP8 e4m3 codes are decoded from the OCP
microscaling element definitions, and every mantissa is rebuilt from its
digits, so a test can compare the images element by element with the
oracle's mantissas and exponents.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32
CHUNK = 13312          # bytes per step of a 128-column weight tile
PART = 4096
TILE_COLS = 128


def _e3m2_table():
    t = np.zeros(64)
    for c in range(64):
        s, e, m = c >> 5, (c >> 2) & 7, c & 3
        v = m / 4 * 2.0 ** -2 if e == 0 else (1 + m / 4) * 2.0 ** (e - 3)
        t[c] = -v if s else v
    return t


def _e4m3_table():
    t = np.zeros(256)
    for c in range(256):
        s, e, m = c >> 7, (c >> 3) & 15, c & 7
        if e == 15 and m == 7:
            t[c] = np.nan
            continue
        v = m / 8 * 2.0 ** -6 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
        t[c] = -v if s else v
    return t


E3M2 = _e3m2_table()
E4M3 = _e4m3_table()


def fp6_values(b24: np.ndarray) -> np.ndarray:
    """[..., 24] bytes -> [..., 32] decoded e3m2 values (element e at bits 6e)."""
    bits = np.unpackbits(b24.astype(np.uint8), axis=-1, bitorder="little")
    bits = bits.reshape(bits.shape[:-1] + (32, 6)).astype(np.int64)
    codes = (bits << np.arange(6)).sum(axis=-1)
    return E3M2[codes]


def fp8_values(b: np.ndarray) -> np.ndarray:
    return E4M3[b.astype(np.int64)]


class Geo:
    def __init__(self, widths):
        w = np.asarray(widths)
        self.n4, self.n6, self.n8 = (int((w == m).sum()) for m in (4, 6, 8))
        self.n4p = -(-self.n4 // 4) * 4
        self.n6p = -(-self.n6 // 2) * 2
        self.s4, self.s6, self.s8 = self.n4p // 4, self.n6p // 2, self.n8
        self.nsteps = self.s4 + self.s6 + self.s8

    def blocks_of_step(self, st):
        """[(block index or None for padding, half, position)] of step st.
        position: 4-bit pair j (0/1); 6-bit and 8-bit 0."""
        out = []
        if st < self.s4:
            for h in (0, 1):
                for j in (0, 1):
                    b = 4 * st + 2 * j + h
                    out.append((b if b < self.n4 else None, h, j))
        elif st < self.s4 + self.s6:
            p = st - self.s4
            for h in (0, 1):
                i = 2 * p + h
                out.append((self.n4 + i if i < self.n6 else None, h, 0))
        else:
            out.append((self.n4 + self.n6 + st - self.s4 - self.s6, None, 0))
        return out


def _decode_lane_block(lane, kind, j=0):
    """q of one 4- or 6-bit block from a lane half's 48 bytes."""
    if kind == 4:
        return fp6_values(lane[..., 24 * j:24 * j + 24]) * 4
    return (fp6_values(lane[..., 0:24]) + fp6_values(lane[..., 24:48])) * 16


def _decode_steps(geo, nb, rows, lane_of, scale_of, weights):
    """Rebuild q [rows, K] and E [rows, nb] from per-step lane data
    lane_of(st, h) -> [rows, 48] and scale_of(st, h) -> [rows, >=2]."""
    q = np.zeros((rows, nb * BLOCK))
    E = np.full((rows, nb), -1, dtype=np.int64)
    ok = True
    for st in range(geo.nsteps):
        lanes = [lane_of(st, h) for h in (0, 1)]
        scs = [scale_of(st, h) for h in (0, 1)]
        for (b, h, j) in geo.blocks_of_step(st):
            if st < geo.s4 + geo.s6:
                kind = 4 if st < geo.s4 else 6
                scale = scs[h][:, j].astype(np.int64)
                if b is None:
                    part = lanes[h][:, 24 * j:24 * j + 24] if kind == 4 else lanes[h]
                    ok &= not part.any() and not scale.any()
                    if kind == 6:
                        ok &= not scs[h][:, 1].any()
                    continue
                q[:, BLOCK * b:BLOCK * b + BLOCK] = _decode_lane_block(lanes[h], kind, j)
                E[:, b] = scale
                if kind == 6:
                    ok &= not scs[h][:, 1].any()
            else:
                vals = []
                for hf in (0, 1):
                    ln = lanes[hf]
                    if weights:
                        ok &= bool(np.array_equal(ln[:, :16], ln[:, 32:48]))
                    else:
                        ok &= not ln[:, 32:48].any()
                    vals.append((fp8_values(ln[:, :16]) + fp8_values(ln[:, 16:32])) * 64)
                q[:, BLOCK * b:BLOCK * b + BLOCK] = np.concatenate(vals, axis=1)
                ok &= bool(np.array_equal(scs[0][:, 0], scs[1][:, 0]))
                ok &= not scs[0][:, 1].any() and not scs[1][:, 1].any()
                E[:, b] = scs[0][:, 0]
    return q, E, ok


ACT_STEP, ACT_SCALE_STEP, ACT_ROWS = 3072, 256, 32


def decode_act(op_img: np.ndarray, sc_img: np.ndarray, widths, M: int):
    """Activation operand image (32-row tiles) and its scale bytes ->
    (q [M, K], E [M, nb], layout_ok)."""
    geo = Geo(widths)
    nt = -(-M // ACT_ROWS)
    assert op_img.size == nt * geo.nsteps * ACT_STEP
    assert sc_img.size == nt * geo.nsteps * ACT_SCALE_STEP
    t = op_img.reshape(nt, geo.nsteps, 3, 2, ACT_ROWS, 16)
    sct = sc_img.reshape(nt, geo.nsteps, 2, ACT_ROWS, 4)

    def lane_of(st, h):
        return t[:, st, :, h].transpose(0, 2, 1, 3).reshape(nt * ACT_ROWS, 48)[:M]

    def scale_of(st, h):
        return sct[:, st, h].reshape(nt * ACT_ROWS, 4)[:M]

    q, E, ok = _decode_steps(geo, len(widths), M, lane_of, scale_of, weights=False)
    for st in range(geo.nsteps):
        for h in (0, 1):
            ok &= not scale_of(st, h)[:, 2:].any()
    return q, E, ok


def w_lane_bytes(img: np.ndarray, geo: Geo, st: int, h: int):
    """Lane data (48 bytes) of step st, half h for every column of the weight
    operand image img (1-D, all tiles).  Returns [ncols_padded, 48]."""
    tile = CHUNK * geo.nsteps
    ntiles = img.size // tile
    t = img[:ntiles * tile].reshape(ntiles, geo.nsteps, CHUNK)[:, st]
    parts = [t[:, j * PART + h * 2048:j * PART + h * 2048 + 2048].reshape(ntiles, TILE_COLS, 16)
             for j in range(3)]
    return np.concatenate(parts, axis=2).reshape(ntiles * TILE_COLS, 48)


def w_scales(img: np.ndarray, geo: Geo, st: int, h: int):
    tile = CHUNK * geo.nsteps
    ntiles = img.size // tile
    t = img[:ntiles * tile].reshape(ntiles, geo.nsteps, CHUNK)[:, st]
    # [lane (c % 32)][column tile (c / 32)][4 bytes] -> columns in order
    s = t[:, 3 * PART + h * 512:3 * PART + h * 512 + 512].reshape(ntiles, 32, 4, 4)
    return s.transpose(0, 2, 1, 3).reshape(ntiles * TILE_COLS, 4)


def decode_weights(img: np.ndarray, widths, N: int):
    """Weight operand image -> (q [Npad128, K], E [Npad128, nb], layout_ok)."""
    geo = Geo(widths)
    tile = CHUNK * geo.nsteps
    ntiles = img.size // tile
    ok = True
    for st in range(geo.nsteps):
        for h in (0, 1):
            ok &= not w_scales(img, geo, st, h)[:, 2:].any()
    q, E, ok2 = _decode_steps(geo, len(widths), ntiles * TILE_COLS,
                              lambda st, h: w_lane_bytes(img, geo, st, h),
                              lambda st, h: w_scales(img, geo, st, h), weights=True)
    return q, E, ok and ok2


# --------------------------------------------------------------------------
# Stream layout (decode GEMM): weight slabs of 16 columns and the 16-row
# activation decode image, step by step in the lane order of the 16x16x128
# scaled matrix-core instruction (lane l = 16 g + line).
# --------------------------------------------------------------------------

W_LANE = {0: 16, 1: 12, 2: 16}
A_LANE = {0: 24, 1: 32, 2: 32}
LANES = 64


GROUP = 4          # steps sharing one 256-byte scale block


class SGeo:
    def __init__(self, widths):
        w = np.asarray(widths)
        self.n = [int((w == m).sum()) for m in (4, 6, 8)]
        self.S = [-(-self.n[0] // 4), -(-self.n[1] // 2), -(-self.n[2] // 2)]
        self.nb = len(w)
        self.base = [0, self.n[0], self.n[0] + self.n[1]]   # first block of each segment

    @staticmethod
    def seg_bytes(S, step_data):
        return S * step_data + -(-S // GROUP) * LANES * 4

    def w_seg_off(self, seg):
        return sum(self.seg_bytes(self.S[s], LANES * W_LANE[s]) for s in range(seg))

    def a_seg_off(self, seg):
        return sum(self.seg_bytes(self.S[s], LANES * A_LANE[s]) for s in range(seg))

    def w_slab_bytes(self):
        return self.w_seg_off(3)

    def a_image_bytes(self):
        return self.a_seg_off(3)


def _step(buf, seg_off, st, step_data):
    """(lane data [step_data bytes], scale bytes [64] of the step) of a
    segment starting at seg_off: groups of GROUP steps, each a scale block
    (lane l's byte for step k at 4 l + k) then the steps' data."""
    g = seg_off + (st // GROUP) * (GROUP * step_data + LANES * 4)
    data = buf[..., g + LANES * 4 + (st % GROUP) * step_data:
               g + LANES * 4 + (st % GROUP + 1) * step_data]
    sc = buf[..., g: g + LANES * 4].reshape(buf.shape[:-1] + (LANES, 4))[..., st % GROUP]
    return data, sc


def _sext(v, bits):
    v = v.astype(np.int64)
    return np.where(v >= (1 << (bits - 1)), v - (1 << bits), v)


def _stream_nibbles(b8):
    """[..., 8] nibble bytes of 16 elements (two dwords; byte k of dword d
    holds elements 8d+k (low) and 8d+k+4 (high)) -> [..., 16] values 0..15."""
    out = np.zeros(b8.shape[:-1] + (16,), np.int64)
    for d in range(2):
        for k in range(4):
            byte = b8[..., 4 * d + k].astype(np.int64)
            out[..., 8 * d + k] = byte & 15
            out[..., 8 * d + k + 4] = byte >> 4
    return out


def _sm_nibble(v):
    """Sign-magnitude 4-bit codes (sign at bit 3) -> values."""
    return np.where(v & 8, -(v & 7), v & 7)


def decode_w_stream(img, widths, N, sm=True):
    """Weight slabs -> (q [Npad16, K], E [Npad16, nb], layout_ok).  sm: 4- and
    6-bit codes are sign-magnitude (symmetric clamp), else two's complement."""
    g = SGeo(widths)
    nsl = -(-N // 16)
    sb = g.w_slab_bytes()
    slabs = img[:nsl * sb].reshape(nsl, sb)
    q = np.zeros((nsl * 16, g.nb * BLOCK), np.int64)
    E = np.full((nsl * 16, g.nb), -1, np.int64)
    ok = True
    for seg in range(3):
        sd = LANES * W_LANE[seg]
        for s in range(g.S[seg]):
            ch, scb = _step(slabs, g.w_seg_off(seg), s, sd)
            sc = scb.reshape(nsl, 4, 16).astype(np.int64)          # [slab, g, col]
            for gg in range(4):
                half = gg & 1
                if seg == 0:
                    lane = ch.reshape(nsl, 4, 16, 16)[:, gg]        # [slab, col, 16]
                    parts = [(4 * s + (gg >> 1), lane[..., 0:8]), (4 * s + 2 + (gg >> 1), lane[..., 8:16])]
                    dec = _sm_nibble if sm else (lambda v: _sext(v, 4))
                    vals = [(blk, dec(_stream_nibbles(p))) for blk, p in parts]
                else:
                    blk = 2 * s + (gg >> 1)
                    if seg == 1:
                        nib = ch[:, :LANES * 8].reshape(nsl, 4, 16, 8)[:, gg]
                        top = ch[:, 512:512 + LANES * 4].reshape(nsl, 4, 16, 4)[:, gg]
                        y = top.astype(np.int64)
                        y = y[..., 0] | (y[..., 1] << 8) | (y[..., 2] << 16) | (y[..., 3] << 24)
                        lo = _stream_nibbles(nib)
                        t2 = np.stack([(y >> (8 * (u % 4) + 2 * (u // 4))) & 3 for u in range(16)],
                                      axis=-1)
                        if sm:      # |q| = 8 t2 + (lo & 7), sign at bit 3 of lo
                            v = np.where(lo & 8, -(8 * t2 + (lo & 7)), 8 * t2 + (lo & 7))
                        else:
                            v = _sext(lo | (t2 << 4), 6)
                    else:
                        v = _sext(ch.reshape(nsl, 4, 16, 16)[:, gg], 8)
                    vals = [(blk, v)]
                for blk, v in vals:
                    v = v.reshape(nsl * 16, 16)
                    if blk < g.n[seg]:
                        b = g.base[seg] + blk
                        q[:, BLOCK * b + 16 * half: BLOCK * b + 16 * half + 16] = v
                    else:
                        ok &= not v.any()
            # lane group gg carries the exponent of block 4s+gg (4-bit) or
            # 2s+(gg&1) (6/8-bit)
            for gg in range(4):
                blk = 4 * s + gg if seg == 0 else 2 * s + (gg & 1)
                e = sc[:, gg].reshape(nsl * 16)
                if blk < g.n[seg]:
                    b = g.base[seg] + blk
                    ok &= bool(np.all((E[:, b] == -1) | (E[:, b] == e)))
                    E[:, b] = e
                else:
                    ok &= not e.any()
        # scale bytes of the missing steps of a short last group are zero
        for s in range(g.S[seg], -(-g.S[seg] // GROUP) * GROUP):
            _, scb = _step(slabs, g.w_seg_off(seg), s, sd)
            ok &= not scb.any()
    return q, E, ok


def decode_act_dimg(img, widths, M):
    """Activation decode image (16 rows) -> (q [M, K], E [M, nb], layout_ok)."""
    g = SGeo(widths)
    assert img.size == g.a_image_bytes()
    q = np.zeros((16, g.nb * BLOCK), np.int64)
    E = np.full((16, g.nb), -1, np.int64)
    ok = True
    for seg in range(3):
        sd = LANES * A_LANE[seg]
        for s in range(g.S[seg]):
            ch, scb = _step(img, g.a_seg_off(seg), s, sd)
            sc = scb.reshape(4, 16).astype(np.int64)
            for gg in range(4):
                if seg == 0:
                    b24 = np.concatenate([ch[:1024].reshape(4, 16, 16)[gg],
                                          ch[1024:1536].reshape(4, 16, 8)[gg]], axis=1)
                    v = fp6_values(b24)[:M] * 4
                    blk, lo, hi = 4 * s + gg, 0, 32
                else:
                    lane = ch[:2048].reshape(4, 16, 32)[gg]
                    hv, lv = fp8_values(lane[:M, :16]), fp8_values(lane[:M, 16:])
                    # digits of q = 16 h + l summing to q 2^-(m-2): h + l/16
                    # (6-bit), h/4 + l/64 (8-bit)
                    f = 16 if seg == 1 else 64
                    v = f * (hv + lv)
                    h, l = hv * f / 16, lv * f
                    ok &= bool(np.all((l >= 0) & (l <= 15) & (h == np.floor(v / 16))))
                    blk, lo, hi = 2 * s + (gg >> 1), 16 * (gg & 1), 16 * (gg & 1) + 16
                if blk < g.n[seg]:           # rows past M are unspecified
                    b = g.base[seg] + blk
                    q[:M, BLOCK * b + lo: BLOCK * b + hi] = v
                else:
                    ok &= not np.any(v)
            for gg in range(4):
                blk = 4 * s + gg if seg == 0 else 2 * s + (gg & 1)
                e = sc[gg]
                if blk < g.n[seg]:
                    b = g.base[seg] + blk
                    ok &= bool(np.all((E[:M, b] == -1) | (E[:M, b] == e[:M])))
                    E[:, b] = e
                else:
                    ok &= not e[:M].any()
    return q[:M], E[:M], ok
