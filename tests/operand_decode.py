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
    return t[:, 3 * PART + h * 512:3 * PART + h * 512 + 512].reshape(ntiles * TILE_COLS, 4)


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
