"""CPU-side checks of the C ABI: the library loads, exports every function
declared in include/mxq.h, and its host-only entry points (sizes, argument
validation) behave as documented.  No device work is enqueued here: every
call either computes a size or fails validation before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mxq.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mxq_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_17733_amd import mxq
    if not os.path.exists(mxq.LIB_PATH):
        from paper_2607_17733_amd import build
        build.build()
    return mxq.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("mxq_quantize_act", "mxq_pack_weights", "mxq_gemm",
              "mxq_unpack_act", "mxq_unpack_weights", "mxq_gemm_partials"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def _fmt(K, widths, round_=0, clamp=0, block=32, reserved=0):
    from paper_2607_17733_amd.mxq import _Fmt
    w = np.ascontiguousarray(widths, dtype=np.uint8)
    f = _Fmt(K, block, round_, clamp, reserved, w.ctypes.data_as(ctypes.c_void_p).value, None)
    return f, w


def layout_sizes(widths, M, N, full=False):
    """Buffer sizes as include/mxq.h states them: four segments (3-, 4-, 6-,
    8-bit blocks) of steps of four (3/4-bit) or two (6/8-bit) blocks, groups
    of four steps; the activation image in 16-row tiles of 64 lanes x 24
    (32 for 8-bit steps) bytes per step plus 256 scale bytes per group; the
    weights in 128-column super-slabs of eight chunks per step plus 2048
    scale bytes per group."""
    n = [sum(1 for w in widths if w == m) for m in (3, 4, 6, 8)]
    S = [-(-n[0] // 4), -(-n[1] // 4), -(-n[2] // 2), -(-n[3] // 2)]
    groups = sum(-(-s // 4) for s in S)
    tiles, supers = -(-M // 16), -(-N // 128)
    chunk = [(768, 1024), (1024, 1536), (768, 1024), (1024, 1024)]
    act = tiles * 64 * (24 * (S[0] + S[1] + S[2]) + 32 * S[3])
    act_exp = tiles * groups * 256
    wb = supers * 8 * sum(s * c[int(full)] for s, c in zip(S, chunk))
    w_exp = supers * groups * 2048
    return act, act_exp, wb, w_exp


def test_sizes(lib):
    w1 = [4] * 6 + [6, 8]
    f, _w = _fmt(256, w1)
    fr = ctypes.byref(f)
    assert lib.mxq_abi_version() == 12
    # S = 0/2/1/1 steps, 3 groups: tiles of 64 x (3 x 24 + 32) bytes
    assert layout_sizes(w1, 16, 128) == (6656, 768, 8 * (2 * 1024 + 768 + 1024), 3 * 2048)
    assert lib.mxq_act_packed_bytes(fr) == 160
    assert lib.mxq_exp_row_bytes(fr) == 16
    for M in (1, 16, 17, 33, 64, 300):
        act, act_exp, _, _ = layout_sizes(w1, M, 1)
        assert lib.mxq_act_bytes(fr, M) == act
        assert lib.mxq_act_exp_bytes(fr, M) == act_exp
    assert lib.mxq_act_bytes(fr, 0) == 0
    assert lib.mxq_act_bytes(fr, -1) == -2
    for N in (1, 17, 128, 129, 250, 256):
        _, _, wb, w_exp = layout_sizes(w1, 1, N)
        assert lib.mxq_weight_bytes(fr, N) == wb
        assert lib.mxq_weight_exp_bytes(fr, N) == w_exp
    f_full, _wf = _fmt(256, w1, clamp=1)
    assert lib.mxq_weight_bytes(ctypes.byref(f_full), 256) == layout_sizes(w1, 1, 256, True)[2]
    w2 = [4] * 102 + [6] * 13 + [8] * 13
    f2, _w2 = _fmt(4096, w2)
    assert lib.mxq_act_packed_bytes(ctypes.byref(f2)) == 2368   # 2360 rounded up to 16
    assert lib.mxq_exp_row_bytes(ctypes.byref(f2)) == 128
    assert lib.mxq_act_bytes(ctypes.byref(f2), 2048) == 128 * 64 * (24 * 33 + 32 * 7)
    assert lib.mxq_act_exp_bytes(ctypes.byref(f2), 2048) == 128 * 11 * 256
    w3 = [3] * 26 + [6] * 4 + [8] * 2
    f3, _w3 = _fmt(1024, w3)
    assert lib.mxq_act_packed_bytes(ctypes.byref(f3)) == 480   # 26 x 12 + 4 x 24 + 2 x 32 = 472
    assert lib.mxq_weight_bytes(ctypes.byref(f3), 128) == layout_sizes(w3, 1, 128)[2]


@pytest.mark.parametrize("counts,N", [((217, 26, 13), 28672), ((761, 90, 45), 8192)])
def test_weights_at_mxint_size(lib, counts, N):
    """The one weight copy is within 5 % of the MXINT bits (mantissas plus
    one exponent byte per block) at the decode workload's 85/10/5 split."""
    n4, n6, n8 = counts
    widths = [4] * n4 + [6] * n6 + [8] * n8
    f, _w = _fmt(32 * len(widths), widths)
    stored = lib.mxq_weight_bytes(ctypes.byref(f), N) + lib.mxq_weight_exp_bytes(ctypes.byref(f), N)
    mxint = N * sum(4 * m + 1 for m in widths)
    assert stored <= 1.05 * mxint, stored / mxint
    assert 8 * stored / (N * 32 * len(widths)) <= 4.9


def test_size_functions_match_oracle_layout(lib, oracle_lib):
    for widths in ([4] * 3 + [6] * 1, [6] * 3, [8] * 5, [4] * 7 + [8], [3] * 2 + [6] + [8],
                   [3, 4, 4, 6]):
        f, _w = _fmt(32 * len(widths), widths)
        assert lib.mxq_act_packed_bytes(ctypes.byref(f)) == oracle_lib.act_row_bytes(widths)


@pytest.mark.parametrize("kwargs,status", [
    (dict(K=250, widths=[4] * 8), 2),            # K % 32
    (dict(K=64, widths=[4, 5]), 3),              # bad width
    (dict(K=64, widths=[8, 4]), 3),              # not grouped
    (dict(K=64, widths=[6, 4]), 3),
    (dict(K=64, widths=[4, 3]), 3),              # 3-bit blocks come first
    (dict(K=64, widths=[2, 4]), 3),
    (dict(K=64, widths=[4, 4], block=16), 6),
    (dict(K=64, widths=[4, 4], round_=2), 6),
    (dict(K=64, widths=[4, 4], clamp=7), 6),
    (dict(K=64, widths=[4, 4], reserved=1), 6),
])
def test_bad_formats_rejected(lib, kwargs, status):
    f, _w = _fmt(**kwargs)
    assert lib.mxq_act_packed_bytes(ctypes.byref(f)) == -status
    assert lib.mxq_act_bytes(ctypes.byref(f), 4) == -status
    # the quantizer rejects the format before touching any pointer
    dummy = ctypes.c_void_p(16)
    assert lib.mxq_quantize_act(ctypes.byref(f), dummy, 4, 4096, dummy, dummy, None) == status


def test_argument_validation_before_launch(lib):
    f, _w = _fmt(64, [4, 8])
    fr = ctypes.byref(f)
    p16 = ctypes.c_void_p(4096)          # never dereferenced: validation fails first
    bad = ctypes.c_void_p(4097)
    assert lib.mxq_quantize_act(None, p16, 4, 64, p16, p16, None) == 1
    assert lib.mxq_quantize_act(fr, None, 4, 64, p16, p16, None) == 1
    assert lib.mxq_quantize_act(fr, p16, 4, 63, p16, p16, None) == 2
    assert lib.mxq_quantize_act(fr, p16, -1, 64, p16, p16, None) == 2
    assert lib.mxq_quantize_act(fr, bad, 4, 64, p16, p16, None) == 5
    assert lib.mxq_quantize_act(fr, p16, 0, 64, None, None, None) == 0   # empty: no-op
    assert lib.mxq_pack_weights(fr, p16, 4, 64, bad, p16, None) == 5
    assert lib.mxq_gemm(fr, 4, 4, p16, p16, p16, p16, p16, 3, None) == 2   # ldy < N
    assert lib.mxq_gemm(fr, 4, 4, p16, None, p16, p16, p16, 4, None) == 1
    assert lib.mxq_gemm(fr, 0, 4, None, None, None, None, None, 4, None) == 0
    assert lib.mxq_gemm(fr, -1, 4, p16, p16, p16, p16, p16, 4, None) == 2
    assert lib.mxq_gemm_partials(fr, 4, 4, p16, p16, p16, p16, bad, None) == 5
    assert lib.mxq_unpack_act(fr, 4, p16, p16, None, p16, None) == 1
    assert lib.mxq_status_str(5).decode().startswith("device pointer")


def test_peak_microbenchmarks_validate_before_launch(lib):
    from paper_2607_17733_amd.mxq import _SIGS  # noqa: F401  (signatures set by lib())
    assert lib.mxq_peak_sink_words() >= 256 * 16 * 64
    fake = ctypes.c_void_p(16)
    ops = ctypes.c_int64(-1)
    assert lib.mxq_peak_stream_read(None, 16, fake, None) == 1          # MXQ_ERR_NULL
    assert lib.mxq_peak_stream_read(fake, 15, fake, None) == 2          # MXQ_ERR_SHAPE
    assert lib.mxq_peak_stream_read(fake, 0, fake, None) == 2
    assert lib.mxq_peak_mfma(3, 1, fake, ctypes.byref(ops), None) == 2
    assert lib.mxq_peak_mfma(0, 0, fake, ctypes.byref(ops), None) == 2
    assert lib.mxq_peak_mfma(0, 1, None, ctypes.byref(ops), None) == 1


def test_attention_validates_before_launch(lib):
    f, _w = _fmt(128, [4, 4, 6, 8])
    fr = ctypes.byref(f)
    p16 = ctypes.c_void_p(4096)          # never dereferenced: validation fails first
    bad = ctypes.c_void_p(4097)
    big = 1 << 40

    def call(fmt=fr, q=p16, B=2, Hq=8, Hkv=2, T=100, scale=0.1, k=p16, work=p16, wb=big):
        return lib.mxq_attn_decode(fmt, q, B, Hq, Hkv, T, scale, k, p16, p16, p16, p16,
                                   work, wb, None)

    # per (sequence, query head) 130 floats per token split; splits <= ceil(T / 64)
    for B, Hq, Hkv, T in [(1, 64, 8, 4096), (16, 64, 8, 4096), (3, 8, 2, 1), (2, 16, 1, 65)]:
        n = lib.mxq_attn_work_bytes(fr, B, Hq, Hkv, T)
        unit = B * Hq * 130 * 4
        assert n > 0 and n % unit == 0 and n // unit <= -(-T // 64), (B, Hq, Hkv, T, n)
    assert lib.mxq_attn_work_bytes(fr, 0, 8, 2, 10) == 0
    assert lib.mxq_attn_work_bytes(fr, 1, 8, 3, 10) == -2            # Hq % Hkv
    assert lib.mxq_attn_work_bytes(fr, 1, 34, 2, 10) == -2           # G > 16
    assert lib.mxq_attn_work_bytes(fr, 1, 8, 2, 0) == -2             # T < 1
    f2, _w2 = _fmt(256, [4] * 8)
    assert lib.mxq_attn_work_bytes(ctypes.byref(f2), 1, 8, 2, 10) == -2   # head dim 256
    assert call(B=0, q=None, k=None, work=None) == 0                 # empty batch: no-op
    assert call(q=None) == 1
    assert call(k=bad) == 5
    assert call(q=ctypes.c_void_p(4098)) == 5                          # q not 16-byte aligned
    assert call(work=bad) == 5
    assert call(wb=16) == 2                                          # short work buffer
    assert call(scale=float("inf")) == 2
    assert call(scale=float("nan")) == 2
    assert call(Hkv=3) == 2
    assert call(T=0) == 2
