"""The allocation-free attention entry point (mxq_attn_decode_static, static
per-GPU scratch) against mxq_attn_decode with a caller work buffer and
against the float64 oracle, through the C ABI: two calls in a row, the second
smaller, so the second reuses scratch the first left behind."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import attn as oattn
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from parity_util import say, to_dev_bf16

pytestmark = pytest.mark.gpu

D = 128


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def _case(seed, B, Hq, Hkv, T, widths):
    say("no-alloc attn seed=%d B=%d Hq=%d Hkv=%d T=%d widths=%s" % (seed, B, Hq, Hkv, T, widths))
    qb, kb, vb = W.attn_inputs(seed, B, Hq, Hkv, T)
    fmt = mxq.Format(D, widths)
    kc = mxq.quantize_rows(to_dev_bf16(kb), fmt)
    vc = mxq.quantize_rows(to_dev_bf16(vb), fmt)
    q = to_dev_bf16(qb.reshape(-1, D)).reshape(B, Hq, D)
    return qb, kb, vb, fmt, kc, vc, q


def _static_call(fmt, q, kc, vc, B, Hq, Hkv, T, scale, out):
    lib = mxq.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return lib.mxq_attn_decode_static(fmt.ref, _p(q), B, Hq, Hkv, T, ctypes.c_float(scale),
                                      _p(kc[0]), _p(kc[1]), _p(vc[0]), _p(vc[1]), _p(out), stream)


def _work_call(fmt, q, kc, vc, B, Hq, Hkv, T, scale, out):
    lib = mxq.lib()
    nw = lib.mxq_attn_work_bytes(fmt.ref, B, Hq, Hkv, T)
    assert 0 < nw <= mxq.ATTN_STATIC_WORK_BYTES
    work = torch.empty(nw, dtype=torch.uint8, device="cuda")
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return lib.mxq_attn_decode(fmt.ref, _p(q), B, Hq, Hkv, T, ctypes.c_float(scale),
                               _p(kc[0]), _p(kc[1]), _p(vc[0]), _p(vc[1]), _p(out), _p(work),
                               nw, stream)


def test_static_scratch_matches_work_buffer_twice():
    cases = [(31, 4, 64, 8, 1000, [4, 4, 6, 8]),      # larger first
             (32, 1, 16, 4, 300, [4, 4, 4, 4])]       # then smaller
    scale = 1.0 / np.sqrt(D)
    for seed, B, Hq, Hkv, T, widths in cases:
        qb, kb, vb, fmt, kc, vc, q = _case(seed, B, Hq, Hkv, T, widths)
        o_static = torch.full((B, Hq, D), float("nan"), device="cuda")
        o_work = torch.full((B, Hq, D), float("nan"), device="cuda")
        assert _static_call(fmt, q, kc, vc, B, Hq, Hkv, T, scale, o_static) == 0
        assert _work_call(fmt, q, kc, vc, B, Hq, Hkv, T, scale, o_work) == 0
        torch.cuda.synchronize()
        # the same kernels with the same split: identical results
        assert torch.equal(o_static, o_work)
        o = o_static.cpu().numpy().astype(np.float64)
        qf = W.bf16_bits_to_f32(qb).astype(np.float64)
        rows = T * Hkv
        for b in range(B):
            sl = slice(b * rows, (b + 1) * rows)
            kd = oattn.dequantize_cache(kb[sl], widths)
            vd = oattn.dequantize_cache(vb[sl], widths)
            ref = oattn.attention(qf[b:b + 1], kd, vd, 1, Hq, Hkv, T, scale)[0]
            vmax = np.abs(vd.reshape(T, Hkv, D)).max(axis=(0, 2))
            err = np.abs(o[b] - ref).max(axis=1) / vmax[np.arange(Hq) // (Hq // Hkv)]
            assert err.max() <= 1e-5, (b, err.max())


def test_static_scratch_rejects_oversize_before_launch():
    lib = mxq.lib()
    fmt = mxq.Format(D, [4, 4, 4, 4])
    B, Hq, Hkv, T = 300, 64, 8, 64
    assert lib.mxq_attn_work_bytes(fmt.ref, B, Hq, Hkv, T) > mxq.ATTN_STATIC_WORK_BYTES
    fake = ctypes.c_void_p(1 << 20)
    st = lib.mxq_attn_decode_static(fmt.ref, fake, B, Hq, Hkv, T, ctypes.c_float(0.1),
                                    fake, fake, fake, fake, fake, None)
    assert st == 8
