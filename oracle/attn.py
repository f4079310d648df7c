"""Oracle of decode attention over an MXINT KV cache.

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the product
library; it shares no code with the GPU path.

Paper: MXSens (arXiv 2607.17733), Appendix A.2: the KV cache is quantized
to MXINT (4 to 8 bits per block); attention then reads it.  One new token
per sequence attends to the T cached tokens of its sequence: with K and V
dequantized block by block (value = q * 2^(E - 127 - (m - 2)), the
quantizer's definition), per query head h of KV group g = h / (Hq / Hkv):
  s_t = (q_h . K_t) * scale,  p = softmax(s) over t,  o_h = sum_t p_t V_t,
in float64 here.
"""
from __future__ import annotations

import numpy as np

import oracle


def dequantize_cache(bits, widths):
    """bf16 cache rows [rows, D] -> the dequantized float64 values the
    attention reads (quantize then dequantize, identity permutation)."""
    q, e = oracle.quantize(bits, widths=widths)
    return oracle.dequantize(q, e, widths)


def attention(qf, kd, vd, B: int, Hq: int, Hkv: int, T: int, scale: float):
    """qf: float [B, Hq, D]; kd, vd: float64 [B * T * Hkv, D] with row
    (b * T + t) * Hkv + h.  Returns o float64 [B, Hq, D]."""
    D = kd.shape[1]
    k = kd.reshape(B, T, Hkv, D)
    v = vd.reshape(B, T, Hkv, D)
    G = Hq // Hkv
    o = np.empty((B, Hq, D), dtype=np.float64)
    for b in range(B):
        for h in range(Hq):
            kh = k[b, :, h // G, :]                       # [T, D]
            s = (kh @ np.asarray(qf[b, h], dtype=np.float64)) * scale
            p = np.exp(s - s.max())
            p /= p.sum()
            o[b, h] = p @ v[b, :, h // G, :]
    return o
