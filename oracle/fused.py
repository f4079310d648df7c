"""Oracle of a quantizer fused into its producer: RMSNorm -> MXINT quantize.

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the product
library; it shares no code with the GPU path.

Paper: MXSens (arXiv 2607.17733), Appendix A.2: the activations of every
decoder linear are quantized, while normalisation layers stay in 16-bit
floating point.  The paper does not spell out the normalisation; this is
the RMS normalisation of the LLaMA models it evaluates, made deterministic
(a reading): for a row x of K bf16 values and a bf16 gain g,
  ms  = (sum of x_k^2) / K in float64: each 32-element block summed in
        order, then the block sums in order (every square is exact);
  r   = float32(1 / sqrt(ms + eps)), the square root and the division in
        IEEE float64, eps the float32 value given;
  h_k = bf16(float32(x_k * r)),  y_k = bf16(float32(g_k * h_k)),
with round-to-nearest-even at every narrowing.  The fused quantizer then
quantizes y exactly as the plain one quantizes its input.
"""
from __future__ import annotations

import numpy as np

BLOCK = 32


def bf16_to_f32(bits) -> np.ndarray:
    return (np.asarray(bits).astype(np.uint32) << 16).view(np.float32)


def f32_to_bf16(x) -> np.ndarray:
    """Round float32 to bf16 bits, nearest-even (NaN stays NaN)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    return np.where(nan, ((u >> 16) | 0x40).astype(np.uint16), r)


def row_inv_rms(x_bits, eps) -> np.ndarray:
    """Per row: float32(1 / sqrt(ms + eps)) with ms in the fixed order."""
    x = bf16_to_f32(x_bits).astype(np.float64)
    M, K = x.shape
    out = np.empty(M, dtype=np.float32)
    for i in range(M):
        acc = 0.0
        for b in range(K // BLOCK):
            part = 0.0
            for v in x[i, BLOCK * b:BLOCK * (b + 1)]:
                part += v * v
            acc += part
        ms = acc / K
        out[i] = np.float32(1.0 / np.sqrt(ms + float(np.float32(eps))))
    return out


def rmsnorm_bf16(x_bits, g_bits, eps) -> np.ndarray:
    """RMS normalisation of bf16 rows with bf16 gain, as bf16 bits."""
    x_bits = np.asarray(x_bits, dtype=np.uint16)
    r = row_inv_rms(x_bits, eps)
    x32 = bf16_to_f32(x_bits)
    h = f32_to_bf16(x32 * r[:, None])                         # float32 products
    g32 = bf16_to_f32(np.asarray(g_bits, dtype=np.uint16))
    return f32_to_bf16(g32[None, :] * bf16_to_f32(h))
