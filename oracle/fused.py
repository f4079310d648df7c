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


# --------------------------------------------------------------------------
# SiLU(gate) * up before the quantizer (the down projection's producer)
#
# Reading: the exponential is not left to a math library, whose last-bit
# results differ between machines; it is a fixed float32 evaluation, the
# classic Cody-Waite reduction and a Taylor polynomial, with every operation
# an IEEE float32 operation rounded on its own (no fused multiply-add):
#   t  = clamp(t, -120, 120)
#   k  = rint(t * (1/ln2))                     (float32 1/ln2 = 0x3FB8AA3B)
#   r  = (t - k * LN2_HI) - k * LN2_LO         (0x3F317200, 0x35BFBE8E)
#   p  = Horner over 1, 1, 1/2!, ..., 1/7! (float32 coefficients)
#   e^t = ldexp(p, k)
# silu(g) = g / (1 + e^(-g)); a = bf16(silu(g)); y = bf16(a * u), float32
# products and round-to-nearest-even; a NaN gate gives a NaN.

F32 = np.float32
INV_LN2 = np.uint32(0x3FB8AA3B).view(np.float32)
LN2_HI = np.uint32(0x3F317200).view(np.float32)
LN2_LO = np.uint32(0x35BFBE8E).view(np.float32)
EXP_COEF = [np.uint32(v).view(np.float32) for v in
            (0x39500D01, 0x3AB60B61, 0x3C088889, 0x3D2AAAAB, 0x3E2AAAAB, 0x3F000000,
             0x3F800000, 0x3F800000)]                # 1/7!, 1/6!, ..., 1/2!, 1, 1


def exp32(t) -> np.ndarray:
    """e^t as defined above (a NaN argument is not defined here; silu32
    handles it)."""
    t = np.asarray(t, dtype=F32)
    t = np.clip(np.where(np.isnan(t), F32(0.0), t), F32(-120.0), F32(120.0))
    k = np.rint(t * INV_LN2).astype(F32)
    r = (t - k * LN2_HI) - k * LN2_LO
    p = np.full_like(r, EXP_COEF[0])
    for c in EXP_COEF[1:]:
        p = p * r + c
    with np.errstate(over="ignore"):
        return np.ldexp(p, k.astype(np.int32)).astype(F32)


def silu32(g) -> np.ndarray:
    g = np.asarray(g, dtype=F32)
    with np.errstate(over="ignore"):
        s = g / (F32(1.0) + exp32(-g))
    return np.where(np.isnan(g), F32(np.nan), s).astype(F32)


def swiglu_bf16(g_bits, u_bits) -> np.ndarray:
    """bf16(bf16(silu(g)) * u) as bf16 bits."""
    a = f32_to_bf16(silu32(bf16_to_f32(g_bits)))
    return f32_to_bf16(bf16_to_f32(a) * bf16_to_f32(u_bits))
