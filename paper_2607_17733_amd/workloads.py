"""Seeded synthetic workloads shared by the tests, the smoke check and the bench.

This module only draws inputs; it contains none of the quantization or GEMM
arithmetic.  Everything is numpy on the host.  Tensors are returned as bf16
bit patterns (``uint16``) plus the offline-calibration outputs the hot path
takes as inputs: a column permutation ``perm`` (``perm[p]`` = source column
placed at position ``p``) and a per-block width map ``widths``.

Shapes and value distributions stand in for the paper's LLaMA workloads
(Section 5: LLaMA-3-8B, LLaMA-2-70B), whose weights and calibration data are
not available:

* activations ``A[r, k] = z[r, k] * c[k]`` with ``z ~ N(0, 1)`` (Student-t
  with 3 degrees of freedom for the heavy-tailed down-projection input) and a
  per-channel scale ``c`` that is 1 except on two disjoint outlier channel
  sets: 1 % of channels with ``c ~ U(20, 100)`` (extreme outliers) and 5 % with
  ``c ~ U(2, 5)`` (mild outliers), after the paper's observation that
  systematic outliers range from rare extremes to frequent mild deviations
  (Sections 1 and 3.1);
* weights ``W ~ N(0, 0.02^2)``, shape ``[N, K]`` (``torch.nn.Linear`` layout);
* width maps from percentages: ``n8 = round(p8 * nb)``, ``n6 = round(p6 * nb)``,
  ``n4 = nb - n6 - n8``; blocks are ordered 4-bit, then 6-bit, then 8-bit;
* the permutation stands in for the column-sensitivity ranking: channels are
  ordered by their drawn scale (largest first, ties in a seeded random
  order); the first ``32 * n8`` go to 8-bit blocks, the next ``32 * n6`` to
  6-bit blocks, the rest to 4-bit blocks (Section 4.1: the most sensitive
  columns form the high-precision blocks).

Random streams: ``numpy.random.Generator(PCG64(SeedSequence(1000 + config,
spawn_key=(k,))))`` with k = 0 outlier channel sets, 1 outlier scales,
2 permutation tie-break, 3 activations, 4 + j weights of linear j,
20 / 21 the K / V cache tensors.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

BLOCK = 32


def rng(config: int, k: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence(1000 + config, spawn_key=(k,))))


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & 1
    return ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32)


def width_counts(nb: int, p6: float, p8: float):
    n8 = int(np.floor(p8 * nb + 0.5))
    n6 = int(np.floor(p6 * nb + 0.5))
    return nb - n6 - n8, n6, n8


def widths_from_counts(n4: int, n6: int, n8: int) -> np.ndarray:
    return np.array([4] * n4 + [6] * n6 + [8] * n8, dtype=np.uint8)


def channel_scales(config: int, K: int, p_extreme=0.01, p_mild=0.05,
                   fixed=None) -> np.ndarray:
    """Per-channel scale vector c (1 outside the outlier channel sets)."""
    c = np.ones(K, np.float64)
    if fixed is not None:                   # (count, scale) -> explicit outliers
        count, scale = fixed
        chans = rng(config, 0).permutation(K)[:count]
        c[chans] = scale
        return c
    n1 = int(round(p_extreme * K))
    n2 = int(round(p_mild * K))
    chans = rng(config, 0).permutation(K)[: n1 + n2]
    g = rng(config, 1)
    c[chans[:n1]] = g.uniform(20.0, 100.0, n1)
    c[chans[n1:]] = g.uniform(2.0, 5.0, n2)
    return c


def permutation_from_scales(config: int, c: np.ndarray, n4: int, n6: int,
                            n8: int) -> np.ndarray:
    K = len(c)
    tiebreak = rng(config, 2).permutation(K)
    order = np.lexsort((tiebreak, -c))      # largest scale first
    s8 = order[: BLOCK * n8]
    s6 = order[BLOCK * n8: BLOCK * (n8 + n6)]
    s4 = order[BLOCK * (n8 + n6):]
    return np.concatenate([s4, s6, s8]).astype(np.int32)


@dataclass
class LinearCase:
    """One quantized linear: activations [M, K], weights [N, K], format."""
    name: str
    M: int
    K: int
    N: int
    a_bits: np.ndarray            # uint16 [M, K]
    w_bits: np.ndarray            # uint16 [N, K]
    perm: np.ndarray              # int32 [K]
    widths: np.ndarray            # uint8 [K/32]
    meta: dict = field(default_factory=dict)


def activations(config: int, M: int, c: np.ndarray, dist: str = "normal",
                stream: int = 3) -> np.ndarray:
    g = rng(config, stream)
    K = len(c)
    if dist == "student_t3":
        z = g.standard_t(3, size=(M, K)).astype(np.float32)
    else:
        z = g.standard_normal((M, K), dtype=np.float32)
    z *= c.astype(np.float32)[None, :]
    return to_bf16_bits(z)


def weights(config: int, N: int, K: int, j: int = 0, std: float = 0.02) -> np.ndarray:
    g = rng(config, 4 + j)
    w = g.standard_normal((N, K), dtype=np.float32) * np.float32(std)
    return to_bf16_bits(w)


def make_linear(config: int, name: str, M: int, K: int, N: int, p6: float,
                p8: float, dist: str = "normal", j: int = 0, counts=None,
                fixed_outliers=None, identity_perm: bool = False) -> LinearCase:
    nb = K // BLOCK
    n4, n6, n8 = counts if counts is not None else width_counts(nb, p6, p8)
    c = channel_scales(config, K, fixed=fixed_outliers)
    perm = (np.arange(K, dtype=np.int32) if identity_perm
            else permutation_from_scales(config, c, n4, n6, n8))
    return LinearCase(name, M, K, N, activations(config, M, c, dist),
                      weights(config, N, K, j), perm,
                      widths_from_counts(n4, n6, n8),
                      {"config": config, "n4": n4, "n6": n6, "n8": n8,
                       "dist": dist})


# --------------------------------------------------------------------------
# The workload table: LLaMA-shaped linears.
# --------------------------------------------------------------------------

def tiny() -> LinearCase:
    """M=16, K=256, N=256; two input channels scaled x50; widths 6/1/1."""
    return make_linear(1, "tiny", 16, 256, 256, 0.0, 0.0, counts=(6, 1, 1),
                       fixed_outliers=(2, 50.0))


def attn_proj(M: int = 2048) -> LinearCase:
    """LLaMA-3-8B attention projection: M=2048, K=N=4096, widths 80/10/10 %."""
    return make_linear(2, "llama3_8b_attn_proj", M, 4096, 4096, 0.10, 0.10)


def mlp_gate_up(M: int = 4096) -> LinearCase:
    """LLaMA-3-8B gate/up projection: M=4096, K=4096, N=14336, 70/15/15 %."""
    return make_linear(3, "llama3_8b_gate_up", M, 4096, 14336, 0.15, 0.15, j=0)


def mlp_down(M: int = 4096) -> LinearCase:
    """LLaMA-3-8B down projection: M=4096, K=14336, N=4096, t3 activations."""
    return make_linear(3, "llama3_8b_down", M, 14336, 4096, 0.15, 0.15,
                       dist="student_t3", j=1)


def decode(M: int, which: str) -> LinearCase:
    """LLaMA-2-70B-shaped decode linears, widths 85/10/5 %."""
    K, N, j = (8192, 28672, 0) if which == "up" else (28672, 8192, 1)
    return make_linear(4, "llama2_70b_decode_%s_m%d" % (which, M), M, K, N,
                       0.10, 0.05, j=j)


LAYER_LINEARS = (
    # name, K, N
    ("q", 8192, 8192), ("k", 8192, 1024), ("v", 8192, 1024),
    ("o", 8192, 8192), ("gate", 8192, 28672), ("up", 8192, 28672),
    ("down", 28672, 8192),
)


def layer_linear(j: int, sensitive: bool, M: int = 8192) -> LinearCase:
    """One linear of a LLaMA-2-70B-shaped decoder layer (hidden 8192, 64 query
    heads, 8 KV heads, head dim 128, FFN 28672); sensitive layers use 30 %
    8-bit blocks, the others 5 %, both with 10 % 6-bit blocks."""
    name, K, N = LAYER_LINEARS[j]
    p8 = 0.30 if sensitive else 0.05
    return make_linear(5, "llama2_70b_%s" % name, M, K, N, 0.10, p8, j=j)


def kv_cache(which: int, tokens: int = 4096, heads: int = 8, head_dim: int = 128):
    """bf16 K (which=0) or V (which=1) cache [tokens * heads, head_dim],
    N(0, 1) values; quantized along the head dimension with 4-bit blocks."""
    g = rng(5, 20 + which)
    x = g.standard_normal((tokens * heads, head_dim), dtype=np.float32)
    return to_bf16_bits(x)


def random_case(seed: int, M: int, K: int, N: int, counts, perm: str = "random",
                outliers: bool = True) -> LinearCase:
    """Small seeded case for parity tests (perm: identity|random|scales)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(
        7000 + seed, spawn_key=(M, K, N))))
    c = np.ones(K)
    if outliers:
        nout = max(1, K // 64)
        ch = g.permutation(K)[:nout]
        c[ch] = g.uniform(2.0, 100.0, nout)
    z = g.standard_normal((M, K), dtype=np.float32) * c.astype(np.float32)
    w = g.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)
    n4, n6, n8 = counts
    if perm == "identity":
        p = np.arange(K, dtype=np.int32)
    elif perm == "scales":
        order = np.lexsort((g.permutation(K), -c))
        p = np.concatenate([order[BLOCK * (n8 + n6):],
                            order[BLOCK * n8: BLOCK * (n8 + n6)],
                            order[: BLOCK * n8]]).astype(np.int32)
    else:
        p = g.permutation(K).astype(np.int32)
    return LinearCase("random_%d" % seed, M, K, N, to_bf16_bits(z),
                      to_bf16_bits(w), p, widths_from_counts(n4, n6, n8),
                      {"seed": seed})


# --------------------------------------------------------------------------
# Device-side generation for the full decoder layer (M = 8192): the same
# recipe as make_linear (outlier channel scales, N(0, 0.02) weights,
# permutation from the channel ranking), with the large tensors drawn by a
# seeded torch generator on the GPU instead of numpy on the host.
# --------------------------------------------------------------------------

@dataclass
class LayerLinearSpec:
    name: str
    K: int
    N: int
    widths: np.ndarray            # uint8 [K/32]
    perm: np.ndarray              # int32 [K]
    scales: np.ndarray            # float64 [K] per-channel activation scale
    seed: int                     # torch generator seed of this linear


def layer_specs(sensitive: bool):
    """Formats of the seven linears of a LLaMA-2-70B-shaped decoder layer:
    sensitive layers use 30 % 8-bit blocks, the others 5 %, both 10 % 6-bit."""
    p8 = 0.30 if sensitive else 0.05
    out = []
    for j, (name, K, N) in enumerate(LAYER_LINEARS):
        n4, n6, n8 = width_counts(K // BLOCK, 0.10, p8)
        c = channel_scales(5, K)
        perm = permutation_from_scales(5, c, n4, n6, n8)
        out.append(LayerLinearSpec(name, K, N, widths_from_counts(n4, n6, n8), perm, c,
                                   5000 + 10 * j + (1 if sensitive else 0)))
    return out


def device_activations(spec: LayerLinearSpec, M: int, device, seed_offset: int = 0):
    """bf16 [M, K] activations z * c on the device (z ~ N(0, 1))."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(spec.seed + seed_offset)
    z = torch.randn((M, spec.K), generator=g, device=device, dtype=torch.float32)
    c = torch.from_numpy(spec.scales.astype(np.float32)).to(device)
    return (z * c[None, :]).to(torch.bfloat16)


def device_weights(spec: LayerLinearSpec, device, std: float = 0.02):
    """bf16 [N, K] weights ~ N(0, std^2) on the device."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(spec.seed + 7)
    w = torch.randn((spec.N, spec.K), generator=g, device=device, dtype=torch.float32)
    return (w * std).to(torch.bfloat16)


def device_kv(which: int, device, tokens: int = 4096, heads: int = 8, head_dim: int = 128):
    """bf16 K (which=0) or V (which=1) cache [tokens * heads, head_dim] ~ N(0, 1)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(5020 + which)
    x = torch.randn((tokens * heads, head_dim), generator=g, device=device,
                    dtype=torch.float32)
    return x.to(torch.bfloat16)


def attn_inputs(seed: int, B: int, Hq: int, Hkv: int, T: int, head_dim: int = 128,
                outlier_channels: int = 2, outlier_scale: float = 8.0):
    """Decode-attention inputs as bf16 bit patterns: q [B, Hq, head_dim] and
    the K and V caches [B * T * Hkv, head_dim] (row (b * T + t) * Hkv + h),
    all N(0, 1); K has a few channels scaled up, as keys of trained models
    show per-channel outliers."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(7000 + seed)))
    q = g.standard_normal((B, Hq, head_dim), dtype=np.float32)
    k = g.standard_normal((B * T * Hkv, head_dim), dtype=np.float32)
    v = g.standard_normal((B * T * Hkv, head_dim), dtype=np.float32)
    if outlier_channels:
        ch = g.choice(head_dim, size=outlier_channels, replace=False)
        k[:, ch] *= outlier_scale
    return to_bf16_bits(q), to_bf16_bits(k), to_bf16_bits(v)


def device_attn_inputs(B: int, Hq: int, Hkv: int, T: int, device, head_dim: int = 128,
                       outlier_scale: float = 8.0):
    """The same distribution generated on the device (bf16 tensors), for sizes
    whose host generation would dominate a benchmark."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(7100 + B * 131 + T)
    q = torch.randn((B, Hq, head_dim), generator=g, device=device, dtype=torch.float32)
    k = torch.randn((B * T * Hkv, head_dim), generator=g, device=device, dtype=torch.float32)
    v = torch.randn((B * T * Hkv, head_dim), generator=g, device=device, dtype=torch.float32)
    k[:, :2] *= outlier_scale
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)
