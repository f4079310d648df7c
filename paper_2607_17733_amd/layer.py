"""The MXINT linears of one decoder layer as one stream of device work.

MXSens (arXiv 2607.17733, Section 5 and Appendix A.2) quantizes the weights
and activations of every linear of a decoder layer (q, k, v, o, gate, up,
down) and the KV cache.  ``LayerSequence`` packs the seven weight matrices
once (offline), then ``run`` enqueues on the current stream, with no host
synchronization, the online activation quantize + GEMM of each linear and
the 4-bit quantize of the K and V caches (blocks of 32 along the head
dimension, identity permutation).  The layer's other operations
(normalization, attention, SiLU) stay in FP16 in the paper and are not part
of this path, so every linear takes its own bf16 input.
"""
from __future__ import annotations

import torch

from . import mxq


class Linear:
    """One quantized linear: its format and packed weights."""

    def __init__(self, name: str, K: int, N: int, widths, perm, w_bf16):
        self.name, self.K, self.N = name, int(K), int(N)
        self.fmt = mxq.Format(self.K, widths, perm)
        self.w_mant, self.w_exp = mxq.pack_weights(w_bf16, self.fmt)


class LayerSequence:
    def __init__(self, linears, M: int, device, kv_head_dim: int = 128):
        """linears: list of Linear (in execution order); M: tokens."""
        self.linears = list(linears)
        self.M = int(M)
        self.kv_fmt = mxq.Format(kv_head_dim, [4] * (kv_head_dim // mxq.BLOCK))
        # one activation buffer pair serves every linear: stream order keeps
        # each GEMM ahead of the next quantize that overwrites it
        ab = max(l.fmt.act_bytes(self.M) for l in self.linears)
        eb = max(l.fmt.act_exp_bytes(self.M) for l in self.linears)
        self.a_mant = torch.empty(ab, dtype=torch.uint8, device=device)
        self.a_exp = torch.empty(eb, dtype=torch.uint8, device=device)
        self.ys = [torch.empty((self.M, l.N), dtype=torch.float32, device=device)
                   for l in self.linears]
        self.kv_out = None

    def run(self, xs, kv=()):
        """xs: one bf16 [M, K] input per linear; kv: bf16 K and V caches
        [rows, head_dim].  Returns the fp32 outputs (reused buffers) and the
        quantized caches."""
        for lin, x, y in zip(self.linears, xs, self.ys):
            mxq.quantize_act(x, lin.fmt, out=(self.a_mant, self.a_exp))
            mxq.gemm(self.a_mant, self.a_exp, lin.w_mant, lin.w_exp, lin.fmt,
                     self.M, lin.N, out=y)
        if self.kv_out is None:
            rb, erb = self.kv_fmt.act_packed_bytes(), self.kv_fmt.exp_row_bytes()
            self.kv_out = [(torch.empty((t.shape[0], rb), dtype=torch.uint8, device=t.device),
                            torch.empty((t.shape[0], erb), dtype=torch.uint8, device=t.device))
                           for t in kv]
        # the caches as packed rows, the layout attention reads
        for t, out in zip(kv, self.kv_out):
            mxq.quantize_rows(t, self.kv_fmt, out=out)
        return self.ys, self.kv_out

    def ops(self) -> float:
        """Algorithmic multiply-add count (2*M*N*K summed over the linears)."""
        return float(sum(2 * self.M * l.N * l.K for l in self.linears))
