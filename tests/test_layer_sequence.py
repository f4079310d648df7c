"""The config-5 decoder layer (LLaMA-2-70B shapes, M = 8192 tokens): seven
quantize + GEMM pairs and the 4-bit K/V cache quantize, enqueued on one
stream with no host synchronization, checked against the oracle on sampled
output rows and columns of every linear and on every cache row."""
import numpy as np
import pytest
import torch

import oracle
from parity_util import check_gemm, say
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from paper_2607_17733_amd.layer import LayerSequence, Linear

M = 8192


def _bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.gpu
@pytest.mark.parametrize("sensitive", [True, False], ids=["sensitive", "insensitive"])
def test_layer_sequence(sensitive):
    dev = "cuda"
    specs = W.layer_specs(sensitive)
    linears, xs, ws = [], [], []
    for s in specs:
        say("layer", "sensitive" if sensitive else "insensitive", s.name, s.K, s.N,
            np.bincount(s.widths, minlength=9)[[4, 6, 8]].tolist())
        w = W.device_weights(s, dev)
        linears.append(Linear(s.name, s.K, s.N, s.widths,
                              torch.from_numpy(s.perm).to(dev), w))
        ws.append(w)
        xs.append(W.device_activations(s, M, dev))
    kv = [W.device_kv(0, dev), W.device_kv(1, dev)]
    seq = LayerSequence(linears, M, dev)
    ys, kvq = seq.run(xs, kv)
    torch.cuda.synchronize()

    g = np.random.Generator(np.random.PCG64(77 + int(sensitive)))
    rows = np.array([0, 4097, M - 1])
    for s, x, w, y in zip(specs, xs, ws, ys):
        cols = np.arange(s.N) if s.N <= 8192 else np.sort(g.choice(s.N, 2048, replace=False))
        say("check", s.name, "rows", rows.tolist(), "cols", len(cols))
        qa, ea = oracle.quantize(_bits(x[torch.from_numpy(rows).to(dev)]), perm=s.perm,
                                 widths=s.widths)
        qw, ew = oracle.quantize(_bits(w[torch.from_numpy(cols).to(dev)]), perm=s.perm,
                                 widths=s.widths)
        Yref = oracle.gemm(qa, ea, qw, ew, s.widths)
        got = y[torch.from_numpy(rows).to(dev)][:, torch.from_numpy(cols).to(dev)]
        check_gemm(got.cpu().numpy(), Yref, qa, ea, qw, ew, s.widths, s.name)

    widths = [4, 4, 4, 4]
    for t, (rows, exps) in zip(kv, kvq):
        q, e = oracle.quantize(_bits(t), widths=widths)
        assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(q, widths))
        assert np.array_equal(exps.cpu().numpy()[:, :4], e)
