"""The quantizer fused with RMS normalisation, against the oracle chain
(normalise on the host, then quantize): every activation buffer bit for bit
(packed rows, exponents, the operand image decoded back, padding), and the
GEMM fed by it against the oracle GEMM."""
import numpy as np
import pytest
import torch

import oracle
from oracle import fused
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from parity_util import check_gemm, check_quant_act, fmt_for, say, to_dev_bf16

pytestmark = pytest.mark.gpu

SHAPES = [
    # M, K, N, (n4, n6, n8), perm, eps
    (1, 64, 32, (1, 0, 1), "random", 1e-5),
    (3, 256, 64, (6, 1, 1), "scales", 1e-6),
    (16, 1024, 128, (25, 5, 2), "random", 1e-5),
    (37, 512, 96, (12, 2, 2), "identity", 0.0),
    (300, 4096, 256, (102, 13, 13), "scales", 1e-5),
    (64, 28672, 64, (761, 90, 45), "scales", 1e-5),
]


@pytest.mark.parametrize("M,K,N,counts,perm,eps", SHAPES)
def test_fused_rmsnorm_quantize(M, K, N, counts, perm, eps):
    say("fused-rmsnorm", M, K, N, counts, perm, eps)
    case = W.random_case(M * 13 + K, M, K, N, counts, perm=perm)
    g = np.random.Generator(np.random.PCG64(K + M))
    gain = fused.f32_to_bf16(g.uniform(0.25, 2.0, size=K).astype(np.float32))
    fmt = fmt_for(case)
    am, ae = mxq.quantize_act_rmsnorm(to_dev_bf16(case.a_bits), to_dev_bf16(gain), eps, fmt)
    wm, we = mxq.pack_weights(to_dev_bf16(case.w_bits), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, N)
    torch.cuda.synchronize()
    # the oracle chain: normalise on the host, then quantize
    y_bits = fused.rmsnorm_bf16(case.a_bits, gain, eps)
    qa, ea = oracle.quantize(y_bits, perm=case.perm, widths=case.widths)
    qw, ew = oracle.quantize(case.w_bits, perm=case.perm, widths=case.widths)
    check_quant_act(case, {"a_mant": am, "a_exp": ae}, qa, ea, fmt)
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths)
    check_gemm(y.cpu().numpy(), Yref, qa, ea, qw, ew, case.widths, case.name + "-fused")


def test_fused_equals_unfused_on_device():
    say("fused-vs-unfused")
    case = W.attn_proj()
    g = np.random.Generator(np.random.PCG64(77))
    gain = fused.f32_to_bf16(g.uniform(0.5, 1.5, size=case.K).astype(np.float32))
    fmt = fmt_for(case)
    am, ae = mxq.quantize_act_rmsnorm(to_dev_bf16(case.a_bits), to_dev_bf16(gain), 1e-5, fmt)
    y_bits = fused.rmsnorm_bf16(case.a_bits[:64], gain, 1e-5)      # a sample of rows
    bm, be = mxq.quantize_act(to_dev_bf16(y_bits), fmt)
    torch.cuda.synchronize()
    # the first 64 rows are the image's first four 16-row tiles
    tb, tsc = fmt.act_bytes(16), fmt.act_exp_bytes(16)
    assert torch.equal(am[:4 * tb], bm[:4 * tb])
    assert torch.equal(ae[:4 * tsc], be[:4 * tsc])


SWIGLU_SHAPES = [
    # M, K, N, (n4, n6, n8), perm
    (1, 64, 32, (1, 0, 1), "random"),
    (5, 256, 64, (6, 1, 1), "scales"),
    (37, 1024, 96, (25, 5, 2), "identity"),
    (300, 4096, 128, (102, 13, 13), "scales"),
    (40, 28672, 64, (761, 90, 45), "random"),
]


@pytest.mark.parametrize("M,K,N,counts,perm", SWIGLU_SHAPES)
def test_fused_swiglu_quantize(M, K, N, counts, perm):
    say("fused-swiglu", M, K, N, counts, perm)
    case = W.random_case(M * 29 + K, M, K, N, counts, perm=perm)
    g = np.random.Generator(np.random.PCG64(K * 3 + M))
    gate = g.normal(size=(M, K)) * 4
    gate.flat[g.choice(M * K, size=min(64, M * K), replace=False)] = g.choice(
        [-1000.0, -150.0, -90.0, 90.0, 150.0, 1000.0], size=min(64, M * K))
    gate = fused.f32_to_bf16(gate.astype(np.float32))
    up = fused.f32_to_bf16((g.normal(size=(M, K)) * g.uniform(0.5, 20, size=K)).astype(np.float32))
    fmt = fmt_for(case)
    am, ae = mxq.quantize_act_swiglu(to_dev_bf16(gate), to_dev_bf16(up), fmt)
    wm, we = mxq.pack_weights(to_dev_bf16(case.w_bits), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, N)
    torch.cuda.synchronize()
    act = fused.swiglu_bf16(gate, up)
    qa, ea = oracle.quantize(act, perm=case.perm, widths=case.widths)
    qw, ew = oracle.quantize(case.w_bits, perm=case.perm, widths=case.widths)
    check_quant_act(case, {"a_mant": am, "a_exp": ae}, qa, ea, fmt)
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths)
    check_gemm(y.cpu().numpy(), Yref, qa, ea, qw, ew, case.widths, case.name + "-swiglu")
