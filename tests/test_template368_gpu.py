"""GPU parity of the 3-6-8 template (3-bit blocks in place of 4-bit ones, the
paper's average-bitwidth study, Section 5) through the C ABI: the
quantizer's packed rows (3-bit blocks at 12 bytes), exponents and operand
image bit-exact against the oracle, the weight buffers (3 bits per element
under the symmetric clamp), the prefill and decode GEMMs against the oracle
GEMM, and attention over 3-bit caches."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from operand_decode import decode_act, decode_weights
from parity_util import check_gemm, say, to_dev_bf16
from test_attn_gpu import _run as attn_run

pytestmark = pytest.mark.gpu


def _case(seed, M, K, N, n3, n6, n8):
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(9000 + seed)))
    c = np.ones(K, np.float32)
    c[g.choice(K, size=max(1, K // 64), replace=False)] = g.uniform(20, 100, max(1, K // 64))
    a = W.to_bf16_bits(g.standard_normal((M, K), dtype=np.float32) * c)
    w = W.to_bf16_bits(g.standard_normal((N, K), dtype=np.float32) * 0.02)
    perm = np.argsort(-c, kind="stable")[::-1].astype(np.int32)   # large channels last (8-bit)
    widths = [3] * n3 + [6] * n6 + [8] * n8
    assert len(widths) * 32 == K
    return a, w, perm, widths


@pytest.mark.parametrize("clamp", ["sym", "full"])
@pytest.mark.parametrize("M", [1, 16, 77])
def test_quantizer_bytes(M, clamp):
    a, _, perm, widths = _case(1, M, 512, 16, 12, 2, 2)
    say("368 quantize M=%d clamp=%s" % (M, clamp))
    fmt = mxq.Format(512, widths, torch.from_numpy(perm).cuda(), clamp=clamp)
    am, ae = mxq.quantize_act(to_dev_bf16(a), fmt)
    rows, exps = mxq.quantize_rows(to_dev_bf16(a), fmt)
    torch.cuda.synchronize()
    q, e = oracle.quantize(a, perm=perm, widths=widths, clamp_mode=1 if clamp == "full" else 0)
    assert rows.shape[1] == 12 * 12 + 24 * 2 + 32 * 2        # 3 bits per 3-bit element
    assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(q, widths))
    assert np.array_equal(exps.cpu().numpy()[:, :16], e)
    qu, eu = mxq.unpack_act(rows, exps, fmt, M)
    assert np.array_equal(qu.cpu().numpy(), q) and np.array_equal(eu.cpu().numpy(), e)
    qi, ei, pad_ok = decode_act(am.cpu().numpy(), ae.cpu().numpy(), widths, M)
    assert np.array_equal(qi, q) and np.array_equal(ei, e) and pad_ok


@pytest.mark.parametrize("clamp", ["sym", "full"])
def test_weight_pack(clamp):
    _, w, perm, widths = _case(2, 4, 1024, 200, 26, 4, 2)
    fmt = mxq.Format(1024, widths, torch.from_numpy(perm).cuda(), clamp=clamp)
    wm, we = mxq.pack_weights(to_dev_bf16(w), fmt)
    qu, eu = mxq.unpack_weights(wm, we, fmt, 200)
    torch.cuda.synchronize()
    q, e = oracle.quantize(w, perm=perm, widths=widths, clamp_mode=1 if clamp == "full" else 0)
    assert np.array_equal(qu.cpu().numpy()[:200], q)
    assert np.array_equal(eu.cpu().numpy()[:200], e)
    qd, ed, ok = decode_weights(wm.cpu().numpy(), we.cpu().numpy(), widths, 200,
                                full=clamp == "full")
    assert ok and np.array_equal(qd[:200], q) and np.array_equal(ed[:200], e)
    if clamp == "sym":
        # 3-bit blocks at 3 bits per element: 26 blocks = 7 steps of 768
        # bytes per slab of 16 columns
        steps = [(7, 768), (2, 768), (1, 1024)]
        assert wm.numel() == 2 * 8 * sum(n * c for n, c in steps)


@pytest.mark.parametrize("M", [1, 4, 16, 17, 300])
def test_gemm(M):
    K, N = 2048, 384
    a, w, perm, widths = _case(3, M, K, N, 52, 8, 4)
    say("368 gemm M=%d" % M)
    fmt = mxq.Format(K, widths, torch.from_numpy(perm).cuda())
    am, ae = mxq.quantize_act(to_dev_bf16(a), fmt)
    wm, we = mxq.pack_weights(to_dev_bf16(w), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, N)
    torch.cuda.synchronize()
    qa, ea = oracle.quantize(a, perm=perm, widths=widths)
    qw, ew = oracle.quantize(w, perm=perm, widths=widths)
    ref = oracle.gemm(qa, ea, qw, ew, widths)
    check_gemm(y.cpu().numpy(), ref, qa, ea, qw, ew, widths, "3-6-8 gemm M=%d" % M)


def test_template_matches_its_definition_at_the_attention_shape():
    # the LLaMA-3-8B attention projection with the 3-6-8 template (102/13/13
    # blocks), M = 2048: sampled rows and columns against the oracle
    K = N = 4096
    a, w, perm, widths = _case(4, 2048, K, N, 102, 13, 13)
    fmt = mxq.Format(K, widths, torch.from_numpy(perm).cuda())
    am, ae = mxq.quantize_act(to_dev_bf16(a), fmt)
    wm, we = mxq.pack_weights(to_dev_bf16(w), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, 2048, N)
    torch.cuda.synchronize()
    rows = np.array([0, 31, 32, 1000, 2047])
    cols = np.array([0, 127, 128, 2049, 4095])
    qa, ea = oracle.quantize(a[rows], perm=perm, widths=widths)
    qw, ew = oracle.quantize(w[cols], perm=perm, widths=widths)
    ref = oracle.gemm(qa, ea, qw, ew, widths)
    check_gemm(y.cpu().numpy()[np.ix_(rows, cols)], ref, qa, ea, qw, ew, widths,
               "3-6-8 attention shape")


@pytest.mark.parametrize("widths", [[3, 3, 3, 3], [3, 3, 6, 8]])
def test_attention_over_three_bit_cache(widths):
    attn_run(20 + widths[2], 2, 64, 8, 600, widths)


@pytest.mark.parametrize("producer", ["rmsnorm", "swiglu"])
@pytest.mark.parametrize("M", [5, 40])
def test_fused_producers(producer, M):
    # the quantizer fused with its producers quantizes 3-bit blocks the same way
    from oracle import fused
    K, N = 1024, 96
    a, w, perm, widths = _case(5 + M, M, K, N, 26, 4, 2)
    say("368 fused %s M=%d" % (producer, M))
    g = np.random.Generator(np.random.PCG64(77 + M))
    fmt = mxq.Format(K, widths, torch.from_numpy(perm).cuda())
    if producer == "rmsnorm":
        gain = fused.f32_to_bf16(g.uniform(0.25, 2.0, size=K).astype(np.float32))
        am, ae = mxq.quantize_act_rmsnorm(to_dev_bf16(a), to_dev_bf16(gain), 1e-5, fmt)
        x = fused.rmsnorm_bf16(a, gain, 1e-5)
    else:
        gate = fused.f32_to_bf16((g.normal(size=(M, K)) * 4).astype(np.float32))
        am, ae = mxq.quantize_act_swiglu(to_dev_bf16(gate), to_dev_bf16(a), fmt)
        x = fused.swiglu_bf16(gate, a)
    wm, we = mxq.pack_weights(to_dev_bf16(w), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, N)
    torch.cuda.synchronize()
    qa, ea = oracle.quantize(x, perm=perm, widths=widths)
    qw, ew = oracle.quantize(w, perm=perm, widths=widths)
    qi, ei, pad_ok = decode_act(am.cpu().numpy(), ae.cpu().numpy(), widths, M)
    assert np.array_equal(qi, qa) and np.array_equal(ei, ea) and pad_ok
    ref = oracle.gemm(qa, ea, qw, ew, widths)
    check_gemm(y.cpu().numpy(), ref, qa, ea, qw, ew, widths, "3-6-8 fused %s" % producer)
