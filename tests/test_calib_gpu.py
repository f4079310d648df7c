"""GPU calibration against the oracle: column sensitivities bit for bit
(the same float64 order), the permutation exactly (ties and NaN included),
and a calibrated format driving the quantize + GEMM path."""
import numpy as np
import pytest
import torch

from oracle import calib
from paper_2607_17733_amd import mxq
from parity_util import say, to_dev_bf16

pytestmark = pytest.mark.gpu


def _samples(seed, n, rows, K, ld=None):
    g = np.random.Generator(np.random.PCG64(seed))
    scale = np.ones(K)
    hot = g.choice(K, size=max(1, K // 100), replace=False)
    scale[hot] = g.uniform(20, 100, size=len(hot))
    out = []
    for _ in range(n):
        a = (g.normal(size=(rows, ld or K)) * np.concatenate([scale, np.ones((ld or K) - K)]))
        bits = (a.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
        out.append(bits)
    return out


@pytest.mark.parametrize("n,rows,K,ld", [(1, 1, 32, None), (3, 37, 96, None),
                                         (4, 128, 4096, None), (2, 300, 1024, 1040),
                                         (1, 64, 28672, None)])
def test_colsq_bit_exact(n, rows, K, ld):
    say("calib-colsq", n, rows, K, ld)
    samples = _samples(rows * 7 + K, n, rows, K, ld)
    s = None
    for i, bits in enumerate(samples):
        x = to_dev_bf16(bits)[:, :K]
        s = mxq.calib_colsq(x, s, accumulate=i > 0)
    torch.cuda.synchronize()
    ref = calib.column_sensitivity([b[:, :K] for b in samples])
    assert np.array_equal(s.cpu().numpy(), ref)


@pytest.mark.parametrize("K,n6,n8", [(32, 0, 1), (256, 2, 1), (4096, 13, 1), (4096, 0, 4),
                                     (28672, 90, 1)])
def test_perm_matches_oracle(K, n6, n8):
    say("calib-perm", K, n6, n8)
    g = np.random.Generator(np.random.PCG64(K + n6))
    s = g.integers(0, max(2, K // 8), size=K).astype(np.float64)   # many ties
    if K >= 256:
        s[[5, 100]] = np.nan
        s[7] = np.inf
    perm = mxq.calib_perm(torch.from_numpy(s).cuda(), n6, n8)
    torch.cuda.synchronize()
    ref, widths = calib.allocate(s, n6, n8)
    assert np.array_equal(perm.cpu().numpy(), ref)
    assert len(widths) == K // 32


def test_calibrated_format_drives_the_path():
    say("calib-end-to-end")
    K, N, M = 1024, 256, 64
    samples = _samples(5, 2, 128, K)
    xs = [to_dev_bf16(b) for b in samples]
    R = mxq.calib_ratio([K, 4096], [0.8, 0.3], 4.5)
    perm, widths = mxq.calibrate(xs, 0.8, R)
    ref_s = calib.column_sensitivity(samples)
    n4, n6, n8 = calib.counts(K, R, 0.8)
    ref_perm, ref_widths = calib.allocate(ref_s, n6, n8)
    assert np.array_equal(perm.cpu().numpy(), ref_perm)
    assert list(widths) == ref_widths.tolist()
    # the format accepts them and the GEMM matches the oracle's
    import oracle
    g = np.random.Generator(np.random.PCG64(9))
    a = (g.normal(size=(M, K)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    w = ((g.normal(size=(N, K)) * 0.02).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    fmt = mxq.Format(K, widths, perm)
    am, ae = mxq.quantize_act(to_dev_bf16(a), fmt)
    wm, we = mxq.pack_weights(to_dev_bf16(w), fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, N).cpu().numpy()
    qa, ea = oracle.quantize(a, perm=ref_perm, widths=ref_widths)
    qw, ew = oracle.quantize(w, perm=ref_perm, widths=ref_widths)
    yref = oracle.gemm(qa, ea, qw, ew, ref_widths)
    assert np.linalg.norm(y - yref) <= 1e-5 * np.linalg.norm(yref)


@pytest.mark.parametrize("n,rows,K", [(1, 5, 64), (6, 37, 96), (16, 128, 4096)])
def test_colsq_samples_equals_per_sample_calls(n, rows, K):
    say("calib-colsq-samples", n, rows, K)
    samples = _samples(n * 31 + rows, n, rows, K)
    x = torch.stack([to_dev_bf16(b) for b in samples])
    s0 = torch.from_numpy(np.arange(K, dtype=np.float64) * 0.5).cuda()
    s = mxq.calib_colsq_samples(x, s0.clone(), accumulate=True)
    torch.cuda.synchronize()
    ref = np.arange(K, dtype=np.float64) * 0.5
    for b in samples:
        ref = ref + calib.sample_sensitivity(b)
    assert np.array_equal(s.cpu().numpy(), ref)
    s1 = mxq.calib_colsq_samples(x)
    torch.cuda.synchronize()
    assert np.array_equal(s1.cpu().numpy(), calib.column_sensitivity(samples))
