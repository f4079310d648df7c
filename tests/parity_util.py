"""Shared helpers of the GPU parity tests: run a LinearCase through the C ABI
(via the Python binding) and through the CPU oracle, and compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd.workloads import LinearCase

BLOCK = 32


def say(*args):
    print("[case]", *args, flush=True)
    sys.stdout.flush()


def to_dev_bf16(bits: np.ndarray, dev="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(dev).view(torch.bfloat16)


def fmt_for(case: LinearCase, round_="rne", clamp="sym", identity=False):
    perm = None if identity else torch.from_numpy(case.perm).to("cuda")
    return mxq.Format(case.K, case.widths, perm, round=round_, clamp=clamp)


def oracle_quant(case: LinearCase, round_="rne", clamp="sym", identity=False):
    rm = 1 if round_ == "rna" else 0
    cm = 1 if clamp == "full" else 0
    perm = None if identity else case.perm
    qa, ea = oracle.quantize(case.a_bits, perm=perm, widths=case.widths,
                             round_mode=rm, clamp_mode=cm)
    qw, ew = oracle.quantize(case.w_bits, perm=perm, widths=case.widths,
                             round_mode=rm, clamp_mode=cm)
    return qa, ea, qw, ew


def gpu_run(case: LinearCase, fmt, want_partials=False, M=None):
    """Quantize A, pack W and run the GEMM on the GPU; return host arrays."""
    a = to_dev_bf16(case.a_bits)
    w = to_dev_bf16(case.w_bits)
    M = case.M if M is None else M
    am, ae = mxq.quantize_act(a, fmt)
    wm, we = mxq.pack_weights(w, fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, case.N)
    out = {"a_mant": am, "a_exp": ae, "w_mant": wm, "w_exp": we, "y": y}
    if want_partials:
        out["p"] = mxq.gemm_partials(am, ae, wm, we, fmt, M, case.N)
    torch.cuda.synchronize()
    return out


def check_y(Y, Yref, S, nb, what=""):
    """The GEMM tolerance: relative error 1e-5 against the fp64 oracle,
    normwise and elementwise (with a small absolute floor for outputs that
    cancel), plus a hard bound from fp32 summation of the block terms."""
    Y = Y.astype(np.float64)
    assert Y.shape == Yref.shape
    nan_ref = np.isnan(Yref)
    assert np.array_equal(np.isnan(Y), nan_ref), what + ": NaN pattern differs"
    Y, Yref, S = Y[~nan_ref], Yref[~nan_ref], S[~nan_ref]
    if Yref.size == 0:
        return
    err = np.abs(Y - Yref)
    ref_inf = np.abs(Yref).max()
    normwise = np.linalg.norm(Y - Yref) / max(np.linalg.norm(Yref), 1e-300)
    assert normwise <= 1e-5, "%s: normwise %.3g" % (what, normwise)
    assert np.all(err <= 1e-5 * np.abs(Yref) + 1e-7 * ref_inf), \
        "%s: elementwise max rel %.3g" % (what, (err / np.maximum(np.abs(Yref), 1e-300)).max())
    # fp32 accumulation of nb exact block terms, any order; 2^-126 covers
    # terms below fp32's normal range
    bound = (nb + 2) * 2.0 ** -24 * S + nb * 2.0 ** -126
    assert np.all(err <= bound), "%s: exceeds fp32 summation bound" % what
    return normwise


def operand_order(widths):
    """Position of each element of a row inside the operand image."""
    pos = []
    for b, m in enumerate(widths):
        for t in range(BLOCK):
            if m == 8:
                pos.append(32 * b + t)
            else:
                pos.append(32 * b + 8 * (t // 8) + (t % 8) // 2 + 4 * (t % 2))
    return np.array(pos)


def check_operand_image(am, ae, qa, ea, widths, canon, erb):
    """The quantizer's matrix-core operand image: every element equals
    q * 2^(8 - m - (ref - E)) exactly, 0 <= ref - E <= 8 - m, and the
    reference is shared over each 16-block chunk whose exponent spread fits
    8 - m (else ref = E)."""
    nb = len(widths)
    K = nb * BLOCK
    op = am[:, canon:canon + K].view(np.int8).astype(np.int64)
    ref = ae[:, erb:erb + nb].astype(np.int64)
    E = ea.astype(np.int64)
    m = np.asarray(widths, dtype=np.int64)
    sh = ref - E
    assert np.all(sh >= 0) and np.all(sh <= 8 - m[None, :]), "reference out of range"
    mult = np.repeat(8 - m[None, :] - sh, BLOCK, axis=1)
    want = qa.astype(np.int64) * (1 << mult)
    got = op[:, operand_order(widths)]
    assert np.array_equal(got, want), "operand image differs"
    # chunk rule
    start = 0
    for w in (4, 6, 8):
        n = int((m == w).sum())
        for c0 in range(0, n, 16):
            sl = slice(start + c0, start + min(n, c0 + 16))
            spread = E[:, sl].max(axis=1) - E[:, sl].min(axis=1)
            shared = spread <= 8 - w
            assert np.all(ref[shared, sl] == E[shared, sl].max(axis=1)[:, None])
            assert np.all(ref[~shared, sl] == E[~shared, sl])
        start += n
    assert not ae[:, erb + nb:].any()


def check_quant_act(case, out, qa, ea, fmt):
    am = out["a_mant"].cpu().numpy()
    ae = out["a_exp"].cpu().numpy()
    nb = case.K // BLOCK
    canon = fmt.act_packed_bytes()
    erb = fmt.exp_row_bytes() // 2
    ref_bytes = oracle.pack_act(qa, case.widths)
    assert am.shape == (case.M, canon + case.K) and ref_bytes.shape == (case.M, canon)
    assert np.array_equal(am[:, :canon], ref_bytes), "packed activation bytes differ"
    assert np.array_equal(ae[:, :nb], ea), "activation exponents differ"
    assert not ae[:, nb:erb].any()
    check_operand_image(am, ae, qa, ea, case.widths, canon, erb)
    q, e = mxq.unpack_act(out["a_mant"], out["a_exp"], fmt, case.M)
    assert np.array_equal(q.cpu().numpy(), qa) and np.array_equal(e.cpu().numpy(), ea)


def check_pack_w(case, out, qw, ew, fmt):
    q, e = mxq.unpack_weights(out["w_mant"], out["w_exp"], fmt, case.N)
    assert np.array_equal(q.cpu().numpy(), qw), "weight mantissas differ"
    assert np.array_equal(e.cpu().numpy(), ew), "weight exponents differ"
