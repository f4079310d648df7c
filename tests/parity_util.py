"""Shared helpers of the GPU parity tests: run a LinearCase through the C ABI
(via the Python binding) and through the CPU oracle, and compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from operand_decode import Geo, decode_act, decode_weights
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
    """Quantize A (operand image and packed rows), pack W and run the GEMM
    on the GPU; return the device buffers."""
    a = to_dev_bf16(case.a_bits)
    w = to_dev_bf16(case.w_bits)
    M = case.M if M is None else M
    am, ae = mxq.quantize_act(a, fmt)
    rows, exps = mxq.quantize_rows(a, fmt)
    wm, we = mxq.pack_weights(w, fmt)
    y = mxq.gemm(am, ae, wm, we, fmt, M, case.N)
    out = {"a_mant": am, "a_exp": ae, "rows": rows, "exps": exps, "w_mant": wm, "w_exp": we,
           "y": y}
    if want_partials:
        out["p"] = mxq.gemm_partials(rows, exps, wm, we, fmt, M, case.N)
    torch.cuda.synchronize()
    return out


def digit_absbound(qa, ea, qw, ew, widths, rows=None, cols=None):
    """T[i, j] = sum_k (|qa|+c)(|qw|+c) 2^(Ea+Ew-254-2(m-2)), an upper bound of
    the sum of |digit products| the matrix core accumulates for Y[i, j]: an
    m-bit mantissa q splits into digits with |8h| + |l| <= |q| + 14 (m = 6)
    and |16h| + |l| <= |q| + 30 (m = 8); 3- and 4-bit mantissas are not
    split."""
    wb = np.asarray(widths)
    c = np.repeat(np.select([wb <= 4, wb == 6], [0, 14], 30), BLOCK).astype(np.float64)
    off = 127 + (wb - 2)
    rows = np.arange(qa.shape[0]) if rows is None else np.asarray(rows)
    cols = np.arange(qw.shape[0]) if cols is None else np.asarray(cols)
    sa = np.repeat(np.clip(ea[rows].astype(np.float64), 0, 254) - off, BLOCK, axis=1)
    sw = np.repeat(np.clip(ew[cols].astype(np.float64), 0, 254) - off, BLOCK, axis=1)
    A = (np.abs(qa[rows].astype(np.float64)) + c) * np.exp2(sa)
    Wm = (np.abs(qw[cols].astype(np.float64)) + c) * np.exp2(sw)
    return A @ Wm.T


def mma_steps(widths):
    """Matrix-core instructions accumulated into each output, the larger of
    the two GEMMs' counts: the prefill kernel's 64-K instructions, two per
    3/4-bit step (four blocks) and four per 6/8-bit step (two blocks, two
    digit planes)."""
    g = Geo(widths)
    return 2 * (g.S[0] + g.S[1]) + 4 * (g.S[2] + g.S[3])


def a14_ratio(Y, Yref):
    """Worst ratio of |Y - Y_ref| to the elementwise gate 1e-5 |Y_ref| +
    1e-7 max|Y_ref| (allclose-style, the second term covering outputs that
    cancel to near zero); <= 1 passes."""
    Y = np.asarray(Y, np.float64)
    Yref = np.asarray(Yref, np.float64)
    keep = ~np.isnan(Yref)
    if not keep.any():
        return 0.0
    err = np.abs(Y[keep] - Yref[keep])
    gate = 1e-5 * np.abs(Yref[keep]) + 1e-7 * np.abs(Yref[keep]).max()
    return float((err / np.maximum(gate, 1e-300)).max())


def check_y(Y, Yref, S, nb, what="", T=None, steps=0, a14=True):
    """The GEMM tolerance against the fp64 oracle:
      - normwise relative error <= 1e-5;
      - elementwise, the gate |Y - Y_ref| <= 1e-5 |Y_ref| + 1e-7 max|Y_ref|
        (enforced unless a14=False, which only the deliberately adversarial
        exponent-spread case uses; its ratio is always reported);
      - elementwise, a bound derived from the arithmetic, always enforced:
          decode path (exact int32 block sums, one fp32 rescale-add each):
            (nb + 2) 2^-24 S with S = sum_b |P_b| 2^(sa+sw);
          prefill path (exact digit products, fp32 accumulation inside each
            matrix-core instruction): 2 * steps * 2^-24 * T, T from
            digit_absbound, i.e. at most two roundings of the running
            absolute sum per instruction;
        plus nb 2^-126 for terms below fp32's normal range."""
    Y = Y.astype(np.float64)
    assert Y.shape == Yref.shape
    nan_ref = np.isnan(Yref)
    assert np.array_equal(np.isnan(Y), nan_ref), what + ": NaN pattern differs"
    keep = ~nan_ref
    Y, Yref, S = Y[keep], Yref[keep], S[keep]
    if Yref.size == 0:
        return
    err = np.abs(Y - Yref)
    normwise = np.linalg.norm(Y - Yref) / max(np.linalg.norm(Yref), 1e-300)
    assert normwise <= 1e-5, "%s: normwise %.3g" % (what, normwise)
    bound = (nb + 2) * 2.0 ** -24 * S + nb * 2.0 ** -126
    if T is not None:
        bound = np.maximum(bound, 2 * steps * 2.0 ** -24 * T[keep] + nb * 2.0 ** -126)
    worst = (err / bound).max()
    assert np.all(err <= bound), "%s: exceeds the accumulation bound (x%.3g)" % (what, worst)
    gate = a14_ratio(Y, Yref)
    say("%s: normwise %.3g, elementwise gate ratio %.3g, derived-bound ratio %.3g"
        % (what, normwise, gate, worst))
    if a14:
        assert gate <= 1.0, "%s: elementwise 1e-5 gate exceeded (x%.3g)" % (what, gate)
    return normwise


def check_gemm(Y, Yref, qa, ea, qw, ew, widths, what, rows=None, cols=None, a14=True):
    """check_y with both accumulation bounds computed from the oracle's
    mantissas and exponents."""
    S = oracle.gemm_absbound(qa, ea, qw, ew, widths, rows=rows, cols=cols)
    T = digit_absbound(qa, ea, qw, ew, widths, rows=rows, cols=cols)
    return check_y(Y, Yref, S, len(widths), what, T=T, steps=mma_steps(widths), a14=a14)


def check_quant_act(case, out, qa, ea, fmt):
    """Bit-exact activation buffers: the operand image decoded on the host
    back to mantissas and scale bytes (zero padding included) and, when
    `out` holds them, the packed rows against the oracle's packing, the
    exponent rows, and mxq_unpack_act."""
    M = case.M
    am = out["a_mant"].cpu().numpy()
    ae = out["a_exp"].cpu().numpy()
    nb = case.K // BLOCK
    assert am.size == fmt.act_bytes(M) and ae.size == fmt.act_exp_bytes(M)
    q, E, pad_ok = decode_act(am, ae, case.widths, M)
    assert np.array_equal(q, qa), "activation operand image differs from the mantissas"
    assert np.array_equal(E, ea.astype(np.int64)), "activation scale bytes differ"
    assert pad_ok, "activation operand padding not zero"
    if "rows" not in out:
        return
    rows = out["rows"].cpu().numpy()
    exps = out["exps"].cpu().numpy()
    assert rows.shape == (M, fmt.act_packed_bytes())
    assert np.array_equal(rows, oracle.pack_act(qa, case.widths)), "packed activation rows differ"
    assert np.array_equal(exps[:, :nb], ea), "activation exponents differ"
    assert not exps[:, nb:].any()
    qd, ed = mxq.unpack_act(out["rows"], out["exps"], fmt, M)
    assert np.array_equal(qd.cpu().numpy(), qa) and np.array_equal(ed.cpu().numpy(), ea)


def check_pack_w(case, out, qw, ew, fmt):
    """Bit-exact weight buffers: mxq_unpack_weights, and the host decoder of
    the documented layout (padding columns and zero blocks included)."""
    N = qw.shape[0]
    q, e = mxq.unpack_weights(out["w_mant"], out["w_exp"], fmt, N)
    assert np.array_equal(q.cpu().numpy(), qw), "weight mantissas differ"
    assert np.array_equal(e.cpu().numpy(), ew), "weight exponents differ"
    qo, eo, ok = decode_weights(out["w_mant"].cpu().numpy(), out["w_exp"].cpu().numpy(),
                                case.widths, N, full=fmt.clamp == 1)
    assert ok, "weight layout / padding"
    assert np.array_equal(qo[:N], qw), "weight buffer differs from the mantissas"
    assert np.array_equal(eo[:N], ew.astype(np.int64)), "weight scale bytes differ"
