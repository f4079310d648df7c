"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bit-exact: the activation operand image and the weight buffers (decoded
on the host back to mantissas and scale bytes), packed activation rows,
exponents, unpacked mantissas and exponents, and the per-block int32 sums.  GEMM outputs: relative error 1e-5 (normwise) against the fp64 oracle
and, elementwise, the accumulation bound of the path that ran.  Small shapes span several tiles and ragged tails; the workload
shapes run at full size with sampled GEMM outputs.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from operand_decode import decode_act
from parity_util import (check_gemm, check_pack_w, check_quant_act, fmt_for,
                         gpu_run, oracle_quant, say, to_dev_bf16)

pytestmark = pytest.mark.gpu


def _full_check(case, round_="rne", clamp="sym", identity=False, partials=True):
    say(case.name, case.M, case.K, case.N, round_, clamp, "identity" if identity else "perm")
    fmt = fmt_for(case, round_, clamp, identity)
    out = gpu_run(case, fmt, want_partials=partials)
    qa, ea, qw, ew = oracle_quant(case, round_, clamp, identity)
    check_quant_act(case, out, qa, ea, fmt)
    check_pack_w(case, out, qw, ew, fmt)
    if partials:
        P = oracle.block_partials(qa, qw)
        assert np.array_equal(out["p"].cpu().numpy(), P), "block partial sums differ"
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths)
    check_gemm(out["y"].cpu().numpy(), Yref, qa, ea, qw, ew, case.widths, case.name)


def test_tiny_config():
    _full_check(W.tiny())


@pytest.mark.parametrize("round_", ["rne", "rna"])
@pytest.mark.parametrize("clamp", ["sym", "full"])
def test_tiny_modes(round_, clamp):
    _full_check(W.tiny(), round_, clamp)


SHAPES = [
    # M, K, N, (n4, n6, n8), perm
    (1, 32, 16, (1, 0, 0), "identity"),
    (3, 96, 40, (1, 1, 1), "random"),
    (16, 256, 256, (6, 1, 1), "scales"),
    (17, 256, 200, (4, 2, 2), "random"),
    (33, 512, 130, (8, 4, 4), "scales"),
    (48, 512, 300, (8, 4, 4), "random"),
    (64, 768, 160, (16, 4, 4), "scales"),
    (65, 256, 96, (4, 2, 2), "identity"),
    (129, 384, 129, (0, 12, 0), "random"),
    (200, 320, 300, (0, 0, 10), "identity"),
    (257, 1024, 272, (24, 5, 3), "scales"),
    (4, 640, 1000, (13, 4, 3), "scales"),
    (16, 1024, 48, (25, 6, 1), "random"),
]


@pytest.mark.parametrize("M,K,N,counts,perm", SHAPES)
def test_random_shapes(M, K, N, counts, perm):
    case = W.random_case(M * 7 + N, M, K, N, counts, perm=perm)
    _full_check(case)


# Prefill kernel variants: small grids take 128-row workgroup tiles, grids of
# at least one 256-row workgroup per CU (256 on MI355X) the 256-row tiles;
# the full clamp always takes the 256-row tiles.  Ragged M and N in each.
PREFILL_VARIANTS = [
    # M, K, N, (n4, n6, n8), perm, round, clamp
    (513, 256, 10900, (4, 2, 2), "random", "rne", "sym"),   # 3 x 86 256-row tiles
    (100, 256, 200, (4, 2, 2), "random", "rne", "full"),
    (300, 320, 150, (6, 2, 2), "scales", "rna", "full"),
    (130, 384, 140, (0, 12, 0), "identity", "rna", "sym"),
]


@pytest.mark.parametrize("M,K,N,counts,perm,round_,clamp", PREFILL_VARIANTS)
def test_prefill_variants(M, K, N, counts, perm, round_, clamp):
    case = W.random_case(M * 11 + N, M, K, N, counts, perm=perm)
    _full_check(case, round_, clamp)


def test_identity_format_matches_explicit_identity():
    case = W.random_case(5, 40, 256, 64, (5, 2, 1), perm="identity")
    _full_check(case, identity=True)


def test_out_of_range_permutation_entries_read_zero():
    case = W.random_case(9, 20, 256, 32, (6, 1, 1), perm="random")
    perm = case.perm.copy()
    perm[[3, 100, 255]] = [256, -5, 1 << 30]
    say("oor-perm")
    fmtg = mxq.Format(case.K, case.widths, torch.from_numpy(perm).cuda())
    a = to_dev_bf16(case.a_bits)
    am, ae = mxq.quantize_act(a, fmtg)
    rows, exps = mxq.quantize_rows(a, fmtg)
    torch.cuda.synchronize()
    # oracle: the same gather from a source padded with a zero column
    src = np.zeros((case.M, case.K + 32), np.uint16)
    src[:, :case.K] = case.a_bits
    p2 = perm.copy()
    p2[[3, 100, 255]] = case.K
    qa, ea = oracle.quantize(src, K=case.K, perm=p2, widths=case.widths)
    assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(qa, case.widths))
    assert np.array_equal(exps.cpu().numpy()[:, :case.K // 32], ea)
    q, E, pad_ok = decode_act(am.cpu().numpy(), ae.cpu().numpy(), case.widths, case.M)
    assert np.array_equal(q, qa) and np.array_equal(E, ea) and pad_ok


def test_long_rows_permutation_from_global_memory():
    """Rows longer than 32767 elements gather the permutation from global
    memory instead of the LDS offset table; an out-of-range entry still
    reads zero."""
    K = 33280
    case = W.random_case(31, 5, K, 16, (K // 32 - 20, 12, 8), perm="random")
    perm = case.perm.copy()
    perm[[7, 20000]] = [K + 3, -1]
    say("long-rows-perm", case.M, K)
    fmtg = mxq.Format(K, case.widths, torch.from_numpy(perm).cuda())
    a = to_dev_bf16(case.a_bits)
    am, ae = mxq.quantize_act(a, fmtg)
    rows, exps = mxq.quantize_rows(a, fmtg)
    torch.cuda.synchronize()
    src = np.zeros((case.M, K + 32), np.uint16)
    src[:, :K] = case.a_bits
    p2 = perm.copy()
    p2[[7, 20000]] = K
    qa, ea = oracle.quantize(src, K=K, perm=p2, widths=case.widths)
    assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(qa, case.widths))
    assert np.array_equal(exps.cpu().numpy()[:, :K // 32], ea)
    q, E, pad_ok = decode_act(am.cpu().numpy(), ae.cpu().numpy(), case.widths, case.M)
    assert np.array_equal(q, qa) and np.array_equal(E, ea) and pad_ok


def test_strided_inputs_and_outputs():
    case = W.random_case(12, 48, 256, 40, (6, 1, 1), perm="scales")
    say("strided")
    fmt = fmt_for(case)
    a_big = torch.zeros((48, 256 + 24), dtype=torch.bfloat16, device="cuda")
    a_big[:, :256] = to_dev_bf16(case.a_bits)
    w_big = torch.zeros((40, 256 + 8), dtype=torch.bfloat16, device="cuda")
    w_big[:, :256] = to_dev_bf16(case.w_bits)
    am, ae = mxq.quantize_act(a_big[:, :256], fmt)
    wm, we = mxq.pack_weights(w_big[:, :256], fmt)
    y_big = torch.full((48, 64), 7.0, device="cuda")
    mxq.gemm(am, ae, wm, we, fmt, 48, 40, out=y_big[:, :40])
    torch.cuda.synchronize()
    qa, ea, qw, ew = oracle_quant(case)
    rows, _ = mxq.quantize_rows(a_big[:, :256], fmt)
    assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(qa, case.widths))
    q, _, _ = decode_act(am.cpu().numpy(), ae.cpu().numpy(), case.widths, 48)
    assert np.array_equal(q, qa)
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths)
    yb = y_big.cpu().numpy()
    check_gemm(yb[:, :40], Yref, qa, ea, qw, ew, case.widths, "strided")
    assert np.all(yb[:, 40:] == 7.0)          # nothing outside N written


def test_special_values():
    """Zero rows, subnormals, huge values, Inf and NaN blocks."""
    g = np.random.default_rng(3)
    M, K, N = 80, 128, 32                           # M > 64: the prefill kernel
    a = g.standard_normal((M, K)).astype(np.float32)
    a[0] = 0.0                                      # zero row
    a[1] = g.standard_normal(K) * 1e-39             # subnormal values
    a[2] = g.standard_normal(K) * 1e37              # near the top of the range
    a[3, 5] = np.inf                                # Inf in block 0
    a[4, 70] = np.nan                               # NaN in block 2
    a[5, :32] = 2.0 ** -130                         # subnormal-only block
    w = (g.standard_normal((N, K)) * 0.02).astype(np.float32)
    case = W.LinearCase("special", M, K, N, W.to_bf16_bits(a), W.to_bf16_bits(w),
                        np.arange(K, dtype=np.int32), np.array([4, 4, 6, 8], np.uint8))
    for rows_m in (M, 16):                           # prefill and decode kernels
        c2 = W.LinearCase(case.name, rows_m, K, N, case.a_bits[:rows_m], case.w_bits,
                          case.perm, case.widths)
        _full_check(c2, identity=True)


def _spread_case(seed, M, K, N, counts, spread=15):
    """Every (row, block) of A and every (column, block) of W scaled by its
    own 2^u, u uniform in [-spread, spread]: block exponents within one
    matrix-core step differ by up to 2 * spread."""
    g = np.random.default_rng(seed)
    nb = K // 32
    a = g.standard_normal((M, K)) * np.repeat(np.exp2(g.integers(-spread, spread + 1, (M, nb))),
                                               32, axis=1)
    w = 0.02 * g.standard_normal((N, K)) * np.repeat(
        np.exp2(g.integers(-spread, spread + 1, (N, nb))), 32, axis=1)
    return W.LinearCase("spread%d" % seed, M, K, N, W.to_bf16_bits(a.astype(np.float32)),
                        W.to_bf16_bits(w.astype(np.float32)), np.arange(K, dtype=np.int32),
                        W.widths_from_counts(*counts))


@pytest.mark.parametrize("M", [8, 40, 100])             # decode, decode, prefill
def test_wide_exponent_spread(M):
    """Adversarial accumulation case: block exponents spread over 30 binades
    inside every matrix-core step.  Bit-exact operands as everywhere; the
    GEMM must meet both the derived accumulation bound and the 1e-5
    elementwise gate."""
    case = _spread_case(100 + M, M, 512, 96, (8, 4, 4))
    say(case.name, M, case.K, case.N, "exponent spread +-15")
    fmt = fmt_for(case, identity=True)
    out = gpu_run(case, fmt, want_partials=True)
    qa, ea, qw, ew = oracle_quant(case, identity=True)
    check_quant_act(case, out, qa, ea, fmt)
    check_pack_w(case, out, qw, ew, fmt)
    assert np.array_equal(out["p"].cpu().numpy(), oracle.block_partials(qa, qw))
    assert (ea.max(axis=1).astype(int) - ea.min(axis=1)).min() >= 20
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths)
    check_gemm(out["y"].cpu().numpy(), Yref, qa, ea, qw, ew, case.widths, case.name)


def test_deterministic_repeat():
    case = W.random_case(77, 300, 1024, 260, (24, 4, 4), perm="scales")
    say("determinism")
    fmt = fmt_for(case)
    o1 = gpu_run(case, fmt)
    o2 = gpu_run(case, fmt)
    assert torch.equal(o1["y"], o2["y"])
    assert torch.equal(o1["w_mant"], o2["w_mant"])


# ---------------------------------------------------------------------------
# Workload shapes at full size; GEMM outputs sampled.
# ---------------------------------------------------------------------------

def _sampled_check(case, n_rows=12, n_cols=384, seed=0):
    say(case.name, case.M, case.K, case.N)
    fmt = fmt_for(case)
    out = gpu_run(case, fmt)
    qa, ea, qw, ew = oracle_quant(case)
    check_quant_act(case, out, qa, ea, fmt)
    check_pack_w(case, out, qw, ew, fmt)
    g = np.random.default_rng(seed)
    rows = np.unique(np.concatenate([[0, case.M - 1],
                                     g.choice(case.M, min(n_rows, case.M), replace=False)]))
    cols = np.unique(np.concatenate([[0, case.N - 1],
                                     g.choice(case.N, min(n_cols, case.N), replace=False)]))
    Yref = oracle.gemm(qa, ea, qw, ew, case.widths, rows=rows, cols=cols)
    Y = out["y"].cpu().numpy()[np.ix_(rows, cols)]
    return check_gemm(Y, Yref, qa, ea, qw, ew, case.widths, case.name, rows=rows, cols=cols)


def test_attn_proj_full():
    _sampled_check(W.attn_proj())


def test_mlp_gate_up_full():
    _sampled_check(W.mlp_gate_up())


def test_mlp_down_full():
    _sampled_check(W.mlp_down())


@pytest.mark.parametrize("which", ["up", "down"])
def test_decode_full(which):
    """LLaMA-2-70B decode shapes, M in {1, 4, 16, 40, 64} (one to four
    16-row activation tiles per weight read); the packed weights are checked
    once, the GEMM at every M."""
    base = W.decode(64, which)
    say(base.name, base.K, base.N)
    fmt = fmt_for(base)
    w = to_dev_bf16(base.w_bits)
    wm, we = mxq.pack_weights(w, fmt)
    qw, ew = oracle.quantize(base.w_bits, perm=base.perm, widths=base.widths)
    check_pack_w(base, {"w_mant": wm, "w_exp": we}, qw, ew, fmt)
    g = np.random.default_rng(1)
    cols = np.unique(np.concatenate([[0, base.N - 1], g.choice(base.N, 2048, replace=False)]))
    for M in (1, 4, 16, 40, 64):
        say(base.name, "M=%d" % M)
        a_bits = base.a_bits[:M]
        am, ae = mxq.quantize_act(to_dev_bf16(a_bits), fmt)
        y = mxq.gemm(am, ae, wm, we, fmt, M, base.N)
        torch.cuda.synchronize()
        qa, ea = oracle.quantize(a_bits, perm=base.perm, widths=base.widths)
        Yref = oracle.gemm(qa, ea, qw, ew, base.widths, cols=cols)
        check_gemm(y.cpu().numpy()[:, cols], Yref, qa, ea, qw, ew, base.widths,
                   "decode M=%d" % M, cols=cols)


# Decode with one unit of 5, 6 or 7 slabs per CU (the slab count of N comes
# to 5-7 per CU on a 256-CU device): units cross from one 128-column
# super-slab into the next; ragged N leaves dead slabs in the last unit.
DECODE_UNIT_PER_CU = [
    # M, K, N, (n4, n6, n8)
    (1, 256, 28632, (4, 2, 2)),      # 7 slabs per CU, last slab ragged
    (16, 256, 25000, (4, 2, 2)),     # 7 slabs per CU, last unit short
    (7, 320, 24000, (6, 2, 2)),      # 6 slabs per CU
    (3, 256, 17000, (4, 2, 2)),      # 5 slabs per CU
]


@pytest.mark.parametrize("M,K,N,counts", DECODE_UNIT_PER_CU)
def test_decode_units_across_superslabs(M, K, N, counts):
    case = W.random_case(M * 13 + N, M, K, N, counts, perm="random")
    _full_check(case, partials=False)


def test_decode_units_across_superslabs_full_clamp():
    """The full clamp's weight records (two's complement 8-bit digits, the
    4-bit record's extra plane) through units that cross super-slabs."""
    case = W.random_case(77, 9, 384, 27000, (6, 3, 3), perm="scales")
    _full_check(case, "rna", "full", partials=False)


def test_kv_cache_quantize():
    """4-bit MXINT along the head dimension for a 4096-token, 8-head cache."""
    for which in (0, 1):
        bits = W.kv_cache(which)
        say("kv", which, bits.shape)
        fmt = mxq.Format(128, [4, 4, 4, 4])
        rows, exps = mxq.quantize_rows(to_dev_bf16(bits), fmt)
        torch.cuda.synchronize()
        q, e = oracle.quantize(bits, widths=[4, 4, 4, 4])
        assert np.array_equal(rows.cpu().numpy(), oracle.pack_act(q, [4, 4, 4, 4]))
        assert np.array_equal(exps.cpu().numpy()[:, :4], e)
