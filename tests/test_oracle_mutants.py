"""Plant plausible mistakes in the oracle (on the CPU) and show that the pins
catch every one of them.

Each mutant is a textual edit of the C oracle compiled into a temporary
library; the module-level oracle functions are pointed at it, every pin is
run, and at least one must fail.  The real oracle is restored afterwards.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "mxq_oracle.c")

# (name, anchor, old, new): replace the first `old` after `anchor`.
MUTANTS = [
    ("exponent off by one", "int ex;", "int e = ex - 1;", "int e = ex;"),
    ("lsb weight", "int e = ex - 1;", "int s = e - (m - 2);", "int s = e - (m - 1);"),
    ("truncating rounding", "double v = ldexp", "nearbyint(v)", "trunc(v)"),
    ("ties-away uses ties-even", "double v = ldexp", "round(v)", "nearbyint(v)"),
    ("no upper clamp", "long qmin", "if (qi > qmax) qi = qmax;", ""),
    ("symmetric clamp ignored", "long qmax",
     "long qmin = clamp_mode == 1 ? -(1L << (m - 1)) : -qmax;",
     "long qmin = -(1L << (m - 1));"),
    ("max ignores sign", "double amax = 0.0;", "double a = fabs(x[t]);",
     "double a = x[t];"),
    ("gemm exponent sign", "int oracle_gemm(", "ldexp((double)acc, sa + sw)",
     "ldexp((double)acc, sa - sw)"),
    ("gemm drops last block", "int oracle_gemm(",
     "for (int64_t b = 0; b < nb; ++b) {\n        int EA",
     "for (int64_t b = 0; b < nb - 1; ++b) {\n        int EA"),
    ("gemm reversed weight index", "int oracle_gemm(",
     "(int64_t)qw[j * K + b * ORACLE_BLOCK + t];",
     "(int64_t)qw[j * K + b * ORACLE_BLOCK + (31 - t)];"),
    ("gemm width offset", "int oracle_gemm(",
     "int sw = EW - 127 - (widths[b] - 2);", "int sw = EW - 127 - widths[b];"),
    ("absbound drops the magnitude", "int oracle_gemm_absbound(",
     "ldexp((double)(acc < 0 ? -acc : acc), sa + sw)", "ldexp((double)acc, sa + sw)"),
    ("absbound exponent sign", "int oracle_gemm_absbound(",
     "ldexp((double)(acc < 0 ? -acc : acc), sa + sw)",
     "ldexp((double)(acc < 0 ? -acc : acc), sa - sw)"),
    ("absbound drops last block", "int oracle_gemm_absbound(",
     "for (int64_t b = 0; b < nb; ++b) {", "for (int64_t b = 0; b < nb - 1; ++b) {"),
    ("absbound width offset", "int oracle_gemm_absbound(",
     "int sw = ew[j * nb + b] - 127 - (widths[b] - 2);",
     "int sw = ew[j * nb + b] - 127 - widths[b];"),
    ("absbound doubles", "int oracle_gemm_absbound(",
     "S[a * nc + c] = s;", "S[a * nc + c] = 2.0 * s;"),
    ("partials drop an element", "int oracle_block_partials(",
     "for (int t = 0; t < ORACLE_BLOCK; ++t)", "for (int t = 1; t < ORACLE_BLOCK; ++t)"),
    ("dequantize width offset", "int oracle_dequantize(",
     "int s = E - 127 - (widths[b] - 2);", "int s = E - 127 - (widths[b] - 1);"),
    ("packed nibbles swapped", "int oracle_pack_act(",
     "(uint8_t)(lo | (hi << 4))", "(uint8_t)(hi | (lo << 4))"),
    ("6-bit top bits misplaced", "int oracle_pack_act(",
     "(h0 << 6) | (h1 << 4) | (h2 << 2) | h3", "(h0 << 6) | (h2 << 4) | (h1 << 2) | h3"),
    ("permutation ignored", "int oracle_quantize(",
     "int64_t col = perm ? perm[p] : p;", "int64_t col = p;"),
]


def _mutate(text, anchor, old, new):
    i = text.index(anchor)
    j = text.index(old, i)
    return text[:j] + new + text[j + len(old):]


@pytest.mark.parametrize("name,anchor,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, oracle_lib, name, anchor, old, new):
    src = open(SRC).read()
    mutated = _mutate(src, anchor, old, new)
    assert mutated != src
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    so = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC",
                           "-shared", "-o", str(so), str(c), "-lm"])
    failures = 0
    oracle.use_library(str(so))
    try:
        for check in pins.ALL_CHECKS:
            try:
                check()
            except (AssertionError, ValueError, IndexError):
                failures += 1
    finally:
        oracle.use_library(None)
    assert failures > 0, "no pin caught the mutant: " + name
