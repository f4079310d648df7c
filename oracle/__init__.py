"""Reference CPU oracle for mixed-mantissa MXINT quantization and GEMM.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and
the CPU-baseline leg of the benchmark, never by the product library.  It
shares no code with the GPU path.  The numerical work lives in plain C
(``mxq_oracle.c``, double precision, OpenMP over rows); this module builds it
with gcc and exposes numpy wrappers.  ``oracle.exact`` is a second, pure
Python implementation in exact rational arithmetic for tiny inputs.

Paper: MXSens (arXiv 2607.17733), Section 2 (MXINT: 32-element blocks sharing a
power-of-two scale, fixed-point integer elements), Section 4.1 (one mantissa
width out of {4, 6, 8} per block, or 3 in the 3-6-8 template of Section 5),
Section 5.1 (8-bit shared exponent, +0.25 bit per element).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

BLOCK = 32
ROUND_RNE, ROUND_RNA = 0, 1
CLAMP_SYMMETRIC, CLAMP_FULL = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mxq_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None
_lib_path = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (no fast-math, no intrinsics)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
             "-fno-fast-math", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def bind(path: str):
    """Bind a compiled oracle library (the default one, or a test variant)."""
    lib = ctypes.CDLL(path)
    _declare(lib)
    return lib


def use_library(path=None):
    """Route the module-level functions to another compiled oracle (tests of
    the pins compile deliberately broken variants); None restores the default."""
    global _lib, _lib_path
    _lib = None if path is None else bind(path)
    _lib_path = path


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        _lib = bind(_LIB)
    return _lib


def _declare(lib):
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    I = ctypes.c_int
    lib.oracle_quantize.argtypes = [P, I64, I64, I64, P, P, I, I, P, P]
    lib.oracle_dequantize.argtypes = [P, P, I64, I64, P, P]
    lib.oracle_block_partials.argtypes = [P, P, I64, I64, I64, P]
    lib.oracle_gemm.argtypes = [P, P, P, P, P, I64, P, I64, P, I64, P]
    lib.oracle_gemm_absbound.argtypes = [P, P, P, P, P, I64, P, I64, P, I64, P]
    lib.oracle_act_row_bytes.argtypes = [P, I64]
    lib.oracle_act_row_bytes.restype = I64
    lib.oracle_pack_act.argtypes = [P, I64, I64, P, P]
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = I
    lib.oracle_set_threads.argtypes = [I]
    lib.oracle_set_threads.restype = None
    for f in ("oracle_quantize", "oracle_dequantize", "oracle_block_partials",
              "oracle_gemm", "oracle_gemm_absbound", "oracle_pack_act"):
        getattr(lib, f).restype = I


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _widths(widths, K):
    w = np.ascontiguousarray(np.asarray(widths, dtype=np.uint8))
    if w.shape != (K // BLOCK,):
        raise ValueError("widths must have K/32 entries")
    return w


def quantize(x_bits, K=None, perm=None, widths=None, round_mode=ROUND_RNE,
             clamp_mode=CLAMP_SYMMETRIC):
    """Quantize rows of a bf16 matrix given as uint16 bit patterns [rows, ld].

    Returns (q int8 [rows, K] in permuted order, e uint8 [rows, K/32]).
    """
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    if x.ndim != 2:
        raise ValueError("x_bits must be 2-D")
    rows, ld = x.shape
    K = ld if K is None else K
    w = _widths(widths, K)
    p = None if perm is None else np.ascontiguousarray(perm, dtype=np.int32)
    q = np.empty((rows, K), np.int8)
    e = np.empty((rows, K // BLOCK), np.uint8)
    rc = _load().oracle_quantize(_ptr(x), rows, ld, K, _ptr(p), _ptr(w),
                                 round_mode, clamp_mode, _ptr(q), _ptr(e))
    if rc:
        raise ValueError("oracle_quantize rejected its arguments (%d)" % rc)
    return q, e


def dequantize(q, e, widths):
    q = np.ascontiguousarray(q, dtype=np.int8)
    e = np.ascontiguousarray(e, dtype=np.uint8)
    rows, K = q.shape
    w = _widths(widths, K)
    out = np.empty((rows, K), np.float64)
    rc = _load().oracle_dequantize(_ptr(q), _ptr(e), rows, K, _ptr(w), _ptr(out))
    if rc:
        raise ValueError("oracle_dequantize failed")
    return out


def block_partials(qa, qw):
    """P[i, j, b] = sum over block b of qa[i, k] * qw[j, k] (int32)."""
    qa = np.ascontiguousarray(qa, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    M, K = qa.shape
    N = qw.shape[0]
    P = np.empty((M, N, K // BLOCK), np.int32)
    rc = _load().oracle_block_partials(_ptr(qa), _ptr(qw), M, N, K, _ptr(P))
    if rc:
        raise ValueError("oracle_block_partials failed")
    return P


def _gemm_common(fn, qa, ea, qw, ew, widths, rows, cols):
    qa = np.ascontiguousarray(qa, dtype=np.int8)
    qw = np.ascontiguousarray(qw, dtype=np.int8)
    ea = np.ascontiguousarray(ea, dtype=np.uint8)
    ew = np.ascontiguousarray(ew, dtype=np.uint8)
    M, K = qa.shape
    N = qw.shape[0]
    w = _widths(widths, K)
    ri = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    ci = None if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
    nr = M if ri is None else len(ri)
    nc = N if ci is None else len(ci)
    Y = np.empty((nr, nc), np.float64)
    rc = fn(_ptr(qa), _ptr(ea), _ptr(qw), _ptr(ew), _ptr(w), K, _ptr(ri), nr,
            _ptr(ci), nc, _ptr(Y))
    if rc:
        raise ValueError("oracle gemm failed")
    return Y


def gemm(qa, ea, qw, ew, widths, rows=None, cols=None):
    """Blockwise MXINT GEMM in float64: Y = Ahat @ What.T (optionally a subset)."""
    return _gemm_common(_load().oracle_gemm, qa, ea, qw, ew, widths, rows, cols)


def gemm_absbound(qa, ea, qw, ew, widths, rows=None, cols=None):
    """sum_b |P_b| 2^(sa+sw): the scale of fp32 rounding in any summation order."""
    return _gemm_common(_load().oracle_gemm_absbound, qa, ea, qw, ew, widths,
                        rows, cols)


def act_row_bytes(widths):
    w = np.ascontiguousarray(np.asarray(widths, dtype=np.uint8))
    return int(_load().oracle_act_row_bytes(_ptr(w), len(w)))


def pack_act(q, widths):
    """Packed activation bytes [rows, row_bytes] in the documented layout."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    rows, K = q.shape
    w = _widths(widths, K)
    out = np.empty((rows, act_row_bytes(w)), np.uint8)
    rc = _load().oracle_pack_act(_ptr(q), rows, K, _ptr(w), _ptr(out))
    if rc:
        raise ValueError("oracle_pack_act failed")
    return out


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use."""
    return int(_load().oracle_num_threads())


def set_threads(n: int) -> None:
    """Threads for the oracle's OpenMP loops (for timing at a stated count)."""
    _load().oracle_set_threads(int(n))
