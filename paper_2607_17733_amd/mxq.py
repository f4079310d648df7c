"""Python binding of libmxq (include/mxq.h): argument marshalling only.

Every step of the quantize / pack / GEMM path runs in the HIP kernels of
``libmxq.so``; torch provides device memory and the current stream.  There
is no fallback: if the library is missing the calls raise ``MxqError``.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmxq.so")
BLOCK = 32
DECODE_MAX_M = 64


class MxqError(RuntimeError):
    pass


class _Fmt(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int64), ("block", ctypes.c_int32),
                ("round", ctypes.c_int32), ("clamp", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("widths", ctypes.c_void_p),
                ("perm", ctypes.c_void_p)]


_lib = None

# name -> (restype, argtypes)
_P, _I64 = ctypes.c_void_p, ctypes.c_int64
_SIGS = {
    "mxq_abi_version": (ctypes.c_int, []),
    "mxq_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "mxq_act_packed_bytes": (_I64, [_P]),
    "mxq_exp_row_bytes": (_I64, [_P]),
    "mxq_act_bytes": (_I64, [_P, _I64]),
    "mxq_act_exp_bytes": (_I64, [_P, _I64]),
    "mxq_weight_bytes": (_I64, [_P, _I64]),
    "mxq_weight_exp_bytes": (_I64, [_P, _I64]),
    "mxq_quantize_act": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P]),
    "mxq_quantize_rows": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P]),
    "mxq_quantize_act_rmsnorm": (ctypes.c_int, [_P, _P, _I64, _I64, _P, ctypes.c_float,
                                                 _P, _P, _P]),
    "mxq_quantize_act_swiglu": (ctypes.c_int, [_P, _P, _P, _I64, _I64, _P, _P, _P]),
    "mxq_pack_weights": (ctypes.c_int, [_P, _P, _I64, _I64, _P, _P, _P]),
    "mxq_gemm": (ctypes.c_int, [_P, _I64, _I64, _P, _P, _P, _P, _P, _I64, _P]),
    "mxq_gemm_partials": (ctypes.c_int, [_P, _I64, _I64, _P, _P, _P, _P, _P, _P]),
    "mxq_unpack_act": (ctypes.c_int, [_P, _I64, _P, _P, _P, _P, _P]),
    "mxq_unpack_weights": (ctypes.c_int, [_P, _I64, _P, _P, _P, _P, _P]),
    "mxq_calib_colsq": (ctypes.c_int, [_P, _I64, _I64, _I64, _P, ctypes.c_int, _P]),
    "mxq_calib_colsq_samples": (ctypes.c_int, [_P, _I64, _I64, _I64, _I64, _I64, _P, _P,
                                               ctypes.c_int, _P]),
    "mxq_calib_ratio": (ctypes.c_int, [ctypes.c_int32, _P, _P, ctypes.c_double, _P]),
    "mxq_calib_counts": (ctypes.c_int, [_I64, ctypes.c_double, ctypes.c_double,
                                        ctypes.c_int32, _P, _P, _P]),
    "mxq_calib_perm": (ctypes.c_int, [_P, _I64, ctypes.c_int32, ctypes.c_int32, _P, _P]),
    "mxq_peak_sink_words": (_I64, []),
    "mxq_peak_stream_read": (ctypes.c_int, [_P, _I64, _P, _P]),
    "mxq_peak_mfma": (ctypes.c_int, [ctypes.c_int, _I64, _P, _P, _P]),
    "mxq_attn_work_bytes": (_I64, [_P, _I64, _I64, _I64, _I64]),
    "mxq_attn_decode": (ctypes.c_int, [_P, _P, _I64, _I64, _I64, _I64, ctypes.c_float,
                                       _P, _P, _P, _P, _P, _P, _I64, _P]),
    "mxq_attn_decode_static": (ctypes.c_int, [_P, _P, _I64, _I64, _I64, _I64, ctypes.c_float,
                                              _P, _P, _P, _P, _P, _P]),
}


def lib(path: str = LIB_PATH):
    """Load libmxq.so (once).  Raises MxqError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise MxqError("libmxq.so is not built (%s); run __graft_entry__.build()"
                           % path)
        handle = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(status: int, what: str):
    if status != 0:
        msg = lib().mxq_status_str(status).decode()
        raise MxqError("%s failed: %s (status %d)" % (what, msg, status))


def _size(v: int, what: str) -> int:
    if v < 0:
        _check(int(-v), what)
    return int(v)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


class Format:
    """Width map + permutation of one quantized linear (include/mxq.h mxq_fmt).

    widths: K/32 entries in {3, 4, 6, 8}, non-decreasing (3-bit blocks are
            the floor of the 3-6-8 template).
    perm:   None (identity) or an int32 device tensor of K source columns.
    """

    def __init__(self, K: int, widths, perm=None, round: str = "rne",
                 clamp: str = "sym"):
        self.K = int(K)
        self.widths = np.ascontiguousarray(np.asarray(widths, dtype=np.uint8))
        if perm is not None:
            if not (isinstance(perm, torch.Tensor) and perm.is_cuda
                    and perm.dtype == torch.int32 and perm.is_contiguous()):
                raise MxqError("perm must be a contiguous int32 device tensor")
        self.perm = perm
        self.round = {"rne": 0, "rna": 1}[round]
        self.clamp = {"sym": 0, "full": 1}[clamp]
        self._c = _Fmt(self.K, BLOCK, self.round, self.clamp, 0,
                       self.widths.ctypes.data_as(ctypes.c_void_p).value,
                       None if perm is None else perm.data_ptr())

    @property
    def ref(self):
        return ctypes.byref(self._c)

    @property
    def nb(self) -> int:
        return self.K // BLOCK

    def act_packed_bytes(self) -> int:
        """Bytes of one packed activation row."""
        return _size(lib().mxq_act_packed_bytes(self.ref), "mxq_act_packed_bytes")

    def exp_row_bytes(self) -> int:
        """Bytes of one row of block exponents."""
        return _size(lib().mxq_exp_row_bytes(self.ref), "mxq_exp_row_bytes")

    def act_bytes(self, M: int) -> int:
        """The activation operand image of M rows (mxq_quantize_act)."""
        return _size(lib().mxq_act_bytes(self.ref, M), "mxq_act_bytes")

    def act_exp_bytes(self, M: int) -> int:
        """Its scale bytes."""
        return _size(lib().mxq_act_exp_bytes(self.ref, M), "mxq_act_exp_bytes")

    def weight_bytes(self, N: int) -> int:
        return _size(lib().mxq_weight_bytes(self.ref, N), "mxq_weight_bytes")

    def weight_exp_bytes(self, N: int) -> int:
        return _size(lib().mxq_weight_exp_bytes(self.ref, N), "mxq_weight_exp_bytes")


def _bf16_2d(t, K, what):
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.bfloat16
            and t.dim() == 2 and t.stride(1) == 1):
        raise MxqError("%s must be a 2-D bf16 device tensor with unit column stride"
                       % what)
    if t.shape[1] < K:
        raise MxqError("%s has fewer than K columns" % what)
    return t


def _dev_bytes(t, n: int, what: str, dev=None):
    """A contiguous uint8 device tensor of at least n bytes (on `dev`)."""
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == torch.uint8
            and t.is_contiguous()):
        raise MxqError("%s must be a contiguous uint8 device tensor" % what)
    if t.numel() < n:
        raise MxqError("%s holds %d bytes, %d needed" % (what, t.numel(), n))
    if dev is not None and t.device != dev:
        raise MxqError("%s is on %s, not %s" % (what, t.device, dev))
    return t


def _act_out(out, fmt: Format, M: int, dev):
    """The caller's (mant, exp) activation buffers, checked, or new ones."""
    if out is None:
        return (torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev),
                torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev))
    mant, exp = out
    _dev_bytes(mant, fmt.act_bytes(M), "activation mantissa buffer", dev)
    _dev_bytes(exp, fmt.act_exp_bytes(M), "activation exponent buffer", dev)
    return mant, exp


def _gemm_operands(a_mant, a_exp, w_mant, w_exp, fmt: Format, M: int, N: int):
    if M < 0 or N < 0:
        raise MxqError("M and N must be non-negative")
    dev = a_mant.device if isinstance(a_mant, torch.Tensor) else None
    _dev_bytes(a_mant, fmt.act_bytes(M), "a_mant", dev)
    _dev_bytes(a_exp, fmt.act_exp_bytes(M), "a_exp", dev)
    _dev_bytes(w_mant, fmt.weight_bytes(N), "w_mant", dev)
    _dev_bytes(w_exp, fmt.weight_exp_bytes(N), "w_exp", dev)
    return dev


def quantize_act(a, fmt: Format, out=None):
    """Online activation quantization: bf16 [M, >=K] -> (mant uint8
    [act_bytes(M)], exp uint8 [act_exp_bytes(M)]) on the current stream."""
    _bf16_2d(a, fmt.K, "activations")
    M = a.shape[0]
    mant, exp = _act_out(out, fmt, M, a.device)
    _check(lib().mxq_quantize_act(fmt.ref, _ptr(a), M, a.stride(0), _ptr(mant),
                                  _ptr(exp), _stream()), "mxq_quantize_act")
    return mant, exp


def quantize_act_rmsnorm(x, gain, eps: float, fmt: Format, out=None):
    """RMS-normalise bf16 rows x with bf16 gain, then quantize them (one
    kernel; the normalised rows are never written)."""
    _bf16_2d(x, fmt.K, "activations")
    if gain.dtype != torch.bfloat16 or gain.numel() < fmt.K or not gain.is_contiguous():
        raise MxqError("gain must be a contiguous bf16 tensor of K elements")
    if not gain.is_cuda or gain.device != x.device:
        raise MxqError("gain must be on the activations' device")
    M = x.shape[0]
    mant, exp = _act_out(out, fmt, M, x.device)
    _check(lib().mxq_quantize_act_rmsnorm(fmt.ref, _ptr(x), M, x.stride(0), _ptr(gain),
                                          float(eps), _ptr(mant), _ptr(exp), _stream()),
           "mxq_quantize_act_rmsnorm")
    return mant, exp


def quantize_act_swiglu(gate, up, fmt: Format, out=None):
    """Quantize SiLU(gate) * up (bf16 rows of the same shape and stride) in
    one kernel; the product rows are never written."""
    _bf16_2d(gate, fmt.K, "gate")
    _bf16_2d(up, fmt.K, "up")
    if up.shape != gate.shape or up.stride() != gate.stride():
        raise MxqError("gate and up must have the same shape and strides")
    if up.device != gate.device:
        raise MxqError("gate and up must be on one device")
    M = gate.shape[0]
    mant, exp = _act_out(out, fmt, M, gate.device)
    _check(lib().mxq_quantize_act_swiglu(fmt.ref, _ptr(gate), _ptr(up), M, gate.stride(0),
                                         _ptr(mant), _ptr(exp), _stream()),
           "mxq_quantize_act_swiglu")
    return mant, exp


def quantize_rows(a, fmt: Format, out=None):
    """The quantizer writing packed rows: bf16 [M, >=K] -> (rows uint8
    [M, act_packed_bytes], exps uint8 [M, exp_row_bytes]) -- the KV-cache
    layout, and the input of unpack_act and gemm_partials."""
    _bf16_2d(a, fmt.K, "activations")
    M = a.shape[0]
    rb, erb = fmt.act_packed_bytes(), fmt.exp_row_bytes()
    if out is None:
        rows = torch.empty((M, rb), dtype=torch.uint8, device=a.device)
        exps = torch.empty((M, erb), dtype=torch.uint8, device=a.device)
    else:
        rows, exps = out
        _dev_bytes(rows, M * rb, "packed row buffer", a.device)
        _dev_bytes(exps, M * erb, "exponent row buffer", a.device)
    _check(lib().mxq_quantize_rows(fmt.ref, _ptr(a), M, a.stride(0), _ptr(rows),
                                   _ptr(exps), _stream()), "mxq_quantize_rows")
    return rows, exps


def pack_weights(w, fmt: Format):
    """Offline weight quantization into the GEMM-tiled packed layout."""
    _bf16_2d(w, fmt.K, "weights")
    N = w.shape[0]
    mant = torch.empty(fmt.weight_bytes(N), dtype=torch.uint8, device=w.device)
    exp = torch.empty(fmt.weight_exp_bytes(N), dtype=torch.uint8, device=w.device)
    _check(lib().mxq_pack_weights(fmt.ref, _ptr(w), N, w.stride(0), _ptr(mant),
                                  _ptr(exp), _stream()), "mxq_pack_weights")
    return mant, exp


def gemm(a_mant, a_exp, w_mant, w_exp, fmt: Format, M: int, N: int, out=None):
    """Y = Ahat @ What^T, fp32 [M, N]."""
    dev = _gemm_operands(a_mant, a_exp, w_mant, w_exp, fmt, M, N)
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=dev)
    if not (isinstance(out, torch.Tensor) and out.is_cuda and out.device == dev
            and out.dim() == 2 and out.stride(1) == 1 and out.dtype == torch.float32):
        raise MxqError("out must be a 2-D fp32 device tensor with unit column stride")
    if out.shape[0] < M or out.shape[1] < N:
        raise MxqError("out is %s, smaller than [M, N] = [%d, %d]" % (tuple(out.shape), M, N))
    _check(lib().mxq_gemm(fmt.ref, M, N, _ptr(a_mant), _ptr(a_exp), _ptr(w_mant),
                          _ptr(w_exp), _ptr(out), out.stride(0), _stream()),
           "mxq_gemm")
    return out


def gemm_partials(rows, exps, w_mant, w_exp, fmt: Format, M: int, N: int):
    """Exact per-block int32 sums P[M, N, K/32] (debug / parity) from packed
    rows (quantize_rows) and the packed weights."""
    if M < 0 or N < 0:
        raise MxqError("M and N must be non-negative")
    dev = rows.device if isinstance(rows, torch.Tensor) else None
    _dev_bytes(rows, M * fmt.act_packed_bytes(), "rows", dev)
    _dev_bytes(exps, M * fmt.exp_row_bytes(), "exps", dev)
    _dev_bytes(w_mant, fmt.weight_bytes(N), "w_mant", dev)
    _dev_bytes(w_exp, fmt.weight_exp_bytes(N), "w_exp", dev)
    a_mant, a_exp = rows, exps
    p = torch.empty((M, N, fmt.nb), dtype=torch.int32, device=dev)
    _check(lib().mxq_gemm_partials(fmt.ref, M, N, _ptr(a_mant), _ptr(a_exp),
                                   _ptr(w_mant), _ptr(w_exp), _ptr(p), _stream()),
           "mxq_gemm_partials")
    return p


def unpack_act(mant, exp, fmt: Format, rows: int):
    """Packed rows and exponent rows (quantize_rows) -> (q int8 [rows, K],
    e uint8 [rows, K/32])."""
    _dev_bytes(mant, rows * fmt.act_packed_bytes(), "rows")
    _dev_bytes(exp, rows * fmt.exp_row_bytes(), "exps", mant.device)
    q = torch.empty((rows, fmt.K), dtype=torch.int8, device=mant.device)
    e = torch.empty((rows, fmt.nb), dtype=torch.uint8, device=mant.device)
    _check(lib().mxq_unpack_act(fmt.ref, rows, _ptr(mant), _ptr(exp), _ptr(q), _ptr(e),
                                _stream()), "mxq_unpack_act")
    return q, e


def unpack_weights(w_mant, w_exp, fmt: Format, N: int):
    _dev_bytes(w_mant, fmt.weight_bytes(N), "w_mant")
    _dev_bytes(w_exp, fmt.weight_exp_bytes(N), "w_exp", w_mant.device)
    q = torch.empty((N, fmt.K), dtype=torch.int8, device=w_mant.device)
    e = torch.empty((N, fmt.nb), dtype=torch.uint8, device=w_mant.device)
    _check(lib().mxq_unpack_weights(fmt.ref, N, _ptr(w_mant), _ptr(w_exp), _ptr(q),
                                    _ptr(e), _stream()), "mxq_unpack_weights")
    return q, e


# --------------------------------------------------------------------------
# Achievable-peak microbenchmarks (measurement only)

def peak_sink(device):
    """A sink buffer large enough for the peak microbenchmarks."""
    return torch.empty(int(lib().mxq_peak_sink_words()), dtype=torch.int32, device=device)


def peak_stream_read(buf, sink):
    """Read every byte of `buf` (a device tensor, nbytes % 16 == 0) once."""
    nbytes = buf.numel() * buf.element_size()
    _check(lib().mxq_peak_stream_read(_ptr(buf), nbytes, _ptr(sink), _stream()),
           "mxq_peak_stream_read")
    return nbytes


PEAK_KINDS = {"int8": 0, "fp6": 1, "fp8": 2}


def peak_mfma(kind: str, iters: int, sink):
    """Matrix-core loop of `kind` ("int8", "fp6", "fp8"); returns the ops of
    one launch."""
    ops = ctypes.c_int64(0)
    _check(lib().mxq_peak_mfma(PEAK_KINDS[kind], int(iters), _ptr(sink),
                               ctypes.byref(ops), _stream()), "mxq_peak_mfma")
    return ops.value


# --------------------------------------------------------------------------
# Calibration (offline): permutation and width map from calibration samples

def calib_colsq(x, s=None, accumulate: bool = False):
    """Column sensitivities of one calibration sample x (bf16 [rows, >=K]):
    s[k] = sum_r x[r, k]^2 in float64 (added to s when accumulate)."""
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise MxqError("calibration samples must be 2-D bf16 with unit column stride")
    rows, K = x.shape
    if s is None:
        if accumulate:
            raise MxqError("accumulate needs the running sensitivities")
        s = torch.empty(K, dtype=torch.float64, device=x.device)
    _check(lib().mxq_calib_colsq(_ptr(x), rows, x.stride(0), K, _ptr(s),
                                 1 if accumulate else 0, _stream()), "mxq_calib_colsq")
    return s


def calib_colsq_samples(x, s=None, accumulate: bool = False, work=None):
    """Column sensitivities of a batch of samples x (bf16 [n, rows, >=K]),
    summed in sample order (equal to one calib_colsq call per sample)."""
    if x.dtype != torch.bfloat16 or x.dim() != 3 or x.stride(2) != 1:
        raise MxqError("calibration samples must be 3-D bf16 with unit column stride")
    n, rows, K = x.shape
    if s is None:
        if accumulate:
            raise MxqError("accumulate needs the running sensitivities")
        s = torch.empty(K, dtype=torch.float64, device=x.device)
    if work is None:
        work = torch.empty(n * K, dtype=torch.float64, device=x.device)
    _check(lib().mxq_calib_colsq_samples(_ptr(x), n, rows, x.stride(1), x.stride(0), K,
                                         _ptr(work), _ptr(s), 1 if accumulate else 0,
                                         _stream()), "mxq_calib_colsq_samples")
    return s


def calib_ratio(d_in, s_layer, B: float) -> float:
    """Theorem A.1's control parameter R for layers of widths d_in."""
    n = len(d_in)
    d = (ctypes.c_int64 * n)(*[int(v) for v in d_in])
    sl = (ctypes.c_double * n)(*[float(v) for v in s_layer])
    R = ctypes.c_double(0.0)
    _check(lib().mxq_calib_ratio(n, d, sl, float(B), ctypes.byref(R)), "mxq_calib_ratio")
    return R.value


def calib_counts(d_in: int, R: float, s_layer: float, n8_blocks: int = 1):
    """(n4, n6, n8) block counts of one layer (Algorithm 2)."""
    out = [ctypes.c_int32(0) for _ in range(3)]
    _check(lib().mxq_calib_counts(int(d_in), float(R), float(s_layer), int(n8_blocks),
                                  *[ctypes.byref(v) for v in out]), "mxq_calib_counts")
    return tuple(v.value for v in out)


def calib_perm(s, n6: int, n8: int, perm=None):
    """The permutation of Algorithm 2 (int32 device tensor [K])."""
    if s.dtype != torch.float64 or s.dim() != 1:
        raise MxqError("sensitivities must be a 1-D float64 tensor")
    K = s.numel()
    if perm is None:
        perm = torch.empty(K, dtype=torch.int32, device=s.device)
    _check(lib().mxq_calib_perm(_ptr(s), K, int(n6), int(n8), _ptr(perm), _stream()),
           "mxq_calib_perm")
    return perm


def calibrate(samples, s_layer: float, R: float, n8_blocks: int = 1):
    """One layer: sensitivities over the samples, the block counts and the
    permutation.  Returns (perm int32 device tensor, widths list)."""
    s = None
    for i, x in enumerate(samples):
        s = calib_colsq(x, s, accumulate=i > 0)
    K = s.numel()
    n4, n6, n8 = calib_counts(K, R, s_layer, n8_blocks)
    perm = calib_perm(s, n6, n8)
    return perm, [4] * n4 + [6] * n6 + [8] * n8


def attn_work_bytes(fmt: Format, B: int, Hq: int, Hkv: int, T: int) -> int:
    """Bytes of the scratch that mxq_attn_decode needs for these sizes."""
    return _size(lib().mxq_attn_work_bytes(fmt.ref, B, Hq, Hkv, T), "mxq_attn_work_bytes")


def attn_decode(q, k_cache, v_cache, fmt: Format, B: int, Hq: int, Hkv: int, T: int,
                scale: float, out=None, work=None):
    """Decode attention over an MXINT KV cache.  q: bf16 [B, Hq, 128] on the
    device; k_cache, v_cache: (rows, exps) as returned by quantize_rows for
    the B * T * Hkv cache rows (row (b * T + t) * Hkv + h).  Returns float32
    [B, Hq, 128] on the current stream."""
    if not (isinstance(q, torch.Tensor) and q.is_cuda and q.dtype == torch.bfloat16
            and q.is_contiguous() and q.numel() == B * Hq * 128):
        raise MxqError("q must be a contiguous bf16 device tensor of B * Hq * 128 elements")
    rows = B * T * Hkv
    for mant, exp in (k_cache, v_cache):
        if mant.numel() < rows * fmt.act_packed_bytes() or exp.numel() < rows * fmt.exp_row_bytes():
            raise MxqError("KV cache buffers are too small for B * T * Hkv rows")
    if out is None:
        out = torch.empty((B, Hq, 128), dtype=torch.float32, device=q.device)
    nw = attn_work_bytes(fmt, B, Hq, Hkv, T)
    if work is None:
        work = torch.empty(max(nw, 16), dtype=torch.uint8, device=q.device)
    _check(lib().mxq_attn_decode(fmt.ref, _ptr(q), B, Hq, Hkv, T, float(scale),
                                 _ptr(k_cache[0]), _ptr(k_cache[1]), _ptr(v_cache[0]),
                                 _ptr(v_cache[1]), _ptr(out), _ptr(work), work.numel(),
                                 _stream()), "mxq_attn_decode")
    return out


ATTN_STATIC_WORK_BYTES = 8 << 20


def attn_decode_static(q, k_cache, v_cache, fmt: Format, B: int, Hq: int, Hkv: int, T: int,
                       scale: float, out):
    """attn_decode without a work buffer: the library's static per-GPU
    scratch holds the split results (calls overlapping on one GPU race).
    `out` (float32 [B, Hq, 128], contiguous, on the device) is required, so
    the call allocates nothing."""
    if not (isinstance(q, torch.Tensor) and q.is_cuda and q.dtype == torch.bfloat16
            and q.is_contiguous() and q.numel() == B * Hq * 128):
        raise MxqError("q must be a contiguous bf16 device tensor of B * Hq * 128 elements")
    if not (isinstance(out, torch.Tensor) and out.is_cuda and out.dtype == torch.float32
            and out.is_contiguous() and out.numel() >= B * Hq * 128):
        raise MxqError("out must be a contiguous float32 device tensor of B * Hq * 128 elements")
    rows = B * T * Hkv
    for mant, exp in (k_cache, v_cache):
        if mant.numel() < rows * fmt.act_packed_bytes() or exp.numel() < rows * fmt.exp_row_bytes():
            raise MxqError("KV cache buffers are too small for B * T * Hkv rows")
    _check(lib().mxq_attn_decode_static(fmt.ref, _ptr(q), B, Hq, Hkv, T, float(scale),
                                        _ptr(k_cache[0]), _ptr(k_cache[1]), _ptr(v_cache[0]),
                                        _ptr(v_cache[1]), _ptr(out), _stream()),
           "mxq_attn_decode_static")
    return out
