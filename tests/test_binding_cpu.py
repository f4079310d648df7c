"""The Python binding and the C ABI reject mismatched or oversized buffers
before anything is launched.  Runs on the CPU: tensors are host tensors
presented as device tensors, and every launching entry point of the library
is replaced by one that fails the test if it is reached."""
import ctypes
from unittest import mock

import numpy as np
import pytest
import torch

from paper_2607_17733_amd import mxq

LAUNCHING = {"mxq_quantize_act", "mxq_quantize_rows", "mxq_quantize_act_rmsnorm",
             "mxq_quantize_act_swiglu",
             "mxq_pack_weights", "mxq_gemm", "mxq_gemm_partials", "mxq_unpack_act",
             "mxq_unpack_weights", "mxq_attn_decode"}


class _NoLaunch:
    def __init__(self, real):
        self._real = real

    def __getattr__(self, name):
        if name in LAUNCHING:
            def fail(*_a, **_k):
                raise AssertionError("%s reached a launch" % name)
            return fail
        return getattr(self._real, name)


@pytest.fixture
def host_as_device():
    real = mxq.lib()
    with mock.patch.object(torch.Tensor, "is_cuda", new_callable=mock.PropertyMock,
                           return_value=True), \
            mock.patch.object(mxq, "lib", lambda path=mxq.LIB_PATH: _NoLaunch(real)):
        yield


def _u8(n):
    return torch.zeros(max(n, 0), dtype=torch.uint8)


def _operands(fmt, M, N):
    return (_u8(fmt.act_bytes(M)), _u8(fmt.act_exp_bytes(M)), _u8(fmt.weight_bytes(N)),
            _u8(fmt.weight_exp_bytes(N)))


def _row_operands(fmt, M, N):
    """The inputs of gemm_partials: packed rows, exponent rows, weights."""
    return (_u8(M * fmt.act_packed_bytes()), _u8(M * fmt.exp_row_bytes()),
            _u8(fmt.weight_bytes(N)), _u8(fmt.weight_exp_bytes(N)))


FMT_ARGS = (256, [4] * 6 + [6, 8])


@pytest.mark.parametrize("short", [0, 1, 2, 3])
@pytest.mark.parametrize("M", [4, 40])
def test_gemm_rejects_short_operands(host_as_device, short, M):
    fmt = mxq.Format(*FMT_ARGS)
    ops = list(_operands(fmt, M, 48))
    ops[short] = ops[short][:-1]
    with pytest.raises(mxq.MxqError, match="needed"):
        mxq.gemm(*ops, fmt, M, 48, out=torch.zeros((M, 48)))
    rops = list(_row_operands(fmt, M, 48))
    rops[short] = rops[short][:-1]
    with pytest.raises(mxq.MxqError, match="needed"):
        mxq.gemm_partials(*rops, fmt, M, 48)


def test_gemm_rejects_small_or_wrong_out(host_as_device):
    fmt = mxq.Format(*FMT_ARGS)
    ops = _operands(fmt, 40, 48)
    for out in (torch.zeros((39, 48)), torch.zeros((40, 47)),
                torch.zeros((40, 48), dtype=torch.float64), torch.zeros((48, 40)).t()):
        with pytest.raises(mxq.MxqError, match="out"):
            mxq.gemm(*ops, fmt, 40, 48, out=out)


def test_gemm_rejects_wrong_dtype(host_as_device):
    fmt = mxq.Format(*FMT_ARGS)
    am, ae, wm, we = _operands(fmt, 40, 48)
    with pytest.raises(mxq.MxqError, match="uint8"):
        mxq.gemm(am, ae, wm.view(torch.int8), we, fmt, 40, 48)


def test_quantizers_reject_short_outputs(host_as_device):
    fmt = mxq.Format(*FMT_ARGS)
    x = torch.zeros((40, 256), dtype=torch.bfloat16)
    gain = torch.ones(256, dtype=torch.bfloat16)
    mant, exp = _u8(fmt.act_bytes(40)), _u8(fmt.act_exp_bytes(40))
    for out in ((mant[:-1], exp), (mant, exp[:-1])):
        with pytest.raises(mxq.MxqError, match="needed"):
            mxq.quantize_act(x, fmt, out=out)
        with pytest.raises(mxq.MxqError, match="needed"):
            mxq.quantize_act_rmsnorm(x, gain, 1e-5, fmt, out=out)
        with pytest.raises(mxq.MxqError, match="needed"):
            mxq.quantize_act_swiglu(x, x, fmt, out=out)
    rows, exps = _u8(40 * fmt.act_packed_bytes()), _u8(40 * fmt.exp_row_bytes())
    for out in ((rows[:-1], exps), (rows, exps[:-1])):
        with pytest.raises(mxq.MxqError, match="needed"):
            mxq.quantize_rows(x, fmt, out=out)


def test_unpack_rejects_short_inputs(host_as_device):
    fmt = mxq.Format(*FMT_ARGS)
    rows, exps, wm, we = _row_operands(fmt, 40, 48)
    with pytest.raises(mxq.MxqError, match="needed"):
        mxq.unpack_act(rows[:-16], exps, fmt, 40)
    with pytest.raises(mxq.MxqError, match="needed"):
        mxq.unpack_act(rows, exps[:-1], fmt, 40)
    with pytest.raises(mxq.MxqError, match="needed"):
        mxq.unpack_weights(wm, we[:-1], fmt, 48)


def test_cpu_tensor_is_not_a_device_tensor():
    fmt = mxq.Format(*FMT_ARGS)
    ops = _operands(fmt, 40, 48)
    with pytest.raises(mxq.MxqError, match="device"):
        mxq.gemm(*ops, fmt, 40, 48)


def test_abi_rejects_offsets_beyond_32_bits():
    """A K so long that sixteen 16-row activation tiles (a prefill
    workgroup's rows) span more than INT32_MAX bytes is refused with
    MXQ_ERR_SHAPE before any pointer is touched."""
    lib = mxq.lib()
    fake = ctypes.c_void_p(1 << 20)    # aligned, never dereferenced
    for nb, rejected in ((131072, True), (131071, True), (131070, False)):
        # 8-bit blocks: a 16-row tile holds 64 lanes x 32 bytes per two blocks
        w = np.full(nb, 8, np.uint8)
        f = mxq._Fmt(32 * nb, 32, 0, 0, 0, w.ctypes.data_as(ctypes.c_void_p).value, None)
        tile = 64 * 32 * -(-nb // 2)
        assert lib.mxq_act_bytes(ctypes.byref(f), 16) == tile
        if rejected:
            assert 16 * tile > 2 ** 31 - 1
            st = lib.mxq_gemm(ctypes.byref(f), 64, 128, fake, fake, fake, fake, fake, 128, None)
            assert st == 2
            st = lib.mxq_gemm_partials(ctypes.byref(f), 64, 128, fake, fake, fake, fake, fake,
                                       None)
            assert st == 2
        else:
            assert 16 * tile <= 2 ** 31 - 1


def test_static_attention_rejects_oversize_on_the_host():
    """mxq_attn_decode_static refuses sizes whose split results exceed its
    static scratch with MXQ_ERR_SCRATCH, before any device call."""
    lib = mxq.lib()
    w = np.array([4, 4, 4, 4], np.uint8)
    f = mxq._Fmt(128, 32, 0, 0, 0, w.ctypes.data_as(ctypes.c_void_p).value, None)
    B, Hq, Hkv, T = 300, 64, 8, 64
    assert lib.mxq_attn_work_bytes(ctypes.byref(f), B, Hq, Hkv, T) > mxq.ATTN_STATIC_WORK_BYTES
    fake = ctypes.c_void_p(1 << 20)
    st = lib.mxq_attn_decode_static(ctypes.byref(f), fake, B, Hq, Hkv, T, ctypes.c_float(0.1),
                                    fake, fake, fake, fake, fake, None)
    assert st == 8
    assert b"static scratch" in lib.mxq_status_str(8)
