"""MI355X-native MXINT 4/6/8 mixed-mantissa quantize + GEMM (MXSens hot path).

The compute path is the HIP library ``libmxq.so`` behind the C ABI in
``include/mxq.h``; ``paper_2607_17733_amd.mxq`` is its Python binding and
``paper_2607_17733_amd.workloads`` draws the seeded synthetic inputs.
"""
_BINDING = ("Format", "MxqError", "quantize_act", "quantize_rows", "pack_weights", "gemm",
            "gemm_partials", "unpack_act", "unpack_weights", "lib")


def __getattr__(name):
    if name in _BINDING:
        from . import mxq
        return getattr(mxq, name)
    raise AttributeError(name)
