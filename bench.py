#!/usr/bin/env python3
"""Benchmark of the MXINT 4/6/8 hot path on one MI355X.

A step is one pass of the online path of a quantized linear on the
LLaMA-3-8B attention-projection shape (M=2048 tokens, K=N=4096, width map
102/13/13 blocks of 4/6/8 bits): MXINT quantization of the bf16 activations
followed by the mixed-mantissa GEMM against pre-packed weights.  Inputs are
seeded synthetic tensors already resident in HBM; the weights are packed once
before timing (offline step, reported separately).

Printed as one JSON line: the step throughput (effective TOPS = 2*M*N*K per
step time), the GEMM kernel against the int8 matrix-core roofline (its launch
duration from HIP events on the launch stream around back-to-back launches of
the kernel alone), the
decode-shape GEMMs against the HBM roofline (M = 1, 4, 16 against both
LLaMA-2-70B shapes, four weight copies rotated so the 256 MB last-level cache
cannot hold them), the LLaMA-2-70B-shaped decoder layer at M=8192 (seven
quantize + GEMM pairs and the K/V cache quantize on one stream, both width
variants), and the CPU oracle timed on the host on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0          # MI355X dense int8 matrix-core peak
FP6_PEAK_TOPS = 10100.0          # MI355X dense FP6 / FP4 matrix-core peak
FP8_PEAK_TOPS = 5000.0           # MI355X dense FP8 matrix-core peak
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E

# Sources of the prefill GEMM kernel: the HBM traffic stored under profiles/
# was counted on a build of exactly these files (sha256 of their contents).
GEMM_SOURCES = ("paper_2607_17733_amd/csrc/gemm_prefill.hip",
                "paper_2607_17733_amd/csrc/mxq_device.h",
                "paper_2607_17733_amd/csrc/mxq_internal.h",
                "paper_2607_17733_amd/csrc/api.cpp")
TRAFFIC_FILE = "profiles/traffic_gemm_prefill_attn_2048x4096x4096.json"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def bf16_dev(bits, dev):
    import numpy as np
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)


def sources_sha256(paths=GEMM_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(p.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per launch of the prefill GEMM from the committed counter
    summary (FETCH_SIZE + WRITE_SIZE, scaled by the same counters on a plain
    copy of known size), or None when the kernel sources changed since."""
    path = os.path.join(ROOT, TRAFFIC_FILE)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("sources_sha256") != sources_sha256():
        return None
    return rec.get("traffic_bytes")


def copy_calibration(dev, mib: int = 512, reps: int = 5):
    """A plain device-to-device copy of known size, for scaling the HBM
    byte counters (run under rocprofv3 --pmc)."""
    import torch
    n = mib << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "reps": reps}),
          flush=True)


def burst_ms(fn, reps: int, warmup: int):
    """Mean milliseconds per call of fn over reps calls launched back to back
    on the current stream, between HIP events on that stream."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def peaks(dev, reps: int = 5):
    """Achievable peaks on this machine: a streaming HBM read of 1 GiB and
    register-resident matrix-core loops (int8, FP6, FP8)."""
    import torch
    from paper_2607_17733_amd import mxq
    sink = mxq.peak_sink(dev)
    buf = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    out = {}

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    nbytes = buf.numel()
    out["hbm_stream_read_GBps"] = nbytes / timed(lambda: mxq.peak_stream_read(buf, sink)) / 1e9
    for kind in ("int8", "fp6", "fp8"):
        ops = [0]

        def run():
            ops[0] = mxq.peak_mfma(kind, 400, sink)
        t = timed(run)
        out["mfma_%s_TOPs" % kind] = ops[0] / t / 1e12
    del buf
    return out


def prefill_issue(meta, M: int, N: int):
    """Matrix-core instructions the prefill GEMM issues (32x32x64, 131072 ops
    each): per 32x32 output tile, 2 FP6 per 3/4-bit step (four blocks), 4 FP6
    per 6-bit step and 4 FP8 per 8-bit step (two blocks each, two digit
    planes).  Rows are padded to 256 and columns to 128 per workgroup."""
    tiles = -(-M // 256) * 8 * -(-N // 128) * 4
    s4, s6, s8 = -(-meta["n4"] // 4), -(-meta["n6"] // 2), -(-meta["n8"] // 2)
    return {"fp6": tiles * (2 * s4 + 4 * s6), "fp8": tiles * 4 * s8, "ops_per_instr": 131072}


def prefill_peak_times_us(meta, M: int, N: int, pk=None):
    """Times the prefill GEMM would take at the matrix cores' peaks:
      dtype_us   the algorithmic work (2*M*N*32 per block) of each block at
                 the datasheet peak of the dtype its block runs on (FP6 for
                 4- and 6-bit blocks, FP8 for 8-bit blocks);
      issued_us  the instructions actually issued at the datasheet peaks;
      measured_floor_us  the same at the loop rates measured on this machine."""
    per_block = 2.0 * M * N * 32
    dtype_us = per_block * ((meta["n4"] + meta["n6"]) / (FP6_PEAK_TOPS * 1e12) +
                            meta["n8"] / (FP8_PEAK_TOPS * 1e12)) * 1e6
    iss = prefill_issue(meta, M, N)
    o = iss["ops_per_instr"]
    out = {"dtype_us": dtype_us,
           "issued_us": (iss["fp6"] * o / (FP6_PEAK_TOPS * 1e12) +
                         iss["fp8"] * o / (FP8_PEAK_TOPS * 1e12)) * 1e6}
    if pk is not None:
        out["measured_floor_us"] = (iss["fp6"] * o / (pk["mfma_fp6_TOPs"] * 1e12) +
                                    iss["fp8"] * o / (pk["mfma_fp8_TOPs"] * 1e12)) * 1e6
    return out


def _rotated(t, copies: int):
    """`copies` distinct device buffers with t's contents."""
    return [t] + [t.clone() for _ in range(copies - 1)]


def prefill_leg(dev, case, reps: int, warmup: int, pk=None, rotate_bytes: int = 0):
    """One prefill linear: quantize + GEMM per step, and each kernel alone
    in a back-to-back burst (HIP events on the launch stream).  With
    rotate_bytes the quantizer is also timed over enough distinct input and
    output buffers to exceed that many bytes, so its rate is HBM's."""
    import torch
    from paper_2607_17733_amd import mxq
    M, K, N = case.M, case.K, case.N
    fmt = mxq.Format(K, case.widths, torch.from_numpy(case.perm).to(dev))
    a = bf16_dev(case.a_bits, dev)
    wm, we = mxq.pack_weights(bf16_dev(case.w_bits, dev), fmt)
    am = torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev)
    y = torch.empty((M, N), dtype=torch.float32, device=dev)

    def quantize():
        mxq.quantize_act(a, fmt, out=(am, ae))

    def gemm():
        mxq.gemm(am, ae, wm, we, fmt, M, N, out=y)

    def step():
        quantize()
        gemm()
    step_ms = burst_ms(step, reps, warmup)
    gemm_ms = burst_ms(gemm, reps, warmup)
    quant_ms = burst_ms(quantize, reps, warmup)
    ops = 2.0 * M * N * K
    meta = {"n4": int((case.widths <= 4).sum()), "n6": int((case.widths == 6).sum()),
            "n8": int((case.widths == 8).sum())}
    t = prefill_peak_times_us(meta, M, N, pk)
    gemm_us = gemm_ms * 1e3
    q_bytes = 2 * M * K + fmt.act_bytes(M) + fmt.act_exp_bytes(M)
    rec = {"M": M, "K": K, "N": N, "widths": [meta["n4"], meta["n6"], meta["n8"]],
           "step_us": step_ms * 1e3, "step_TOPs": ops / (step_ms * 1e-3) / 1e12,
           "gemm_us": gemm_us, "gemm_TOPs": ops / (gemm_ms * 1e-3) / 1e12,
           "frac_int8_peak": ops / (gemm_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS,
           "frac_dtype_peak": t["dtype_us"] / gemm_us,
           "frac_issued_peak": t["issued_us"] / gemm_us,
           "quantize_us": quant_ms * 1e3,
           "quantize_algorithmic_bytes": q_bytes,
           "quantize_GBps_cached": q_bytes / (quant_ms * 1e-3) / 1e9,
           "weight_bytes": wm.numel() + we.numel(),
           "weight_bits_per_element": 8.0 * (wm.numel() + we.numel()) / (N * K)}
    rec.update({k: v for k, v in t.items()})
    if rotate_bytes:
        per = 2 * M * K + am.numel() + ae.numel()
        R = max(2, -(-rotate_bytes // per))
        ins = _rotated(a, R)
        outs = [(am, ae)] + [(torch.empty_like(am), torch.empty_like(ae)) for _ in range(R - 1)]
        it = [0]

        def quant_rot():
            i = it[0] % R
            it[0] += 1
            mxq.quantize_act(ins[i], fmt, out=outs[i])
        qr_ms = burst_ms(quant_rot, max(reps, 2 * R), 2 * R)
        rec["quantize_rotated"] = {"us": qr_ms * 1e3, "copies": R,
                                   "GBps": q_bytes / (qr_ms * 1e-3) / 1e9,
                                   "frac_hbm_peak": q_bytes / (qr_ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
        del ins, outs
    del a, wm, we, am, ae, y
    torch.cuda.empty_cache()
    return rec


def calib_bench(dev, samples: int = 128, rows: int = 2048, K: int = 4096, reps: int = 3):
    """Offline calibration of one attention-shape layer: column sensitivities
    over `samples` calibration samples of `rows` tokens (the paper uses 128
    samples), then the permutation; reported, not part of a step."""
    import torch
    from paper_2607_17733_amd import mxq
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    x = torch.randn((samples, rows, K), generator=g, device=dev).to(torch.bfloat16)
    work = torch.empty(samples * K, dtype=torch.float64, device=dev)
    s = torch.empty(K, dtype=torch.float64, device=dev)

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    ms = timed(lambda: mxq.calib_colsq_samples(x, s, work=work))
    nbytes = x.numel() * 2
    out = {"sensitivity_ms": ms, "sensitivity_GBps": nbytes / (ms * 1e-3) / 1e9,
           "sensitivity_frac_hbm_peak": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    del x, work
    for kk in (4096, 28672):
        sk = torch.rand(kk, generator=g, device=dev, dtype=torch.float64)
        out["perm_K%d_us" % kk] = timed(lambda: mxq.calib_perm(sk, 2, 1)) * 1e3
    out["workload"] = ("one layer, K=%d: %d samples x %d tokens bf16 (%.2f GB), then the "
                       "permutation for K=4096 and K=28672" % (K, samples, rows, nbytes / 1e9))
    return out


def fused_bench(dev, case, fmt, reps: int = 50):
    """RMS normalisation fused into the quantizer against the two-kernel
    path (torch's RMS normalisation to bf16, then the quantizer) on the
    attention shape."""
    import torch
    import torch.nn.functional as F
    from paper_2607_17733_amd import mxq
    M, K = case.M, case.K
    x = bf16_dev(case.a_bits, dev)
    g = torch.Generator(device=dev)
    g.manual_seed(4321)
    gain = (torch.rand(K, generator=g, device=dev) + 0.5).to(torch.bfloat16)
    am = torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev)

    def fused():
        mxq.quantize_act_rmsnorm(x, gain, 1e-5, fmt, out=(am, ae))

    def unfused():
        mxq.quantize_act(F.rms_norm(x, (K,), gain, 1e-5), fmt, out=(am, ae))

    out = {"fused_us": burst_ms(fused, reps, 10) * 1e3,
           "unfused_us": burst_ms(unfused, reps, 10) * 1e3}
    out["saved_bytes"] = 2 * 2 * M * K            # the normalised rows, written and read back
    out["workload"] = ("RMS normalisation + quantize, M=%d K=%d; unfused = torch rms_norm "
                       "to bf16, then mxq_quantize_act" % (M, K))
    return out


def swiglu_bench(dev, M: int = 2048, K: int = 28672, reps: int = 20):
    """SiLU(gate)*up fused into the quantizer against torch's SiLU and product
    followed by the quantizer, at the down projection's K (LLaMA-2-70B)."""
    import numpy as np
    import torch
    import torch.nn.functional as F
    from paper_2607_17733_amd import mxq
    from paper_2607_17733_amd import workloads as W
    case = W.decode(16, "down")                 # K = 28672 and its width map
    fmt = mxq.Format(case.K, case.widths, torch.from_numpy(case.perm).to(dev))
    g = torch.Generator(device=dev)
    g.manual_seed(99)
    gate = (torch.randn((M, K), generator=g, device=dev) * 3).to(torch.bfloat16)
    up = torch.randn((M, K), generator=g, device=dev).to(torch.bfloat16)
    am = torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev)

    def fused():
        mxq.quantize_act_swiglu(gate, up, fmt, out=(am, ae))

    def unfused():
        mxq.quantize_act(F.silu(gate) * up, fmt, out=(am, ae))

    out = {"fused_us": burst_ms(fused, reps, 5) * 1e3,
           "unfused_us": burst_ms(unfused, reps, 5) * 1e3,
           "saved_bytes": 2 * 2 * M * K,
           "workload": "SiLU(gate)*up + quantize, M=%d K=%d (widths %d/%d/%d); unfused = "
                       "torch silu(gate)*up in bf16, then mxq_quantize_act" % (
                           M, K, case.meta["n4"], case.meta["n6"], case.meta["n8"])}
    return out


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


_MLP = []


def mlp_cases():
    """The LLaMA-3-8B MLP linears at M=4096 (generated once per run)."""
    if not _MLP:
        from paper_2607_17733_amd import workloads as W
        _MLP.extend([W.mlp_gate_up(), W.mlp_down()])
    return _MLP


def oracle_case_times(case, rows=None):
    """The oracle as it stands on one linear: activation quantize, weight
    quantize (the pack), and the blockwise GEMM over all rows or the first
    `rows` rows (then extrapolated linearly in M)."""
    import numpy as np
    import oracle
    t0 = time.perf_counter()
    qa, ea = oracle.quantize(case.a_bits if rows is None else case.a_bits[:rows],
                             perm=case.perm, widths=case.widths)
    if rows is not None:
        rows = qa.shape[0]
    t_quant = time.perf_counter() - t0
    t0 = time.perf_counter()
    qw, ew = oracle.quantize(case.w_bits, perm=case.perm, widths=case.widths)
    t_pack = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.gemm(qa, ea, qw, ew, case.widths)
    t_gemm = time.perf_counter() - t0
    n = case.M if rows is None else rows
    scale = case.M / n
    step = (t_quant + t_gemm) * scale
    rec = {"M": case.M, "K": case.K, "N": case.N, "threads": oracle.num_threads(),
           "quantize_s": t_quant * scale, "pack_s": t_pack, "gemm_s": t_gemm * scale,
           "TOPs": 2.0 * case.M * case.N * case.K / step / 1e12}
    if rows is not None:
        rec["extrapolated"] = "first %d of %d rows, linear in M" % (n, case.M)
    return rec


def oracle_plan(layer: bool = False):
    """The oracle timed on the host cores: full runs of the tiny linear, the
    attention projection, both MLP linears and the decode linears (M = 1, 4,
    16), one-thread runs of the tiny linear and the decode linears at M = 16,
    and (with `layer`) a 256-row sample of the 70B-shaped layer."""
    import oracle
    from paper_2607_17733_amd import workloads as W
    oracle.build(force=False)
    nthreads = oracle.num_threads()
    out = {"cpu_model": cpu_model(), "threads": nthreads}
    out["tiny"] = oracle_case_times(W.tiny())
    out["attn_proj"] = oracle_case_times(W.attn_proj())
    out["mlp_gate_up"] = oracle_case_times(mlp_cases()[0])
    out["mlp_down"] = oracle_case_times(mlp_cases()[1])
    for which in ("up", "down"):
        base = W.decode(16, which)
        for M in (1, 4, 16):
            c = W.LinearCase(base.name, M, base.K, base.N, base.a_bits[:M], base.w_bits,
                             base.perm, base.widths, base.meta)
            out["decode_%s_M%d" % (which, M)] = oracle_case_times(c)
    oracle.set_threads(1)
    try:
        out["tiny_1thread"] = oracle_case_times(W.tiny())
        for which in ("up", "down"):
            out["decode_%s_M16_1thread" % which] = oracle_case_times(W.decode(16, which))
    finally:
        oracle.set_threads(nthreads)
    if layer:
        rec = {}
        for j in range(len(W.LAYER_LINEARS)):
            c = W.layer_linear(j, True, M=256)
            c.M = 8192                         # the layer's M; 256 rows are computed
            rec[c.name] = oracle_case_times(c, rows=256)
        out["layer_sensitive"] = rec
    return out


def decode_bench(dev, which: str = "up", reps: int = 50):
    """Decode GEMM (M in 1, 4, 16, and 64: four 16-row activation tiles per
    weight read) streaming packed weights of one LLaMA-2-70B-shaped linear
    ("up": K=8192, N=28672; "down": K=28672, N=8192)."""
    import torch
    from paper_2607_17733_amd import mxq
    from paper_2607_17733_amd import workloads as W
    case = W.decode(64, which)
    fmt = mxq.Format(case.K, case.widths, torch.from_numpy(case.perm).to(dev))
    wm0, we0 = mxq.pack_weights(bf16_dev(case.w_bits, dev), fmt)
    copies = [(wm0, we0)] + [(wm0.clone(), we0.clone()) for _ in range(3)]
    # algorithmic bytes: the MXINT weights, 4 m bytes per block and column
    # plus one exponent byte per block; the decode kernel streams the whole
    # weight buffer (the same bits, blocks padded to whole steps)
    w_bytes = case.N * sum(4 * int(m) + 1 for m in case.widths)
    buf_bytes = wm0.numel() + we0.numel()
    out = {}
    for M in (1, 4, 16, 64):
        am, ae = mxq.quantize_act(bf16_dev(case.a_bits[:M], dev), fmt)
        y = torch.empty((M, case.N), dtype=torch.float32, device=dev)
        for i in range(8):
            wm, we = copies[i % 4]
            mxq.gemm(am, ae, wm, we, fmt, M, case.N, out=y)
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            wm, we = copies[i % 4]
            mxq.gemm(am, ae, wm, we, fmt, M, case.N, out=y)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        gbs = w_bytes / (ms * 1e-3) / 1e9
        out["M%d" % M] = {"us": ms * 1e3, "packed_weight_GBps": gbs,
                          "frac_hbm_peak": gbs / HBM_PEAK_GBS}
    # What a pure streaming read reaches over the same bytes per launch (the
    # buffer's size, four rotated copies): a short launch pays its ramp-up
    # and tail, which the 1 GiB figure of `peaks` hides.
    sink = mxq.peak_sink(dev)
    srcs = [torch.empty(buf_bytes // 16 * 16, dtype=torch.uint8, device=dev) for _ in range(4)]
    for b in srcs:
        b.fill_(1)
    for i in range(8):
        mxq.peak_stream_read(srcs[i % 4], sink)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(reps):
        mxq.peak_stream_read(srcs[i % 4], sink)
    e1.record()
    torch.cuda.synchronize()
    s_us = e0.elapsed_time(e1) / reps * 1e3
    del srcs
    out["stream_read_same_bytes"] = {"us": s_us, "GBps": buf_bytes / (s_us * 1e-6) / 1e9}
    for M in (1, 4, 16, 64):
        out["M%d" % M]["frac_stream_read_same_bytes"] = s_us / out["M%d" % M]["us"]
    out["workload"] = "LLaMA-2-70B %s-projection decode K=%d N=%d widths %d/%d/%d, " \
                      "4 weight buffers rotated (%.1f MB of packed weights and " \
                      "exponents streamed per launch)" % (
                          which, case.K, case.N, case.meta["n4"], case.meta["n6"],
                          case.meta["n8"], w_bytes / 1e6)
    out["packed_weight_bytes"] = w_bytes
    out["weight_buffer_bytes"] = buf_bytes
    out["weight_bits_per_element"] = 8.0 * buf_bytes / (case.N * case.K)
    out["buffer_over_mxint"] = buf_bytes / w_bytes
    return out


def attn_bench(dev, reps: int = 50):
    """Decode attention over the MXINT KV cache at the LLaMA-2-70B attention
    shape: 64 query heads, 8 KV heads, head dim 128, 4096 cached tokens per
    sequence, batches of 1, 4 and 16 sequences."""
    import torch
    from paper_2607_17733_amd import mxq
    from paper_2607_17733_amd import workloads as W
    Hq, Hkv, T, D = 64, 8, 4096, 128
    out = {}
    for widths in ([4, 4, 4, 4], [4, 4, 6, 8]):
        fmt = mxq.Format(D, widths)
        rb, erb = fmt.act_packed_bytes(), fmt.exp_row_bytes()
        # bytes the attention needs per cache row: the mantissas and the four
        # block exponents
        row_alg = sum(4 * m for m in widths) + len(widths)
        rec = {}
        for B in (1, 4, 16):
            rows = B * T * Hkv
            per_copy = 2 * rows * (rb + erb)
            R = max(2, -(-600_000_000 // per_copy))   # rotate > 2x the 256 MB last-level cache
            q, k, v = W.device_attn_inputs(B * R, Hq, Hkv, T, dev)
            q = q[:B].contiguous()
            kc = mxq.quantize_rows(k, fmt)
            vc = mxq.quantize_rows(v, fmt)
            del k, v
            o = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
            work = torch.empty(max(mxq.attn_work_bytes(fmt, B, Hq, Hkv, T), 16),
                               dtype=torch.uint8, device=dev)

            mxq.attn_decode(q, kc, vc, fmt, B, Hq, Hkv, T, D ** -0.5, out=o, work=work)
            # the C ABI called directly with pre-marshalled arguments, so that
            # host-side argument checks do not pace the launches
            L = mxq.lib()
            args = [(fmt.ref, mxq._ptr(q), B, Hq, Hkv, T, D ** -0.5,
                     kc[0].data_ptr() + c * rows * rb, kc[1].data_ptr() + c * rows * erb,
                     vc[0].data_ptr() + c * rows * rb, vc[1].data_ptr() + c * rows * erb,
                     mxq._ptr(o), mxq._ptr(work), work.numel(), mxq._stream())
                    for c in range(R)]

            def call(i):
                L.mxq_attn_decode(*args[i % R])
            for i in range(2 * R):
                call(i)
            torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for i in range(reps):
                call(i)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / reps
            alg = 2 * rows * row_alg + 2 * q.numel() + 4 * o.numel()
            gbs = alg / (ms * 1e-3) / 1e9
            rec["B%d" % B] = {"us": ms * 1e3, "algorithmic_bytes": alg, "GBps": gbs,
                              "frac_hbm_peak": gbs / HBM_PEAK_GBS,
                              "bf16_cache_bytes": 2 * rows * 2 * D, "rotated_copies": R}
            del kc, vc, q
            torch.cuda.empty_cache()
        rec["widths"] = widths
        out["w" + "".join(str(m) for m in widths)] = rec
    out["workload"] = ("decode attention, 64 query / 8 KV heads, head dim 128, 4096 cached "
                       "tokens per sequence, K and V MXINT (widths per 32-block of the head "
                       "dimension), caches rotated so none stays in the last-level cache; "
                       "bytes = mantissas + block exponents of K and V, q in, o out")
    return out


def template368_bench(dev, case, reps: int = 50):
    """The 3-6-8 template (3-bit blocks in place of the 4-bit ones, the same
    counts and permutation): the attention-projection step, the bytes of its
    weights and activation image against the 4-6-8 map's, and the
    LLaMA-2-70B up-projection decode GEMM at M = 1, whose time follows the
    weight bytes."""
    import torch
    from paper_2607_17733_amd import mxq
    from paper_2607_17733_amd import workloads as W
    widths = [3 if m == 4 else int(m) for m in case.widths]
    fmt = mxq.Format(case.K, widths, torch.from_numpy(case.perm).to(dev))
    fmt4 = mxq.Format(case.K, case.widths, torch.from_numpy(case.perm).to(dev))
    a = bf16_dev(case.a_bits, dev)
    wm, we = mxq.pack_weights(bf16_dev(case.w_bits, dev), fmt)
    am = torch.empty(fmt.act_bytes(case.M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(case.M), dtype=torch.uint8, device=dev)
    y = torch.empty((case.M, case.N), dtype=torch.float32, device=dev)

    def step():
        mxq.quantize_act(a, fmt, out=(am, ae))
        mxq.gemm(am, ae, wm, we, fmt, case.M, case.N, out=y)
    ms = burst_ms(step, reps, 10)
    ops = 2.0 * case.M * case.N * case.K
    nk = case.N * case.K
    out = {"ms_per_step": ms, "TOPs": ops / (ms * 1e-3) / 1e12,
           "widths": [case.meta["n4"], case.meta["n6"], case.meta["n8"]],
           "weight_bits_per_element": 8.0 * (fmt.weight_bytes(case.N) +
                                             fmt.weight_exp_bytes(case.N)) / nk,
           "weight_bits_per_element_468": 8.0 * (fmt4.weight_bytes(case.N) +
                                                 fmt4.weight_exp_bytes(case.N)) / nk,
           "activation_image_bytes": fmt.act_bytes(case.M) + fmt.act_exp_bytes(case.M),
           "activation_image_bytes_468": fmt4.act_bytes(case.M) + fmt4.act_exp_bytes(case.M),
           "workload": "attention projection M=%d K=%d N=%d, 3-bit/6-bit/8-bit blocks "
                       "%d/%d/%d (3 bits per element in the weights)" % (
                           case.M, case.K, case.N, case.meta["n4"], case.meta["n6"],
                           case.meta["n8"])}
    # decode: the up projection with its 4-bit blocks made 3-bit
    dc = W.decode(1, "up")
    rec = {}
    for tag, ws in (("368", [3 if m == 4 else int(m) for m in dc.widths]),
                    ("468", [int(m) for m in dc.widths])):
        f = mxq.Format(dc.K, ws, torch.from_numpy(dc.perm).to(dev))
        w0 = mxq.pack_weights(bf16_dev(dc.w_bits, dev), f)
        copies = [w0] + [(w0[0].clone(), w0[1].clone()) for _ in range(3)]
        xa, xe = mxq.quantize_act(bf16_dev(dc.a_bits[:1], dev), f)
        yd = torch.empty((1, dc.N), dtype=torch.float32, device=dev)
        it = [0]

        def dstep():
            wmc, wec = copies[it[0] % 4]
            it[0] += 1
            mxq.gemm(xa, xe, wmc, wec, f, 1, dc.N, out=yd)
        dms = burst_ms(dstep, 40, 8)
        nbytes = copies[0][0].numel() + copies[0][1].numel()
        rec[tag] = {"us": dms * 1e3, "weight_buffer_bytes": nbytes,
                    "GBps": nbytes / (dms * 1e-3) / 1e9}
        del copies, w0
    rec["workload"] = ("LLaMA-2-70B up-projection decode, M=1, K=%d N=%d, blocks %d/%d/%d "
                       "(3- or 4-bit / 6-bit / 8-bit), 4 weight buffers rotated" % (
                           dc.K, dc.N, dc.meta["n4"], dc.meta["n6"], dc.meta["n8"]))
    out["decode_up_M1"] = rec
    return out


def layer_bench(dev, sensitive: bool, reps: int = 5):
    """The config-5 decoder layer: seven online quantize + GEMM pairs and the
    K/V cache quantize on one stream (inputs drawn on the device, weights
    packed once before timing)."""
    import numpy as np
    import torch
    from paper_2607_17733_amd import workloads as W
    from paper_2607_17733_amd.layer import LayerSequence, Linear
    M = 8192
    specs = W.layer_specs(sensitive)
    linears, xs = [], []
    for s in specs:
        w = W.device_weights(s, dev)
        linears.append(Linear(s.name, s.K, s.N, s.widths,
                              torch.from_numpy(s.perm).to(dev), w))
        del w
        xs.append(W.device_activations(s, M, dev))
    kv = [W.device_kv(0, dev), W.device_kv(1, dev)]
    seq = LayerSequence(linears, M, dev)
    for _ in range(2):
        seq.run(xs, kv)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        seq.run(xs, kv)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"ms": ms, "effective_TOPs": seq.ops() / (ms * 1e-3) / 1e12,
            "ops": seq.ops(),
            "workload": "LLaMA-2-70B-shaped decoder layer, M=8192: q/k/v/o/gate/up/down "
                        "(%s: %s) + 4-bit K/V cache quantize [32768, 128] x 2, one stream"
                        % ("sensitive" if sensitive else "insensitive",
                           ", ".join("%s %d/%d/%d" % (s.name, *np.bincount(
                               s.widths, minlength=9)[[4, 6, 8]].tolist()) for s in specs))}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    # The default warm-up is about 0.1 s of steps: the device reaches its
    # steady clocks only after tens of milliseconds of work (after 10 steps
    # a step still takes about 12 % longer, after 200 about 5 %).
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=2000)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-layer", action="store_true")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--no-calib", action="store_true")
    ap.add_argument("--no-fused", action="store_true")
    ap.add_argument("--no-attn", action="store_true")
    ap.add_argument("--no-template", action="store_true")
    ap.add_argument("--no-mlp", action="store_true")
    ap.add_argument("--no-paper-point", action="store_true")
    ap.add_argument("--oracle-layer", action="store_true",
                    help="also time the oracle on a 256-row sample of the 70B layer")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 512 MiB device copy (counter scaling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the MXINT quantize + GEMM path runs on "
              "a single device (no collectives); run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_17733_amd import mxq
    from paper_2607_17733_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("device", torch.cuda.get_device_name(dev))
    if args.copy_calibration:
        copy_calibration(dev)
        return
    case = W.attn_proj()
    M, K, N = case.M, case.K, case.N
    log("workload", case.name, M, K, N, case.meta)
    fmt = mxq.Format(K, case.widths, torch.from_numpy(case.perm).to(dev))
    a = bf16_dev(case.a_bits, dev)
    w = bf16_dev(case.w_bits, dev)

    # offline: pack the weights (timed, not part of the step)
    wm, we = mxq.pack_weights(w, fmt)
    torch.cuda.synchronize()
    p0 = torch.cuda.Event(enable_timing=True)
    p1 = torch.cuda.Event(enable_timing=True)
    p0.record()
    for _ in range(5):
        mxq.pack_weights(w, fmt)
    p1.record()
    torch.cuda.synchronize()
    pack_ms = p0.elapsed_time(p1) / 5

    am = torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev)
    y = torch.empty((M, N), dtype=torch.float32, device=dev)

    def quantize():
        mxq.quantize_act(a, fmt, out=(am, ae))

    def gemm():
        mxq.gemm(am, ae, wm, we, fmt, M, N, out=y)

    def step():
        quantize()
        gemm()

    # The timed region: K steps launched back to back on one stream, no host
    # synchronization or events inside.  (Replaying the step from a HIP graph
    # measured slower on this stack: each graph node adds a few microseconds.)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = start.elapsed_time(end) / args.steps

    # Per-kernel launch durations: each kernel alone, K launches back to
    # back between HIP events on the launch stream.
    gemm_ms = burst_ms(gemm, args.steps, args.warmup)
    quant_ms = burst_ms(quantize, args.steps, args.warmup)

    ops = 2.0 * M * N * K
    value = ops / (ms_per_step * 1e-3) / 1e12
    gemm_tops = ops / (gemm_ms * 1e-3) / 1e12
    # quantizer: bf16 in; packed rows, operand image, exponents and scales out
    q_bytes = 2 * M * K + fmt.act_bytes(M) + fmt.act_exp_bytes(M)
    log("step %.3f ms (alone: quantize %.3f, gemm %.3f), wall %.3f s" %
        (ms_per_step, quant_ms, gemm_ms, wall))

    result = {
        "metric": "MXINT mixed GEMM effective TOPS (prefill) + packed-weight GB/s "
                  "(decode), 1 GPU",
        "value": value,
        "unit": "TOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "mxint4/6/8 as fp6/fp8 mfma digits, fp32 accumulate",
        "data": "synthetic",
        "config": {
            "workload": "LLaMA-3-8B attention projection, online activation "
                        "quantize + MXINT GEMM, M=2048 K=4096 N=4096, width map "
                        "102/13/13 blocks (4/6/8-bit), bf16 N(0,1) activations "
                        "with 1%% x U(20,100) and 5%% x U(2,5) outlier channels, "
                        "weights N(0,0.02)",
            "M": M, "K": K, "N": N,
            "widths": [case.meta["n4"], case.meta["n6"], case.meta["n8"]],
        },
        "roofline": {
            "kernel": "gemm_prefill (mxq_gemm, M > 16)",
            "bound": "mfma",
            "achieved": gemm_tops,
            "unit": "TOP/s",
            "traffic": measured_traffic(),
            "avg_launch_us": gemm_ms * 1e3,
            "frac_int8_peak": gemm_tops / INT8_PEAK_TOPS,
        },
        "gemm_only_tops": gemm_tops,
        "quantize": {"us": quant_ms * 1e3,
                     "GBps": q_bytes / (quant_ms * 1e-3) / 1e9,
                     "frac_hbm_peak": q_bytes / (quant_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "algorithmic_bytes": q_bytes},
        "pack_weights_ms": pack_ms,
    }
    pk = None
    if not args.no_peaks:
        log("achievable peaks")
        pk = peaks(dev)
        result["peaks"] = pk
    t = prefill_peak_times_us(case.meta, M, N, pk)
    gemm_us = gemm_ms * 1e3
    # the contraction's own dtypes: 4- and 6-bit blocks run FP6, 8-bit blocks
    # FP8, so the peak is the blend of their datasheet peaks over this width map
    blended = ops / (t["dtype_us"] * 1e-6) / 1e12
    result["roofline"]["peak"] = blended
    result["roofline"]["frac"] = gemm_tops / blended
    result["roofline"]["frac_issued_peak"] = t["issued_us"] / gemm_us
    result["roofline"]["algorithmic"] = (
        "2*M*N*K = %.4g ops per launch (MXINT multiply-adds); peak = the same ops "
        "at the datasheet peak of the dtype each block runs on (FP6 10.1 POP/s for "
        "the %d 4-bit and %d 6-bit blocks, FP8 5.0 POP/s for the %d 8-bit blocks), "
        "%.2f us; frac_int8_peak prices them at the dense int8 peak (5.0 POP/s); "
        "frac_issued_peak = the instructions actually issued (digit products "
        "included) at their dtype peaks, %.2f us, over the launch time" % (
            ops, case.meta["n4"], case.meta["n6"], case.meta["n8"], t["dtype_us"],
            t["issued_us"]))
    if pk is not None:
        result["roofline"]["achievable"] = {
            "int8_loop_TOPs": pk["mfma_int8_TOPs"],
            "frac_int8_loop": gemm_tops / pk["mfma_int8_TOPs"],
            "kernel_mfma_floor_us": t["measured_floor_us"],
            "frac_of_mfma_floor": t["measured_floor_us"] / gemm_us,
        }
    result["weight_bits_per_element"] = 8.0 * (wm.numel() + we.numel()) / (N * K)
    if not args.no_mlp:
        log("MLP linears (gate/up, down) at M=4096")
        result["mlp"] = {"gate_up": prefill_leg(dev, mlp_cases()[0], 20, 5, pk),
                         "down": prefill_leg(dev, mlp_cases()[1], 20, 5, pk)}
    log("paper operating point and rotated quantizer at the attention shape")
    if not args.no_paper_point:
        pp = W.make_linear(2, "paper_point_127_0_1", M, K, N, 0.0, 0.0, counts=(127, 0, 1))
        result["paper_point"] = prefill_leg(dev, pp, args.steps, args.warmup, pk)
        result["paper_point"]["workload"] = (
            "the paper's operating point (one 8-bit block of 32 columns, the rest 4-bit: "
            "127/0/1 blocks) at the attention-projection shape M=2048 K=N=4096")
    result["quantize"]["rotated"] = prefill_leg(
        dev, case, 10, 2, pk, rotate_bytes=600 << 20)["quantize_rotated"]
    if not args.no_fused:
        log("fused normalisation + quantize")
        result["fused_rmsnorm_quantize"] = fused_bench(dev, case, fmt)
        result["fused_swiglu_quantize"] = swiglu_bench(dev)
    if not args.no_calib:
        log("calibration")
        result["calibration"] = calib_bench(dev)
    if not args.no_decode:
        log("decode bench")
        result["decode"] = {"up": decode_bench(dev, "up"),
                            "down": decode_bench(dev, "down")}
        if pk is not None:
            for which in ("up", "down"):
                for key, rec in result["decode"][which].items():
                    if key.startswith("M"):
                        rec["frac_achievable_hbm"] = (rec["packed_weight_GBps"] /
                                                      pk["hbm_stream_read_GBps"])
    if not args.no_template:
        log("3-6-8 template")
        result["template_368"] = template368_bench(dev, case)
    if not args.no_attn:
        log("attention over the MXINT KV cache")
        result["attention"] = attn_bench(dev)
        if pk is not None:
            for key, rec in result["attention"].items():
                if isinstance(rec, dict):
                    for b, r in rec.items():
                        if b.startswith("B"):
                            r["frac_achievable_hbm"] = r["GBps"] / pk["hbm_stream_read_GBps"]
    if not args.no_layer:
        log("layer sequence")
        result["layer"] = {"sensitive": layer_bench(dev, True),
                           "insensitive": layer_bench(dev, False)}
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        plan = oracle_plan(layer=args.oracle_layer)
        att = plan["attn_proj"]
        result["cpu_baseline"] = {
            "value": att["TOPs"], "unit": "TOP/s", "cores": att["threads"], "kind": "oracle",
            "cpu_model": plan["cpu_model"],
            "sample": "the whole step on the host: quantize all %d rows (%.2f s) + blockwise "
                      "GEMM on all %d rows (%.2f s); the other linears under oracle_plan"
                      % (M, att["quantize_s"], M, att["gemm_s"])}
        result["oracle_plan"] = plan
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
