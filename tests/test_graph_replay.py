"""The quantize + GEMM step captured in a HIP graph and replayed.

The library launches on the caller's stream and neither allocates nor clears
memory with memset nodes, so a serving loop (and the benchmark) can capture a
step once and replay it.  Every replay must reproduce the eager result bit for
bit, also with eager work and synchronizations between replays.
"""
import pytest
import torch

from paper_2607_17733_amd import mxq
from paper_2607_17733_amd import workloads as W
from parity_util import say, to_dev_bf16

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M", [8, 300])
def test_step_graph_replays_match_eager(M):
    # a prefill-shaped case (M > 16) and a decode-shaped one (M <= 16)
    case = W.random_case(31 + M, M, 1024, 384, (24, 5, 3), perm="random")
    say("graph-replay", M, case.K, case.N)
    dev = torch.device("cuda:0")
    fmt = mxq.Format(case.K, case.widths, torch.from_numpy(case.perm).to(dev))
    a = to_dev_bf16(case.a_bits)
    wm, we = mxq.pack_weights(to_dev_bf16(case.w_bits), fmt)
    am = torch.empty(fmt.act_bytes(M), dtype=torch.uint8, device=dev)
    ae = torch.empty(fmt.act_exp_bytes(M), dtype=torch.uint8, device=dev)
    y = torch.empty((M, case.N), dtype=torch.float32, device=dev)

    def step():
        mxq.quantize_act(a, fmt, out=(am, ae))
        mxq.gemm(am, ae, wm, we, fmt, M, case.N, out=y)

    step()
    torch.cuda.synchronize()
    # the packed rows and exponent rows are fully specified; the operand
    # image's padding rows are not, so the image is checked through the GEMM
    n_rows, n_exp = M * fmt.act_packed_bytes(), M * fmt.exp_row_bytes()
    ref = (y.clone(), am[:n_rows].clone(), ae[:n_exp].clone())

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        # eager work between the replays overwrites every output
        y.fill_(float("nan"))
        am.fill_(0xA5)
        ae.fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref[0]), "replay %d: GEMM output differs" % r
        assert torch.equal(am[:n_rows], ref[1]), "replay %d: packed rows differ" % r
        assert torch.equal(ae[:n_exp], ref[2]), "replay %d: exponent rows differ" % r


def test_attention_graph_replays_match_eager():
    # decode attention over an MXINT cache: its split partials live in the
    # caller's work buffer, so a captured call replays without allocations
    B, Hq, Hkv, T, D = 2, 16, 2, 700, 128
    say("graph-replay attention", B, Hq, Hkv, T)
    dev = torch.device("cuda:0")
    qb, kb, vb = W.attn_inputs(41, B, Hq, Hkv, T)
    fmt = mxq.Format(D, [4, 4, 6, 8])
    kc = mxq.quantize_rows(to_dev_bf16(kb), fmt)
    vc = mxq.quantize_rows(to_dev_bf16(vb), fmt)
    q = to_dev_bf16(qb.reshape(-1, D)).reshape(B, Hq, D)
    o = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    work = torch.empty(mxq.attn_work_bytes(fmt, B, Hq, Hkv, T), dtype=torch.uint8, device=dev)

    def step():
        mxq.attn_decode(q, kc, vc, fmt, B, Hq, Hkv, T, D ** -0.5, out=o, work=work)

    step()
    torch.cuda.synchronize()
    ref = o.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for r in range(4):
        o.fill_(float("nan"))
        work.fill_(0xA5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref), "replay %d: attention output differs" % r
