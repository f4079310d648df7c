"""The achievable-peak microbenchmarks that the benchmark's roofline figures
use: the streaming read touches every byte exactly once (an XOR checksum
over the buffer: a missed or repeated word changes it), and the matrix-core
loops report the op count of their launch."""
import numpy as np
import pytest
import torch

from paper_2607_17733_amd import mxq
from parity_util import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, 3 << 20])
def test_stream_read_reads_every_word_once(nbytes):
    say("peak-stream", nbytes)
    g = np.random.Generator(np.random.PCG64(nbytes))
    host = g.integers(0, 2**32, size=nbytes // 4, dtype=np.uint32)
    buf = torch.from_numpy(host.view(np.int32)).cuda()
    sink = mxq.peak_sink(buf.device)
    assert mxq.peak_stream_read(buf, sink) == nbytes
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == np.bitwise_xor.reduce(host)


@pytest.mark.parametrize("kind,per", [("int8", 2 * 32 * 32 * 32), ("fp6", 2 * 32 * 32 * 64),
                                      ("fp8", 2 * 32 * 32 * 64)])
def test_mfma_loop_op_count(kind, per):
    say("peak-mfma", kind)
    sink = mxq.peak_sink(torch.device("cuda:0"))
    words = int(mxq.lib().mxq_peak_sink_words())
    ops = mxq.peak_mfma(kind, 3, sink)
    torch.cuda.synchronize()
    # eight accumulators per wave, four waves per workgroup, one sink word a thread
    assert ops == per * 8 * 3 * (words // 64)
    assert torch.isfinite(sink.view(torch.float32)).all()
