"""GPU read-stream yardstick (the HBM read ceiling the weight kernels are compared with):
it must read every 16-byte word it is given, which the XOR fold written to the sink shows."""
import pytest

from _gpu_util import say, torch_cuda

pytestmark = pytest.mark.gpu

MAGIC = 0x9E3779B9   # the fold value that makes a lane write the sink


@pytest.mark.parametrize("words,grid,at", [(4096, 1, 0), (4096, 1, 4095), (100_003, 0, 77_777),
                                           (1 << 20, 64, (1 << 20) - 1), (1 << 20, 0, 12345)])
def test_read_stream_reads_every_word(words, grid, at):
    torch = torch_cuda()
    import paper_2512_16473_amd as moe
    say("read_stream", words, grid, at)
    buf = torch.zeros((words, 4), dtype=torch.int32, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    moe.read_stream(buf, words * 16, sink, grid=grid)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0            # every fold is 0: nothing written
    # one word whose fold is the magic value: the lane that reads it writes the sink
    buf[at, 0] = MAGIC - (1 << 32)
    moe.read_stream(buf, words * 16, sink, grid=grid)
    torch.cuda.synchronize()
    assert int(sink.item()) & 0xFFFFFFFF == MAGIC
    # the same word outside the range read: not seen
    sink.zero_()
    moe.read_stream(buf, at * 16, sink, grid=grid)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0
