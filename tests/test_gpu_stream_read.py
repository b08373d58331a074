"""The attainable-bandwidth probe reads every byte it is given.

A zero buffer holds one word 0x9e3779b9 and nothing else, so exactly one
block's xor of what it read equals that value and only that block writes
its sink entry.  Every grid size, loads in flight and access order is
checked with the word at the first, a middle and the last position of a
length that is not a whole number of 1 KB wave loads.
"""
import pytest
import torch

import paper_2404_08763_amd as P

from gpu_util import say

pytestmark = pytest.mark.gpu

MAGIC = 0x9E3779B9 - (1 << 32)  # as int32


@pytest.mark.parametrize("blocks", [1, 3, 256, 1024])
@pytest.mark.parametrize("inflight", [4, 8, 16])
@pytest.mark.parametrize("runs", [False, True])
def test_stream_read_covers_every_byte(blocks, inflight, runs):
    nbytes = (1 << 20) + 48
    buf = torch.zeros(nbytes // 4, dtype=torch.int32, device="cuda")
    for pos in (0, nbytes // 8 + 3, nbytes // 4 - 1):
        say("stream read", blocks, inflight, runs, pos)
        buf.zero_()
        buf[pos] = MAGIC
        sink = torch.full((blocks,), -1, dtype=torch.int32, device="cuda")
        P.stream_read(buf, blocks, inflight, runs, sink)
        got = sink.cpu()
        hit = (got == MAGIC).nonzero().flatten().tolist()
        assert len(hit) == 1, (pos, hit)
        assert int((got == -1).sum()) == blocks - 1
