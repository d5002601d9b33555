"""GPU check of the streaming-read probe: the XOR of its sink words is the XOR
of every 32-bit word of the bytes it read (so it read each of them), on sizes
below one load per lane of the grid, across several grid strides, and at an
offset into a larger buffer."""
import numpy as np
import pytest
import torch

import paper_2609_21704_amd as sq

pytestmark = pytest.mark.gpu


def xor_words(a: np.ndarray) -> int:
    return int(np.bitwise_xor.reduce(a.view(np.uint32))) if a.size else 0


@pytest.mark.parametrize("nbytes,offset", [(16, 0), (4096, 16), ((1 << 20) + 16, 0), (37 * (1 << 20) + 48, 1024),
                                           (200 << 20, 0)])
def test_probe_reads_every_word(nbytes, offset):
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2**32, size=(offset + nbytes + 64) // 4, dtype=np.uint32)
    src = torch.from_numpy(host.view(np.int32)).cuda()
    sink = sq.sq_probe_stream_read(src, nbytes, offset)
    torch.cuda.synchronize()
    got = xor_words(sink.cpu().numpy())
    want = xor_words(host.view(np.uint8)[offset:offset + nbytes].copy())
    assert got == want
