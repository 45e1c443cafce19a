"""The read-ceiling measurement aid reads every byte exactly once: its per-chunk
XOR of 32-bit words equals numpy's over the same bytes, for sizes that end
inside a chunk and inside a loop step."""

import numpy as np
import pytest
import torch

import paper_2608_00531_amd as pc
from parity_util import say

pytestmark = pytest.mark.gpu

CHUNK = 256 << 10


@pytest.mark.parametrize("nbytes", [16, 4096, 8192 + 16, CHUNK, CHUNK + 48, 5 * CHUNK - 16,
                                    (64 << 20) + 4096])
def test_chunk_xor_matches_numpy(nbytes):
    say("read ceiling", nbytes)
    rng = np.random.default_rng(nbytes)
    host = rng.integers(0, 2**32, nbytes // 4, dtype=np.uint32)
    dev = torch.from_numpy(host.view(np.int32)).cuda()
    got = pc.cure_read_ceiling(dev).cpu().numpy().view(np.uint32)
    chunks = (nbytes + CHUNK - 1) // CHUNK
    assert len(got) == chunks
    for c in range(chunks):
        part = host[c * CHUNK // 4:(c + 1) * CHUNK // 4]
        assert int(got[c]) == int(np.bitwise_xor.reduce(part)), c
