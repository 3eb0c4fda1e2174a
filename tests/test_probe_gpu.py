"""The streaming-read probe (a measurement helper, not part of the method):
its pass covers every word of the buffer exactly once -- the XOR of the
workgroups' results equals the XOR of all words -- at sizes below one
grid-stride round, with a ragged tail, and over 256 MiB."""

import numpy as np
import pytest
import torch

from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n_words", [4, 4 * 1000, 4 * 1_000_003, 64 << 20])
def test_read_probe_covers_every_word(n_words):
    dev = G.device()
    g = torch.Generator(device="cpu").manual_seed(n_words)
    host = torch.randint(-2**31, 2**31 - 1, (n_words,), dtype=torch.int32, generator=g)
    G.say(f"read probe over {n_words * 4} bytes")
    buf = host.to(dev)
    sink = W.hbm_read_probe(buf)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host.numpy().view(np.uint32))
    assert got == want
