"""The allocation-free windowed call (wmtp_draft_attn_windowed_noalloc)
against the workspace call it varies (wmtp_draft_attn_windowed), through the
C ABI: two calls in a row on the same static scratch, the second with a
smaller input, each bit for bit equal to the workspace call and within the
parity bar of the oracle."""

import numpy as np
import pytest
import torch

from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


CASES = [
    # (B, Hq, Hkv, d, lens, W, sink): the 1M workload's head shape on a batch of
    # lengths around the window threshold, then a smaller call
    (6, 32, 2, 256, [0, 3, 2052, 2053, 9000, 40000], 2048, 4),
    (2, 16, 2, 128, [700, 5], 512, 4),
]


def _run(dev, case, seed):
    B, Hq, Hkv, d, lens, Wn, sink = case
    S_max = max(lens) + 2
    q = I.normal_bf16((B, Hq, d), seed, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), seed + 1, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), seed + 2, dev)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    out_na = torch.full((B, Hq, d), 7.0, dtype=torch.bfloat16, device=dev)
    lse_na = torch.full((B, Hq), 7.0, dtype=torch.float32, device=dev)
    W.draft_attn_windowed_noalloc(q, k, v, lt, Wn, sink, out_na, lse=lse_na, err=err)
    lse_ws = torch.empty_like(lse_na)
    out_ws = W.draft_attn_windowed(q, k, v, lt, Wn, sink, lse=lse_ws, err=err)
    torch.cuda.synchronize()
    assert err.item() == 0
    assert torch.equal(out_na, out_ws) and torch.equal(lse_na, lse_ws)
    qb = I.bf16_bits(q)
    scale = 1.0 / np.sqrt(d)
    refs = [G.oracle_seq(qb[b], k[b], v[b], lens[b], scale, "windowed", Wn, sink) for b in range(B)]
    e = G.assert_attn_close(out_na, np.stack([r[0] for r in refs]), lse_na, np.stack([r[1] for r in refs]),
                            what=f"noalloc B={B} d={d}")
    G.say(f"noalloc B={B} Hq={Hq} d={d} lens={lens}: equal to the workspace call; oracle err {e}")


def test_noalloc_two_calls_then_smaller(dev, wpath):
    G.say("noalloc: two calls in a row, the second smaller")
    _run(dev, CASES[0], 900)
    _run(dev, CASES[1], 910)


def test_noalloc_rejects_oversized_batch(dev):
    B, Hq, Hkv, d = 4096, 32, 2, 256
    assert W.workspace_bytes(B, Hq, Hkv, d, 64, 2048, 4, variant=W.VARIANT_WINDOWED) > W.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((B, Hq, d), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((B, 64, Hkv, d), dtype=torch.bfloat16, device=dev)
    out = torch.empty_like(q)
    with pytest.raises(W.WmtpError) as ei:
        W.draft_attn_windowed_noalloc(q, k, k, G.lens_tensor([64] * B, dev), 2048, 4, out)
    assert ei.value.status == W.ESCRATCH
