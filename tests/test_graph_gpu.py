"""The draft loop (append, then attend, gamma times) captured once in a HIP
graph and replayed: every replay must equal the eager run bit for bit.

The library does nothing a capture forbids (no allocation, no
synchronisation, no memset), and lengths advance on the device, so the
graph replays the whole loop without the host (the paper requires the
windowing change to be graph-safe, Section 4 "Mechanism").  Replays are
interleaved with eager work and synchronisations, and each one is checked.
"""

import pytest
import torch

from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager():
    dev = G.device()
    Hq, Hkv, d, S, gamma, Wn, sink = 32, 2, 256, 70000, 3, 2048, 4
    q = I.normal_bf16((gamma, 1, Hq, d), 1, dev)
    k0 = torch.zeros((1, S + gamma, Hkv, d), dtype=torch.bfloat16, device=dev)
    k0[:, :S] = I.normal_bf16((1, S, Hkv, d), 2, dev)
    v0 = torch.zeros_like(k0)
    v0[:, :S] = I.normal_bf16((1, S, Hkv, d), 3, dev)
    kn = I.normal_bf16((gamma, 1, 1, Hkv, d), 4, dev)
    vn = I.normal_bf16((gamma, 1, 1, Hkv, d), 5, dev)
    ones = torch.ones(1, dtype=torch.int32, device=dev)
    lens0 = torch.tensor([S], dtype=torch.int32, device=dev)

    k, v = k0.clone(), v0.clone()
    lens = lens0.clone()
    outs_f = torch.empty((gamma, 1, Hq, d), dtype=torch.bfloat16, device=dev)
    outs_w = torch.empty_like(outs_f)
    ws_f = torch.empty(W.workspace_bytes(W.VARIANT_FULL, 1, Hq, Hkv, d, S + gamma), dtype=torch.uint8, device=dev)
    ws_w = torch.empty(W.workspace_bytes(W.VARIANT_WINDOWED, 1, Hq, Hkv, d, S + gamma, Wn, sink),
                       dtype=torch.uint8, device=dev)

    def loop():
        for j in range(gamma):
            W.cache_append(k, v, kn[j], vn[j], ones, lens)
            W.draft_attn_full(q[j], k, v, lens, out=outs_f[j], ws=ws_f)
            W.draft_attn_windowed(q[j], k, v, lens, Wn, sink, out=outs_w[j], ws=ws_w)

    loop()
    torch.cuda.synchronize()
    ref_f, ref_w, ref_k = outs_f.clone(), outs_w.clone(), k.clone()

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        k.copy_(k0)
        v.copy_(v0)
        lens.copy_(lens0)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=s):
            loop()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        k.copy_(k0)
        v.copy_(v0)
        lens.copy_(lens0)
        outs_f.zero_()
        outs_w.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert lens.item() == S + gamma, f"replay {rep}"
        assert torch.equal(outs_f, ref_f), f"replay {rep}: full"
        assert torch.equal(outs_w, ref_w), f"replay {rep}: windowed"
        assert torch.equal(k, ref_k), f"replay {rep}: cache"
        _ = (k0.float().sum() + 1).item()  # unrelated eager work between replays
