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


def test_graph_replay_matches_eager(wpath):
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
    ws_f = torch.zeros(W.workspace_bytes(1, Hq, Hkv, d, S + gamma, variant=W.VARIANT_FULL), dtype=torch.uint8, device=dev)
    ws_w = torch.zeros(W.workspace_bytes(1, Hq, Hkv, d, S + gamma, Wn, sink, variant=W.VARIANT_WINDOWED),
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


def _graph_matches_eager(reset, body, outputs, state=lambda: [], reps=3):
    """Run body eagerly after reset, capture it in a graph, replay `reps`
    times (each after reset, with eager work in between) and require every
    tensor in outputs() (cleared before each replay) and state() (restored by
    reset) to equal the eager values bit for bit."""
    reset()
    body()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outputs() + state()]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        reset()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=s):
            body()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(reps):
        reset()
        for t in outputs():
            t.fill_(0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (t, r) in enumerate(zip(outputs() + state(), ref)):
            assert torch.equal(t, r), f"replay {rep}: tensor {i}"
        _ = (ref[0].float().sum() + 1).item()  # unrelated eager work between replays


def test_graph_extend_dense_and_ring(wpath):
    dev = G.device()
    B, Hq, Hkv, d, Wn, sink, qm = 3, 16, 2, 128, 64, 4, 5
    R_w = Wn + qm
    S0 = [0, 90, 400]
    k0 = I.normal_bf16((B, 500, Hkv, d), 11, dev)
    v0 = I.normal_bf16((B, 500, Hkv, d), 12, dev)
    kn = I.normal_bf16((B, qm, Hkv, d), 13, dev)
    vn = I.normal_bf16((B, qm, Hkv, d), 14, dev)
    n_new = G.lens_tensor([5, 2, 3], dev)
    q = I.normal_bf16((B, qm, Hq, d), 15, dev)
    k, v = k0.clone(), v0.clone()
    kr = torch.zeros((B, sink + R_w, Hkv, d), dtype=torch.bfloat16, device=dev)
    vr = torch.zeros_like(kr)
    lens, lens_r = G.lens_tensor(S0, dev), G.lens_tensor(S0, dev)
    outs = [torch.empty_like(q) for _ in range(4)]
    ws = torch.zeros(W.workspace_bytes(B * qm, Hq, Hkv, d, 500, variant=W.VARIANT_FULL), dtype=torch.uint8, device=dev)
    # the full-context extend with items sized per sequence (its own workspace)
    ws_x = torch.zeros(W.extend_workspace_bytes(B, qm, Hq, Hkv, d, 500), dtype=torch.uint8, device=dev)
    ws_w = torch.zeros(W.workspace_bytes(B * qm, Hq, Hkv, d, 500, Wn, sink, variant=W.VARIANT_WINDOWED),
                       dtype=torch.uint8, device=dev)

    def reset():
        k.copy_(k0)
        v.copy_(v0)
        kr.zero_()
        vr.zero_()
        lens.copy_(G.lens_tensor(S0, dev))
        lens_r.copy_(G.lens_tensor(S0, dev))

    def body():
        W.cache_append(k, v, kn, vn, n_new, lens)
        W.draft_extend_full(q, k, v, lens, n_q=n_new, out=outs[0], ws=ws)
        W.draft_extend_full(q, k, v, lens, n_q=n_new, out=outs[3], ws=ws_x)
        W.draft_extend_windowed(q, k, v, lens, Wn, sink, n_q=n_new, out=outs[1], ws=ws_w)
        W.ring_append(kr, vr, kn, vn, n_new, lens_r, sink, R_w)
        W.ring_extend(q, kr, vr, lens_r, Wn, sink, R_w, n_q=n_new, out=outs[2], ws=ws_w)

    _graph_matches_eager(reset, body, lambda: outs, lambda: [k, kr, lens, lens_r])


def test_graph_paged_index_build_and_attention():
    dev = G.device()
    B, Hq, Hkv, d, Wn, sink, C = 3, 16, 2, 128, 64, 4, 700
    lens = G.lens_tensor([1, 300, 690], dev)
    P = B * C
    g = torch.Generator(device="cpu").manual_seed(3)
    table = torch.randperm(P, generator=g)[: B * C].view(B, C).to(torch.int32).to(dev)
    kp = I.normal_bf16((P, Hkv, d), 21, dev)
    vp = I.normal_bf16((P, Hkv, d), 22, dev)
    q = I.normal_bf16((B, Hq, d), 23, dev)
    indptr = [torch.empty(B + 1, dtype=torch.int32, device=dev) for _ in range(2)]
    idx = [torch.empty(B * C, dtype=torch.int32, device=dev) for _ in range(2)]
    outs = [torch.empty_like(q) for _ in range(2)]
    ws = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, C, variant=W.VARIANT_PAGED_FULL), dtype=torch.uint8, device=dev)
    ws_w = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, C, Wn, sink, variant=W.VARIANT_PAGED_WINDOWED),
                       dtype=torch.uint8, device=dev)

    def body():
        W.build_kv_indices(table, lens, W.VARIANT_PAGED_FULL, indptr=indptr[0], indices=idx[0])
        W.build_kv_indices(table, lens, W.VARIANT_PAGED_WINDOWED, Wn, sink, indptr=indptr[1], indices=idx[1])
        W.paged_attn_full(q, kp, vp, table, lens, out=outs[0], ws=ws)
        W.paged_attn_windowed(q, kp, vp, table, lens, Wn, sink, out=outs[1], ws=ws_w)

    def reset():
        for t in indptr + idx:
            t.fill_(-7)

    n_full = 1 + 300 + 690
    n_win = 1 + 68 + 68
    _graph_matches_eager(reset, body, lambda: outs, lambda: indptr + [idx[0][:n_full], idx[1][:n_win]])


def test_graph_fp8_append_and_attention():
    dev = G.device()
    B, Hq, Hkv, d, Wn, sink, gamma = 2, 32, 2, 256, 64, 4, 3
    R_w = Wn + gamma
    S0 = [100, 3000]
    S_max = 3000 + gamma
    k0 = I.normal_fp8((B, S_max, Hkv, d), 31, dev)
    v0 = I.normal_fp8((B, S_max, Hkv, d), 32, dev)
    k, v = k0.clone(), v0.clone()
    kr = torch.zeros((B, sink + R_w, Hkv, d), dtype=torch.uint8, device=dev)
    vr = torch.zeros_like(kr)
    kn = I.normal_bf16((gamma, B, 1, Hkv, d), 33, dev)
    vn = I.normal_bf16((gamma, B, 1, Hkv, d), 34, dev)
    q = I.normal_bf16((gamma, B, Hq, d), 35, dev)
    ones = G.lens_tensor([1, 1], dev)
    lens, lens_r = G.lens_tensor(S0, dev), G.lens_tensor(S0, dev)
    outs = [torch.empty_like(q) for _ in range(3)]
    ws = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, S_max, variant=W.VARIANT_FULL), dtype=torch.uint8, device=dev)
    ws_w = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, S_max, Wn, sink, variant=W.VARIANT_WINDOWED),
                       dtype=torch.uint8, device=dev)

    def reset():
        k.copy_(k0)
        v.copy_(v0)
        kr.zero_()
        vr.zero_()
        lens.copy_(G.lens_tensor(S0, dev))
        lens_r.copy_(G.lens_tensor(S0, dev))

    def body():
        for j in range(gamma):
            W.cache_append_fp8(k, v, kn[j], vn[j], ones, lens, 0.5, 2.0)
            W.draft_attn_full_fp8(q[j], k, v, lens, 0.5, 2.0, out=outs[0][j], ws=ws)
            W.draft_attn_windowed_fp8(q[j], k, v, lens, Wn, sink, 0.5, 2.0, out=outs[1][j], ws=ws_w)
            W.ring_append_fp8(kr, vr, kn[j], vn[j], ones, lens_r, sink, R_w, 0.5, 2.0)
            W.ring_attn_fp8(q[j], kr, vr, lens_r, Wn, sink, R_w, 0.5, 2.0, out=outs[2][j], ws=ws_w)

    _graph_matches_eager(reset, body, lambda: outs, lambda: [k, v, kr, lens, lens_r])


def test_graph_tree_speculation_round(wpath):
    dev = G.device()
    B, width, dd, Hq, Hkv, d, Wn, sink = 2, 3, 4, 16, 2, 128, 64, 4
    R_w = Wn + dd
    kr0 = I.normal_bf16((B, sink + R_w, Hkv, d), 41, dev)
    vr0 = I.normal_bf16((B, sink + R_w, Hkv, d), 42, dev)
    kr, vr = kr0.clone(), vr0.clone()
    kb = torch.zeros((B, (width - 1) * dd, Hkv, d), dtype=torch.bfloat16, device=dev)
    vb = torch.zeros_like(kb)
    kn = I.normal_bf16((dd, B, width, Hkv, d), 43, dev)
    vn = I.normal_bf16((dd, B, width, Hkv, d), 44, dev)
    q = I.normal_bf16((dd, B, width, Hq, d), 45, dev)
    lens = G.lens_tensor([30, 500], dev)
    depth = G.lens_tensor([0, 0], dev)
    drop = G.lens_tensor([2, 0], dev)
    outs = torch.empty_like(q)
    ws = torch.zeros(W.workspace_bytes(B * width, Hq, Hkv, d, 0, Wn, sink, variant=W.VARIANT_TREE), dtype=torch.uint8,
                     device=dev)
    depth_seen = torch.empty((dd, B), dtype=torch.int32, device=dev)

    def reset():
        kr.copy_(kr0)
        vr.copy_(vr0)
        kb.zero_()
        vb.zero_()
        lens.copy_(G.lens_tensor([30, 500], dev))
        depth.zero_()

    def body():
        for i in range(dd):
            W.tree_append(kr, vr, kb, vb, kn[i], vn[i], lens, depth, Wn, sink, R_w, dd)
            W.tree_attn(q[i], kr, vr, kb, vb, lens, depth, Wn, sink, R_w, dd, out=outs[i], ws=ws)
            depth_seen[i].copy_(depth)
        W.tree_reset(depth)
        W.ring_rollback(lens, drop)

    _graph_matches_eager(reset, body, lambda: [outs, depth_seen], lambda: [kr, kb, lens, depth])
