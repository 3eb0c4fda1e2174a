"""The ring workload: B=8, Hq=32, Hkv=2, d=256, ring of sink=4 + R_w=2048
slots, 1000 speculative iterations each appending a seeded accepted count in
[1, 8] of N(0,1) K/V rows to every sequence, then attending.

Every iteration checks, on the HIP path:
  * the selection export (positions and ring slots) equals the oracle's,
    exactly;
  * ring attention is bit-identical to windowed attention over an
    uncompacted dense cache holding the same rows (same kept keys, same
    order, same split plan);
  * the lengths advanced by the accepted counts.
Every 20th iteration (and the first 12, where the sequences cross the sink,
the threshold and the first wrap) also checks the ring's bytes at every live
slot against the oracle's replay, and the outputs against the oracle.
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import ring as R
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


def test_ring_b8_1000_iterations(dev):
    wl = I.WORKLOADS["ring_b8"]
    B, Hq, Hkv, d, Wn, sink, R_w = wl.B, wl.Hq, wl.Hkv, wl.d, wl.W, wl.sink, wl.R_w
    n_max = wl.max_accept
    acc = I.accept_counts(wl.iterations, B, n_max, I.stream_seed(wl.seed, I.STREAM_ACCEPT))
    S_cap = int(acc.sum(axis=0).max())
    kr = torch.zeros((B, sink + R_w, Hkv, d), dtype=torch.bfloat16, device=dev)
    vr = torch.zeros_like(kr)
    kd = torch.zeros((B, S_cap, Hkv, d), dtype=torch.bfloat16, device=dev)
    vd = torch.zeros_like(kd)
    lens_r = torch.zeros(B, dtype=torch.int32, device=dev)
    lens_d = torch.zeros(B, dtype=torch.int32, device=dev)
    err = G.err_word(dev)
    out_r = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    out_d = torch.empty_like(out_r)
    lse_r = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    lse_d = torch.empty_like(lse_r)
    ws_r = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, sink + R_w, Wn, sink, variant=W.VARIANT_RING),
                       dtype=torch.uint8, device=dev)
    ws_d = torch.zeros(W.workspace_bytes(B, Hq, Hkv, d, S_cap, Wn, sink, variant=W.VARIANT_WINDOWED),
                       dtype=torch.uint8, device=dev)
    replay = [R.ReplayCache(Hkv, d) for _ in range(B)]
    host_len = np.zeros(B, dtype=np.int64)
    checked = 0
    for it in range(wl.iterations):
        n_new = torch.as_tensor(acc[it], device=dev)
        k_new = I.normal_bf16((B, n_max, Hkv, d), I.stream_seed(wl.seed, I.STREAM_KNEW, it), dev)
        v_new = I.normal_bf16((B, n_max, Hkv, d), I.stream_seed(wl.seed, I.STREAM_VNEW, it), dev)
        q = I.normal_bf16((B, Hq, d), I.stream_seed(wl.seed, I.STREAM_Q, it), dev)
        W.ring_append(kr, vr, k_new, v_new, n_new, lens_r, sink, R_w, err=err)
        W.cache_append(kd, vd, k_new, v_new, n_new, lens_d, err=err)
        W.ring_attn(q, kr, vr, lens_r, Wn, sink, R_w, out=out_r, lse=lse_r, ws=ws_r, err=err)
        W.draft_attn_windowed(q, kd, vd, lens_d, Wn, sink, out=out_d, lse=lse_d, ws=ws_d, err=err)
        pos, slot, n_sel = W.select_indices(lens_r, Wn, sink, R_w)
        torch.cuda.synchronize()
        host_len += acc[it]
        assert lens_r.cpu().numpy().tolist() == host_len.tolist(), f"iteration {it}"
        assert torch.equal(lens_r, lens_d)
        assert torch.equal(out_r, out_d), f"iteration {it}: ring != windowed on full cache"
        assert torch.equal(lse_r, lse_d)
        pos, slot, n_sel = pos.cpu().numpy(), slot.cpu().numpy(), n_sel.cpu().numpy()
        knb, vnb = I.bf16_bits(k_new), I.bf16_bits(v_new)
        for b in range(B):
            replay[b].append(knb[b, :acc[it, b]], vnb[b, :acc[it, b]])
            exp = A.selected_positions(int(host_len[b]), Wn, sink)
            assert n_sel[b] == exp.size
            assert np.array_equal(pos[b, :exp.size], exp), f"iteration {it} b={b}: positions"
            assert np.array_equal(slot[b, :exp.size], R.ring_slots(exp, sink, R_w)), f"iteration {it} b={b}: slots"
        if it < 12 or it % 20 == 0 or it == wl.iterations - 1:
            krb, vrb = I.bf16_bits(kr), I.bf16_bits(vr)
            qb = I.bf16_bits(q)
            o_ref, l_ref = [], []
            for b in range(B):
                S = int(host_len[b])
                live = [p for p in range(S) if p < sink or p >= S - R_w]
                lk, lv = replay[b].rows(live)
                sl = R.ring_slots(live, sink, R_w)
                assert np.array_equal(krb[b, sl], lk) and np.array_equal(vrb[b, sl], lv), \
                    f"iteration {it} b={b}: ring bytes"
                o, l = replay[b].attend_windowed(qb[b], wl.scale, Wn, sink)
                o_ref.append(o)
                l_ref.append(l)
            G.assert_attn_close(out_r, np.stack(o_ref), lse_r, np.stack(l_ref), f"ring iteration {it}")
            checked += 1
        if it % 100 == 0:
            G.say(f"ring iteration {it}: lens {host_len.tolist()}")
    assert err.item() == 0
    assert checked >= 60
    # the run covered the short, threshold and wrapped regimes
    assert host_len.min() > 2 * (sink + R_w)
