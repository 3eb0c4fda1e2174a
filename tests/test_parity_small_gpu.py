"""GPU parity at small sizes: every head size, a spread of GQA shapes,
ragged and degenerate lengths, windows and sinks, against the float64 oracle.

Each case spans several 16-key tiles, several work items and a ragged tail;
lengths include 0 (empty), 1, shorter than the sink, exactly sink + W and
sink + W + 1 (the threshold of the Appendix A rule).
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

SHAPES = [  # (d, Hq, Hkv)
    (64, 1, 1),
    (64, 6, 2),
    (128, 16, 2),
    (128, 16, 1),
    (128, 4, 4),
    (256, 32, 2),
    (256, 12, 3),
    (256, 8, 8),
]
WINDOWS = [(64, 4), (1, 0), (100, 7), (3000, 2)]


@pytest.fixture(scope="module")
def dev():
    return G.device()


def _make(dev, B, Hq, Hkv, d, S_max, seed):
    q = I.normal_bf16((B, Hq, d), seed, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), seed + 1, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), seed + 2, dev)
    return q, k, v


def _lens_for(W_, sink):
    return [0, 1, 3, sink + W_, sink + W_ + 1, 17, 1000, 5003]


@pytest.mark.parametrize("d,Hq,Hkv", SHAPES)
def test_full_and_windowed_vs_oracle(dev, d, Hq, Hkv, wpath):
    seed = 100 * d + 10 * Hq + Hkv
    for W_, sink in WINDOWS:
        lens = _lens_for(W_, sink)
        B = len(lens)
        S_max = max(lens) + 5
        G.say(f"case d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} lens={lens}")
        q, k, v = _make(dev, B, Hq, Hkv, d, S_max, seed)
        lt = G.lens_tensor(lens, dev)
        scale = 1.0 / np.sqrt(d)
        qb = I.bf16_bits(q)
        for variant in ("full", "windowed"):
            lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
            if variant == "full":
                out = W.draft_attn_full(q, k, v, lt, lse=lse)
            else:
                out = W.draft_attn_windowed(q, k, v, lt, W_, sink, lse=lse)
            torch.cuda.synchronize()
            refs = [G.oracle_seq(qb[b], k[b], v[b], lens[b], scale, variant, W_, sink, spread=True)
                    for b in range(B)]
            o_ref = np.stack([r[0] for r in refs])
            l_ref = np.stack([r[1] for r in refs])
            G.assert_attn_close(out, o_ref, lse, l_ref, what=f"{variant} d={d} G={Hq // Hkv} W={W_}",
                                spread=np.stack([r[2] for r in refs]))
            # empty sequence: exact zeros
            assert torch.count_nonzero(out[0]) == 0
        if W_ == 64:  # the window really drops keys past the threshold
            ow = W.draft_attn_windowed(q, k, v, lt, W_, sink)
            of = W.draft_attn_full(q, k, v, lt)
            diff = (ow[-1].float() - of[-1].float()).norm() / of[-1].float().norm()
            assert diff > 0.1


def _ring_from_dense(k, lens, sink, R_w):
    """Build a ring store from a dense cache with the oracle's slot map (torch
    copies only): row p of sequence b goes to slot ring_slot(p) for every
    position the ring still holds."""
    B, _, Hkv, d = k.shape
    ring = torch.zeros((B, sink + R_w, Hkv, d), dtype=k.dtype, device=k.device)
    for b, S in enumerate(lens):
        live = [p for p in range(S) if p < sink or p >= S - R_w]
        if not live:
            continue
        slots = R.ring_slots(live, sink, R_w)
        ring[b, torch.as_tensor(slots, device=k.device)] = k[b, torch.as_tensor(live, device=k.device)]
    return ring


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 6, 2), (128, 16, 2), (256, 32, 2)])
@pytest.mark.parametrize("W_,sink,slack", [(64, 4, 0), (64, 4, 7), (1, 0, 0), (100, 7, 3)])
def test_ring_equals_windowed_bitwise(dev, d, Hq, Hkv, W_, sink, slack, wpath):
    R_w = W_ + slack
    lens = [0, 1, 3, sink + W_, sink + W_ + 1, sink + R_w + 1, 777, 5003]
    B = len(lens)
    S_max = max(lens) + 2
    G.say(f"ring d={d} Hq={Hq} W={W_} sink={sink} R_w={R_w}")
    q, k, v = _make(dev, B, Hq, Hkv, d, S_max, 7 * d + W_ + slack)
    lt = G.lens_tensor(lens, dev)
    kr = _ring_from_dense(k, lens, sink, R_w)
    vr = _ring_from_dense(v, lens, sink, R_w)
    lse_w = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    lse_r = torch.empty_like(lse_w)
    ow = W.draft_attn_windowed(q, k, v, lt, W_, sink, lse=lse_w)
    orr = W.ring_attn(q, kr, vr, lt, W_, sink, R_w, lse=lse_r)
    torch.cuda.synchronize()
    assert torch.equal(orr, ow)
    assert torch.equal(lse_r, lse_w)
    qb = I.bf16_bits(q)
    scale = 1.0 / np.sqrt(d)
    refs = [G.oracle_seq(qb[b], k[b], v[b], lens[b], scale, "windowed", W_, sink, spread=True)
            for b in range(B)]
    G.assert_attn_close(orr, np.stack([r[0] for r in refs]), lse_r, np.stack([r[1] for r in refs]),
                        what="ring", spread=np.stack([r[2] for r in refs]))


def test_select_indices_export_exact(dev):
    rng = np.random.default_rng(0)
    for W_, sink, R_w in [(8, 3, 8), (8, 3, 13), (1, 0, 1), (2048, 4, 2048), (2048, 4, 2055), (5, 9, 6)]:
        lens = np.concatenate([np.arange(0, 40), rng.integers(0, 1 << 20, size=60)]).astype(np.int32)
        lt = G.lens_tensor(lens, dev)
        pos, slot, n_sel = W.select_indices(lt, W_, sink, R_w)
        pos, slot, n_sel = pos.cpu().numpy(), slot.cpu().numpy(), n_sel.cpu().numpy()
        for b, S in enumerate(lens):
            exp = A.selected_positions(int(S), W_, sink)
            assert n_sel[b] == exp.size
            assert np.array_equal(pos[b, :exp.size], exp)
            assert np.all(pos[b, exp.size:] == -1)
            assert np.array_equal(slot[b, :exp.size], R.ring_slots(exp, sink, R_w))
            assert np.all(slot[b, exp.size:] == -1)


def test_length_out_of_range_is_clamped_and_flagged(dev, wpath):
    d, Hq, Hkv, S_max = 128, 16, 2, 300
    q, k, v = _make(dev, 3, Hq, Hkv, d, S_max, 5)
    err = G.err_word(dev)
    bad = G.lens_tensor([S_max + 50, -7, 100], dev)
    good = G.lens_tensor([S_max, 0, 100], dev)
    o_bad = W.draft_attn_full(q, k, v, bad, err=err)
    o_good = W.draft_attn_full(q, k, v, good)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_LEN_RANGE
    assert torch.equal(o_bad, o_good)
    err.zero_()
    W.draft_attn_full(q, k, v, good, err=err)
    torch.cuda.synchronize()
    assert err.item() == 0


def test_determinism(dev, wpath):
    d, Hq, Hkv = 256, 32, 2
    lens = [70000, 12345, 1]
    q, k, v = _make(dev, 3, Hq, Hkv, d, max(lens), 9)
    lt = G.lens_tensor(lens, dev)
    a = W.draft_attn_full(q, k, v, lt)
    b = W.draft_attn_full(q, k, v, lt)
    c = W.draft_attn_windowed(q, k, v, lt, 2048, 4)
    e = W.draft_attn_windowed(q, k, v, lt, 2048, 4)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(c, e)


def test_cache_append_exact_and_capacity(dev):
    B, Hkv, d, S_max, n_max = 4, 2, 128, 40, 6
    k = torch.zeros((B, S_max, Hkv, d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    ref_k, ref_v = k.clone(), v.clone()
    lens = [0, 10, 37, 40]
    lt = G.lens_tensor(lens, dev)
    kn = I.normal_bf16((B, n_max, Hkv, d), 1, dev)
    vn = I.normal_bf16((B, n_max, Hkv, d), 2, dev)
    nn = G.lens_tensor([6, 0, 5, 1], dev)
    err = G.err_word(dev)
    W.cache_append(k, v, kn, vn, nn, lt, err=err)
    torch.cuda.synchronize()
    exp_lens = [6, 10, 40, 40]
    assert lt.cpu().tolist() == exp_lens
    assert err.item() & W.DERR_CAPACITY
    for b, (L0, n) in enumerate(zip(lens, [6, 0, 5, 1])):
        m = min(n, S_max - L0)
        ref_k[b, L0:L0 + m] = kn[b, :m]
        ref_v[b, L0:L0 + m] = vn[b, :m]
    assert torch.equal(k, ref_k) and torch.equal(v, ref_v)
    # n_new out of range is clamped to [0, n_max] and flagged
    err.zero_()
    lt2 = G.lens_tensor([0, 0, 0, 0], dev)
    W.cache_append(k, v, kn, vn, G.lens_tensor([-1, 9, 2, 0], dev), lt2, err=err)
    torch.cuda.synchronize()
    assert lt2.cpu().tolist() == [0, 6, 2, 0]
    assert err.item() & W.DERR_NNEW_RANGE


@pytest.mark.parametrize("sink,R_w,L0,n", [(4, 16, 0, 3), (4, 16, 2, 30), (4, 16, 10, 50),
                                             (0, 8, 5, 20), (3, 5, 100, 7), (4, 2048, 0, 6000)])
def test_ring_bulk_append_equals_sequential(dev, sink, R_w, L0, n):
    """A bulk append (n > R_w, the pruned draft prefill of Section 7) leaves
    the ring exactly as appending the rows one by one would (last write wins)."""
    Hkv, d = 2, 64
    kr = I.normal_bf16((1, sink + R_w, Hkv, d), 11, dev)  # stale content
    vr = kr.clone()
    kn = I.normal_bf16((1, n, Hkv, d), 12, dev)
    lt = G.lens_tensor([L0], dev)
    W.ring_append(kr, vr, kn, kn, G.lens_tensor([n], dev), lt, sink, R_w)
    torch.cuda.synchronize()
    assert lt.item() == L0 + n
    ref = I.bf16_bits(I.normal_bf16((1, sink + R_w, Hkv, d), 11, dev)).copy()  # the stale rows
    knb = I.bf16_bits(kn)
    sim = R.RingSimulator(sink, R_w)
    sim.append(L0)
    for i, (p, s) in enumerate(sim.append(n)):
        ref[0, s] = knb[0, i]
    assert np.array_equal(I.bf16_bits(kr), ref)


def _vs_oracle(dev, d, Hq, Hkv, lens, variant, W_=None, sink=None, seed=7):
    B = len(lens)
    q, k, v = _make(dev, B, Hq, Hkv, d, max(lens) + 3, seed)
    lt = G.lens_tensor(lens, dev)
    scale = 1.0 / np.sqrt(d)
    lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    if variant == "full":
        out = W.draft_attn_full(q, k, v, lt, lse=lse)
    else:
        out = W.draft_attn_windowed(q, k, v, lt, W_, sink, lse=lse)
    torch.cuda.synchronize()
    qb = I.bf16_bits(q)
    refs = [G.oracle_seq(qb[b], k[b], v[b], lens[b], scale, variant, W_, sink, spread=True)
            for b in range(B)]
    G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                        what=f"{variant} d={d} lens={lens[:6]}", spread=np.stack([r[2] for r in refs]))


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2)])
def test_windowed_merge_in_several_batches(dev, d, Hq, Hkv, wpath):
    """A 65536-key window: at most 1024 keys per work item, so a row has at
    least 65 items and the one-launch kernel's merger combines them in
    several batches of registers (rows past, at and below the threshold)."""
    W_, sink = 65536, 4
    lens = [W_ + sink + 3001, W_ + sink, 40007, 5]
    G.say(f"windowed merge batches d={d} W={W_} lens={lens}")
    _vs_oracle(dev, d, Hq, Hkv, lens, "windowed", W_, sink)


@pytest.mark.parametrize("n_sel", [63 * 64, 64 * 64, 64 * 64 + 1, 65 * 64 + 17])
def test_merge_around_one_item_per_slot_wide(dev, n_sel):
    """One long row (the 1024-thread merge, 64 item slots): with 64-key items
    the row has 63, 64, 65 and 66 items -- the merge's one-round path up to 64,
    its two-pass path beyond."""
    G.say(f"wide merge boundary n_sel={n_sel}")
    _vs_oracle(dev, 256, 32, 2, [n_sel], "full")
    _vs_oracle(dev, 256, 32, 2, [n_sel + 500], "windowed", n_sel - 4, 4)


def test_merge_around_one_item_per_slot_rows(dev):
    """Many short rows (the 256-thread row merge, 4 item slots): rows of 4, 5
    and 6 items of 64 keys and ragged tails."""
    lens = [4 * 64 - 1, 4 * 64, 4 * 64 + 1, 5 * 64, 5 * 64 + 3, 6 * 64 + 63, 64, 1] * 4
    G.say(f"row merge boundary lens={lens[:8]}")
    _vs_oracle(dev, 128, 16, 2, lens, "full")
