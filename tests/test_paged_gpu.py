"""GPU parity of the paged token pool (page size 1): the draft's index
builder and attention read through req_to_token.

* build_kv_indices equals the oracle's index list exactly (full and
  windowed), for a batch of requests whose rows are scattered over the pool;
* paged attention equals dense attention over the same rows bit for bit (same
  kept keys, same order, same split) and the oracle within tolerance;
* a table entry outside the pool is flagged and never dereferenced;
* a 1M-token request scattered over a shuffled pool;
* an fp8 (E4M3) pool: equal bit for bit to the fp8 dense cache over the same
  rows, and to the oracle's paged attention over the dequantized pool.
"""

import numpy as np
import pytest
import torch

from oracle import fp8 as F
from oracle import paged as Pg
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


def _scatter(dense, lens, P, seed):
    """Pool [P, Hkv, d] holding every request's rows at random distinct slots,
    and the table [B, C] naming them (torch copies only)."""
    B, C, Hkv, d = dense.shape
    g = torch.Generator(device="cpu").manual_seed(seed)
    perm = torch.randperm(P, generator=g)[: B * C].view(B, C).to(torch.int32)
    pool = torch.zeros((P, Hkv, d), dtype=dense.dtype, device=dense.device)
    table = perm.to(dense.device)
    for b, S in enumerate(lens):
        if S:
            pool[table[b, :S].long()] = dense[b, :S]
    return pool, table


@pytest.mark.parametrize("variant", ["full", "windowed"])
def test_index_builder_exact(dev, variant):
    rng = np.random.default_rng(3)
    lens = [0, 1, 5, 68, 69, 3000, 9000, 20001] + [int(x) for x in rng.integers(0, 40000, size=40)]
    B, C = len(lens), 40004
    g = torch.Generator(device="cpu").manual_seed(7)
    table_cpu = torch.randint(0, 1 << 30, (B, C), generator=g, dtype=torch.int32)
    table = table_cpu.to(dev)
    Wn, sink = 64, 4
    vid = W.VARIANT_PAGED_FULL if variant == "full" else W.VARIANT_PAGED_WINDOWED
    err = G.err_word(dev)
    indptr, idx = W.build_kv_indices(table, G.lens_tensor(lens, dev), vid, Wn, sink, err=err)
    torch.cuda.synchronize()
    e_ptr, e_idx = Pg.kv_indices(table_cpu.numpy(), lens, variant, Wn, sink)
    assert indptr.cpu().numpy().tolist() == e_ptr.tolist()
    assert np.array_equal(idx[: e_ptr[-1]].cpu().numpy(), e_idx)
    assert err.item() == 0
    # a length past the table is clamped and flagged
    err.zero_()
    indptr2, _ = W.build_kv_indices(table[:1], G.lens_tensor([C + 9], dev), vid, Wn, sink, err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_LEN_RANGE
    assert indptr2[1].item() == (C if variant == "full" else Wn + sink)


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2), (64, 6, 2)])
def test_paged_attention_equals_dense(dev, d, Hq, Hkv, wpath):
    lens = [0, 1, 3, 68, 69, 1000, 5003, 12000]
    B, C = len(lens), max(lens) + 5
    P = B * C + 777
    G.say(f"paged d={d} Hq={Hq} Hkv={Hkv}")
    q = I.normal_bf16((B, Hq, d), 61, dev)
    kd = I.normal_bf16((B, C, Hkv, d), 62, dev)
    vd = I.normal_bf16((B, C, Hkv, d), 63, dev)
    kp, table = _scatter(kd, lens, P, 1)
    vp, _ = _scatter(vd, lens, P, 1)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    Wn, sink = 64, 4
    lse_p = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    lse_d = torch.empty_like(lse_p)
    for variant in ("full", "windowed"):
        if variant == "full":
            op = W.paged_attn_full(q, kp, vp, table, lt, lse=lse_p, err=err)
            od = W.draft_attn_full(q, kd, vd, lt, lse=lse_d)
        else:
            op = W.paged_attn_windowed(q, kp, vp, table, lt, Wn, sink, lse=lse_p, err=err)
            od = W.draft_attn_windowed(q, kd, vd, lt, Wn, sink, lse=lse_d)
        torch.cuda.synchronize()
        assert torch.equal(op, od), variant
        assert torch.equal(lse_p, lse_d), variant
        qb = I.bf16_bits(q)
        refs = [Pg.attend_paged(qb[b], G.HostRows(kp), G.HostRows(vp), table[b].cpu().numpy(), S,
                                1.0 / np.sqrt(d), variant, Wn, sink, spread=True) for b, S in enumerate(lens)]
        G.assert_attn_close(op, np.stack([r[0] for r in refs]), lse_p, np.stack([r[1] for r in refs]),
                            what=f"paged {variant}", spread=np.stack([r[2] for r in refs]))
    assert err.item() == 0


def test_slot_outside_pool_is_flagged(dev, wpath):
    Hq, Hkv, d, P = 16, 2, 128, 1000
    q = I.normal_bf16((1, Hq, d), 1, dev)
    kp = I.normal_bf16((P, Hkv, d), 2, dev)
    table = torch.arange(300, dtype=torch.int32, device=dev).view(1, 300).clone()
    table[0, 5] = P + 10
    table[0, 6] = -3
    err = G.err_word(dev)
    W.paged_attn_full(q, kp, kp, table, G.lens_tensor([300], dev), err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_SLOT_RANGE


def test_paged_1m_shuffled_pool(dev):
    wl = I.WORKLOADS["draft_loop_s1m"]
    G.say("paged 1M: generating")
    case = I.decode_case(wl, dev, steps=1)
    S = wl.S
    C = case["S_max"]
    kp, table = _scatter(case["k"], [S], C, 5)
    vp, _ = _scatter(case["v"], [S], C, 5)
    del case["v"]
    q = case["q"][0]
    lt = G.lens_tensor([S], dev)
    ow_p = W.paged_attn_windowed(q, kp, vp, table, lt, wl.W, wl.sink)
    of_p = W.paged_attn_full(q, kp, vp, table, lt)
    of_d = W.draft_attn_full(q, case["k"], _dense_v(vp, table, S, C), lt)
    torch.cuda.synchronize()
    assert torch.equal(of_p, of_d)
    qb = I.bf16_bits(q)
    o_ref, l_ref = Pg.attend_paged(qb[0], G.HostRows(kp), G.HostRows(vp), table[0].cpu().numpy(), S,
                                   wl.scale, "windowed", wl.W, wl.sink)
    G.say(f"paged 1M windowed err {G.assert_attn_close(ow_p, o_ref[None], what='paged 1M windowed')}")


def _dense_v(vp, table, S, C):
    v = torch.zeros((1, C) + tuple(vp.shape[1:]), dtype=vp.dtype, device=vp.device)
    v[0, :S] = vp[table[0, :S].long()]
    return v


class _HostCodes:
    """Host view of a device fp8 pool [P, Hkv, d]: indexing returns the rows'
    codes as a uint8 numpy array."""

    def __init__(self, t: torch.Tensor):
        self.t = t
        self.shape = tuple(t.shape)

    def __getitem__(self, rows):
        idx = torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int64)).to(self.t.device)
        return self.t.index_select(0, idx).cpu().numpy()


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2), (64, 6, 2)])
def test_paged_fp8_equals_dense_fp8(dev, d, Hq, Hkv, wpath):
    lens = [0, 1, 3, 68, 69, 1000, 5003, 12000]
    B, C = len(lens), max(lens) + 5
    P = B * C + 333
    ks, vs = 0.75, 1.5
    G.say(f"paged fp8 d={d} Hq={Hq} Hkv={Hkv}")
    q = I.normal_bf16((B, Hq, d), 71, dev)
    kd = I.normal_fp8((B, C, Hkv, d), 72, dev)
    vd = I.normal_fp8((B, C, Hkv, d), 73, dev)
    kp, table = _scatter(kd, lens, P, 2)
    vp, _ = _scatter(vd, lens, P, 2)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    Wn, sink = 64, 4
    scale = 1.0 / np.sqrt(d)
    lse_p = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    lse_d = torch.empty_like(lse_p)
    qb = I.bf16_bits(q)
    for variant in ("full", "windowed"):
        if variant == "full":
            op = W.paged_attn_full_fp8(q, kp, vp, table, lt, ks, vs, lse=lse_p, err=err)
            od = W.draft_attn_full_fp8(q, kd, vd, lt, ks, vs, lse=lse_d)
        else:
            op = W.paged_attn_windowed_fp8(q, kp, vp, table, lt, Wn, sink, ks, vs, lse=lse_p, err=err)
            od = W.draft_attn_windowed_fp8(q, kd, vd, lt, Wn, sink, ks, vs, lse=lse_d)
        torch.cuda.synchronize()
        assert torch.equal(op, od), variant
        assert torch.equal(lse_p, lse_d), variant
        kv = F.DequantizedRows(_HostCodes(kp), ks), F.DequantizedRows(_HostCodes(vp), vs)
        refs = [Pg.attend_paged(qb[b], kv[0], kv[1], table[b].cpu().numpy(), S, scale, variant, Wn, sink,
                                spread=True) for b, S in enumerate(lens)]
        G.assert_attn_close(op, np.stack([r[0] for r in refs]), lse_p, np.stack([r[1] for r in refs]),
                            what=f"paged fp8 {variant}", spread=np.stack([r[2] for r in refs]))
        assert torch.count_nonzero(op[0]) == 0
    assert err.item() == 0
    # a table entry outside the pool is flagged
    bad = table.clone()
    bad[7, 11] = P + 5
    W.paged_attn_full_fp8(q, kp, vp, bad, lt, ks, vs, err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_SLOT_RANGE
