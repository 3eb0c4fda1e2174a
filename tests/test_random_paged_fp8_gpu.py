"""GPU parity over seeded random shapes for the paged token pool (page size
1) and the fp8 (E4M3) caches: GQA groups from 1 to 16, 1 to 8 KV heads,
every head size, batches with empty, short, threshold and long sequences,
windows and sinks of any size.

* paged attention (bf16 and fp8 pools, full and windowed, rows scattered
  over a shuffled pool) equals the dense call over the same rows bit for
  bit, and the oracle's paged attention within the elementwise bound of
  tests/_gpu.py;
* fp8 full, windowed and ring attention against the oracle over the
  dequantized rows, ring == windowed bit for bit;
* fp8 draft-extends (ragged new-row counts, empty sequences): full and
  windowed against the oracle, the ring extend (ring of W + q_max - 1 rows)
  == the windowed extend bit for bit.

Both windowed paths (one launch, split + merge) run every case.
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import fp8 as F
from oracle import paged as Pg
from oracle import ring as R
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


def _case(seed):
    rng = np.random.default_rng(5000 + seed)
    d = int(rng.choice([64, 128, 256]))
    Hkv = int(rng.choice([1, 2, 3, 4, 8]))
    Gq = int(rng.integers(1, 17))
    B = int(rng.integers(1, 6))
    W_ = int(rng.choice([1, 3, 64, 100, 513, 2048]))
    sink = int(rng.choice([0, 1, 4, 9]))
    th = sink + W_
    pool = [0, 1, 2, th - 1, th, th + 1, 700, 4001, 9000]
    lens = [max(0, int(rng.choice(pool))) for _ in range(B)]
    return d, Hkv, Gq, B, W_, sink, lens


class _HostCodes:
    """Host view of a device fp8 tensor's rows: codes as numpy."""

    def __init__(self, t):
        self.t = t
        self.shape = tuple(t.shape)

    def __getitem__(self, rows):
        idx = torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int64)).to(self.t.device)
        return self.t.index_select(0, idx).cpu().numpy()


def _scatter(dense, lens, P, seed):
    """Pool [P, Hkv, d] holding every sequence's rows at distinct random slots,
    and the table [B, C] naming them (torch copies only)."""
    B, C = dense.shape[:2]
    g = torch.Generator(device="cpu").manual_seed(seed)
    table = torch.randperm(P, generator=g)[: B * C].view(B, C).to(torch.int32).to(dense.device)
    pool = torch.zeros((P,) + tuple(dense.shape[2:]), dtype=dense.dtype, device=dense.device)
    for b, S in enumerate(lens):
        if S:
            pool[table[b, :S].long()] = dense[b, :S]
    return pool, table


def _ring_from_dense(x, lens, sink, R_w):
    B, _, Hkv, d = x.shape
    ring = torch.zeros((B, sink + R_w, Hkv, d), dtype=x.dtype, device=x.device)
    for b, S in enumerate(lens):
        live = [p for p in range(S) if p < sink or p >= S - R_w]
        if live:
            ring[b, torch.as_tensor(R.ring_slots(live, sink, R_w), device=x.device)] = \
                x[b, torch.as_tensor(live, device=x.device)]
    return ring


def _check_paged(dev, seed, fp8, wpath):
    d, Hkv, Gq, B, W_, sink, lens = _case(seed + (100 if fp8 else 0))
    Hq = Hkv * Gq
    C = max(lens) + 3
    P = B * C + 101
    scale = 1.0 / np.sqrt(d)
    ks, vs = 0.625, 1.75
    G.say(f"random paged {'fp8 ' if fp8 else ''}{seed}: d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} lens={lens} "
          f"path={wpath}")
    q = I.normal_bf16((B, Hq, d), 300 + seed, dev)
    gen = I.normal_fp8 if fp8 else I.normal_bf16
    kd, vd = gen((B, C, Hkv, d), 301 + seed, dev), gen((B, C, Hkv, d), 302 + seed, dev)
    kp, table = _scatter(kd, lens, P, 17 + seed)
    vp, _ = _scatter(vd, lens, P, 17 + seed)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    qb = I.bf16_bits(q)
    if fp8:
        kv = F.DequantizedRows(_HostCodes(kp), ks), F.DequantizedRows(_HostCodes(vp), vs)
    else:
        kv = G.HostRows(kp), G.HostRows(vp)
    for variant in ("full", "windowed"):
        lse_p = torch.empty(B, Hq, dtype=torch.float32, device=dev)
        lse_d = torch.empty_like(lse_p)
        if fp8 and variant == "full":
            op = W.paged_attn_full_fp8(q, kp, vp, table, lt, ks, vs, lse=lse_p, err=err)
            od = W.draft_attn_full_fp8(q, kd, vd, lt, ks, vs, lse=lse_d)
        elif fp8:
            op = W.paged_attn_windowed_fp8(q, kp, vp, table, lt, W_, sink, ks, vs, lse=lse_p, err=err)
            od = W.draft_attn_windowed_fp8(q, kd, vd, lt, W_, sink, ks, vs, lse=lse_d)
        elif variant == "full":
            op = W.paged_attn_full(q, kp, vp, table, lt, lse=lse_p, err=err)
            od = W.draft_attn_full(q, kd, vd, lt, lse=lse_d)
        else:
            op = W.paged_attn_windowed(q, kp, vp, table, lt, W_, sink, lse=lse_p, err=err)
            od = W.draft_attn_windowed(q, kd, vd, lt, W_, sink, lse=lse_d)
        torch.cuda.synchronize()
        what = f"paged {'fp8 ' if fp8 else ''}{seed} {variant}"
        assert torch.equal(op, od) and torch.equal(lse_p, lse_d), f"{what}: paged != dense"
        table_h = table.cpu().numpy()
        refs = [Pg.attend_paged(qb[b], kv[0], kv[1], table_h[b], S, scale, variant, W_, sink, spread=True)
                for b, S in enumerate(lens)]
        G.assert_attn_close(op, np.stack([r[0] for r in refs]), lse_p, np.stack([r[1] for r in refs]),
                            what=what, spread=np.stack([r[2] for r in refs]))
    assert err.item() == 0, f"paged {seed}: device error word {err.item():#x}"


@pytest.mark.parametrize("seed", range(12))
def test_random_paged_vs_dense_and_oracle(dev, seed, wpath):
    _check_paged(dev, seed, False, wpath)


@pytest.mark.parametrize("seed", range(12))
def test_random_paged_fp8_vs_dense_and_oracle(dev, seed, wpath):
    _check_paged(dev, seed, True, wpath)


@pytest.mark.parametrize("seed", range(12))
def test_random_fp8_cache_vs_oracle(dev, seed, wpath):
    d, Hkv, Gq, B, W_, sink, lens = _case(200 + seed)
    Hq = Hkv * Gq
    S_max = max(lens) + 3
    scale = 1.0 / np.sqrt(d)
    ks, vs = 0.375, 2.5
    G.say(f"random fp8 {seed}: d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} lens={lens} path={wpath}")
    q = I.normal_bf16((B, Hq, d), 400 + seed, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 401 + seed, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 402 + seed, dev)
    R_w = W_ + 2
    kr, vr = _ring_from_dense(k8, lens, sink, R_w), _ring_from_dense(v8, lens, sink, R_w)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    qb = I.bf16_bits(q)
    outs = {}
    for variant in ("full", "windowed", "ring"):
        lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_attn_full_fp8(q, k8, v8, lt, ks, vs, lse=lse, err=err)
        elif variant == "windowed":
            out = W.draft_attn_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, lse=lse, err=err)
        else:
            out = W.ring_attn_fp8(q, kr, vr, lt, W_, sink, R_w, ks, vs, lse=lse, err=err)
        torch.cuda.synchronize()
        outs[variant] = (out, lse)
        ref_variant = "full" if variant == "full" else "windowed"
        refs = [F.attend_sequence_fp8(qb[b], _HostCodes(k8[b]), _HostCodes(v8[b]), S, scale, ks, vs, ref_variant,
                                      W_, sink, spread=True) for b, S in enumerate(lens)]
        G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                            what=f"random fp8 {seed} {variant}", spread=np.stack([r[2] for r in refs]))
    assert torch.equal(outs["ring"][0], outs["windowed"][0]), f"random fp8 {seed}: ring != windowed"
    assert torch.equal(outs["ring"][1], outs["windowed"][1]), f"random fp8 {seed}: ring lse != windowed"
    assert err.item() == 0, f"random fp8 {seed}: device error word {err.item():#x}"


@pytest.mark.parametrize("seed", range(10))
def test_random_fp8_extend_vs_oracle(dev, seed, wpath):
    d, Hkv, Gq, B, W_, sink, lens = _case(300 + seed)
    rng = np.random.default_rng(9000 + seed)
    q_max = int(rng.integers(1, 9))
    n_q = [min(int(rng.integers(1, q_max + 1)), S) for S in lens]
    Hq = Hkv * Gq
    S_max = max(lens) + 3
    scale = 1.0 / np.sqrt(d)
    ks, vs = 0.875, 1.125
    G.say(f"random fp8 extend {seed}: d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} lens={lens} n_q={n_q} "
          f"path={wpath}")
    q = I.normal_bf16((B, q_max, Hq, d), 500 + seed, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 501 + seed, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 502 + seed, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    err = G.err_word(dev)
    qb = I.bf16_bits(q)
    rows = [(F.DequantizedRows(_HostCodes(k8[b]), ks), F.DequantizedRows(_HostCodes(v8[b]), vs)) for b in range(B)]
    outs = {}
    for variant in ("full", "windowed"):
        lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_extend_full_fp8(q, k8, v8, lt, ks, vs, n_q=nt, lse=lse, err=err)
        else:
            out = W.draft_extend_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, n_q=nt, lse=lse, err=err)
        torch.cuda.synchronize()
        outs[variant] = (out, lse)
        o_ref, l_ref, spread = [], [], []
        for b in range(B):
            if n_q[b] == 0:  # an empty sequence: every row is padding
                o_ref.append(np.zeros((q_max, Hq, d)))
                l_ref.append(np.full((q_max, Hq), -np.inf))
                spread.append(np.zeros((q_max, Hq, d)))
                continue
            o, l = A.attend_extend(qb[b], *rows[b], lens[b], n_q[b], scale, variant, W_, sink)
            o_ref.append(o)
            l_ref.append(l)
            spread.append(A.extend_spread(qb[b], *rows[b], lens[b], n_q[b], scale, variant, W_, sink))
        G.assert_attn_close(out, np.stack(o_ref), lse, np.stack(l_ref), what=f"random fp8 extend {seed} {variant}",
                            spread=np.stack(spread))
    R_w = W_ + q_max - 1
    kr, vr = _ring_from_dense(k8, lens, sink, R_w), _ring_from_dense(v8, lens, sink, R_w)
    lse_r = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
    orr = W.ring_extend_fp8(q, kr, vr, lt, W_, sink, R_w, ks, vs, n_q=nt, lse=lse_r, err=err)
    torch.cuda.synchronize()
    assert torch.equal(orr, outs["windowed"][0]), f"random fp8 extend {seed}: ring != windowed"
    assert torch.equal(lse_r, outs["windowed"][1]), f"random fp8 extend {seed}: ring lse != windowed"
    assert err.item() == 0, f"random fp8 extend {seed}: device error word {err.item():#x}"
