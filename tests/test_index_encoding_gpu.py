"""Closed-form index-encoding checks: the kernels read exactly the rows the
selection rule names, at the real shapes (Hq=32, Hkv=2, d=256) up to 1M keys.

With every key zero, every kept key gets weight exactly 1/n (all logits are
0), so the output is the mean of the kept value rows and lse = ln(n).  The
value rows encode their own position:
  * residue code (windowed and ring, any length): channel c < 127 is
    [(p + 37 g) mod 127 == c], channel 127 + c is [(p + 41 g) mod 128 == c]
    for KV head g, channel 255 is 1.  Each output channel is an exact count
    over the kept positions divided by n; a wrong, stale or missing row moves
    at least two counts by one (>= 6% at n = 2052).
  * block code (full, 1M keys): channel c is [p * d // S == c] (+ g shift);
    a skipped or repeated work item shows in its channel, and lse must equal
    ln(S) within 3 float32 ulps, which pins the number of keys read to a few.
Expected values are exact counts computed here from the oracle's selection.
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

Hq, Hkv, d = 32, 2, 256


@pytest.fixture(scope="module")
def dev():
    return G.device()


def _residue_rows(pos, dev):
    """Value rows [len(pos), Hkv, d] bf16 encoding each position."""
    p = torch.as_tensor(np.asarray(pos, dtype=np.int64), device=dev)
    out = torch.zeros((p.numel(), Hkv, d), dtype=torch.bfloat16, device=dev)
    c = torch.arange(128, device=dev)
    for g in range(Hkv):
        out[:, g, :127] = (((p + 37 * g) % 127)[:, None] == c[None, :127]).to(torch.bfloat16)
        out[:, g, 127:255] = (((p + 41 * g) % 128)[:, None] == c[None, :128]).to(torch.bfloat16)
        out[:, g, 255] = 1.0
    return out


def _residue_expected(positions):
    e = np.zeros((Hkv, d))
    n = len(positions)
    p = np.asarray(positions, dtype=np.int64)
    for g in range(Hkv):
        e[g, :127] = np.bincount((p + 37 * g) % 127, minlength=127)
        e[g, 127:255] = np.bincount((p + 41 * g) % 128, minlength=128)
        e[g, 255] = n
    return e / n


def _check_exact(out, exp_per_kv, what):
    """out [Hq, d] bf16 vs exact expected values: within one bf16 ulp."""
    o = out.float().cpu().numpy().astype(np.float64)
    G_ = Hq // Hkv
    ref = np.repeat(exp_per_kv, G_, axis=0)
    ulp = np.where(ref > 0, 2.0 ** (np.floor(np.log2(np.maximum(ref, 1e-30))) - 7), 0.0)
    bad = np.abs(o - ref) > ulp
    assert not bad.any(), f"{what}: {bad.sum()} channels off, first at {np.argwhere(bad)[:4].tolist()}"


@pytest.mark.parametrize("S", [1, 3, 2052, 2053, 5000, 131075, 1048576 + 7])
def test_windowed_reads_the_right_rows(dev, S, wpath):
    G.say(f"index encoding windowed S={S}")
    sink, Wn = 4, 2048
    S_max = S
    k = torch.zeros((1, S_max, Hkv, d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    keep = A.selected_positions(S, Wn, sink)
    v[0, torch.as_tensor(keep, device=dev)] = _residue_rows(keep, dev)
    # rows outside the key set carry a poison code (a different residue)
    drop = np.setdiff1d(np.arange(max(0, S - 3 * Wn), S), keep)[:4096]
    if drop.size:
        v[0, torch.as_tensor(drop, device=dev)] = _residue_rows(drop + 5, dev)
    q = I.normal_bf16((1, Hq, d), 3, dev)
    lse = torch.empty((1, Hq), dtype=torch.float32, device=dev)
    out = W.draft_attn_windowed(q, k, v, G.lens_tensor([S], dev), Wn, sink, lse=lse)
    torch.cuda.synchronize()
    _check_exact(out[0], _residue_expected(keep), f"windowed S={S}")
    assert np.allclose(lse.cpu().numpy(), np.log(keep.size), rtol=0, atol=4e-6)


@pytest.mark.parametrize("S", [5, 2052, 2060, 4100, 1048576 + 3])
@pytest.mark.parametrize("R_w", [2048, 2056])
def test_ring_reads_the_right_slots(dev, S, R_w, wpath):
    G.say(f"index encoding ring S={S} R_w={R_w}")
    sink, Wn = 4, 2048
    kr = torch.zeros((1, sink + R_w, Hkv, d), dtype=torch.bfloat16, device=dev)
    # every slot holds the newest position that maps to it (what appends leave)
    live = np.array([p for p in range(max(0, S - R_w - sink), S) if p < sink or p >= S - R_w])
    live = np.union1d(np.arange(min(sink, S)), live)
    slots = R.ring_slots(live, sink, R_w)
    vr = torch.zeros_like(kr)
    vr[0, torch.as_tensor(slots, device=dev)] = _residue_rows(live, dev)
    q = I.normal_bf16((1, Hq, d), 4, dev)
    lse = torch.empty((1, Hq), dtype=torch.float32, device=dev)
    out = W.ring_attn(q, kr, vr, G.lens_tensor([S], dev), Wn, sink, R_w, lse=lse)
    torch.cuda.synchronize()
    keep = A.selected_positions(S, Wn, sink)
    _check_exact(out[0], _residue_expected(keep), f"ring S={S} R_w={R_w}")


@pytest.mark.parametrize("S", [700, 4096])
def test_full_small_reads_every_row(dev, S):
    k = torch.zeros((1, S + 9, Hkv, d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    v[0, :S] = _residue_rows(np.arange(S), dev)
    v[0, S:] = _residue_rows(np.arange(S, S + 9) + 11, dev)  # beyond the length: never read
    q = I.normal_bf16((1, Hq, d), 5, dev)
    out = W.draft_attn_full(q, k, v, G.lens_tensor([S], dev))
    torch.cuda.synchronize()
    _check_exact(out[0], _residue_expected(np.arange(S)), f"full S={S}")


def test_full_1m_block_code_and_count(dev):
    S = 1 << 20
    G.say("index encoding full S=1M")
    k = torch.zeros((1, S, Hkv, d), dtype=torch.bfloat16, device=dev)
    v = torch.zeros_like(k)
    p = torch.arange(S, device=dev)
    blk = (p * d) // S  # 4096 keys per channel
    for g in range(Hkv):
        v[0, :, g, :] = (((blk + 7 * g) % d)[:, None] == torch.arange(d, device=dev)[None, :]).to(torch.bfloat16)
    q = I.normal_bf16((1, Hq, d), 6, dev)
    lse = torch.empty((1, Hq), dtype=torch.float32, device=dev)
    out = W.draft_attn_full(q, k, v, G.lens_tensor([S], dev), lse=lse)
    torch.cuda.synchronize()
    exp = np.zeros((Hkv, d))
    pn = np.arange(S, dtype=np.int64)
    for g in range(Hkv):
        exp[g] = np.bincount(((pn * d) // S + 7 * g) % d, minlength=d) / S
    _check_exact(out[0], exp, "full 1M")
    ln_s = np.float32(np.log(S))
    ulp = np.spacing(ln_s)
    assert np.all(np.abs(lse.cpu().numpy().astype(np.float64) - np.log(S)) <= 3 * ulp)
