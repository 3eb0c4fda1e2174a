"""GPU parity over seeded random shapes: GQA groups of every size from 1 to
16 (including ones that do not divide the 16-wide MFMA tile), 1 to 8 KV
heads, every head size, batches with empty, short, threshold and long
sequences, windows and sinks of any size, and draft-extends with ragged row
counts; full, windowed, ring and both extend forms against the float64
oracle (elementwise bound as in tests/_gpu.py), and ring == windowed bit for
bit.  Each case is small enough for the oracle to run in well under a
second.
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


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    d = int(rng.choice([64, 128, 256]))
    Hkv = int(rng.choice([1, 2, 3, 4, 8]))
    Gq = int(rng.integers(1, 17))
    B = int(rng.integers(1, 5))
    W_ = int(rng.choice([1, 2, 7, 64, 100, 513]))
    sink = int(rng.choice([0, 1, 4, 9]))
    q_max = int(rng.integers(1, 7))
    th = sink + W_
    pool = [0, 1, 2, q_max, th - 1, th, th + 1, th + 2, 300, 1500, 2999]
    lens = [max(0, int(rng.choice(pool))) for _ in range(B)]
    n_q = [int(rng.integers(1, q_max + 1)) if S else 0 for S in lens]
    n_q = [min(n, S) for n, S in zip(n_q, lens)]
    return d, Hkv, Gq, B, W_, sink, q_max, lens, n_q


def _ring_from_dense(k, lens, sink, R_w):
    B, _, Hkv, d = k.shape
    ring = torch.zeros((B, sink + R_w, Hkv, d), dtype=k.dtype, device=k.device)
    for b, S in enumerate(lens):
        live = [p for p in range(S) if p < sink or p >= S - R_w]
        if live:
            ring[b, torch.as_tensor(R.ring_slots(live, sink, R_w), device=k.device)] = \
                k[b, torch.as_tensor(live, device=k.device)]
    return ring


@pytest.mark.parametrize("seed", range(40))
def test_random_shape_vs_oracle(dev, seed, wpath):
    d, Hkv, Gq, B, W_, sink, q_max, lens, n_q = _case(seed)
    Hq = Hkv * Gq
    S_max = max(lens) + 3
    scale = 1.0 / np.sqrt(d)
    G.say(f"random case {seed}: d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} lens={lens} q_max={q_max} n_q={n_q}")
    q = I.normal_bf16((B, Hq, d), 50 + seed, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), 51 + seed, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 52 + seed, dev)
    lt = G.lens_tensor(lens, dev)
    err = G.err_word(dev)
    qb = I.bf16_bits(q)

    # single-row calls
    R_w = W_ + q_max - 1
    kr, vr = _ring_from_dense(k, lens, sink, R_w), _ring_from_dense(v, lens, sink, R_w)
    outs = {}
    for variant in ("full", "windowed", "ring"):
        lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_attn_full(q, k, v, lt, lse=lse, err=err)
        elif variant == "windowed":
            out = W.draft_attn_windowed(q, k, v, lt, W_, sink, lse=lse, err=err)
        else:
            out = W.ring_attn(q, kr, vr, lt, W_, sink, R_w, lse=lse, err=err)
        torch.cuda.synchronize()
        outs[variant] = out
        ref_variant = "full" if variant == "full" else "windowed"
        refs = [G.oracle_seq(qb[b], k[b], v[b], lens[b], scale, ref_variant, W_, sink, spread=True)
                for b in range(B)]
        G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                            what=f"case {seed} {variant}", spread=np.stack([r[2] for r in refs]))
    assert torch.equal(outs["ring"], outs["windowed"]), f"case {seed}: ring != windowed"

    # draft-extend over n_q[b] causal rows (full and windowed)
    qx = I.normal_bf16((B, q_max, Hq, d), 53 + seed, dev)
    nt = G.lens_tensor(n_q, dev)
    qxb = I.bf16_bits(qx)
    for variant in ("full", "windowed"):
        lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_extend_full(qx, k, v, lt, n_q=nt, lse=lse, err=err)
        else:
            out = W.draft_extend_windowed(qx, k, v, lt, W_, sink, n_q=nt, lse=lse, err=err)
        torch.cuda.synchronize()
        o_ref, l_ref, spread = [], [], []
        for b in range(B):
            K, V = G.HostRows(k[b]), G.HostRows(v[b])
            if n_q[b] == 0:  # an empty sequence: every row is padding
                o_ref.append(np.zeros((q_max, Hq, d)))
                l_ref.append(np.full((q_max, Hq), -np.inf))
                spread.append(np.zeros((q_max, Hq, d)))
                continue
            o, l = A.attend_extend(qxb[b], K, V, lens[b], n_q[b], scale, variant, W_, sink)
            o_ref.append(o)
            l_ref.append(l)
            spread.append(A.extend_spread(qxb[b], K, V, lens[b], n_q[b], scale, variant, W_, sink))
        G.assert_attn_close(out, np.stack(o_ref), lse, np.stack(l_ref), what=f"case {seed} extend {variant}",
                            spread=np.stack(spread))
    assert err.item() == 0, f"case {seed}: device error word {err.item():#x}"
