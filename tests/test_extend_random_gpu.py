"""GPU parity of the full-context draft-extend over seeded random shapes of
moderate length (thousands to tens of thousands of keys), where rows have
many work items: the multi-row kernel with items sized per sequence, its
loads issued a step ahead, and the merge on its wide (1024-thread), middle
(512-thread, 128-wide slices) or row (256-thread) shape, whichever the grid
gives.  Ragged new-row counts, G from 1 to 16, d = 128 and 256, both cache
types; every output and lse against the float64 oracle (elementwise bound as
in tests/_gpu.py).
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import fp8 as F
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


class _HostCodes:
    """Host view of one sequence of a device fp8 cache: rows' codes as numpy."""

    def __init__(self, t):
        self.t = t
        self.shape = tuple(t.shape)

    def __getitem__(self, rows):
        idx = torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int64)).to(self.t.device)
        return self.t.index_select(0, idx).cpu().numpy()


def _case(seed):
    rng = np.random.default_rng(7000 + seed)
    d = int(rng.choice([128, 256]))
    Hkv = int(rng.choice([1, 2]))
    Gq = int(rng.choice([1, 4, 8, 16]))
    B = int(rng.integers(1, 3))
    q_max = int(rng.integers(2, 9))
    lens = [int(rng.integers(3000, 40000)) for _ in range(B)]
    n_q = [int(rng.integers(1, q_max + 1)) for _ in range(B)]
    return d, Hkv, Gq, B, q_max, lens, n_q


# Fixed shapes for the merge shapes the seeds above do not reach: 2 x 8 rows
# at Hq = 32, d = 256 (the row shape), and an fp8 cache with 8 rows at
# Hq = 32 (the middle shape).
FIXED = {"row": (256, 2, 16, 2, 8, [9001, 30011], [8, 5]), "mid_fp8": (256, 2, 16, 1, 8, [20003], [8])}


@pytest.mark.parametrize("seed", list(range(10)) + ["row"])
def test_random_full_extend_vs_oracle(dev, seed):
    d, Hkv, Gq, B, q_max, lens, n_q = FIXED[seed] if seed in FIXED else _case(seed)
    Hq = Hkv * Gq
    S_max = max(lens) + 5
    scale = 1.0 / np.sqrt(d)
    G.say(f"random extend {seed}: d={d} Hq={Hq} Hkv={Hkv} B={B} q_max={q_max} lens={lens} n_q={n_q}")
    sd = 50 if isinstance(seed, str) else seed
    q = I.normal_bf16((B, q_max, Hq, d), 90 + sd, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), 91 + sd, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 92 + sd, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    err = G.err_word(dev)
    lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
    out = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse, err=err)
    torch.cuda.synchronize()
    qb = I.bf16_bits(q)
    o_ref, l_ref, spread = [], [], []
    for b in range(B):
        K, V = G.HostRows(k[b]), G.HostRows(v[b])
        o, l = A.attend_extend(qb[b], K, V, lens[b], n_q[b], scale, "full")
        o_ref.append(o)
        l_ref.append(l)
        spread.append(A.extend_spread(qb[b], K, V, lens[b], n_q[b], scale, "full"))
    G.assert_attn_close(out, np.stack(o_ref), lse, np.stack(l_ref), what=f"random extend {seed}",
                        spread=np.stack(spread))
    assert err.item() == 0


@pytest.mark.parametrize("seed", list(range(4)) + ["mid_fp8"])
def test_random_full_extend_fp8_vs_oracle(dev, seed):
    d, Hkv, Gq, B, q_max, lens, n_q = FIXED[seed] if seed in FIXED else _case(100 + seed)
    Hq = Hkv * Gq
    S_max = max(lens) + 5
    scale, ks, vs = 1.0 / np.sqrt(d), 0.5, 1.25
    G.say(f"random fp8 extend {seed}: d={d} Hq={Hq} Hkv={Hkv} B={B} q_max={q_max} lens={lens} n_q={n_q}")
    sd = 50 if isinstance(seed, str) else seed
    q = I.normal_bf16((B, q_max, Hq, d), 95 + sd, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 96 + sd, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 97 + sd, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
    out = W.draft_extend_full_fp8(q, k8, v8, lt, ks, vs, n_q=nt, lse=lse)
    torch.cuda.synchronize()
    qb = I.bf16_bits(q)
    for b in range(B):
        for t in range(q_max):
            if t >= n_q[b]:  # padding rows: zeros and -inf
                assert torch.count_nonzero(out[b, t]) == 0
                assert torch.isneginf(lse[b, t]).all()
                continue
            L = lens[b] - n_q[b] + t + 1
            o, l, sp = F.attend_sequence_fp8(qb[b, t], _HostCodes(k8[b]), _HostCodes(v8[b]), L, scale, ks, vs,
                                             "full", spread=True)
            G.assert_attn_close(out[b, t], o, lse[b, t], l, what=f"random fp8 extend {seed} row ({b}, {t})",
                                spread=sp)
