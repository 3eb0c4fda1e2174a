"""GPU parity of speculative draft rows: chain rollback and tree-width rings.

* chain: speculative rows appended to the ring (lens advancing), attention
  after each, rollback of the rejected rows, a bonus row; every output
  against the oracle's logical sequences (oracle.spec.SpecSequences) over
  many rounds with random accept counts per request, R_w = W + gamma;
* tree: width-k candidates written with tree_append (candidate 0 in place,
  the others in private runs), every candidate's attention against the
  oracle after each draft step, then the verify: depth reset, the accepted
  candidate's rows plus a bonus row appended and attended by the
  draft-extend (ring_extend) -- against the oracle, over many rounds;
* the chain and tree rounds over seeded random shapes (gamma 1-8, widths
  1-6, depths 1-8, windows down to one key, sinks from none, G 1-16);
* a width-1 tree equals the chain path bit for bit;
* a request at the largest depth is flagged and left unchanged.
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import spec as P
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


class Rows:
    """Seeded bf16 rows [B, n, Hkv, d] (device) with their host bit patterns."""

    def __init__(self, dev, Hkv, d):
        self.dev, self.Hkv, self.d, self.seed = dev, Hkv, d, 7000

    def draw(self, B, n):
        self.seed += 2
        k = I.normal_bf16((B, n, self.Hkv, self.d), self.seed, self.dev)
        v = I.normal_bf16((B, n, self.Hkv, self.d), self.seed + 1, self.dev)
        return k, v, I.bf16_bits(k), I.bf16_bits(v)


def _check(out, lse, refs, what):
    o_ref = np.stack([r[0] for r in refs])
    l_ref = np.stack([r[1] for r in refs])
    G.assert_attn_close(out, o_ref, lse, l_ref, what=what, spread=np.stack([r[2] for r in refs]))


def _prefill(dev, rows, kr, vr, lens, seqs, S0, sink, R_w):
    """Committed prompt rows through the bulk ring append (oracle: verify)."""
    B = len(S0)
    n_max = max(S0)
    k, v, kb, vb = rows.draw(B, n_max)
    W.ring_append(kr, vr, k, v, G.lens_tensor(S0, dev), lens, sink, R_w)
    for b in range(B):
        seqs[b].verify([(kb[b, i], vb[b, i]) for i in range(S0[b])])


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2)])
def test_chain_speculate_rollback(dev, d, Hq, Hkv, wpath):
    _chain_rounds(dev, d, Hq, Hkv, 64, 4, 5, [0, 3, 70, 250], 30, d)


@pytest.mark.parametrize("seed", range(6))
def test_chain_random_shapes(dev, seed, wpath):
    """The chain rounds over seeded random shapes: gamma 1-8, windows down to
    one key, sinks from none, G from 1 to 16."""
    rng = np.random.default_rng(8500 + seed)
    d = int(rng.choice([64, 128, 256]))
    Hkv = int(rng.choice([1, 2, 4]))
    Hq = Hkv * int(rng.integers(1, 17))
    gamma = int(rng.integers(1, 9))
    Wn = int(rng.choice([1, 2, 5, 64, 129]))
    sink = int(rng.choice([0, 1, 4, 7]))
    S0 = [int(rng.choice([0, 1, sink + 1, sink + Wn, sink + Wn + 3, 250])) for _ in range(int(rng.integers(1, 5)))]
    S0[-1] = max(S0[-1], 1)  # at least one prompt row drawn
    G.say(f"random chain {seed}: d={d} Hq={Hq} Hkv={Hkv} gamma={gamma} W={Wn} sink={sink} S0={S0}")
    _chain_rounds(dev, d, Hq, Hkv, Wn, sink, gamma, S0, 10, 55 + seed)


def _chain_rounds(dev, d, Hq, Hkv, Wn, sink, gamma, S0, n_rounds, seed):
    B = len(S0)
    R_w = Wn + gamma
    scale = 1.0 / np.sqrt(d)
    rows = Rows(dev, Hkv, d)
    rng = np.random.default_rng(seed)
    kr = torch.zeros((B, sink + R_w, Hkv, d), dtype=torch.bfloat16, device=dev)
    vr = torch.zeros_like(kr)
    lens = G.lens_tensor([0] * B, dev)
    err = G.err_word(dev)
    seqs = [P.SpecSequences(1) for _ in range(B)]
    _prefill(dev, rows, kr, vr, lens, seqs, S0, sink, R_w)
    ones = G.lens_tensor([1] * B, dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    for rnd in range(n_rounds):
        G.say(f"chain d={d} round {rnd}")
        for j in range(gamma):
            k, v, kb, vb = rows.draw(B, 1)
            W.ring_append(kr, vr, k, v, ones, lens, sink, R_w, err=err)
            q = I.normal_bf16((B, Hq, d), 100 * rnd + j, dev)
            out = W.ring_attn(q, kr, vr, lens, Wn, sink, R_w, lse=lse, err=err)
            torch.cuda.synchronize()
            qb = I.bf16_bits(q)
            refs = []
            for b in range(B):
                seqs[b].speculate([(kb[b, 0], vb[b, 0])])
                refs.append(seqs[b].attend(qb[b], 0, scale, Wn, sink, spread=True))
            _check(out, lse, refs, f"chain round {rnd} step {j}")
        acc = rng.integers(0, gamma + 1, size=B)
        W.ring_rollback(lens, G.lens_tensor(gamma - acc, dev), err=err)
        k, v, kb, vb = rows.draw(B, 1)  # the bonus token's row
        W.ring_append(kr, vr, k, v, ones, lens, sink, R_w, err=err)
        q = I.normal_bf16((B, Hq, d), 100 * rnd + 99, dev)
        out = W.ring_attn(q, kr, vr, lens, Wn, sink, R_w, lse=lse, err=err)
        torch.cuda.synchronize()
        qb = I.bf16_bits(q)
        refs = []
        for b in range(B):
            kept = seqs[b].spec[0][: acc[b]] + [(kb[b, 0], vb[b, 0])]
            seqs[b].verify(kept)
            refs.append(seqs[b].attend(qb[b], 0, scale, Wn, sink, spread=True))
        _check(out, lse, refs, f"chain round {rnd} after rollback")
        assert lens.cpu().numpy().tolist() == [s.S for s in seqs]
    assert err.item() == 0


def _tree_state(dev, B, width, dd, Hkv, d, sink, R_w):
    kr = torch.zeros((B, sink + R_w, Hkv, d), dtype=torch.bfloat16, device=dev)
    vr = torch.zeros_like(kr)
    kb = torch.zeros((B, max(width - 1, 0) * dd, Hkv, d), dtype=torch.bfloat16, device=dev)
    vb = torch.zeros_like(kb)
    return kr, vr, kb, vb


@pytest.mark.parametrize("d,Hq,Hkv,width,dd", [(128, 16, 2, 3, 4), (256, 32, 2, 4, 3), (64, 6, 2, 2, 7)])
def test_tree_candidates_and_verify(dev, d, Hq, Hkv, width, dd, wpath):
    _tree_rounds(dev, d, Hq, Hkv, width, dd, 64, 4, [2, 66, 300], 20, width * 10 + dd)


def _random_tree_case(seed):
    rng = np.random.default_rng(8000 + seed)
    d = int(rng.choice([64, 128, 256]))
    Hkv = int(rng.choice([1, 2, 4]))
    Gq = int(rng.integers(1, 17))
    width = int(rng.integers(1, 7))
    dd = int(rng.integers(1, 9))
    Wn = int(rng.choice([1, 2, 5, 64, 129]))
    sink = int(rng.choice([0, 1, 4, 7]))
    B = int(rng.integers(1, 5))
    S0 = [int(rng.choice([1, 2, sink + 1, sink + Wn, sink + Wn + 3, 250])) for _ in range(B)]
    return d, Hkv * Gq, Hkv, width, dd, Wn, sink, S0


@pytest.mark.parametrize("seed", range(8))
def test_tree_random_shapes(dev, seed, wpath):
    """The tree rounds over seeded random shapes: widths 1-6, depths 1-8,
    windows down to one key, sinks from none, G from 1 to 16."""
    d, Hq, Hkv, width, dd, Wn, sink, S0 = _random_tree_case(seed)
    G.say(f"random tree {seed}: d={d} Hq={Hq} Hkv={Hkv} width={width} depth_max={dd} W={Wn} sink={sink} S0={S0}")
    _tree_rounds(dev, d, Hq, Hkv, width, dd, Wn, sink, S0, 8, 77 + seed)


def _tree_rounds(dev, d, Hq, Hkv, width, dd, Wn, sink, S0, n_rounds, seed):
    B = len(S0)
    R_w = Wn + dd
    scale = 1.0 / np.sqrt(d)
    rows = Rows(dev, Hkv, d)
    rng = np.random.default_rng(seed)
    kr, vr, kbr, vbr = _tree_state(dev, B, width, dd, Hkv, d, sink, R_w)
    lens = G.lens_tensor([0] * B, dev)
    depth = G.lens_tensor([0] * B, dev)
    err = G.err_word(dev)
    seqs = [P.SpecSequences(width) for _ in range(B)]
    _prefill(dev, rows, kr, vr, lens, seqs, S0, sink, R_w)
    lse = torch.empty((B, width, Hq), dtype=torch.float32, device=dev)
    for rnd in range(n_rounds):
        G.say(f"tree d={d} width={width} dd={dd} round {rnd}")
        n_steps = int(rng.integers(1, dd + 1))
        for i in range(n_steps):
            k, v, kb, vb = rows.draw(B, width)
            W.tree_append(kr, vr, kbr, vbr, k, v, lens, depth, Wn, sink, R_w, dd, err=err)
            q = I.normal_bf16((B, width, Hq, d), 1000 * rnd + i, dev)
            out = W.tree_attn(q, kr, vr, kbr, vbr, lens, depth, Wn, sink, R_w, dd, lse=lse, err=err)
            torch.cuda.synchronize()
            qb = I.bf16_bits(q)
            refs = []
            for b in range(B):
                seqs[b].speculate([(kb[b, c], vb[b, c]) for c in range(width)])
                refs.append([seqs[b].attend(qb[b, c], c, scale, Wn, sink, spread=True) for c in range(width)])
            o_ref = np.stack([[r[0] for r in rr] for rr in refs])
            l_ref = np.stack([[r[1] for r in rr] for rr in refs])
            spread = np.stack([[r[2] for r in rr] for rr in refs])
            G.assert_attn_close(out, o_ref, lse, l_ref, what=f"tree round {rnd} step {i}", spread=spread)
        assert depth.cpu().numpy().tolist() == [n_steps] * B
        # verify: candidate cb[b] wins with acc[b] accepted rows, plus a bonus row
        cb = rng.integers(0, width, size=B)
        acc = rng.integers(0, n_steps + 1, size=B)
        W.tree_reset(depth)
        n_new = acc + 1
        n_max = int(n_new.max())
        kx, vx, kxb, vxb = rows.draw(B, n_max)
        k_acc = torch.zeros((B, n_max, Hkv, d), dtype=torch.bfloat16, device=dev)
        v_acc = torch.zeros_like(k_acc)
        accepted = []
        for b in range(B):
            spec = seqs[b].spec[cb[b]][: acc[b]]
            rows_b = spec + [(kxb[b, 0], vxb[b, 0])]
            accepted.append(rows_b)
            k_acc[b, : len(rows_b)] = I.from_bits(np.stack([r[0] for r in rows_b]), dev)
            v_acc[b, : len(rows_b)] = I.from_bits(np.stack([r[1] for r in rows_b]), dev)
        nn = G.lens_tensor(n_new, dev)
        W.ring_append(kr, vr, k_acc, v_acc, nn, lens, sink, R_w, err=err)
        qx = I.normal_bf16((B, n_max, Hq, d), 1000 * rnd + 500, dev)
        lse_x = torch.empty((B, n_max, Hq), dtype=torch.float32, device=dev)
        ox = W.ring_extend(qx, kr, vr, lens, Wn, sink, R_w, n_q=nn, lse=lse_x, err=err)
        torch.cuda.synchronize()
        qxb = I.bf16_bits(qx)
        o_ref = np.zeros((B, n_max, Hq, d))
        l_ref = np.full((B, n_max, Hq), -np.inf)
        spread = np.zeros((B, n_max, Hq, d))
        for b in range(B):
            seqs[b].verify(accepted[b])
            K = np.stack([r[0] for r in seqs[b].committed])
            V = np.stack([r[1] for r in seqs[b].committed])
            o_ref[b], l_ref[b] = A.attend_extend(qxb[b], K, V, seqs[b].S, int(n_new[b]), scale, "windowed",
                                                 Wn, sink)
            spread[b] = A.extend_spread(qxb[b], K, V, seqs[b].S, int(n_new[b]), scale, "windowed", Wn, sink)
        G.assert_attn_close(ox, o_ref, lse_x, l_ref, what=f"tree round {rnd} extend", spread=spread)
        assert lens.cpu().numpy().tolist() == [s.S for s in seqs]
    assert err.item() == 0


def test_width_one_tree_equals_chain_bitwise(dev, wpath):
    B, Hq, Hkv, d, Wn, sink, dd = 2, 16, 2, 128, 64, 4, 6
    R_w = Wn + dd
    rows = Rows(dev, Hkv, d)
    kr, vr, _, _ = _tree_state(dev, B, 1, dd, Hkv, d, sink, R_w)
    kc, vc = torch.zeros_like(kr), torch.zeros_like(vr)
    k0, v0, _, _ = rows.draw(B, 200)
    S0 = G.lens_tensor([150, 200], dev)
    lens_t = G.lens_tensor([0, 0], dev)
    lens_c = G.lens_tensor([0, 0], dev)
    W.ring_append(kr, vr, k0, v0, S0, lens_t, sink, R_w)
    W.ring_append(kc, vc, k0, v0, S0, lens_c, sink, R_w)
    depth = G.lens_tensor([0, 0], dev)
    ones = G.lens_tensor([1, 1], dev)
    for i in range(dd):
        k, v, _, _ = rows.draw(B, 1)
        W.tree_append(kr, vr, None, None, k, v, lens_t, depth, Wn, sink, R_w, dd)
        W.ring_append(kc, vc, k, v, ones, lens_c, sink, R_w)
        q = I.normal_bf16((B, 1, Hq, d), 40 + i, dev)
        ot = W.tree_attn(q, kr, vr, None, None, lens_t, depth, Wn, sink, R_w, dd)
        oc = W.ring_attn(q[:, 0].contiguous(), kc, vc, lens_c, Wn, sink, R_w)
        torch.cuda.synchronize()
        assert torch.equal(ot[:, 0], oc), i
        assert torch.equal(kr, kc) and torch.equal(vr, vc)


def test_append_past_largest_depth_is_flagged(dev, wpath):
    B, Hkv, d, Wn, sink, dd, width = 2, 2, 64, 8, 2, 2, 3
    R_w = Wn + dd
    rows = Rows(dev, Hkv, d)
    kr, vr, kb, vb = _tree_state(dev, B, width, dd, Hkv, d, sink, R_w)
    lens = G.lens_tensor([5, 9], dev)
    depth = G.lens_tensor([dd, 1], dev)
    err = G.err_word(dev)
    k, v, _, _ = rows.draw(B, width)
    before = (kr.clone(), kb.clone())
    W.tree_append(kr, vr, kb, vb, k, v, lens, depth, Wn, sink, R_w, dd, err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_DEPTH
    assert depth.cpu().numpy().tolist() == [dd, 2]
    assert torch.equal(kr[0], before[0][0]) and torch.equal(kb[0], before[1][0])  # request 0 untouched
    assert not torch.equal(kb[1], before[1][1])  # request 1 written
    W.tree_reset(depth)
    torch.cuda.synchronize()
    assert depth.cpu().numpy().tolist() == [0, 0]
    err.zero_()
    W.ring_rollback(lens, G.lens_tensor([7, -1], dev), err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_NNEW_RANGE
    assert lens.cpu().numpy().tolist() == [0, 9]  # over-long drop clamps to 0, a negative one is ignored
