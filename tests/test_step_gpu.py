"""GPU parity of the fused draft step (append + attention in one call).

* bit for bit against the unfused path (wmtp_cache_append / wmtp_ring_append
  followed by the attention call): outputs, lse, cache contents and lengths,
  over several steps with ragged append counts (0 to 6 rows), lengths 0,
  short and past the window; and ring steps whose append is longer than the
  ring (the fused kernel writes only the rows that stay resident);
* the million-token windowed and full draft loop through the fused step
  against the oracle;
* a dense cache that would grow past its capacity keeps the rows that fit and
  raises WMTP_DERR_CAPACITY.
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


class Spliced:
    """Rows [0, S0) from a host view, rows >= S0 from a host array."""

    def __init__(self, base, S0, tail):
        self.base, self.S0, self.tail = base, S0, np.asarray(tail)
        self.shape = (S0 + len(self.tail),) + tuple(base.shape[1:])

    def __getitem__(self, rows):
        rows = np.asarray(rows, dtype=np.int64)
        out = np.empty((rows.size,) + self.shape[1:], dtype=np.uint16)
        lo = rows < self.S0
        if lo.any():
            out[lo] = self.base[rows[lo]]
        if (~lo).any():
            out[~lo] = self.tail[rows[~lo] - self.S0]
        return out


@pytest.mark.parametrize("variant", ["full", "windowed", "ring"])
@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2), (64, 6, 2)])
def test_step_equals_append_then_attention(dev, variant, d, Hq, Hkv, wpath):
    Wn, sink = 64, 4
    R_w = Wn + 3
    lens0 = [0, 3, 70, 5000]
    B, n_max = len(lens0), 6
    S_max = max(lens0) + 5 * n_max
    G.say(f"step {variant} d={d} Hq={Hq}")
    rows = S_max if variant != "ring" else sink + R_w
    k0 = I.normal_bf16((B, rows, Hkv, d), 3 * d, dev)
    v0 = I.normal_bf16((B, rows, Hkv, d), 3 * d + 1, dev)
    k_f, v_f = k0.clone(), v0.clone()  # fused
    k_u, v_u = k0.clone(), v0.clone()  # unfused
    lens_a = G.lens_tensor(lens0, dev)
    lens_b = torch.empty_like(lens_a)
    lens_u = G.lens_tensor(lens0, dev)
    err_f, err_u = G.err_word(dev), G.err_word(dev)
    counts = [[1, 0, 2, 1], [2, 1, 0, 6], [1, 1, 1, 1], [0, 0, 0, 0], [6, 2, 5, 1]]
    for step, nn in enumerate(counts):
        kn = I.normal_bf16((B, n_max, Hkv, d), 100 * step + 7, dev)
        vn = I.normal_bf16((B, n_max, Hkv, d), 100 * step + 8, dev)
        q = I.normal_bf16((B, Hq, d), 100 * step + 9, dev)
        n_new = G.lens_tensor(nn, dev)
        lse_f = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        lse_u = torch.empty_like(lse_f)
        lin, lout = (lens_a, lens_b) if step % 2 == 0 else (lens_b, lens_a)
        if variant == "full":
            of = W.draft_step_full(q, k_f, v_f, kn, vn, n_new, lin, lout, lse=lse_f, err=err_f)
            W.cache_append(k_u, v_u, kn, vn, n_new, lens_u, err=err_u)
            ou = W.draft_attn_full(q, k_u, v_u, lens_u, lse=lse_u, err=err_u)
        elif variant == "windowed":
            of = W.draft_step_windowed(q, k_f, v_f, kn, vn, n_new, lin, lout, Wn, sink, lse=lse_f, err=err_f)
            W.cache_append(k_u, v_u, kn, vn, n_new, lens_u, err=err_u)
            ou = W.draft_attn_windowed(q, k_u, v_u, lens_u, Wn, sink, lse=lse_u, err=err_u)
        else:
            of = W.ring_step(q, k_f, v_f, kn, vn, n_new, lin, lout, Wn, sink, R_w, lse=lse_f, err=err_f)
            W.ring_append(k_u, v_u, kn, vn, n_new, lens_u, sink, R_w, err=err_u)
            ou = W.ring_attn(q, k_u, v_u, lens_u, Wn, sink, R_w, lse=lse_u, err=err_u)
        torch.cuda.synchronize()
        assert torch.equal(lout, lens_u), step
        assert torch.equal(of, ou), step
        assert torch.equal(lse_f, lse_u), step
        assert torch.equal(k_f, k_u) and torch.equal(v_f, v_u), step
    assert err_f.item() == 0 and err_u.item() == 0


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 16, 2), (256, 32, 2)])
def test_ring_step_append_longer_than_ring(dev, d, Hq, Hkv, wpath):
    """n_new up to R_w + sink + 3 rows in one fused ring step, from lengths
    0, below the sink, past the window and far past it: positions that a
    later row of the same append overwrites must not be written."""
    Wn, sink = 16, 4
    R_w = Wn
    lens0 = [0, 2, 30, 200]
    B, n_max = len(lens0), R_w + sink + 3
    k0 = I.normal_bf16((B, sink + R_w, Hkv, d), 11 * d, dev)
    v0 = I.normal_bf16((B, sink + R_w, Hkv, d), 11 * d + 1, dev)
    k_f, v_f = k0.clone(), v0.clone()
    k_u, v_u = k0.clone(), v0.clone()
    lens_a = G.lens_tensor(lens0, dev)
    lens_b = torch.empty_like(lens_a)
    lens_u = G.lens_tensor(lens0, dev)
    err_f, err_u = G.err_word(dev), G.err_word(dev)
    counts = [[n_max, R_w + 1, n_max, R_w], [1, n_max, 0, n_max], [R_w + 2, 3, n_max - 1, 5]]
    for step, nn in enumerate(counts):
        G.say(f"ring step longer than the ring d={d} step {step} n_new={nn}")
        kn = I.normal_bf16((B, n_max, Hkv, d), 300 + 10 * step, dev)
        vn = I.normal_bf16((B, n_max, Hkv, d), 301 + 10 * step, dev)
        q = I.normal_bf16((B, Hq, d), 302 + 10 * step, dev)
        n_new = G.lens_tensor(nn, dev)
        lse_f = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        lse_u = torch.empty_like(lse_f)
        lin, lout = (lens_a, lens_b) if step % 2 == 0 else (lens_b, lens_a)
        of = W.ring_step(q, k_f, v_f, kn, vn, n_new, lin, lout, Wn, sink, R_w, lse=lse_f, err=err_f)
        W.ring_append(k_u, v_u, kn, vn, n_new, lens_u, sink, R_w, err=err_u)
        ou = W.ring_attn(q, k_u, v_u, lens_u, Wn, sink, R_w, lse=lse_u, err=err_u)
        torch.cuda.synchronize()
        assert torch.equal(lout, lens_u), step
        assert torch.equal(of, ou), step
        assert torch.equal(lse_f, lse_u), step
        assert torch.equal(k_f, k_u) and torch.equal(v_f, v_u), step
    assert err_f.item() == 0 and err_u.item() == 0


def test_step_capacity_is_flagged(dev):
    B, Hq, Hkv, d = 2, 16, 2, 128
    S_max = 50
    k = I.normal_bf16((B, S_max, Hkv, d), 1, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 2, dev)
    k0 = k.clone()
    kn = I.normal_bf16((B, 3, Hkv, d), 3, dev)
    vn = I.normal_bf16((B, 3, Hkv, d), 4, dev)
    q = I.normal_bf16((B, Hq, d), 5, dev)
    lin = G.lens_tensor([49, 10], dev)
    lout = torch.empty_like(lin)
    err = G.err_word(dev)
    out = W.draft_step_full(q, k, v, kn, vn, G.lens_tensor([3, 3], dev), lin, lout, err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_CAPACITY
    assert lout.cpu().numpy().tolist() == [50, 13]
    assert torch.equal(k[0, 49], kn[0, 0]) and torch.equal(k[0, :49], k0[0, :49])
    assert torch.equal(k[1, 10:13], kn[1]) and torch.equal(k[1, 13:], k0[1, 13:])
    ref = W.draft_attn_full(q, k, v, G.lens_tensor([50, 13], dev))
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_step_1m_draft_loop_vs_oracle(dev):
    wl = I.WORKLOADS["draft_loop_s1m"]
    g = wl.gamma
    G.say("step 1M: generating")
    case = I.decode_case(wl, dev, steps=g)
    k, v = case["k"], case["v"]
    q, kn, vn = case["q"], case["k_new"], case["v_new"]
    kn_bits = np.stack([I.bf16_bits(kn[j])[0, 0] for j in range(g)])
    vn_bits = np.stack([I.bf16_bits(vn[j])[0, 0] for j in range(g)])
    lens = [G.lens_tensor([wl.S], dev), G.lens_tensor([0], dev)]
    ones = G.lens_tensor([1], dev)
    err = G.err_word(dev)
    for j in range(g):
        lin, lout = lens[j % 2], lens[(j + 1) % 2]
        lse = torch.empty((1, wl.Hq), dtype=torch.float32, device=dev)
        if j < g - 1:
            out = W.draft_step_windowed(q[j], k, v, kn[j], vn[j], ones, lin, lout, wl.W, wl.sink, lse=lse,
                                        err=err)
            variant = "windowed"
        else:
            out = W.draft_step_full(q[j], k, v, kn[j], vn[j], ones, lin, lout, lse=lse, err=err)
            variant = "full"
        torch.cuda.synchronize()
        S = wl.S + j + 1
        assert lout.item() == S
        G.say(f"step 1M {variant} {j}: oracle")
        # the oracle reads the generator's rows: the cache below the old
        # length (never written here) and the appended rows from k_new / v_new
        Kv = Spliced(G.HostRows(k[0]), wl.S, kn_bits[: j + 1])
        Vv = Spliced(G.HostRows(v[0]), wl.S, vn_bits[: j + 1])
        mask = None if variant == "full" else A.window_mask(S, wl.W, wl.sink)
        o_ref, l_ref = A.attend_sequence(I.bf16_bits(q[j])[0], Kv, Vv, S, wl.scale, mask)
        e = G.assert_attn_close(out, o_ref[None], lse, l_ref[None], what=f"step 1M {variant} {j}")
        G.say(f"step 1M {variant} {j}: max err {e}")
    assert err.item() == 0
