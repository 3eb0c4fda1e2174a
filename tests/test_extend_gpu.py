"""GPU parity of draft-extend attention (several causal query rows per
sequence): full, windowed and ring, against the float64 oracle.

Covers ragged new-row counts (padding rows give 0 / -inf), rows whose
length crosses the window threshold, a ring sized exactly W + q_max - 1,
bitwise equality of ring and windowed extend, and of a one-row extend with
the decode call.  A 1M-token case checks the windowed rows at full size and
two full-context rows.
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


def _ring_from_dense(k, lens, sink, R_w):
    B, _, Hkv, d = k.shape
    ring = torch.zeros((B, sink + R_w, Hkv, d), dtype=k.dtype, device=k.device)
    for b, S in enumerate(lens):
        live = [p for p in range(S) if p < sink or p >= S - R_w]
        if live:
            ring[b, torch.as_tensor(R.ring_slots(live, sink, R_w), device=k.device)] = \
                k[b, torch.as_tensor(live, device=k.device)]
    return ring


def _oracle(q, k, v, lens, n_q, scale, variant, W_=None, sink=None):
    """Oracle outputs, lse and value spreads of every sequence's new rows."""
    qb = I.bf16_bits(q)
    outs, lses, spreads = [], [], []
    for b, (S, n) in enumerate(zip(lens, n_q)):
        K, V = G.HostRows(k[b]), G.HostRows(v[b])
        o, l = A.attend_extend(qb[b], K, V, S, n, scale, variant, W_, sink)
        outs.append(o)
        lses.append(l)
        spreads.append(A.extend_spread(qb[b], K, V, S, n, scale, variant, W_, sink))
    return np.stack(outs), np.stack(lses), np.stack(spreads)


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 6, 2), (128, 16, 2), (256, 32, 2), (256, 8, 8)])
@pytest.mark.parametrize("q_max", [1, 3, 8])
def test_extend_vs_oracle(dev, d, Hq, Hkv, q_max, wpath):
    W_, sink = 64, 4
    rng = np.random.default_rng(d + q_max)
    lens = [1, q_max, 50, sink + W_, sink + W_ + 2, 700, 4099]
    n_q = [1] + [int(rng.integers(1, q_max + 1)) for _ in lens[1:]]
    n_q = [min(n, S) for n, S in zip(n_q, lens)]
    B = len(lens)
    S_max = max(lens) + 3
    G.say(f"extend d={d} Hq={Hq} Hkv={Hkv} q_max={q_max} lens={lens} n_q={n_q}")
    q = I.normal_bf16((B, q_max, Hq, d), 31, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), 32, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 33, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    scale = 1.0 / np.sqrt(d)
    err = G.err_word(dev)
    for variant in ("full", "windowed"):
        lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse, err=err)
        else:
            out = W.draft_extend_windowed(q, k, v, lt, W_, sink, n_q=nt, lse=lse, err=err)
        torch.cuda.synchronize()
        o_ref, l_ref, spread = _oracle(q, k, v, lens, n_q, scale, variant, W_, sink)
        G.assert_attn_close(out, o_ref, lse, l_ref, what=f"extend {variant}", spread=spread)
    assert err.item() == 0
    # a ring sized exactly W + q_max - 1 gives the windowed result bit for bit
    R_w = W_ + q_max - 1
    kr, vr = _ring_from_dense(k, lens, sink, R_w), _ring_from_dense(v, lens, sink, R_w)
    ow = W.draft_extend_windowed(q, k, v, lt, W_, sink, n_q=nt)
    orr = W.ring_extend(q, kr, vr, lt, W_, sink, R_w, n_q=nt)
    torch.cuda.synchronize()
    assert torch.equal(orr, ow)


@pytest.mark.parametrize("scale", [-1.0 / 16, 0.0, 0.5])
def test_full_extend_any_scale(dev, scale):
    """The multi-row kernel folds the logit scale into its exponent and needs
    it positive: a negative scale goes into the queries' sign, a zero one is
    replaced by the smallest normal float.  Negative, zero and large scales
    against the oracle (the zero scale averages the visible values), with
    rows ending inside a 64-key step, where keys are masked."""
    d, Hq, Hkv, q_max = 256, 32, 2, 8
    lens = [q_max, 77, 3000, 9000 + 13]
    n_q = [q_max, 5, q_max, 3]
    B = len(lens)
    S_max = max(lens) + 2
    G.say(f"full extend scale={scale} lens={lens} n_q={n_q}")
    q = I.normal_bf16((B, q_max, Hq, d), 71, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), 72, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 73, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    err = G.err_word(dev)
    lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
    out = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse, scale=scale, err=err)
    torch.cuda.synchronize()
    o_ref, l_ref, spread = _oracle(q, k, v, lens, n_q, scale, "full")
    G.assert_attn_close(out, o_ref, lse, l_ref, what=f"full extend scale {scale}", spread=spread)
    assert err.item() == 0


@pytest.mark.parametrize("d,Hq,Hkv", [(128, 12, 2), (256, 32, 2)])
@pytest.mark.parametrize("q_max", [12, 20])
def test_full_extend_many_rows(dev, d, Hq, Hkv, q_max):
    """More new rows than one pass of the multi-row kernel takes (eight), ragged
    row counts, and rows whose lengths straddle item boundaries."""
    lens = [q_max + 1, 130, 4099, 20000, 64 * 37 + 5]
    n_q = [q_max, q_max, 9, q_max - 3, 7]
    B = len(lens)
    S_max = max(lens) + 1
    G.say(f"extend many rows d={d} Hq={Hq} Hkv={Hkv} q_max={q_max} lens={lens} n_q={n_q}")
    q = I.normal_bf16((B, q_max, Hq, d), 61, dev)
    k = I.normal_bf16((B, S_max, Hkv, d), 62, dev)
    v = I.normal_bf16((B, S_max, Hkv, d), 63, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
    err = G.err_word(dev)
    out = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse, err=err)
    # the same call with only the per-row workspace: items sized from every
    # row's keys (the coarser decomposition)
    ws_rows = torch.zeros(W.workspace_bytes(B * q_max, Hq, Hkv, d, S_max, variant=W.VARIANT_FULL),
                          dtype=torch.uint8, device=dev)
    assert ws_rows.numel() < W.extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max)
    lse_c = torch.empty_like(lse)
    out_c = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse_c, err=err, ws=ws_rows)
    torch.cuda.synchronize()
    o_ref, l_ref, spread = _oracle(q, k, v, lens, n_q, 1.0 / np.sqrt(d), "full")
    G.assert_attn_close(out, o_ref, lse, l_ref, what="extend many rows", spread=spread)
    G.assert_attn_close(out_c, o_ref, lse_c, l_ref, what="extend many rows, per-row items", spread=spread)
    assert err.item() == 0


def test_one_row_extend_is_the_decode_step(dev, wpath):
    Hq, Hkv, d = 32, 2, 256
    lens = [5000, 70000, 1, 3000]
    q = I.normal_bf16((4, 1, Hq, d), 41, dev)
    k = I.normal_bf16((4, max(lens), Hkv, d), 42, dev)
    v = I.normal_bf16((4, max(lens), Hkv, d), 43, dev)
    lt = G.lens_tensor(lens, dev)
    assert torch.equal(W.draft_extend_full(q, k, v, lt)[:, 0], W.draft_attn_full(q[:, 0].contiguous(), k, v, lt))
    assert torch.equal(W.draft_extend_windowed(q, k, v, lt, 2048, 4)[:, 0],
                       W.draft_attn_windowed(q[:, 0].contiguous(), k, v, lt, 2048, 4))


def test_ring_extend_rejects_small_ring(dev):
    q = torch.zeros((1, 8, 16, 128), dtype=torch.bfloat16, device=dev)
    kr = torch.zeros((1, 4 + 70, 2, 128), dtype=torch.bfloat16, device=dev)
    with pytest.raises(W.WmtpError):
        W.ring_extend(q, kr, kr, G.lens_tensor([10], dev), 64, 4, 70)  # needs R_w >= 71


def test_extend_flags_bad_row_counts(dev, wpath):
    q = I.normal_bf16((2, 4, 16, 128), 1, dev)
    k = I.normal_bf16((2, 100, 2, 128), 2, dev)
    err = G.err_word(dev)
    out = W.draft_extend_full(q, k, k, G.lens_tensor([2, 50], dev), n_q=G.lens_tensor([3, 9], dev), err=err)
    torch.cuda.synchronize()
    assert err.item() & W.DERR_NNEW_RANGE and err.item() & W.DERR_LEN_RANGE
    # sequence 0 has 2 cached rows for 3 new ones: row 0 would see 0 rows;
    # row 3 is padding.  Both are zero; rows 1, 2 see 1 and 2 rows.
    assert torch.count_nonzero(out[0, 0]) == 0 and torch.count_nonzero(out[0, 3]) == 0
    assert torch.count_nonzero(out[0, 1]) > 0


def test_extend_s1m_draft_depth8(dev):
    """1M-token cache, 8 new rows (gamma + 1 accepted), Hq=32, d=256."""
    wl = I.WORKLOADS["draft_loop_s1m"]
    S, q_max = wl.S, 8
    G.say("extend 1M: generating")
    case = I.decode_case(wl, dev, steps=1)
    k, v = case["k"], case["v"]
    q = I.normal_bf16((1, q_max, wl.Hq, wl.d), 51, dev)
    lt, nt = G.lens_tensor([S], dev), G.lens_tensor([q_max], dev)
    lse_w = torch.empty(1, q_max, wl.Hq, dtype=torch.float32, device=dev)
    lse_f = torch.empty_like(lse_w)
    ow = W.draft_extend_windowed(q, k, v, lt, wl.W, wl.sink, n_q=nt, lse=lse_w)
    of = W.draft_extend_full(q, k, v, lt, n_q=nt, lse=lse_f)
    torch.cuda.synchronize()
    o_ref, l_ref, _ = _oracle(q, k, v, [S], [q_max], wl.scale, "windowed", wl.W, wl.sink)
    G.say(f"extend 1M windowed err {G.assert_attn_close(ow, o_ref, lse_w, l_ref, 'extend 1M windowed')}")
    qb = I.bf16_bits(q)
    for t in (0, 3, q_max - 1):
        L = S - q_max + t + 1
        o1, l1 = A.attend_sequence(qb[0, t], G.HostRows(k[0]), G.HostRows(v[0]), L, wl.scale, None)
        e = G.assert_attn_close(of[0, t], o1, lse_f[0, t], l1, f"extend 1M full row {t}")
        G.say(f"extend 1M full row {t} err {e}")


def test_full_extend_many_kv_heads_takes_the_per_row_kernel(dev):
    """With 64 token rows of all KV heads spanning 4 GiB or more (here
    Hkv = 131072 at d = 256, G = 1) the multi-row kernel's 32-bit offsets
    would not reach; the call takes the per-row split kernel instead.  Its
    rows against a float32 reference computed here (elementwise products, no
    batched matmul) over the causal keys of each row, to the parity bar's
    elementwise bound (tests/_gpu.py; with two or three keys per row the
    outputs reach |o| ~ 5, where rounding to bf16 alone moves them by up to
    2^-8 |o|)."""
    Hkv = Hq = 131072
    d, q_max, S_max = 256, 2, 4
    lens, n_q = [3], [2]
    q = I.normal_bf16((1, q_max, Hq, d), 81, dev)
    k = I.normal_bf16((1, S_max, Hkv, d), 82, dev)
    v = I.normal_bf16((1, S_max, Hkv, d), 83, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    err = G.err_word(dev)
    out = W.draft_extend_full(q, k, v, lt, n_q=nt, err=err)
    torch.cuda.synchronize()
    assert err.item() == 0
    scale = 1.0 / np.sqrt(d)
    for t in range(q_max):
        L = lens[0] - n_q[0] + t + 1
        qt = q[0, t].float()                                     # [H, d]
        kt, vt = k[0, :L].float(), v[0, :L].float()              # [L, H, d]
        s = (qt[None] * kt).sum(-1) * scale                      # [L, H]
        p = torch.softmax(s, dim=0)
        ref = (p[..., None] * vt).sum(0)                         # [H, d]
        spread = (p[..., None] * (vt - ref[None]).abs()).sum(0)  # sum_p w_p |v_p - o|
        bound = G.elementwise_bound(ref.double().cpu().numpy(), spread.double().cpu().numpy())
        err_t = (out[0, t].float() - ref).abs().double().cpu().numpy()
        assert (err_t <= bound).all(), (t, float(err_t.max()), float((err_t - bound).max()))
