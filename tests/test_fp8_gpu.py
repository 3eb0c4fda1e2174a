"""GPU parity of the fp8 (OCP E4M3, per-tensor scale) draft KV cache.

* the format's element conversions, exhaustively: every code widened to
  bf16, every finite bf16 value quantised with several scales -- bit-exact
  against the oracle;
* fp8 appends (dense cache and ring): the bytes written and the lengths,
  bit-exact against the oracle's quantisation of the same rows;
* fp8 attention (full, windowed, ring) against the float64 oracle over the
  dequantized cache, on every head size and a spread of GQA shapes, ragged
  and degenerate lengths, non-trivial scales; ring == windowed bitwise;
* closed-form index encoding through fp8 codes (zero keys, value rows that
  encode their position), windowed at 1M + 7 keys and the ring after wraps;
* fp8 draft-extend (full, windowed, ring) against the oracle's per-row
  causal attention over the dequantized cache; ring == windowed bitwise;
* the million-token draft loop with an fp8 cache: gamma quantising appends,
  windowed attention every step and full attention at the last, against
  the oracle (appended rows taken from the oracle's own quantisation).
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import fp8 as F
from oracle import ring as R
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


class HostCodes:
    """Host view of one sequence of a device fp8 cache [rows, Hkv, d]:
    indexing returns the rows' codes as a uint8 numpy array."""

    def __init__(self, t: torch.Tensor):
        self.t = t
        self.shape = tuple(t.shape)

    def __getitem__(self, rows):
        idx = torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int64)).to(self.t.device)
        return self.t.index_select(0, idx).cpu().numpy()


class SplicedCodes:
    """Rows [0, S0) from a host view, rows >= S0 from a host array (the
    oracle's own quantisation of the appended rows)."""

    def __init__(self, base, S0, tail):
        self.base, self.S0, self.tail = base, S0, np.asarray(tail)
        self.shape = (S0 + len(self.tail),) + tuple(base.shape[1:])

    def __getitem__(self, rows):
        rows = np.asarray(rows, dtype=np.int64)
        out = np.empty((rows.size,) + self.shape[1:], dtype=np.uint8)
        lo = rows < self.S0
        if lo.any():
            out[lo] = self.base[rows[lo]]
        if (~lo).any():
            out[~lo] = self.tail[rows[~lo] - self.S0]
        return out


def _finite_bf16_bits():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    return bits[(bits & 0x7F80) != 0x7F80]


# ----------------------------------------------------------- conversions
def test_dequantize_every_code(dev):
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8).repeat(2).to(dev)
    out = W.fp8_dequantize(codes)
    torch.cuda.synchronize()
    got = I.bf16_bits(out)[:256].astype(np.uint32)
    ref = F.decode(np.arange(256, dtype=np.uint8))
    nan = np.isnan(ref)
    exp = (ref[~nan].astype(np.float32).view(np.uint32) >> 16)
    assert np.array_equal(got[~nan], exp)
    g_nan = got[nan]
    assert np.all((g_nan & 0x7F80) == 0x7F80) and np.all(g_nan & 0x7F)  # NaN codes give NaN


@pytest.mark.parametrize("scale", [1.0, 0.5, 0.0625, 0.7, 3.0, 1e-3, 300.0])
def test_quantize_every_bf16(dev, scale):
    bits = _finite_bf16_bits()
    assert bits.size % 8 == 0
    x = I.from_bits(bits, dev)
    codes = W.fp8_quantize(x, scale)
    torch.cuda.synchronize()
    got = codes.cpu().numpy()
    with np.errstate(over="ignore"):
        exp = F.quantize(bits, scale)
    bad = np.flatnonzero(got != exp)
    assert bad.size == 0, f"{bad.size} codes differ, e.g. x bits {bits[bad[:4]]}: {got[bad[:4]]} vs {exp[bad[:4]]}"


# --------------------------------------------------------------- appends
@pytest.mark.parametrize("ring", [False, True])
def test_append_quantizes_exactly(dev, ring):
    B, Hkv, d = 5, 2, 128
    sink, R_w, S_max = 4, 40, 300
    lens0 = [0, 3, 39, 44, 250]
    n_new = [0, 1, 7, 20, 50]
    n_max = max(n_new)
    ks, vs = 0.37, 2.5
    k_new = I.normal_bf16((B, n_max, Hkv, d), 21, dev) * 3
    v_new = I.normal_bf16((B, n_max, Hkv, d), 22, dev)
    rows = sink + R_w if ring else S_max
    k8 = torch.full((B, rows, Hkv, d), 0x11, dtype=torch.uint8, device=dev)
    v8 = torch.full_like(k8, 0x22)
    exp_k, exp_v = k8.cpu().numpy().copy(), v8.cpu().numpy().copy()
    lens = G.lens_tensor(lens0, dev)
    nn = G.lens_tensor(n_new, dev)
    err = G.err_word(dev)
    if ring:
        W.ring_append_fp8(k8, v8, k_new, v_new, nn, lens, sink, R_w, ks, vs, err=err)
    else:
        W.cache_append_fp8(k8, v8, k_new, v_new, nn, lens, ks, vs, err=err)
    torch.cuda.synchronize()
    kb, vb = I.bf16_bits(k_new), I.bf16_bits(v_new)
    for b in range(B):
        for i in range(n_new[b]):  # rows written in order: a slot keeps its last writer
            p = lens0[b] + i
            s = R.ring_slot(p, sink, R_w) if ring else p
            exp_k[b, s] = F.quantize(kb[b, i], ks)
            exp_v[b, s] = F.quantize(vb[b, i], vs)
    assert np.array_equal(k8.cpu().numpy(), exp_k)
    assert np.array_equal(v8.cpu().numpy(), exp_v)
    assert lens.cpu().numpy().tolist() == [a + n for a, n in zip(lens0, n_new)]
    assert err.item() == 0


# ------------------------------------------------------------- attention
SHAPES = [(64, 1, 1), (64, 6, 2), (128, 16, 2), (128, 4, 4), (256, 32, 2), (256, 12, 3)]


@pytest.mark.parametrize("d,Hq,Hkv", SHAPES)
@pytest.mark.parametrize("ks,vs", [(1.0, 1.0), (0.75, 1.5)])
def test_fp8_attention_vs_oracle(dev, d, Hq, Hkv, ks, vs, wpath):
    seed = 31 * d + Hq + 7 * Hkv
    for W_, sink in ((64, 4), (100, 7)):
        lens = [0, 1, 3, sink + W_, sink + W_ + 1, 17, 1000, 5003]
        B, S_max = len(lens), max(lens) + 5
        G.say(f"fp8 d={d} Hq={Hq} Hkv={Hkv} W={W_} sink={sink} scales=({ks},{vs})")
        q = I.normal_bf16((B, Hq, d), seed, dev)
        k8 = I.normal_fp8((B, S_max, Hkv, d), seed + 1, dev)
        v8 = I.normal_fp8((B, S_max, Hkv, d), seed + 2, dev)
        lt = G.lens_tensor(lens, dev)
        scale = 1.0 / np.sqrt(d)
        qb = I.bf16_bits(q)
        for variant in ("full", "windowed"):
            lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
            if variant == "full":
                out = W.draft_attn_full_fp8(q, k8, v8, lt, ks, vs, lse=lse)
            else:
                out = W.draft_attn_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, lse=lse)
            torch.cuda.synchronize()
            refs = [F.attend_sequence_fp8(qb[b], HostCodes(k8[b]), HostCodes(v8[b]), lens[b], scale, ks, vs,
                                          variant, W_, sink, spread=True) for b in range(B)]
            G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                                what=f"fp8 {variant} d={d} G={Hq // Hkv} W={W_}",
                                spread=np.stack([r[2] for r in refs]))
            assert torch.count_nonzero(out[0]) == 0


def test_fp8_windowed_merge_in_several_batches(dev, wpath):
    """A 65536-key window over an fp8 cache: at least 65 items per row, so the
    one-launch kernel's merger combines them in several batches."""
    d, Hq, Hkv, W_, sink, ks, vs = 256, 32, 2, 65536, 4, 0.5, 0.25
    lens = [W_ + sink + 3001, W_ + sink, 40007, 5]
    B, S_max = len(lens), max(lens) + 3
    G.say(f"fp8 windowed merge batches W={W_} lens={lens}")
    q = I.normal_bf16((B, Hq, d), 71, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 72, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 73, dev)
    lt = G.lens_tensor(lens, dev)
    scale = 1.0 / np.sqrt(d)
    lse = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    out = W.draft_attn_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, lse=lse)
    torch.cuda.synchronize()
    qb = I.bf16_bits(q)
    refs = [F.attend_sequence_fp8(qb[b], HostCodes(k8[b]), HostCodes(v8[b]), lens[b], scale, ks, vs,
                                  "windowed", W_, sink, spread=True) for b in range(B)]
    G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                        what="fp8 windowed, several merge batches", spread=np.stack([r[2] for r in refs]))


def _ring_from_dense(x, lens, sink, R_w):
    B, _, Hkv, d = x.shape
    ring = torch.zeros((B, sink + R_w, Hkv, d), dtype=x.dtype, device=x.device)
    for b, S in enumerate(lens):
        live = [p for p in range(S) if p < sink or p >= S - R_w]
        if live:
            ring[b, torch.as_tensor(R.ring_slots(live, sink, R_w), device=x.device)] = \
                x[b, torch.as_tensor(live, device=x.device)]
    return ring


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 6, 2), (128, 16, 2), (256, 32, 2)])
def test_fp8_ring_equals_windowed_bitwise(dev, d, Hq, Hkv, wpath):
    W_, sink, R_w = 64, 4, 71
    lens = [0, 1, 3, sink + W_, sink + W_ + 1, sink + R_w + 1, 777, 5003]
    B, S_max = len(lens), max(lens) + 2
    G.say(f"fp8 ring d={d} Hq={Hq}")
    q = I.normal_bf16((B, Hq, d), 5 * d, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 5 * d + 1, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 5 * d + 2, dev, spread=4.0)
    lt = G.lens_tensor(lens, dev)
    kr, vr = _ring_from_dense(k8, lens, sink, R_w), _ring_from_dense(v8, lens, sink, R_w)
    lse_w = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    lse_r = torch.empty_like(lse_w)
    ow = W.draft_attn_windowed_fp8(q, k8, v8, lt, W_, sink, 0.5, 0.25, lse=lse_w)
    orr = W.ring_attn_fp8(q, kr, vr, lt, W_, sink, R_w, 0.5, 0.25, lse=lse_r)
    torch.cuda.synchronize()
    assert torch.equal(orr, ow) and torch.equal(lse_r, lse_w)
    qb = I.bf16_bits(q)
    refs = [F.attend_ring_fp8(qb[b], kr[b].cpu().numpy(), vr[b].cpu().numpy(), lens[b], 1.0 / np.sqrt(d), 0.5,
                              0.25, W_, sink, R_w, spread=True) for b in range(B)]
    G.assert_attn_close(orr, np.stack([r[0] for r in refs]), lse_r, np.stack([r[1] for r in refs]),
                        what=f"fp8 ring d={d}", spread=np.stack([r[2] for r in refs]))


# -------------------------------------------------------- index encoding
Hq_e, Hkv_e, d_e = 32, 2, 256
ONE = 0x38  # E4M3 code of 1.0


def _residue_codes(pos, dev):
    p = torch.as_tensor(np.asarray(pos, dtype=np.int64), device=dev)
    out = torch.zeros((p.numel(), Hkv_e, d_e), dtype=torch.uint8, device=dev)
    c = torch.arange(128, device=dev)
    for g in range(Hkv_e):
        out[:, g, :127] = (((p + 37 * g) % 127)[:, None] == c[None, :127]).to(torch.uint8) * ONE
        out[:, g, 127:255] = (((p + 41 * g) % 128)[:, None] == c[None, :128]).to(torch.uint8) * ONE
        out[:, g, 255] = ONE
    return out


def _residue_expected(positions, v_scale):
    e = np.zeros((Hkv_e, d_e))
    p = np.asarray(positions, dtype=np.int64)
    for g in range(Hkv_e):
        e[g, :127] = np.bincount((p + 37 * g) % 127, minlength=127)
        e[g, 127:255] = np.bincount((p + 41 * g) % 128, minlength=128)
        e[g, 255] = p.size
    return e / p.size * v_scale


def _check_exact(out, exp_per_kv, what):
    o = out.float().cpu().numpy().astype(np.float64)
    ref = np.repeat(exp_per_kv, Hq_e // Hkv_e, axis=0)
    ulp = np.where(ref > 0, 2.0 ** (np.floor(np.log2(np.maximum(ref, 1e-30))) - 7), 0.0)
    bad = np.abs(o - ref) > ulp
    assert not bad.any(), f"{what}: {bad.sum()} channels off, first at {np.argwhere(bad)[:4].tolist()}"


@pytest.mark.parametrize("S", [3, 2053, 1048576 + 7])
def test_fp8_windowed_reads_the_right_rows(dev, S, wpath):
    G.say(f"fp8 index encoding windowed S={S}")
    sink, Wn = 4, 2048
    k8 = torch.zeros((1, S, Hkv_e, d_e), dtype=torch.uint8, device=dev)
    v8 = torch.zeros_like(k8)
    keep = A.selected_positions(S, Wn, sink)
    v8[0, torch.as_tensor(keep, device=dev)] = _residue_codes(keep, dev)
    drop = np.setdiff1d(np.arange(max(0, S - 3 * Wn), S), keep)[:4096]
    if drop.size:
        v8[0, torch.as_tensor(drop, device=dev)] = _residue_codes(drop + 5, dev)
    q = I.normal_bf16((1, Hq_e, d_e), 3, dev)
    lse = torch.empty((1, Hq_e), dtype=torch.float32, device=dev)
    out = W.draft_attn_windowed_fp8(q, k8, v8, G.lens_tensor([S], dev), Wn, sink, 1.0, 0.5, lse=lse)
    torch.cuda.synchronize()
    _check_exact(out[0], _residue_expected(keep, 0.5), f"fp8 windowed S={S}")
    assert np.allclose(lse.cpu().numpy(), np.log(keep.size), rtol=0, atol=4e-6)


@pytest.mark.parametrize("S", [2060, 1048576 + 3])
def test_fp8_ring_reads_the_right_slots(dev, S, wpath):
    G.say(f"fp8 index encoding ring S={S}")
    sink, Wn, R_w = 4, 2048, 2056
    kr = torch.zeros((1, sink + R_w, Hkv_e, d_e), dtype=torch.uint8, device=dev)
    live = np.array([p for p in range(max(0, S - R_w - sink), S) if p < sink or p >= S - R_w])
    live = np.union1d(np.arange(min(sink, S)), live)
    vr = torch.zeros_like(kr)
    vr[0, torch.as_tensor(R.ring_slots(live, sink, R_w), device=dev)] = _residue_codes(live, dev)
    q = I.normal_bf16((1, Hq_e, d_e), 4, dev)
    out = W.ring_attn_fp8(q, kr, vr, G.lens_tensor([S], dev), Wn, sink, R_w, 2.0, 1.0)
    torch.cuda.synchronize()
    _check_exact(out[0], _residue_expected(A.selected_positions(S, Wn, sink), 1.0), f"fp8 ring S={S}")


# ------------------------------------------------------ 1M draft loop
def test_fp8_draft_loop_1m(dev):
    wl = I.WORKLOADS["draft_loop_s1m"]
    g = wl.gamma
    ks, vs = 0.5, 0.25
    G.say("fp8 1M draft loop: generating")
    case = I.decode_case(wl, dev, steps=g)
    S0 = wl.S
    k8 = I.fp8_codes(case["k"].float() / ks)
    del case["k"]
    v8 = I.fp8_codes(case["v"].float() / vs)
    del case["v"]
    torch.cuda.empty_cache()
    q, kn, vn = case["q"], case["k_new"], case["v_new"]
    lens = G.lens_tensor([S0], dev)
    ones = G.lens_tensor([1], dev)
    err = G.err_word(dev)
    tail_k = [F.quantize(I.bf16_bits(kn[j])[0, 0], ks) for j in range(g)]
    tail_v = [F.quantize(I.bf16_bits(vn[j])[0, 0], vs) for j in range(g)]
    for j in range(g):
        W.cache_append_fp8(k8, v8, kn[j], vn[j], ones, lens, ks, vs, err=err)
        S = S0 + j + 1
        lse = torch.empty((1, wl.Hq), dtype=torch.float32, device=dev)
        ow = W.draft_attn_windowed_fp8(q[j], k8, v8, lens, wl.W, wl.sink, ks, vs, lse=lse)
        torch.cuda.synchronize()
        assert np.array_equal(k8[0, S - 1].cpu().numpy(), tail_k[j])
        assert np.array_equal(v8[0, S - 1].cpu().numpy(), tail_v[j])
        Kv = SplicedCodes(HostCodes(k8[0]), S0, np.stack(tail_k[: j + 1]))
        Vv = SplicedCodes(HostCodes(v8[0]), S0, np.stack(tail_v[: j + 1]))
        qb = I.bf16_bits(q[j])[0]
        o_ref, l_ref = F.attend_sequence_fp8(qb, Kv, Vv, S, wl.scale, ks, vs, "windowed", wl.W, wl.sink)
        e = G.assert_attn_close(ow, o_ref[None], lse, l_ref[None], what=f"fp8 1M windowed step {j}")
        G.say(f"fp8 1M windowed step {j}: max err {e}")
        if j == g - 1:
            lse_f = torch.empty_like(lse)
            of = W.draft_attn_full_fp8(q[j], k8, v8, lens, ks, vs, lse=lse_f)
            torch.cuda.synchronize()
            G.say("fp8 1M full: oracle")
            o_ref, l_ref = F.attend_sequence_fp8(qb, Kv, Vv, S, wl.scale, ks, vs, "full")
            e = G.assert_attn_close(of, o_ref[None], lse_f, l_ref[None], what="fp8 1M full")
            G.say(f"fp8 1M full: max err {e}")
    assert lens.item() == S0 + g
    assert err.item() == 0


@pytest.mark.parametrize("d,Hq,Hkv", [(64, 6, 2), (128, 16, 2), (256, 32, 2)])
@pytest.mark.parametrize("q_max", [3, 8, 12])
def test_fp8_extend_vs_oracle(dev, d, Hq, Hkv, q_max, wpath):
    W_, sink, ks, vs = 64, 4, 0.75, 1.5
    rng = np.random.default_rng(3 * d + q_max)
    lens = [1, q_max, 50, sink + W_, sink + W_ + 2, 700, 4099]
    n_q = [1] + [int(rng.integers(1, q_max + 1)) for _ in lens[1:]]
    n_q = [min(n, S) for n, S in zip(n_q, lens)]
    B, S_max = len(lens), max(lens) + 3
    G.say(f"fp8 extend d={d} Hq={Hq} Hkv={Hkv} q_max={q_max} lens={lens} n_q={n_q}")
    q = I.normal_bf16((B, q_max, Hq, d), 41, dev)
    k8 = I.normal_fp8((B, S_max, Hkv, d), 42, dev)
    v8 = I.normal_fp8((B, S_max, Hkv, d), 43, dev)
    lt, nt = G.lens_tensor(lens, dev), G.lens_tensor(n_q, dev)
    scale = 1.0 / np.sqrt(d)
    qb = I.bf16_bits(q)
    err = G.err_word(dev)
    for variant in ("full", "windowed"):
        lse = torch.empty(B, q_max, Hq, dtype=torch.float32, device=dev)
        if variant == "full":
            out = W.draft_extend_full_fp8(q, k8, v8, lt, ks, vs, n_q=nt, lse=lse, err=err)
        else:
            out = W.draft_extend_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, n_q=nt, lse=lse, err=err)
        torch.cuda.synchronize()
        rows = [(F.DequantizedRows(HostCodes(k8[b]), ks), F.DequantizedRows(HostCodes(v8[b]), vs))
                for b in range(B)]
        refs = [A.attend_extend(qb[b], *rows[b], S, n, scale, variant, W_, sink)
                for b, (S, n) in enumerate(zip(lens, n_q))]
        spread = [A.extend_spread(qb[b], *rows[b], S, n, scale, variant, W_, sink)
                  for b, (S, n) in enumerate(zip(lens, n_q))]
        G.assert_attn_close(out, np.stack([r[0] for r in refs]), lse, np.stack([r[1] for r in refs]),
                            what=f"fp8 extend {variant}", spread=np.stack(spread))
    assert err.item() == 0
    # a ring sized exactly W + q_max - 1 gives the windowed result bit for bit
    R_w = W_ + q_max - 1
    kr, vr = _ring_from_dense(k8, lens, sink, R_w), _ring_from_dense(v8, lens, sink, R_w)
    ow = W.draft_extend_windowed_fp8(q, k8, v8, lt, W_, sink, ks, vs, n_q=nt)
    orr = W.ring_extend_fp8(q, kr, vr, lt, W_, sink, R_w, ks, vs, n_q=nt)
    torch.cuda.synchronize()
    assert torch.equal(orr, ow)
