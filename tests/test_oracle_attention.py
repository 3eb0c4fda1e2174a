"""Pins for the oracle's float64 masked-softmax GQA decode attention.

Each test ties the oracle to something other than itself: hand-computed
values (tests/golden/attention_worked.txt), closed forms (zero keys, identical
keys, one dominant key, constant values), a pure-Python brute force, a library
routine (torch scaled_dot_product_attention in float64 on the CPU, with a
boolean mask and GQA head expansion), and invariants the paper states
(windowed equals full when S <= W + sink, Section 7; the reduced key set is
the whole key set, Section 4 "Mechanism").
"""

import math

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import attention as A
from paper_2607_21535_amd import inputs as I


def _rand_case(seed, S, Hq=4, Hkv=2, d=8, bf16=True):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = rng.standard_normal((S, Hkv, d))
    if bf16:
        # Exercise the bit-pattern input path with real bf16 inputs.
        q = I.bf16_bits(torch.from_numpy(q).to(torch.bfloat16))
        K = I.bf16_bits(torch.from_numpy(K).to(torch.bfloat16))
        V = I.bf16_bits(torch.from_numpy(V).to(torch.bfloat16))
    return q, K, V


def test_worked_example(golden):
    q = np.array([[1.0]])
    K = np.array([0.0, math.log(2.0), math.log(3.0)]).reshape(3, 1, 1)
    V = np.array([6.0, 0.0, 12.0]).reshape(3, 1, 1)
    for variant, W, sink, o_exp, Z in golden("attention_worked.txt"):
        mask = None if variant == "full" else A.window_mask(3, int(W), int(sink))
        o, lse = A.attend_sequence(q, K, V, 3, 1.0, mask)
        assert o[0, 0] == pytest.approx(float(o_exp), rel=1e-14)
        assert math.exp(lse[0]) == pytest.approx(float(Z), rel=1e-14)


def test_bf16_widening_matches_torch():
    x = torch.randn(4096) * 37.0
    xb = x.to(torch.bfloat16)
    ref = xb.to(torch.float64).numpy()
    assert np.array_equal(A.bf16_to_f64(I.bf16_bits(xb)), ref)
    specials = torch.tensor([0.0, -0.0, 1e-40, 3.0e38, -2.5], dtype=torch.bfloat16)
    assert np.array_equal(A.bf16_to_f64(I.bf16_bits(specials)), specials.to(torch.float64).numpy())


def _sdpa_reference(q, K, V, S, scale, mask):
    """torch SDPA (float64, CPU) with a boolean key mask and GQA expansion."""
    qf = torch.from_numpy(A.bf16_to_f64(q) if q.dtype == np.uint16 else q)
    Kf = torch.from_numpy(A.bf16_to_f64(K[:S]) if K.dtype == np.uint16 else K[:S])
    Vf = torch.from_numpy(A.bf16_to_f64(V[:S]) if V.dtype == np.uint16 else V[:S])
    Hq = qf.shape[0]
    Hkv = Kf.shape[1]
    qq = qf.reshape(1, Hq, 1, -1)
    kk = Kf.permute(1, 0, 2).unsqueeze(0).contiguous()
    vv = Vf.permute(1, 0, 2).unsqueeze(0).contiguous()
    m = torch.ones(S, dtype=torch.bool) if mask is None else torch.from_numpy(mask)
    out = torch.nn.functional.scaled_dot_product_attention(
        qq, kk, vv, attn_mask=m.view(1, 1, 1, S), scale=scale, enable_gqa=(Hq != Hkv))
    return out.reshape(Hq, -1).numpy()


@pytest.mark.parametrize("S,W,sink", [(1, 4, 2), (7, 4, 2), (37, 8, 3), (200, 16, 4), (513, 64, 0)])
@pytest.mark.parametrize("Hq,Hkv", [(4, 2), (8, 1), (6, 3), (2, 2)])
def test_matches_torch_sdpa(S, W, sink, Hq, Hkv):
    q, K, V = _rand_case(S * 31 + Hq, S, Hq=Hq, Hkv=Hkv, d=16)
    scale = 1.0 / 4.0
    for mask in (None, A.window_mask(S, W, sink)):
        o, _ = A.attend_sequence(q, K, V, S, scale, mask)
        ref = _sdpa_reference(q, K, V, S, scale, mask)
        np.testing.assert_allclose(o, ref, rtol=0, atol=1e-12)


def _brute_force(q, K, V, S, scale, keep):
    """Pure-Python loops, one head at a time (tiny sizes only)."""
    Hq, d = len(q), len(q[0])
    Hkv = len(K[0])
    G = Hq // Hkv
    o = [[0.0] * d for _ in range(Hq)]
    lse = []
    for h in range(Hq):
        g = h // G
        logits = []
        for p in keep:
            logits.append(scale * sum(q[h][c] * K[p][g][c] for c in range(d)))
        mx = max(logits)
        ws = [math.exp(z - mx) for z in logits]
        tot = sum(ws)
        for c in range(d):
            o[h][c] = sum(w * V[p][g][c] for w, p in zip(ws, keep)) / tot
        lse.append(mx + math.log(tot))
    return np.array(o), np.array(lse)


@pytest.mark.parametrize("S", [1, 2, 5, 9, 16, 23])
def test_brute_force_tiny(S):
    rng = np.random.default_rng(S)
    Hq, Hkv, d = 4, 2, 3
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = rng.standard_normal((S, Hkv, d))
    for W, sink in [(3, 1), (4, 0), (2, 2), (30, 3)]:
        if S > sink + W:
            keep = list(range(sink)) + list(range(S - W, S))
        else:
            keep = list(range(S))
        o, lse = A.attend_sequence(q, K, V, S, 0.7, A.window_mask(S, W, sink))
        bo, blse = _brute_force(q.tolist(), K.tolist(), V.tolist(), S, 0.7, keep)
        np.testing.assert_allclose(o, bo, rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse, blse, rtol=0, atol=1e-13)
    o, lse = A.attend_sequence(q, K, V, S, 0.7, None)
    bo, blse = _brute_force(q.tolist(), K.tolist(), V.tolist(), S, 0.7, list(range(S)))
    np.testing.assert_allclose(o, bo, rtol=0, atol=1e-13)


@pytest.mark.parametrize("S,W,sink", [(100, 10, 4), (64, 64, 4), (5, 10, 2), (3000, 512, 4)])
def test_zero_keys_give_mean_of_kept_values(S, W, sink):
    # All logits 0 -> every kept key has weight 1/n: o is the mean of the kept
    # value rows and lse = ln(n).
    _, _, V = _rand_case(S, S, Hq=4, Hkv=2, d=8, bf16=False)
    K = np.zeros((S, 2, 8))
    q = np.ones((4, 8))
    mask = A.window_mask(S, W, sink)
    keep = np.flatnonzero(mask)
    o, lse = A.attend_sequence(q, K, V, S, 0.3, mask)
    for h in range(4):
        np.testing.assert_allclose(o[h], V[keep, h // 2].mean(axis=0), atol=1e-13)
    np.testing.assert_allclose(lse, np.log(keep.size), atol=1e-13)


def test_identical_keys_give_mean():
    S = 50
    rng = np.random.default_rng(3)
    u = rng.standard_normal(8)
    K = np.broadcast_to(u, (S, 1, 8)).copy()
    V = rng.standard_normal((S, 1, 8))
    q = rng.standard_normal((2, 8))
    o, lse = A.attend_sequence(q, K, V, S, 0.5, A.window_mask(S, 10, 2))
    keep = A.selected_positions(S, 10, 2)
    for h in range(2):
        np.testing.assert_allclose(o[h], V[keep, 0].mean(axis=0), atol=1e-13)
        assert lse[h] == pytest.approx(0.5 * q[h] @ u + math.log(keep.size), abs=1e-12)


def test_dominant_key_returns_its_value():
    S, d = 300, 4
    rng = np.random.default_rng(5)
    q = np.zeros((1, d))
    q[0, 0] = 1.0
    K = rng.standard_normal((S, 1, d)) * 0.1
    V = rng.standard_normal((S, 1, d))
    for star in (0, 1, 150, 299):
        K2 = K.copy()
        K2[star, 0, 0] = 45.0  # logit about 45 above the rest
        o, _ = A.attend_sequence(q, K2, V, S, 1.0)
        np.testing.assert_allclose(o[0], V[star, 0], atol=1e-15 * S + 1e-17)
    # A dominant key outside the window is not seen by the windowed draft.
    K2 = K.copy()
    K2[150, 0, 0] = 45.0
    o, _ = A.attend_sequence(q, K2, V, S, 1.0, A.window_mask(S, 20, 4))
    assert np.abs(o[0] - V[150, 0]).max() > 0.1


def test_constant_values_and_convexity():
    S = 400
    q, K, _ = _rand_case(9, S, bf16=False)
    V = np.ones((S, 2, 8))
    for mask in (None, A.window_mask(S, 32, 4)):
        o, _ = A.attend_sequence(q, K, V, S, 0.35, mask)
        np.testing.assert_allclose(o, 1.0, atol=1e-14)  # weights sum to 1
    _, _, V = _rand_case(10, S, bf16=False)
    o, _ = A.attend_sequence(q, K, V, S, 0.35)
    for h in range(4):
        g = h // 2
        assert np.all(o[h] <= V[:, g].max(axis=0) + 1e-12)
        assert np.all(o[h] >= V[:, g].min(axis=0) - 1e-12)


@given(S=st.integers(1, 300), W=st.integers(1, 64), sink=st.integers(0, 8), seed=st.integers(0, 10**6))
@settings(max_examples=60, deadline=None)
def test_windowed_equals_attention_on_reduced_cache(S, W, sink, seed):
    # Section 4 "Mechanism": the reduced table is the key set.  Windowed
    # attention must equal full attention over a cache that physically holds
    # only the kept rows (taken with the printed ranges).
    q, K, V = _rand_case(seed, S, d=8)
    keep = list(range(sink)) + list(range(S - W, S)) if S > sink + W else list(range(S))
    o1, l1 = A.attend_sequence(q, K, V, S, 0.3, A.window_mask(S, W, sink))
    o2, l2 = A.attend_sequence(q, K[keep], V[keep], len(keep), 0.3, None)
    np.testing.assert_allclose(o1, o2, atol=1e-13)
    np.testing.assert_allclose(l1, l2, atol=1e-13)


@pytest.mark.parametrize("S", [1, 30, 68])
def test_windowed_degenerates_to_full(S):
    # Section 7 "When to window": S <= W + sink -> identical to native.
    q, K, V = _rand_case(S, S)
    o1, l1 = A.attend_sequence(q, K, V, S, 0.3, A.window_mask(S, 64, 4))
    o2, l2 = A.attend_sequence(q, K, V, S, 0.3, None)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_windowed_differs_from_full_past_threshold():
    S = 4000
    q, K, V = _rand_case(1, S)
    o1, _ = A.attend_sequence(q, K, V, S, 0.3, A.window_mask(S, 256, 4))
    o2, _ = A.attend_sequence(q, K, V, S, 0.3, None)
    assert np.linalg.norm(o1 - o2) > 0.1 * np.linalg.norm(o2)


def test_logit_shift_invariance():
    # Adding one vector u to every key shifts each head's logits by a
    # constant: the output is unchanged and lse moves by scale * <q_h, u>.
    S = 257
    q, K, V = _rand_case(2, S, bf16=False)
    u = np.random.default_rng(0).standard_normal(8) * 3
    for mask in (None, A.window_mask(S, 40, 3)):
        o1, l1 = A.attend_sequence(q, K, V, S, 0.4, mask)
        o2, l2 = A.attend_sequence(q, K + u, V, S, 0.4, mask)
        np.testing.assert_allclose(o1, o2, atol=1e-12)
        np.testing.assert_allclose(l2 - l1, 0.4 * (q @ u), atol=1e-11)


def test_scale_is_applied_to_logits():
    S = 90
    q, K, V = _rand_case(4, S, bf16=False)
    o1, l1 = A.attend_sequence(q, K, V, S, 0.5)
    o2, l2 = A.attend_sequence(2.0 * q, K, V, S, 0.25)
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    np.testing.assert_allclose(l1, l2, atol=1e-13)


def test_gqa_grouping_is_consecutive():
    # Reading: query head h uses KV head h // G.  Heads of one group see the
    # same keys: giving every head of a group the same query gives the same
    # output, and a group's output only depends on its own KV head.
    S = 120
    q, K, V = _rand_case(6, S, Hq=6, Hkv=3, bf16=False)
    q[1] = q[0]
    q[3] = q[2]
    o, _ = A.attend_sequence(q, K, V, S, 0.3)
    np.testing.assert_allclose(o[0], o[1], atol=1e-15)
    np.testing.assert_allclose(o[2], o[3], atol=1e-15)
    K2, V2 = K.copy(), V.copy()
    K2[:, 2] += 1.0
    V2[:, 2] *= -1.0
    o2, _ = A.attend_sequence(q, K2, V2, S, 0.3)
    np.testing.assert_allclose(o2[:4], o[:4], atol=0)
    assert np.abs(o2[4:] - o[4:]).max() > 1e-3


def test_chunked_passes_equal_single_pass():
    S = 1000
    q, K, V = _rand_case(8, S)
    for mask in (None, A.window_mask(S, 300, 5)):
        o1, l1 = A.attend_sequence(q, K, V, S, 0.3, mask, chunk=7)
        o2, l2 = A.attend_sequence(q, K, V, S, 0.3, mask, chunk=1 << 20)
        np.testing.assert_allclose(o1, o2, atol=1e-14)
        np.testing.assert_allclose(l1, l2, atol=1e-13)


def test_empty_sequence():
    q, K, V = _rand_case(0, 4)
    for mask in (None, A.window_mask(0, 4, 2)):
        o, lse = A.attend_sequence(q, K, V, 0, 0.3, mask)
        assert np.all(o == 0) and np.all(np.isneginf(lse))


def test_sink_bias_case():
    wl = I.WORKLOADS["draft_loop_s1m"]
    case = I.decode_case(wl, "cpu", S=600, steps=1)
    kb = I.bf16_bits(case["k"])
    # The x4 bias rows are exact in bf16.
    raw = I.normal_bf16((600, 2, 256), I.stream_seed(wl.seed, I.STREAM_K, 0))
    assert np.array_equal(A.bf16_to_f64(kb[0, :4]), 4.0 * raw[:4].to(torch.float64).numpy())


# ---------------------------------------------------------------- extend
def _sdpa_extend(q, K, V, S, n, scale, W=None, sink=None):
    """torch SDPA (float64) over all new rows at once with an explicit
    [n, S] boolean mask built from positions: row t is the token at position
    S - n + t; it may see p <= S - n + t, and under the window only the sink
    and the last W of those."""
    qf = torch.from_numpy(A.bf16_to_f64(q[:n]))             # [n, Hq, d]
    Kf = torch.from_numpy(A.bf16_to_f64(K[:S]))
    Vf = torch.from_numpy(A.bf16_to_f64(V[:S]))
    n_, Hq, d = qf.shape
    Hkv = Kf.shape[1]
    me = torch.arange(S - n, S).view(n, 1)                  # each row's own position
    p = torch.arange(S).view(1, S)
    m = p <= me
    if W is not None:
        L = me + 1
        m = m & ((L <= sink + W) | (p < sink) | (p >= L - W))
    out = torch.nn.functional.scaled_dot_product_attention(
        qf.permute(1, 0, 2).unsqueeze(0), Kf.permute(1, 0, 2).unsqueeze(0).contiguous(),
        Vf.permute(1, 0, 2).unsqueeze(0).contiguous(), attn_mask=m.view(1, 1, n, S), scale=scale,
        enable_gqa=(Hq != Hkv))
    return out[0].permute(1, 0, 2).numpy()


@pytest.mark.parametrize("S,n,q_max", [(1, 1, 1), (5, 3, 4), (40, 8, 8), (300, 5, 8), (2100, 4, 4)])
@pytest.mark.parametrize("W,sink", [(None, None), (16, 2), (1, 0), (64, 4)])
def test_extend_matches_causal_sdpa(S, n, q_max, W, sink):
    q, K, V = _rand_case(S + n, S, Hq=4, Hkv=2, d=8)
    qr = I.bf16_bits(torch.from_numpy(np.random.default_rng(S).standard_normal((q_max, 4, 8))).to(torch.bfloat16))
    variant = "full" if W is None else "windowed"
    o, lse = A.attend_extend(qr, K, V, S, n, 0.3, variant, W, sink)
    ref = _sdpa_extend(qr, K, V, S, n, 0.3, W, sink)
    np.testing.assert_allclose(o[:n], ref, atol=1e-12)
    assert np.all(o[n:] == 0) and np.all(np.isneginf(lse[n:]))


def test_extend_rows_are_decode_steps():
    # Row t of an extend equals a decode step at length S - n + t + 1, and a
    # one-row extend is exactly the decode step.
    S, n = 500, 6
    q, K, V = _rand_case(1, S, Hq=4, Hkv=2, d=8)
    qr = np.stack([I.bf16_bits(torch.randn(4, 8).to(torch.bfloat16)) for _ in range(n)])
    o, lse = A.attend_extend(qr, K, V, S, n, 0.3, "windowed", 32, 3)
    for t in range(n):
        L = S - n + t + 1
        od, ld = A.attend_sequence(qr[t], K, V, L, 0.3, A.window_mask(L, 32, 3))
        assert np.array_equal(o[t], od) and np.array_equal(lse[t], ld)
    assert A.extend_lengths(S, 1, 1) == [S]
    assert A.extend_lengths(10, 3, 5) == [8, 9, 10, 0, 0]


# ---------------------------------------------------------- value spread
# value_spread sizes the effect of perturbed weights in the GPU tolerances;
# it is pinned by closed forms that do not restate its definition.
def test_spread_of_binary_values_is_bernoulli():
    # values in {0, 1}: for any weights, o = P(v = 1) and the mean absolute
    # deviation of a Bernoulli variable about its mean is 2 o (1 - o)
    rng = np.random.default_rng(5)
    Hq, Hkv, d, S = 6, 2, 16, 90
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = (rng.random((S, Hkv, d)) < np.linspace(0.05, 0.95, d)).astype(np.float64)
    for mask in (None, A.window_mask(S, 20, 3)):
        o, _ = A.attend_sequence(q, K, V, S, 0.4, mask)
        s = A.value_spread(q, K, V, S, 0.4, mask)
        np.testing.assert_allclose(s, 2 * o * (1 - o), atol=1e-13)


def test_spread_of_two_keys_closed_form():
    # two keys with logits z1, z2: w1 = 1 / (1 + e^(z2 - z1)), w2 = 1 - w1 and
    # |v1 - o| = w2 |v1 - v2|, |v2 - o| = w1 |v1 - v2|, so spread = 2 w1 w2 |v1 - v2|
    rng = np.random.default_rng(6)
    Hq, Hkv, d = 4, 2, 8
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((2, Hkv, d))
    V = rng.standard_normal((2, Hkv, d)) * 3
    s = A.value_spread(q, K, V, 2, 0.9)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        z1, z2 = 0.9 * float(q[h] @ K[0, g]), 0.9 * float(q[h] @ K[1, g])
        w1 = 1.0 / (1.0 + np.exp(z2 - z1))
        np.testing.assert_allclose(s[h], 2 * w1 * (1 - w1) * np.abs(V[0, g] - V[1, g]), rtol=1e-12, atol=1e-15)


def test_spread_shift_scale_and_degenerate_cases():
    rng = np.random.default_rng(7)
    Hq, Hkv, d, S = 4, 1, 8, 40
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = rng.standard_normal((S, Hkv, d))
    s = A.value_spread(q, K, V, S, 0.5)
    np.testing.assert_allclose(A.value_spread(q, K, V + 7.5, S, 0.5), s, atol=1e-12)   # deviation about o
    np.testing.assert_allclose(A.value_spread(q, K, -3.0 * V, S, 0.5), 3.0 * s, rtol=1e-12)
    const = np.broadcast_to(rng.standard_normal((1, Hkv, d)), (S, Hkv, d))
    assert np.abs(A.value_spread(q, K, const, S, 0.5)).max() < 1e-13                  # no deviation
    assert np.all(A.value_spread(q, K, V, 1, 0.5) == 0)                               # one key
    assert np.all(A.value_spread(q, K, V, 0, 0.5) == 0)                               # no key
    # a dominant key (logit +40 above every other) leaves almost no spread
    Kd = np.zeros((S, Hkv, d))
    Kd[11, 0, :] = 40.0 / 0.5 / np.abs(q[0]).sum() * np.sign(q[0])   # q[0] . k = 80: logit 40
    qd = np.tile(q[:1], (Hq, 1))
    assert np.abs(A.value_spread(qd, Kd, V, S, 0.5)).max() < 1e-12
    # chunking does not change it
    np.testing.assert_allclose(A.value_spread(q, K, V, S, 0.5, chunk=7), s, atol=1e-14)


def test_extend_spread_rows_are_decode_steps():
    S, n = 300, 5
    q, K, V = _rand_case(1, S, Hq=4, Hkv=2, d=8)
    qr = np.stack([I.bf16_bits(torch.randn(4, 8).to(torch.bfloat16)) for _ in range(n + 2)])
    sp = A.extend_spread(qr, K, V, S, n, 0.3, "windowed", 32, 3)
    for t in range(n):
        L = S - n + t + 1
        assert np.array_equal(sp[t], A.value_spread(qr[t], K, V, L, 0.3, A.window_mask(L, 32, 3)))
    assert np.all(sp[n:] == 0)
