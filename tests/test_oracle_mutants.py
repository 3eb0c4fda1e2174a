"""The oracle's pins catch plausible mistakes.

Each mutant below plants one mistake in the oracle (on the CPU, through
monkeypatching) -- an off-by-one window start, a non-strict threshold, a
dropped sink, a transposed GQA grouping, a missing scale, a dropped key, a
naive ring modulus, a value spread taken about zero, with unnormalised
weights or over the wrong KV group -- and the test asserts that at least one of the pin
checks (golden fixtures, the printed rule, torch SDPA, closed forms, the
operational ring) then fails.
"""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import ring as R

from .conftest import read_golden

_orig_mask = A.window_mask
_orig_attend = A.attend_sequence
_orig_slot = R.ring_slot
_orig_spread = A.value_spread


# ---------------------------------------------------------------- pin checks
def _pin_golden_selection():
    for S, W, sink, kept, _ in read_golden("selection_examples.txt"):
        exp = [int(x) for x in kept.split()] if kept else []
        if np.flatnonzero(A.window_mask(int(S), int(W), int(sink))).tolist() != exp:
            return False
    return True


def _pin_count_closed_form():
    for S in range(0, 60, 3):
        for W in (1, 4, 9):
            for sink in (0, 2, 5):
                if int(A.window_mask(S, W, sink).sum()) != min(S, W + sink):
                    return False
    return True


def _pin_sdpa():
    rng = np.random.default_rng(0)
    Hq, Hkv, d, S = 4, 2, 8, 40
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = rng.standard_normal((S, Hkv, d))
    for mask in (None, A.window_mask(S, 9, 2)):
        o, _ = A.attend_sequence(q, K, V, S, 0.3, mask)
        m = torch.ones(S, dtype=torch.bool) if mask is None else torch.from_numpy(mask)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q).view(1, Hq, 1, d),
            torch.from_numpy(K).permute(1, 0, 2).unsqueeze(0).contiguous(),
            torch.from_numpy(V).permute(1, 0, 2).unsqueeze(0).contiguous(),
            attn_mask=m.view(1, 1, 1, S), scale=0.3, enable_gqa=True).reshape(Hq, d).numpy()
        if not np.allclose(o, ref, rtol=0, atol=1e-12):
            return False
    return True


def _pin_zero_keys():
    rng = np.random.default_rng(1)
    S = 50
    V = rng.standard_normal((S, 1, 4))
    mask = A.window_mask(S, 7, 3)
    o, lse = A.attend_sequence(np.ones((1, 4)), np.zeros((S, 1, 4)), V, S, 1.0, mask)
    keep = np.flatnonzero(mask)
    return np.allclose(o[0], V[keep, 0].mean(axis=0), atol=1e-13) and abs(lse[0] - np.log(keep.size)) < 1e-12


def _pin_ring():
    for sink, R_w, positions, slots in read_golden("ring_examples.txt"):
        got = [R.ring_slot(int(p), int(sink), int(R_w)) for p in positions.split()]
        if got != [int(x) for x in slots.split()]:
            return False
    sim = R.RingSimulator(3, 7)
    for p, slot in sim.append(40):
        if slot != R.ring_slot(p, 3, 7):
            return False
    return True


def _pin_spread_bernoulli():
    # binary values: the weighted mean absolute deviation is 2 o (1 - o)
    rng = np.random.default_rng(3)
    Hq, Hkv, d, S = 6, 2, 8, 50
    q = rng.standard_normal((Hq, d))
    K = rng.standard_normal((S, Hkv, d))
    V = (rng.random((S, Hkv, d)) < 0.4).astype(np.float64)
    V[:, 1] = 1.0 - V[:, 1]  # the two KV groups differ
    for mask in (None, A.window_mask(S, 9, 2)):
        o, _ = _orig_attend(q, K, V, S, 0.5, mask)
        if not np.allclose(A.value_spread(q, K, V, S, 0.5, mask), 2 * o * (1 - o), rtol=0, atol=1e-12):
            return False
    return True


def _pin_spread_two_keys():
    rng = np.random.default_rng(4)
    q = rng.standard_normal((2, 4))
    K = rng.standard_normal((2, 1, 4))
    V = rng.standard_normal((2, 1, 4))
    s = A.value_spread(q, K, V, 2, 0.7)
    for h in range(2):
        w1 = 1.0 / (1.0 + np.exp(0.7 * float(q[h] @ (K[1, 0] - K[0, 0]))))
        if not np.allclose(s[h], 2 * w1 * (1 - w1) * np.abs(V[0, 0] - V[1, 0]), rtol=1e-12, atol=1e-15):
            return False
    return True


PINS = [_pin_golden_selection, _pin_count_closed_form, _pin_sdpa, _pin_zero_keys, _pin_ring,
        _pin_spread_bernoulli, _pin_spread_two_keys]


# ------------------------------------------------------------------- mutants
def _mask_window_off_by_one(S, W, sink):
    p = np.arange(S)
    if S > sink + W:
        return (p < sink) | (p > S - W)
    return np.ones(S, dtype=bool)


def _mask_non_strict(S, W, sink):
    p = np.arange(S)
    if S >= sink + W and S > 0:
        return (p < sink) | (p >= S - W + 1)
    return np.ones(S, dtype=bool)


def _mask_no_sink(S, W, sink):
    p = np.arange(S)
    if S > sink + W:
        return p >= S - W
    return np.ones(S, dtype=bool)


def _mask_window_includes_sink(S, W, sink):
    p = np.arange(S)
    if S > W:
        return (p < sink) | (p >= S - W + sink)
    return np.ones(S, dtype=bool)


def _attend_grouping_mod(q, K, V, S, scale, mask=None, chunk=65536):
    # query head h served by KV head h % Hkv instead of h // G
    Hq, Hkv = q.shape[0], K.shape[1]
    G = Hq // Hkv
    perm = np.array([(h % Hkv) * G + h // Hkv for h in range(Hq)])
    o, lse = _orig_attend(np.asarray(q)[perm], K, V, S, scale, mask, chunk)
    inv = np.argsort(perm)
    return o[inv], lse[inv]


def _attend_no_scale(q, K, V, S, scale, mask=None, chunk=65536):
    return _orig_attend(q, K, V, S, 1.0, mask, chunk)


def _attend_drop_last_key(q, K, V, S, scale, mask=None, chunk=65536):
    if mask is None:
        mask = np.ones(S, dtype=bool)
    m = np.array(mask, copy=True)
    if S:
        m[S - 1] = False
    return _orig_attend(q, K, V, S, scale, m, chunk)


def _spread_with(q, K, V, S, scale, mask, weight, about_output=True, group=None):
    """value_spread with one planted change: the weights (normalised or not),
    the deviation about the output or the raw magnitude, the KV group."""
    qf = np.asarray(q, dtype=np.float64)
    Hq, d = qf.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    keep = np.arange(S) if mask is None else np.flatnonzero(np.asarray(mask)[:S])
    out = np.zeros((Hq, d))
    if keep.size == 0:
        return out
    o, lse = _orig_attend(q, K, V, S, scale, mask)
    for h in range(Hq):
        g = h // G if group is None else group(h, Hkv)
        z = scale * (np.asarray(K[keep], dtype=np.float64)[:, g, :] @ qf[h])
        w = weight(z, lse[h])
        Vk = np.asarray(V[keep], dtype=np.float64)[:, g, :]
        out[h] = w @ (np.abs(Vk - o[h]) if about_output else np.abs(Vk))
    return out


def _spread_magnitude(q, K, V, S, scale, mask=None, chunk=4096):
    return _spread_with(q, K, V, S, scale, mask, lambda z, lse: np.exp(z - lse), about_output=False)


def _spread_unnormalised(q, K, V, S, scale, mask=None, chunk=4096):
    return _spread_with(q, K, V, S, scale, mask, lambda z, lse: np.exp(z - z.max()))


def _spread_grouping_mod(q, K, V, S, scale, mask=None, chunk=4096):
    return _spread_with(q, K, V, S, scale, mask, lambda z, lse: np.exp(z - lse), group=lambda h, Hkv: h % Hkv)


def _slot_naive_modulus(p, sink, R_w):
    return int(p) % (sink + R_w)


def _slot_absolute(p, sink, R_w):
    p = int(p)
    return p if p < sink else sink + p % R_w


MUTANTS = [
    ("window_mask", _mask_window_off_by_one),
    ("window_mask", _mask_non_strict),
    ("window_mask", _mask_no_sink),
    ("window_mask", _mask_window_includes_sink),
    ("attend_sequence", _attend_grouping_mod),
    ("attend_sequence", _attend_no_scale),
    ("attend_sequence", _attend_drop_last_key),
    ("value_spread", _spread_magnitude),
    ("value_spread", _spread_unnormalised),
    ("value_spread", _spread_grouping_mod),
    ("ring_slot", _slot_naive_modulus),
    ("ring_slot", _slot_absolute),
]


def test_pins_pass_on_the_oracle():
    assert all(pin() for pin in PINS)


@pytest.mark.parametrize("target,mutant", MUTANTS, ids=[m.__name__ for _, m in MUTANTS])
def test_each_mutant_fails_a_pin(monkeypatch, target, mutant):
    module = R if target == "ring_slot" else A
    monkeypatch.setattr(module, target, mutant)
    failed = [pin.__name__ for pin in PINS if not pin()]
    assert failed, f"mutant {mutant.__name__} passed every pin"
