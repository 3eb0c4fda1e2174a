"""Pins for the oracle's ring-buffer model of the compact draft KV store.

The closed-form slot map is checked against an operational simulator (fixed
sink slots plus a wrapping write pointer), the hand-worked fixture, the
footprint the paper prints (n_sink + W + d slots, Figure "window" and
Section 6 "Memory"), and the spec invariant that windowed attention over
the ring's logical content equals windowed attention over the uncompacted
full cache.
"""

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import attention as A
from oracle import ring as R


def test_golden_slot_examples(golden):
    for sink, R_w, positions, slots in golden("ring_examples.txt"):
        pos = [int(x) for x in positions.split()]
        exp = [int(x) for x in slots.split()]
        assert R.ring_slots(pos, int(sink), int(R_w)).tolist() == exp


def test_golden_footprint(golden):
    for name, args, expected, _cite in golden("paper_numbers.txt"):
        if name != "ring_slots":
            continue
        kv = {k: int(v) for k, v in (a.split("=") for a in args.split())}
        R_w = kv["W"] + kv["dd"]  # the window plus the draft-depth headroom
        sim = R.RingSimulator(kv["sink"], R_w)
        sim.append(3 * (kv["sink"] + R_w) + 17)  # many wraps
        assert len(sim.owner) == int(expected)
        assert max(sim.owner) + 1 == int(expected)


@given(sink=st.integers(0, 9), R_w=st.integers(1, 40),
       chunks=st.lists(st.integers(0, 25), min_size=1, max_size=40))
@settings(max_examples=300, deadline=None)
def test_closed_form_matches_operational_ring(sink, R_w, chunks):
    sim = R.RingSimulator(sink, R_w)
    for c in chunks:
        for p, slot in sim.append(c):
            assert slot == R.ring_slot(p, sink, R_w)
        # every row still held is found where the closed form says
        for p in sim.live_positions():
            assert sim.owner[R.ring_slot(p, sink, R_w)] == p
    # footprint never exceeds sink + R_w slots
    assert len(sim.owner) == min(sim.length, sink + R_w)
    assert all(0 <= s < sink + R_w for s in sim.owner)


@given(sink=st.integers(0, 9), W=st.integers(1, 30), extra=st.integers(0, 8), S=st.integers(0, 400))
@settings(max_examples=300, deadline=None)
def test_window_fits_in_ring_without_collision(sink, W, extra, S):
    # With R_w >= W every selected position has its own slot, so the ring
    # holds the whole key set of the windowed draft.
    R_w = W + extra
    pos = A.selected_positions(S, W, sink)
    slots = R.ring_slots(pos, sink, R_w)
    assert len(set(slots.tolist())) == pos.size
    sim = R.RingSimulator(sink, R_w)
    sim.append(S)
    for p, s in zip(pos, slots):
        assert sim.owner[int(s)] == int(p)


def test_ring_too_small_loses_window_rows():
    # R_w < W: two window positions share a slot (the reading needs R_w >= W).
    pos = A.selected_positions(100, 10, 2)
    slots = R.ring_slots(pos, 2, 9)
    assert len(set(slots.tolist())) < pos.size


@pytest.mark.parametrize("sink,R_w", [(4, 2048), (0, 16), (3, 5)])
def test_layout_equals_full_cache_prefix_before_first_wrap(sink, R_w):
    for p in range(sink + R_w):
        assert R.ring_slot(p, sink, R_w) == p
    assert R.ring_slot(sink + R_w, sink, R_w) == sink


def _rows(rng, n, Hkv=2, d=8):
    return rng.standard_normal((n, Hkv, d)), rng.standard_normal((n, Hkv, d))


@given(seed=st.integers(0, 10**6), sink=st.integers(0, 5), W=st.integers(1, 24),
       extra=st.integers(0, 4), counts=st.lists(st.integers(1, 8), min_size=1, max_size=30))
@settings(max_examples=80, deadline=None)
def test_ring_attention_equals_windowed_on_full_cache(seed, sink, W, extra, counts):
    rng = np.random.default_rng(seed)
    Hq, Hkv, d = 4, 2, 8
    cache = R.ReplayCache(Hkv, d, dtype=np.float64)
    full_k, full_v = [], []
    for c in counts:
        k, v = _rows(rng, c, Hkv, d)
        cache.append(k, v)
        full_k.append(k)
        full_v.append(v)
        K = np.concatenate(full_k)
        V = np.concatenate(full_v)
        q = rng.standard_normal((Hq, d))
        o1, l1 = cache.attend_windowed(q, 0.35, W, sink)
        o2, l2 = A.attend_sequence(q, K, V, K.shape[0], 0.35, A.window_mask(K.shape[0], W, sink))
        np.testing.assert_allclose(o1, o2, atol=1e-13)
        np.testing.assert_allclose(l1, l2, atol=1e-13)


def test_physical_ring_content_reproduces_logical_rows():
    # Write rows into a physical slot array with the closed-form map, one by
    # one, then read the windowed key set back through the map: the rows are
    # the logical ones (no live row was overwritten).
    rng = np.random.default_rng(11)
    sink, W, R_w, Hkv, d = 4, 16, 19, 2, 8
    phys = np.full((sink + R_w, Hkv, d), np.nan)
    cache = R.ReplayCache(Hkv, d, dtype=np.float64)
    S = 0
    for c in rng.integers(1, 9, size=60):
        k, v = _rows(rng, int(c), Hkv, d)
        cache.append(k, v)
        for i in range(int(c)):
            phys[R.ring_slot(S + i, sink, R_w)] = k[i]
        S += int(c)
        pos = A.selected_positions(S, W, sink)
        got = phys[R.ring_slots(pos, sink, R_w)]
        exp, _ = cache.rows(pos)
        assert np.array_equal(got, exp)
