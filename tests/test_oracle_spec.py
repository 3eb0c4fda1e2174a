"""Pins of the speculation oracle (oracle.spec): chain rollback and
tree-width rings.

* the footprint the paper prints as a formula (n_sink + W + d k, Section 7)
  against the operational store filled over many speculate/verify rounds;
* tree_slot (closed form) against the operational store: after every write,
  every candidate reads every key of its window from a slot that holds
  exactly that row -- brute force over small shapes and random rounds;
* the sizing is tight: one slot less and a draft-extend over d + 1 rows
  clobbers a window row;
* the chain ring with rollback: the operational ring's write pointer steps
  back and forth as the paper's chain speculates and rejects, and its slots
  always equal the closed form; the window survives a rollback exactly when
  R_w >= W + (rows written past the committed length);
* candidate attention: a candidate whose rows equal another's attends
  identically, and k = 1 equals the plain windowed replay (oracle.ring).
"""

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import attention as A
from oracle import ring as R
from oracle import spec as P

from .conftest import read_golden


def _rounds(rng, n, d):
    """[(depth, accepted)] per round: depth in [1, d], accepted in [0, depth]."""
    out = []
    for _ in range(n):
        depth = int(rng.integers(1, d + 1))
        out.append((depth, int(rng.integers(0, depth + 1))))
    return out


def _run(sink, W, d, k, rounds, R_w=None, check=True):
    """Drive the operational store through speculate / verify rounds and
    compare every candidate's reads with tree_slot.  Returns (store, ok)."""
    store = P.SlotStore(sink, W, d, k, R_w)
    S = 0
    for depth, acc in rounds:
        for i in range(depth):
            for b in range(k):
                store.write_speculative(b, S + i)
            L = S + i + 1
            for b in range(k):
                for p in A.selected_positions(L, W, sink):
                    want = ("c", p) if p < S else ("s", b, p)
                    if store.read(P.tree_slot(p, S, b, sink, W, d, R_w)) != want:
                        if check:
                            raise AssertionError((sink, W, d, k, S, i, b, p))
                        return store, False
        store.verify()
        # the draft-extend step: the accepted rows plus the bonus token are
        # written first, then each of them attends causally
        for p in range(S, S + acc + 1):
            store.write_committed(p)
        for t in range(acc + 1):
            for p in A.selected_positions(S + t + 1, W, sink):
                if store.read(P.tree_slot(p, S + acc + 1, 0, sink, W, d, R_w)) != ("c", p):
                    if check:
                        raise AssertionError(("extend", S, t, p))
                    return store, False
        S += acc + 1
    return store, True


def test_golden_tree_footprint():
    rows = [r for r in read_golden("paper_numbers.txt") if r[0] == "tree_ring_slots"]
    assert len(rows) >= 2
    for _, args, expected, _cite in rows:
        kv = {a.split("=")[0]: int(a.split("=")[1]) for a in args.split()}
        assert P.tree_slots_total(kv["sink"], kv["W"], kv["dd"], kv["k"]) == int(expected)
        # the operational store, driven to full depth over many wraps, uses
        # exactly that many slots (scaled-down W keeps this fast; the count
        # is linear in W)
        small_W = 40
        rounds = [(kv["dd"], kv["dd"] - 1)] * 30
        store, ok = _run(kv["sink"], small_W, kv["dd"], kv["k"], rounds, check=False)
        assert ok
        used = len(store.content)
        assert used == int(expected) - kv["W"] + small_W
        assert max(store.content) + 1 == used


@pytest.mark.parametrize("sink,W,d,k", [(0, 1, 1, 1), (2, 5, 3, 2), (4, 9, 4, 3), (1, 3, 7, 4), (3, 16, 2, 5)])
def test_closed_form_equals_store_under_random_rounds(sink, W, d, k):
    rng = np.random.default_rng(sink * 100 + W * 10 + d + k)
    _run(sink, W, d, k, _rounds(rng, 60, d))


@given(sink=st.integers(0, 5), W=st.integers(1, 12), d=st.integers(1, 6), k=st.integers(1, 4),
       seed=st.integers(0, 10_000))
@settings(max_examples=150, deadline=None)
def test_closed_form_equals_store_hypothesis(sink, W, d, k, seed):
    _run(sink, W, d, k, _rounds(np.random.default_rng(seed), 25, d))


@pytest.mark.parametrize("sink,W,d,k", [(2, 5, 3, 1), (4, 9, 4, 3), (0, 7, 2, 2)])
def test_one_slot_less_clobbers_a_window_row(sink, W, d, k):
    # rounds at full depth whose verify accepts everything: the extend's d + 1
    # rows then reach one slot further than the window leaves free
    _, ok = _run(sink, W, d, k, [(d, d)] * 20, R_w=W + d - 1, check=False)
    assert not ok


def test_chain_rollback_walks_the_ring_like_the_closed_form():
    rng = np.random.default_rng(3)
    for sink, R_w in ((0, 5), (3, 8), (4, 16)):
        ring = P.ChainRing(sink, R_w)
        for _ in range(200):
            g = int(rng.integers(1, 6))
            for p, slot in ring.append(g):
                assert slot == R.ring_slot(p, sink, R_w)
            ring.rollback(int(rng.integers(0, g + 1)))
            for p, slot in ring.append(int(rng.integers(0, 3))):
                assert slot == R.ring_slot(p, sink, R_w)


def _window_survives(sink, W, R_w, S, gamma, a):
    """Append gamma speculative rows past committed length S, roll back to
    S + a: is every kept position still held by its own row?"""
    ring = P.ChainRing(sink, R_w)
    ring.append(S + gamma)
    ring.rollback(gamma - a)
    L = S + a
    return all(ring.owner.get(R.ring_slot(p, sink, R_w)) == p for p in A.selected_positions(L, W, sink))


@pytest.mark.parametrize("sink,W,gamma", [(0, 6, 3), (4, 20, 7), (2, 9, 1)])
def test_chain_rollback_needs_window_plus_gamma(sink, W, gamma):
    for S in range(0, 3 * (W + gamma) + sink, 3):
        for a in range(0, gamma + 1):
            assert _window_survives(sink, W, W + gamma, S, gamma, a), (S, a)
    # one slot less: rejecting everything loses a window row once S is large
    assert not all(_window_survives(sink, W, W + gamma - 1, S, gamma, 0)
                   for S in range(sink + W, 3 * (W + gamma) + sink))


def _rows(rng, n, Hkv=2, d=8):
    return [(rng.standard_normal((Hkv, d)), rng.standard_normal((Hkv, d))) for _ in range(n)]


def test_candidate_attention_is_windowed_attention_of_its_sequence():
    rng = np.random.default_rng(9)
    W, sink, k = 6, 2, 3
    seqs = P.SpecSequences(k)
    replay = R.ReplayCache(2, 8, dtype=np.float64)
    for rnd in range(8):
        depth = int(rng.integers(1, 4))
        for i in range(depth):
            rows = _rows(rng, 1) * k  # every candidate writes the same row
            seqs.speculate(rows)
            q = rng.standard_normal((4, 8))
            outs = [seqs.attend(q, b, 0.3, W, sink) for b in range(k)]
            for b in range(1, k):
                assert np.array_equal(outs[b][0], outs[0][0])
            # equals the plain replay of the committed rows plus the chain
            r2 = R.ReplayCache(2, 8, dtype=np.float64)
            seq = seqs.sequence(0)
            r2.append([x[0] for x in seq], [x[1] for x in seq])
            o, l = r2.attend_windowed(q, 0.3, W, sink)
            assert np.array_equal(o, outs[0][0]) and np.array_equal(l, outs[0][1])
        acc = _rows(rng, int(rng.integers(1, depth + 2)))
        seqs.verify(acc)
        replay.append([x[0] for x in acc], [x[1] for x in acc])
        assert seqs.S == replay.length and seqs.depth == 0


# ------------------------------------------------------------------ mutants
def _pins_fail(monkeypatch, fn):
    monkeypatch.setattr(P, "tree_slot", fn)
    rng = np.random.default_rng(1)
    try:
        for sink, W, d, k in [(2, 5, 3, 2), (4, 9, 4, 3), (1, 3, 7, 4)]:
            _run(sink, W, d, k, _rounds(rng, 40, d))
            _run(sink, W, d, k, [(d, d)] * 10)
    except AssertionError:
        return True
    return False


def test_mutant_overlapping_private_runs(monkeypatch):
    orig = P.tree_slot
    def bad(p, S, b, sink, W, d, R_w=None):
        if p < S or b == 0:
            return orig(p, S, b, sink, W, d, R_w)
        return sink + (W + d if R_w is None else R_w) + (b - 1) * (d - 1) + (p - S)
    assert _pins_fail(monkeypatch, bad)


def test_mutant_every_candidate_in_place(monkeypatch):
    orig = P.tree_slot
    assert _pins_fail(monkeypatch, lambda p, S, b, sink, W, d, R_w=None: orig(p, S, 0, sink, W, d, R_w))


def test_mutant_ring_without_headroom(monkeypatch):
    orig = P.tree_slot
    assert _pins_fail(monkeypatch, lambda p, S, b, sink, W, d, R_w=None: orig(p, S, b, sink, W, d, W))


def test_mutant_private_run_indexed_from_zero_length(monkeypatch):
    orig = P.tree_slot
    def bad(p, S, b, sink, W, d, R_w=None):
        if p < S or b == 0:
            return orig(p, S, b, sink, W, d, R_w)
        return sink + W + d + (b - 1) * d + (p % d)
    assert _pins_fail(monkeypatch, bad)


def test_spread_option_over_binary_rows():
    rng = np.random.default_rng(8)
    Hkv, d = 2, 8
    seqs = P.SpecSequences(3)
    row = lambda: (rng.standard_normal((Hkv, d)), (rng.random((Hkv, d)) < 0.5).astype(np.float64))
    seqs.verify([row() for _ in range(40)])
    seqs.speculate([row() for _ in range(3)])
    q = rng.standard_normal((4, d))
    for b in range(3):
        o, lse, s = seqs.attend(q, b, 0.3, 16, 2, spread=True)
        o2, lse2 = seqs.attend(q, b, 0.3, 16, 2)
        assert np.array_equal(o, o2) and np.array_equal(lse, lse2)
        np.testing.assert_allclose(s, 2 * o * (1 - o), atol=1e-13)
    empty = P.SpecSequences(1)
    o, lse, s = empty.attend(q, 0, 0.3, 16, 2, spread=True)
    assert np.all(s == 0) and np.all(np.isneginf(lse))
