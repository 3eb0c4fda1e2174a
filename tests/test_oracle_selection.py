"""Pins for the oracle's key selection (sink + recent window).

The oracle builds a boolean mask; these tests check it against the paper's
printed rule written as ranges (Appendix A pseudocode), the hand-worked
fixtures in tests/golden/, the closed form min(S, W + n_sink) (Section 6
"Memory") and structural properties of a sliding window.
"""

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import attention as A


def _ints(field):
    return [int(x) for x in field.split()] if field else []


def test_golden_selection_examples(golden):
    rows = golden("selection_examples.txt")
    assert len(rows) >= 8
    for S, W, sink, kept, _note in rows:
        got = A.selected_positions(int(S), int(W), int(sink)).tolist()
        assert got == _ints(kept), (S, W, sink)


def test_golden_paper_counts(golden):
    for name, args, expected, _cite in golden("paper_numbers.txt"):
        kv = dict(a.split("=") for a in args.split())
        kv = {k: int(v) for k, v in kv.items()}
        if name == "n_selected":
            assert A.n_selected(kv["S"], kv["W"], kv["sink"]) == int(expected)


def _pseudocode_ranges(S, W, sink):
    # The Appendix A rule exactly as printed: concatenated Python ranges.
    if S > sink + W:
        keep = list(range(0, sink)) + list(range(S - W, S))
    else:
        keep = list(range(0, S))
    return keep


@pytest.mark.parametrize("S", range(0, 41))
def test_mask_equals_printed_rule_exhaustive(S):
    for W in range(1, 9):
        for sink in range(0, 5):
            assert A.selected_positions(S, W, sink).tolist() == _pseudocode_ranges(S, W, sink)


@given(S=st.integers(0, 5000), W=st.integers(1, 600), sink=st.integers(0, 70))
@settings(max_examples=300, deadline=None)
def test_count_closed_form(S, W, sink):
    # Section 6 "Memory": the windowed draft reads min(seq, W + n_sink) tokens.
    assert A.n_selected(S, W, sink) == min(S, W + sink)


@given(S=st.integers(1, 3000), W=st.integers(1, 300), sink=st.integers(0, 40))
@settings(max_examples=300, deadline=None)
def test_structure(S, W, sink):
    pos = A.selected_positions(S, W, sink)
    assert pos[0] >= 0 and pos[-1] == S - 1          # current token always attended
    assert np.all(np.diff(pos) > 0)                   # ascending, no repeats
    head = np.arange(min(sink, S))
    assert np.array_equal(pos[: head.size], head)     # the sink is always kept
    tail = pos[head.size:]
    if tail.size:
        assert np.all(np.diff(tail) == 1)             # the window is contiguous
        assert tail.size <= max(W, S - sink)


@given(S=st.integers(0, 2000), W=st.integers(1, 200), sink=st.integers(0, 20))
@settings(max_examples=200, deadline=None)
def test_window_slides_by_one(S, W, sink):
    # One more token: the window gains S and, past the threshold, loses S - W.
    a = set(A.selected_positions(S, W, sink).tolist())
    b = set(A.selected_positions(S + 1, W, sink).tolist())
    assert S in b
    assert b - {S} <= a
    lost = a - b
    if S + 1 > sink + W:
        assert lost == {S - W}
    else:
        assert lost == set()


def test_degenerate_short_sequences_keep_everything():
    # Section 7 "When to window": once S <= W (+ sink) the window spans the
    # whole sequence and windowed degenerates to native.
    for S in range(0, 69):
        assert A.selected_positions(S, 64, 4).tolist() == list(range(S))
    assert A.selected_positions(69, 64, 4).tolist() != list(range(69))


def test_full_mask_counts():
    for S in (0, 1, 17, 1000):
        assert A.full_mask(S).sum() == S
