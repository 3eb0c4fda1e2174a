"""Speculative draft rows in the compact ring: rollback of a rejected chain
and tree-width rings -- the oracle's model.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper facts this follows (Windowed-MTP):
  * Section 7, "Compatibility with tree speculation": the window decides
    which rows the draft reads, and is independent of how the candidates
    branch.  Sizing: all candidates read one common set of sink and window
    rows and keep private only their latest d draft rows, so one chain
    needs n_sink + W + d ring slots per request and each extra candidate
    adds d more (n_sink + W + d k for k candidates).
  * Appendix A pseudocode, ring comment: the chain ring's modulus is
    n_sink + W + d.
  * Section 3 (per-step latency model): each draft step writes its token's
    K/V row, then attends.

Readings (the paper gives no more detail):
  * Per request the state is the committed length S (rows the target has
    accepted) and the speculative depth i (draft steps since the last
    verify, 0 <= i <= d).  Candidate b's sequence is the committed rows
    [0, S) followed by its own rows at positions S .. S + i - 1; its draft
    step attends the windowed key set of that sequence at length S + i,
    after writing its row (oracle.attention.window_mask).
  * Layout: the chain ring of the Appendix A comment (sink slots plus a
    circular region of R_w = W + d slots, oracle.ring.ring_slot) holds the
    committed rows and candidate 0's speculative rows, which are written in
    place at the ring slot of their position, as a chain writes them; each
    further candidate b = 1 .. k-1 owns a private run of d slots, position
    S + t at slot t of run b - 1.  Total n_sink + W + d k (Section 7).
  * After the verify, the speculative depth returns to 0 (rollback: the rows
    stay and are overwritten later) and the accepted tokens' draft rows are
    written at their committed positions through the ring map (the
    draft-extend step, at most d + 1 rows: the accepted ones and the bonus
    token), which advances S.  R_w = W + d is exactly what that step needs:
    its first row's window must survive the writes of the last.
  * A chain that appends its speculative rows to the ring and advances the
    length with each (oracle.ring.RingSimulator) rolls back by lowering the
    length by the rejected count.

Two statements of the layout live here and are checked against each other by
the CPU tests: tree_slot() (closed form) and SlotStore (an operational store
that records, for every slot, which row was written there last).
SpecSequences is the logical model used for attention parity: plain lists of
committed and per-candidate rows, and oracle.attention's windowed attention
over candidate b's concatenated sequence.
"""

from __future__ import annotations

import numpy as np

from . import attention
from . import ring

__all__ = ["tree_slots_total", "tree_slot", "SlotStore", "SpecSequences", "ChainRing"]


def tree_slots_total(sink: int, W: int, d: int, k: int) -> int:
    """Slots one request reserves: sink + (W + d) ring + (k - 1) d private."""
    return int(sink) + int(W) + int(d) * int(k)


def tree_slot(p: int, S: int, b: int, sink: int, W: int, d: int, R_w: int | None = None) -> int:
    """Slot that candidate b reads position p from, committed length S
    (ring region of R_w = W + d slots, then the private runs).  R_w may be
    overridden to study undersized rings."""
    R_w = int(W) + int(d) if R_w is None else int(R_w)
    p, S, b = int(p), int(S), int(b)
    if p < S or b == 0:
        return ring.ring_slot(p, sink, R_w)
    return int(sink) + R_w + (b - 1) * int(d) + (p - S)


class SlotStore:
    """Operational store: remembers the row identity last written to each
    slot.  Writes follow the layout rules (a chain writes in place; private
    runs for candidates b >= 1) without tree_slot: a ring position is folded
    into the circular region by repeated subtraction, and a candidate's
    private run is filled by a cursor that every verify resets."""

    def __init__(self, sink: int, W: int, d: int, k: int, R_w: int | None = None):
        self.sink, self.W, self.d, self.k = int(sink), int(W), int(d), int(k)
        self.R_w = self.W + self.d if R_w is None else int(R_w)
        self.content: dict[int, tuple] = {}
        self._cursor = [0] * self.k

    def _ring_slot(self, p: int) -> int:
        # the circular region is walked position by position from the first
        # non-sink position: offset = number of non-sink positions before p,
        # folded by repeated subtraction of the region size
        if p < self.sink:
            return p
        off = p - self.sink
        while off >= self.R_w:
            off -= self.R_w
        return self.sink + off

    def write_committed(self, p: int):
        self.content[self._ring_slot(p)] = ("c", p)

    def write_speculative(self, b: int, p: int):
        if b == 0:
            slot = self._ring_slot(p)
        else:
            slot = self.sink + self.R_w + (b - 1) * self.d + self._cursor[b]
            self._cursor[b] += 1
        self.content[slot] = ("s", b, p)

    def verify(self):
        self._cursor = [0] * self.k

    def read(self, slot: int):
        return self.content.get(slot)


class SpecSequences:
    """Logical rows of one request: committed rows and each candidate's
    speculative rows, as plain lists ([Hkv, d] arrays)."""

    def __init__(self, k: int):
        self.k = int(k)
        self.committed: list[tuple] = []
        self.spec: list[list[tuple]] = [[] for _ in range(self.k)]

    @property
    def S(self) -> int:
        return len(self.committed)

    @property
    def depth(self) -> int:
        return len(self.spec[0])

    def speculate(self, rows):
        """One draft step: rows[b] = (k_row, v_row) of candidate b."""
        for b in range(self.k):
            self.spec[b].append((np.asarray(rows[b][0]), np.asarray(rows[b][1])))

    def verify(self, accepted_rows):
        """Rollback (depth -> 0), then commit the accepted tokens' rows."""
        self.spec = [[] for _ in range(self.k)]
        for kr, vr in accepted_rows:
            self.committed.append((np.asarray(kr), np.asarray(vr)))

    def sequence(self, b: int):
        return self.committed + self.spec[b]

    def attend(self, q, b: int, scale: float, W: int, sink: int, spread: bool = False):
        """Candidate b's windowed draft attention at length S + depth (with
        spread=True also oracle.attention.value_spread over the same rows)."""
        seq = self.sequence(b)
        L = len(seq)
        keep = attention.selected_positions(L, W, sink)
        if keep.size == 0:
            Hq, d = np.asarray(q).shape
            empty = (np.zeros((Hq, d)), np.full(Hq, -np.inf))
            return empty + (np.zeros((Hq, d)),) if spread else empty
        K = np.stack([seq[p][0] for p in keep])
        V = np.stack([seq[p][1] for p in keep])
        o, lse = attention.attend_sequence(q, K, V, keep.size, scale, None)
        if not spread:
            return o, lse
        return o, lse, attention.value_spread(q, K, V, keep.size, scale, None)


class ChainRing(ring.RingSimulator):
    """A chain's speculative appends through the operational ring, with
    rollback: the write pointer steps back over the rejected rows (a row
    that lands in the sink slots steps the sink cursor back)."""

    def rollback(self, n: int):
        n = int(n)
        if n < 0 or n > self.length:
            raise ValueError("cannot roll back more rows than were appended")
        for _ in range(n):
            self.length -= 1
            if self.length < self.sink:
                self._next_sink -= 1
            else:
                self._ptr = self.R_w - 1 if self._ptr == 0 else self._ptr - 1
