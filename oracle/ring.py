"""The compact ring-buffer draft KV store -- the oracle's model of it.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper facts this follows (Windowed-MTP):
  * Section 4 "Memory" and Section 6 "Memory": the windowed draft never reads
    anything but the sink and the recent window, so its KV pool is stored as
    a compact per-request ring of n_sink + W + d slots (d = gamma + 1 is the
    draft depth headroom); the Figure "window" caption says the same.
  * Appendix A pseudocode, ring comment: a request's rows live at
    ring_base(r) plus a slot derived from the logical position, with modulus
    n_sink + W + d.

Reading of that comment (the paper gives no further detail): the sink rows
are pinned to slots [0, sink) and never overwritten;
the other positions cycle through a circular region of R_w slots that follows
the sink, R_w = W + d in the paper's chain setting (any R_w >= W keeps the
whole window resident):

    slot(p) = p                          if p < sink
            = sink + ((p - sink) mod R_w) otherwise

Two independent statements of the ring live here and are checked against each
other by the CPU tests:
  * ring_slot()     -- the closed form above;
  * RingSimulator   -- an operational store: fixed sink slots filled in
                       arrival order, then a write pointer that walks the
                       circular region and wraps at its end, remembering which
                       logical position each slot last received.
ReplayCache is the logical model used for attention parity: every appended
row is kept in a plain list in position order, and the windowed attention of
oracle.attention is applied to that list.  A bulk append is the same as
appending its rows one by one (the last write to a slot wins).
"""

from __future__ import annotations

import numpy as np

from . import attention

__all__ = ["ring_slot", "ring_slots", "RingSimulator", "ReplayCache"]


def ring_slot(p: int, sink: int, R_w: int) -> int:
    """Slot of logical position p inside one request's ring (closed form)."""
    p = int(p)
    if p < sink:
        return p
    return sink + (p - sink) % R_w


def ring_slots(positions, sink: int, R_w: int) -> np.ndarray:
    """ring_slot applied to each position, as an int64 array."""
    return np.array([ring_slot(p, sink, R_w) for p in np.asarray(positions).ravel()],
                    dtype=np.int64)


class RingSimulator:
    """Operational ring of `sink` fixed slots plus a circular region of R_w.

    Rows arrive in logical order.  The first `sink` rows go to the fixed slots
    0, 1, ..., sink - 1 in arrival order; every later row goes to the slot the
    write pointer designates, after which the pointer advances and wraps back
    to the start of the circular region.  owner[slot] is the logical position
    last written into that slot.
    """

    def __init__(self, sink: int, R_w: int):
        if R_w < 1:
            raise ValueError("R_w must be >= 1")
        self.sink = int(sink)
        self.R_w = int(R_w)
        self.length = 0          # logical length (rows appended so far)
        self._next_sink = 0      # next fixed sink slot
        self._ptr = 0            # next offset inside the circular region
        self.owner: dict[int, int] = {}

    def append(self, count: int):
        """Append `count` rows; returns [(position, slot), ...] in order."""
        placed = []
        for _ in range(int(count)):
            p = self.length
            if self._next_sink < self.sink:
                slot = self._next_sink
                self._next_sink += 1
            else:
                slot = self.sink + self._ptr
                self._ptr += 1
                if self._ptr == self.R_w:
                    self._ptr = 0
            self.owner[slot] = p
            placed.append((p, slot))
            self.length += 1
        return placed

    def live_positions(self) -> np.ndarray:
        """Positions whose row is still held: the sink and the last R_w rows."""
        S = self.length
        p = np.arange(S)
        return p[(p < self.sink) | (p >= S - self.R_w)]


class ReplayCache:
    """Logical per-sequence draft KV: every appended row, in position order.

    k_rows / v_rows hold arrays of shape [Hkv, d] (bf16 bits or floats).
    """

    def __init__(self, Hkv: int, d: int, dtype=np.uint16):
        self.Hkv, self.d = int(Hkv), int(d)
        self._k: list[np.ndarray] = []
        self._v: list[np.ndarray] = []
        self._dtype = dtype

    @property
    def length(self) -> int:
        return len(self._k)

    def append(self, k_rows, v_rows):
        """Append rows k_rows[i], v_rows[i] (each [Hkv, d]) in order."""
        for kr, vr in zip(np.asarray(k_rows), np.asarray(v_rows)):
            self._k.append(np.array(kr, dtype=self._dtype))
            self._v.append(np.array(vr, dtype=self._dtype))

    def rows(self, positions):
        """Stacked (K, V) rows at the given logical positions."""
        idx = np.asarray(positions, dtype=np.int64)
        if idx.size == 0:
            shape = (0, self.Hkv, self.d)
            return np.zeros(shape, self._dtype), np.zeros(shape, self._dtype)
        return (np.stack([self._k[i] for i in idx]),
                np.stack([self._v[i] for i in idx]))

    def attend_windowed(self, q, scale: float, W: int, sink: int):
        """Windowed draft attention of query q [Hq, d] over this sequence."""
        S = self.length
        mask = attention.window_mask(S, W, sink)
        keep = np.flatnonzero(mask)
        # Only the kept rows are materialised; positions are renumbered
        # 0..n-1 in the same ascending order, and all of them are attended.
        K, V = self.rows(keep)
        return attention.attend_sequence(q, K, V, keep.size, scale, mask=None)
