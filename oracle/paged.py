"""The paged draft KV (token pool with page size 1) -- the oracle's model.

TEST INFRASTRUCTURE ONLY (see the package docstring).

In the paper's serving setup every request's KV rows live in a shared pool
and req_to_token[r, p] names the pool row of position p of request r.
Windowed-MTP changes only the draft's index construction (Section 4
"Mechanism"; Appendix A pseudocode): kv_index = req_to_token[r, keep], with
keep the full range natively or the sink followed by the recent window.  The
attention itself is unchanged: it attends exactly the listed rows, in order.
"""

from __future__ import annotations

import numpy as np

from . import attention

__all__ = ["keep_positions", "kv_indices", "attend_paged"]


def keep_positions(S: int, variant: str, W: int | None = None, sink: int | None = None) -> np.ndarray:
    """Positions the draft attends at length S: all of them, or the window rule."""
    if variant == "full":
        return np.arange(int(S), dtype=np.int64)
    return attention.selected_positions(S, W, sink)


def kv_indices(table, lens, variant: str, W: int | None = None, sink: int | None = None):
    """(kv_indptr [B+1], kv_indices): request after request, the pool rows of
    the kept positions in ascending order."""
    table = np.asarray(table)
    indptr = [0]
    parts = []
    for b, S in enumerate(np.asarray(lens)):
        rows = table[b, keep_positions(int(S), variant, W, sink)]
        parts.append(rows)
        indptr.append(indptr[-1] + rows.size)
    idx = np.concatenate(parts) if parts else np.zeros(0, dtype=table.dtype)
    return np.asarray(indptr, dtype=np.int64), idx.astype(np.int64)


def attend_paged(q, K_pool, V_pool, table_row, S: int, scale: float, variant: str,
                 W: int | None = None, sink: int | None = None, spread: bool = False):
    """Attention of one request over the pool rows its index list names
    (with spread=True also oracle.attention.value_spread over those rows)."""
    rows = np.asarray(table_row)[keep_positions(int(S), variant, W, sink)]
    K = np.asarray(K_pool[rows])
    V = np.asarray(V_pool[rows])
    o, lse = attention.attend_sequence(q, K, V, rows.size, scale, None)
    if not spread:
        return o, lse
    return o, lse, attention.value_spread(q, K, V, rows.size, scale, None)
