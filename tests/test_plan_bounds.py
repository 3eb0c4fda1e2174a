"""The workspace bound of the full-context extend against its decomposition
(CPU; no GPU needed).

The kernels cut each sequence's keys into items on the device, from the
device-resident lengths, and write one partial per (query row, item it
sees); the library sizes the workspace on the host for every length the
call could meet.  This test restates the item rule (the chunk is the summed
key count over the one-per-CU target, rounded up to 64 keys and clamped to
[64, 9216]; the per-row rule sums every row's keys, the per-sequence rule
only each sequence's last row, the one that sees every key) and checks, over
random batches, that the partials and the multi-row kernel's work items fit
what wmtp_workspace_bytes / wmtp_extend_workspace_bytes provide.  A bound
that is too small would send the kernels' partial stores past the end of the
workspace, so it is pinned here rather than found on the device.
"""

import math

import numpy as np
import pytest

from paper_2607_21535_amd import wmtp as W

CUS = 256          # what the library assumes without a device
QUANTUM = 64       # work items are multiples of this many keys
CAP = 9216         # largest work item
TICKETS = 1 << 20  # counter bytes at the start of every workspace


def _up(x):
    return (x + 255) // 256 * 256


def _bytes_for(items, Hkv, G, d):
    """Workspace bytes whose partial arrays hold `items` partials per KV head
    (the layout of the split plan: three fp32 scalars and d fp32 values)."""
    rows = items * Hkv * G
    return TICKETS + 3 * _up(rows * 4) + _up(rows * d * 4)


def _chunk(total, Hkv):
    T = max(1, CUS // Hkv)
    c = -(-total // T)
    c = -(-c // QUANTUM) * QUANTUM
    return min(max(c, QUANTUM), CAP)


def _one_launch(rows, Hkv, d, S_max):
    """Whether a full-context call takes the one-launch kernel instead of
    the split ones (at most four query rows x KV heads over a short cache:
    16384 rows per sequence at d = 256, 4096 below); its workspace holds that
    kernel's records, not the split partials this test restates."""
    return rows * Hkv <= 4 and 0 < S_max <= (16384 if d >= 256 else 4096)


def _row_lengths(lens, n_q, q_max):
    """Visible length of every query row (row t of sequence b sees
    lens[b] - n + t + 1 keys; rows t >= n see none)."""
    out = []
    for S, n in zip(lens, n_q):
        out.append([S - n + t + 1 if t < n and S > 0 else 0 for t in range(q_max)])
    return out


@pytest.mark.parametrize("seed", range(40))
def test_extend_partials_fit_the_workspace(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 9))
    q_max = int(rng.choice([2, 3, 5, 8, 12, 20]))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 8, 16]))
    d = int(rng.choice([64, 128, 256]))
    S_max = int(rng.choice([q_max + 1, 700, 9000, 131072, 1 << 20]))
    lens = [int(rng.integers(0, S_max + 1)) for _ in range(B)]
    if rng.random() < 0.5:
        lens[int(rng.integers(0, B))] = S_max  # a sequence at full capacity
    n_q = [int(rng.integers(1, q_max + 1)) if S else 0 for S in lens]
    n_q = [min(n, S) for n, S in zip(n_q, lens)]
    rows = _row_lengths(lens, n_q, q_max)
    Hq = Hkv * G

    coarse_ws = W.workspace_bytes(B * q_max, Hq, Hkv, d, S_max, variant=W.VARIANT_FULL)
    fine_ws = W.extend_workspace_bytes(B, q_max, Hq, Hkv, d, S_max)
    assert fine_ws >= coarse_ws > 0
    if _one_launch(B * q_max, Hkv, d, S_max):
        return

    T = max(1, CUS // Hkv)
    for per_seq, ws in ((False, coarse_ws), (True, fine_ws)):
        if per_seq:
            total = sum(r[n - 1] for r, n in zip(rows, n_q) if n > 0)
        else:
            total = sum(sum(r) for r in rows)
        c = _chunk(total, Hkv)
        partials = sum(math.ceil(L / c) for r in rows for L in r)
        assert _bytes_for(partials, Hkv, G, d) <= ws, (per_seq, c, partials)
        # the multi-row kernel's items (one per chunk of each sequence's last
        # row) fit the grid the library launches for them
        items = sum(math.ceil(r[n - 1] / c) for r, n in zip(rows, n_q) if n > 0)
        grid = min(B * math.ceil(S_max / QUANTUM), max(T + B, B * math.ceil(S_max / CAP)))
        assert items <= grid, (per_seq, items, grid)


def test_per_sequence_items_fill_the_device_at_one_sequence():
    """One sequence of 8 rows at 128K: the per-row rule leaves 16 items per
    KV head (1/8 of the one-per-CU target); the per-sequence rule gives 128."""
    S, q, Hkv = 131072, 8, 2
    rows = _row_lengths([S], [q], q)
    coarse = _chunk(sum(rows[0]), Hkv)
    fine = _chunk(rows[0][-1], Hkv)
    assert (math.ceil(S / coarse), math.ceil(S / fine)) == (16, 128)
