"""Exact masked-softmax GQA decode attention in float64 -- the oracle.

TEST INFRASTRUCTURE ONLY (see the package docstring): nothing on the product
path imports this module.

What is computed (Windowed-MTP paper):
  * Section 4 "Mechanism": at each draft decode step the draft attention sees
    a reduced key set, the first n_sink tokens plus the most recent W tokens;
    the reduced set *is* the key set, with no further causal window mask, and
    the scores themselves are unchanged (RoPE is already baked into the cached
    keys, so a key's place in the reduced set does not change its score).
  * Appendix A, pseudocode of the windowing change: the reduction applies only
    when S > n_sink + W; otherwise all S keys are kept.
  * Section 3 / Section 6 "Memory": the windowed draft reads min(S, W + n_sink)
    keys per step.
  * The native (full-context) draft attends all S cached keys (Section 3,
    "Per-step latency model"; Figure "window").
  * Draft-extend (the draft forward over several accepted tokens after a
    verify step; Appendix B kernel attribution table, Section 6 "The backend
    is not the confound"): each new row is an autoregressive decode step of
    its own -- the token at position p sees positions [0, p] -- with the
    selection rule applied at that row's length.

Everything else is the textbook single-query softmax attention, written out:
    z_p = scale * <q_h, k_p>            for kept positions p
    m   = max_p z_p,  w_p = exp(z_p - m),  l = sum_p w_p
    o_h = sum_p (w_p / l) v_p,  lse_h = m + ln l

Readings where the paper is silent:
  * GQA grouping: query head h uses KV head g = h // G with G = Hq / Hkv
    (consecutive grouping).
  * W counts only the recent window, not the sink: |keep| = n_sink + W.
  * S is the sequence length after the current draft row has been appended,
    so the window range(S - W, S) includes the current token.
  * The scale is an explicit argument (1/sqrt(d) by default in the callers);
    no soft-cap, bias or positional transform is applied.
  * An empty sequence (S = 0) attends nothing: o = 0 and lse = -inf.

Inputs may be bfloat16 bit patterns (uint16 / int16 arrays) -- widened exactly
to float64 here -- or ordinary float arrays.  Long sequences are processed in
two passes over key chunks (all logits and their maximum first, then the
weighted sum of values); that is the same arithmetic as the formula above, with
no online rescaling.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_to_f64",
    "full_mask",
    "window_mask",
    "selected_positions",
    "n_selected",
    "attend_sequence",
    "value_spread",
    "extend_lengths",
    "attend_extend",
    "extend_spread",
]

# Keys processed per chunk when forming logits and the value sum.
_CHUNK = 65536


def bf16_to_f64(bits) -> np.ndarray:
    """Widen bfloat16 bit patterns to float64, exactly.

    A bfloat16 value is the upper 16 bits of an IEEE binary32 value, so
    shifting the pattern into the high half of a 32-bit word gives the float32
    with the same value, which float64 then represents exactly.
    """
    u16 = np.ascontiguousarray(bits).view(np.uint16)
    return (u16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _as_f64(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype in (np.uint16, np.int16):
        return bf16_to_f64(x)
    return x.astype(np.float64)


def full_mask(S: int) -> np.ndarray:
    """Native draft: every cached key [0, S) is attended (Section 3)."""
    return np.ones(int(S), dtype=bool)


def window_mask(S: int, W: int, sink: int) -> np.ndarray:
    """Keys attended by the windowed draft at sequence length S.

    Section 4 "Mechanism" and the Appendix A pseudocode: when S > sink + W the
    kept keys are the sink [0, sink) and the recent window [S - W, S);
    otherwise every key [0, S) is kept.
    """
    S = int(S)
    p = np.arange(S)
    if S > sink + W:
        return (p < sink) | (p >= S - W)
    return np.ones(S, dtype=bool)


def selected_positions(S: int, W: int, sink: int) -> np.ndarray:
    """Logical positions of the windowed key set, ascending (sink first)."""
    return np.flatnonzero(window_mask(S, W, sink)).astype(np.int64)


def n_selected(S: int, W: int, sink: int) -> int:
    """Number of keys the windowed draft reads at length S."""
    return int(window_mask(S, W, sink).sum())


def attend_sequence(q, K, V, S: int, scale: float, mask=None, chunk: int = _CHUNK):
    """Single-token GQA attention of one sequence's query over its cached keys.

    q    : [Hq, d]            query (float64, or bf16 bits)
    K, V : [>= S, Hkv, d]     cached keys / values in logical position order
    S    : number of valid cached rows
    mask : bool [S] of kept keys, or None for the full context
    Returns (o [Hq, d] float64, lse [Hq] float64).
    """
    qf = _as_f64(q)
    Hq, d = qf.shape
    Hkv = K.shape[1]
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    G = Hq // Hkv
    S = int(S)
    keep = np.arange(S) if mask is None else np.flatnonzero(np.asarray(mask)[:S])
    n = keep.size
    o = np.zeros((Hq, d), dtype=np.float64)
    lse = np.full(Hq, -np.inf, dtype=np.float64)
    if n == 0:
        return o, lse

    # Pass 1: every kept logit z[h, j] = scale * <q_h, k_keep[j]>.
    z = np.empty((Hq, n), dtype=np.float64)
    for c0 in range(0, n, chunk):
        rows = keep[c0:c0 + chunk]
        Kc = _as_f64(np.asarray(K[rows]))  # [c, Hkv, d]
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            z[hs, c0:c0 + rows.size] = scale * (qf[hs] @ Kc[:, g, :].T)
    m = z.max(axis=1)
    w = np.exp(z - m[:, None])
    l = w.sum(axis=1)

    # Pass 2: sum of the values weighted by w.
    for c0 in range(0, n, chunk):
        rows = keep[c0:c0 + chunk]
        Vc = _as_f64(np.asarray(V[rows]))
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            o[hs] += w[hs, c0:c0 + rows.size] @ Vc[:, g, :]
    o /= l[:, None]
    lse = m + np.log(l)
    return o, lse


def value_spread(q, K, V, S: int, scale: float, mask=None, chunk: int = 4096):
    """Weighted mean absolute deviation of the attended values about the output.

        spread[h, c] = sum_p w_p |V[p, g(h), c] - o[h, c]|,   w_p = exp(z_p - lse_h)

    over the same kept keys, normalised weights (they sum to 1) and output o
    as attend_sequence.  This is not part of the method: it sizes the effect
    of perturbing the weights.  If every weight moves by a relative amount of
    at most r and the result is renormalised, o moves by at most
    r / (1 - r) * spread (because sum_p w_p (V_p - o) = 0).  The GPU tests use
    it to bound the effect of rounding the weights to bfloat16.
    Returns spread [Hq, d] float64 (zero for an empty key set).
    """
    qf = _as_f64(q)
    Hq, d = qf.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    S = int(S)
    keep = np.arange(S) if mask is None else np.flatnonzero(np.asarray(mask)[:S])
    spread = np.zeros((Hq, d), dtype=np.float64)
    if keep.size == 0:
        return spread
    o, lse = attend_sequence(q, K, V, S, scale, mask)
    for c0 in range(0, keep.size, chunk):
        rows = keep[c0:c0 + chunk]
        Kc = _as_f64(np.asarray(K[rows]))
        Vc = _as_f64(np.asarray(V[rows]))
        for g in range(Hkv):
            hs = slice(g * G, (g + 1) * G)
            w = np.exp(scale * (qf[hs] @ Kc[:, g, :].T) - lse[hs, None])        # [G, c]
            dev = np.abs(Vc[None, :, g, :] - o[hs, None, :])                   # [G, c, d]
            spread[hs] += np.einsum("hp,hpc->hc", w, dev)
    return spread


def extend_lengths(S: int, n: int, q_max: int):
    """Visible length of each new query row in a draft-extend call.

    Autoregressive attention over n new rows appended at the end of a
    sequence that now holds S rows: row t (0-based among the new rows) is
    the token at position S - n + t and sees positions [0, S - n + t + 1).
    Rows t >= n (padding up to q_max) see nothing.
    """
    return [S - n + t + 1 if t < n else 0 for t in range(q_max)]


def attend_extend(q_rows, K, V, S: int, n: int, scale: float, variant: str = "full",
                  W: int | None = None, sink: int | None = None):
    """Draft-extend attention of one sequence: q_rows [q_max, Hq, d].

    Each new row attends causally; under the windowed variant each row
    applies the sink + window rule at its own length (Section 4 "Mechanism",
    Appendix A pseudocode, with S the row's own length).
    Returns (o [q_max, Hq, d], lse [q_max, Hq]); padding rows give 0 / -inf.
    """
    q_rows = np.asarray(q_rows)
    q_max, Hq, d = q_rows.shape
    o = np.zeros((q_max, Hq, d))
    lse = np.full((q_max, Hq), -np.inf)
    for t, L in enumerate(extend_lengths(S, n, q_max)):
        if L <= 0:
            continue
        mask = None if variant == "full" else window_mask(L, W, sink)
        o[t], lse[t] = attend_sequence(q_rows[t], K, V, L, scale, mask)
    return o, lse


def extend_spread(q_rows, K, V, S: int, n: int, scale: float, variant: str = "full",
                  W: int | None = None, sink: int | None = None):
    """value_spread of every new row of a draft-extend (rows as attend_extend;
    padding rows give 0).  Returns [q_max, Hq, d]."""
    q_rows = np.asarray(q_rows)
    q_max, Hq, d = q_rows.shape
    out = np.zeros((q_max, Hq, d))
    for t, L in enumerate(extend_lengths(S, n, q_max)):
        if L <= 0:
            continue
        mask = None if variant == "full" else window_mask(L, W, sink)
        out[t] = value_spread(q_rows[t], K, V, L, scale, mask)
    return out
