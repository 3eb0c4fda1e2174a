"""Helpers shared by the GPU parity tests (not collected by pytest).

Parity bar (floating point, all variants):
  * max |o - o_ref| <= 1e-2 over every output element (the contract) on the
    five workloads, where |o_ref| < 1; for the small edge cases (a handful
    of keys, |o_ref| up to ~4) the elementwise bar is
    max(1e-2, 2^-8 |o_ref| + 1e-4): bf16 output rounding alone moves an
    element by up to 2^-8 of its magnitude, 1.6e-2 at |o| = 4;
  * per (b, h): ||o - o_ref||_2 <= 5e-3 * ||o_ref||_2.  Rounding the output
    to bfloat16 alone moves each element by at most 2^-8 of its magnitude
    (half an ulp with 8 significant bits), i.e. <= 3.9e-3 normwise; the fp32
    logits and sums add far less (< 1e-5 relative at 1M keys);
  * lse: |lse - lse_ref| <= 1e-4 * max(1, |lse_ref|), -inf exactly for empty
    sequences.
Integer, index and byte results (selected positions, ring slots, cache
contents after appends, lengths, error words) must match exactly.
"""

from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from oracle import attention as A
from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

ATOL = 1e-2
NREL = 5e-3
LSE_REL = 1e-4
BF16_REL = 2.0 ** -8


def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    W.load_library()  # a GPU run without the library fails loudly here
    return torch.device("cuda:0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class HostRows:
    """Host view of one sequence of a device cache [rows, Hkv, d] for the
    oracle: indexing returns the rows' bf16 bit patterns as numpy."""

    def __init__(self, t: torch.Tensor):
        self.t = t
        self.shape = tuple(t.shape)

    def __getitem__(self, rows):
        idx = torch.from_numpy(np.ascontiguousarray(rows, dtype=np.int64)).to(self.t.device)
        return I.bf16_bits(self.t.index_select(0, idx))


def oracle_seq(q_bits, k_dev_seq, v_dev_seq, S, scale, variant, W_=None, sink=None):
    """Oracle output for one sequence whose cache lives on the device."""
    mask = None if variant == "full" else A.window_mask(S, W_, sink)
    return A.attend_sequence(q_bits, HostRows(k_dev_seq), HostRows(v_dev_seq), S, scale, mask)


def assert_attn_close(out, o_ref, lse=None, lse_ref=None, what="", strict=True, v_max=None):
    """Output within the contract's max-abs tolerance (strict) or, for small
    cases with large outputs, within the bf16 rounding of the output itself;
    v_max (the largest |value| the call can combine) adds the error of the
    weights entering the PV product rounded to bf16: each moves by at most
    2^-9 relative, so the output moves by at most 2^-9 max_i |v_i - o|, and
    that is at most 2^-8 v_max.  Rows with few keys and a wide spread of
    values reach it.  Also checks the normwise error per row and the lse."""
    o = out.detach().float().cpu().numpy().astype(np.float64)
    o_ref = np.asarray(o_ref, dtype=np.float64).reshape(o.shape)
    d = o.shape[-1]
    err = np.abs(o - o_ref)
    assert np.all(np.isfinite(o)), f"{what}: non-finite output"
    bound = ATOL if strict else np.maximum(ATOL, BF16_REL * np.abs(o_ref) + 1e-4)
    if v_max is not None:
        bound = bound + 2.0 ** -8 * float(v_max)
    assert np.all(err <= bound), f"{what}: max abs err {err.max():.3e} (|o_ref| max {np.abs(o_ref).max():.2f})"
    num = np.linalg.norm((o - o_ref).reshape(-1, d), axis=1)
    den = np.linalg.norm(o_ref.reshape(-1, d), axis=1)
    bad = num > NREL * den
    assert not bad.any(), (f"{what}: normwise rel err {np.max(num / np.maximum(den, 1e-300)):.3e} "
                           f"> {NREL} at rows {np.flatnonzero(bad)[:8]}")
    if lse is not None and lse_ref is not None:
        l = lse.detach().cpu().numpy().astype(np.float64).reshape(-1)
        lr = np.asarray(lse_ref, dtype=np.float64).reshape(-1)
        inf_ref = np.isneginf(lr)
        assert np.array_equal(np.isneginf(l), inf_ref), f"{what}: lse -inf mismatch"
        fin = ~inf_ref
        if fin.any():
            lerr = np.abs(l[fin] - lr[fin])
            tol = LSE_REL * np.maximum(1.0, np.abs(lr[fin]))
            assert np.all(lerr <= tol), f"{what}: lse err {lerr.max():.3e}"
    return float(err.max()), float(np.max(num / np.maximum(den, 1e-300)))


def lens_tensor(lens, dev):
    return torch.as_tensor(np.asarray(lens, dtype=np.int32), device=dev)


def err_word(dev):
    return torch.zeros(1, dtype=torch.int32, device=dev)
