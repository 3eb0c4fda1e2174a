"""Helpers shared by the GPU parity tests (not collected by pytest).

Parity bar (floating point, all variants):
  * max |o - o_ref| <= 1e-2 over every output element (the contract).  Where
    the oracle also supplies the value spread (oracle.attention.value_spread,
    s = sum_p w_p |v_p - o_ref| per element), an element may instead be
    within the rounding the kernels' arithmetic provably allows, if that is
    larger (rows with a handful of keys and large values):
        e   = r / (1 - r) * s + 2^-12 * (s + 2 |o_ref|)
        bound = max(1e-2, 2^-8 (|o_ref| + e) + e),   r = 2^-8 + 2^-10.
    Derivation: the weights enter the value product rounded to bfloat16 and
    the output is normalised by the sum of the same rounded weights; a
    relative perturbation of at most r per weight moves the normalised sum
    by at most r / (1 - r) * s.  Round to nearest even to bfloat16 has unit
    roundoff 2^-8 (8 significant bits); the remaining 2^-10 of r covers the
    fp32 logits (d products summed in fp32, the scale folded in fp32), the
    hardware exp2 and the fp32 rescaling factors.  2^-12 covers the fp32
    sums of the weighted values and of the weights (a few hundred additions
    deep: the tiles of a work item, the waves, the items of the merge), and
    the final bfloat16 rounding adds 2^-8 of the value rounded;
  * per (b, h): ||o - o_ref||_2 <= 5e-3 * ||o_ref||_2.  Rounding the output
    to bfloat16 alone moves each element by at most 2^-8 of its magnitude
    (half an ulp with 8 significant bits), i.e. <= 3.9e-3 normwise;
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
U_BF16 = 2.0 ** -8          # unit roundoff of round-to-nearest-even to bfloat16
R_WEIGHT = 2.0 ** -8 + 2.0 ** -10  # relative perturbation budget of one weight
R_SUM = 2.0 ** -12          # fp32 summation budget


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


def oracle_seq(q_bits, k_dev_seq, v_dev_seq, S, scale, variant, W_=None, sink=None, spread=False):
    """Oracle output for one sequence whose cache lives on the device;
    with spread=True also the value spread (for the elementwise bound)."""
    mask = None if variant == "full" else A.window_mask(S, W_, sink)
    K, V = HostRows(k_dev_seq), HostRows(v_dev_seq)
    o, lse = A.attend_sequence(q_bits, K, V, S, scale, mask)
    if not spread:
        return o, lse
    return o, lse, A.value_spread(q_bits, K, V, S, scale, mask)


def elementwise_bound(o_ref, spread):
    """Per-element bound: the 1e-2 contract, or the provable rounding of the
    kernels' arithmetic when that is larger (see the module docstring)."""
    o_abs = np.abs(o_ref)
    s = np.asarray(spread, dtype=np.float64).reshape(o_abs.shape)
    e = R_WEIGHT / (1.0 - R_WEIGHT) * s + R_SUM * (s + 2.0 * o_abs)
    return np.maximum(ATOL, U_BF16 * (o_abs + e) + e)


def assert_attn_close(out, o_ref, lse=None, lse_ref=None, what="", spread=None):
    """Output within the contract's max-abs tolerance, or (spread given)
    within elementwise_bound; also the normwise error per row and the lse."""
    o = out.detach().float().cpu().numpy().astype(np.float64)
    o_ref = np.asarray(o_ref, dtype=np.float64).reshape(o.shape)
    d = o.shape[-1]
    err = np.abs(o - o_ref)
    assert np.all(np.isfinite(o)), f"{what}: non-finite output"
    bound = ATOL if spread is None else elementwise_bound(o_ref, spread)
    bad = err > bound
    assert not bad.any(), (f"{what}: max abs err {err.max():.3e} (|o_ref| max {np.abs(o_ref).max():.2f}); "
                           f"worst excess {np.max(err - bound):.3e} at {np.argwhere(bad)[:4].tolist()}")
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


WINDOW_PATH_ENV = "WMTP_WIN_ONE_LAUNCH_ROWS"
WINDOW_PATHS = ("one_launch", "split")


class window_path:
    """Context manager: windowed calls take the one-launch kernel
    ("one_launch") or the split-K + merge kernels ("split") whatever their
    row count (the library reads the threshold at every call)."""

    def __init__(self, path):
        self.value = {"one_launch": str(1 << 30), "split": "0"}[path]

    def __enter__(self):
        import os
        self.old = os.environ.get(WINDOW_PATH_ENV)
        os.environ[WINDOW_PATH_ENV] = self.value
        return self

    def __exit__(self, *exc):
        import os
        if self.old is None:
            os.environ.pop(WINDOW_PATH_ENV, None)
        else:
            os.environ[WINDOW_PATH_ENV] = self.old
        return False
