"""Pins for the oracle's paged-pool model (index list and attention)."""

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import paged as Pg
from paper_2607_21535_amd import inputs as I

TABLE = [list(range(40, 52)), [7, 3, 9, 1, 5] + [0] * 7]


def test_golden_index_lists(golden):
    rows = golden("kv_index_examples.txt")
    assert len(rows) >= 6
    for req, S, variant, W, sink, idx in rows:
        table = np.array([TABLE[int(req)]])
        indptr, got = Pg.kv_indices(table, [int(S)], variant, int(W), int(sink))
        exp = [int(x) for x in idx.split()] if idx else []
        assert got.tolist() == exp and indptr.tolist() == [0, len(exp)]


def test_index_list_is_packed_in_request_order():
    table = np.array(TABLE)
    indptr, idx = Pg.kv_indices(table, [10, 5], "windowed", 3, 2)
    assert indptr.tolist() == [0, 5, 10]
    assert idx.tolist() == [40, 41, 47, 48, 49, 7, 3, 9, 1, 5]


def _case(seed, S, P, Hq=4, Hkv=2, d=8):
    rng = np.random.default_rng(seed)
    q = I.bf16_bits(torch.from_numpy(rng.standard_normal((Hq, d))).to(torch.bfloat16))
    Kp = I.bf16_bits(torch.from_numpy(rng.standard_normal((P, Hkv, d))).to(torch.bfloat16))
    Vp = I.bf16_bits(torch.from_numpy(rng.standard_normal((P, Hkv, d))).to(torch.bfloat16))
    return rng, q, Kp, Vp


@pytest.mark.parametrize("variant", ["full", "windowed"])
def test_identity_table_is_the_dense_cache(variant):
    S = 300
    _, q, Kp, Vp = _case(1, S, S)
    o1, l1 = Pg.attend_paged(q, Kp, Vp, np.arange(S), S, 0.3, variant, 32, 4)
    mask = None if variant == "full" else A.window_mask(S, 32, 4)
    o2, l2 = A.attend_sequence(q, Kp, Vp, S, 0.3, mask)
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    np.testing.assert_allclose(l1, l2, atol=1e-13)


@pytest.mark.parametrize("variant", ["full", "windowed"])
def test_relabelling_the_pool_changes_nothing(variant):
    # Moving every row to another pool slot and rewriting the table to match
    # leaves the attention unchanged; a table that points elsewhere does not.
    S, P = 200, 500
    rng, q, Kp, Vp = _case(2, S, P)
    table = rng.permutation(P)[:S]
    o1, _ = Pg.attend_paged(q, Kp, Vp, table, S, 0.3, variant, 16, 2)
    perm = rng.permutation(P)           # new slot of old row r is perm[r]
    Kq, Vq = np.empty_like(Kp), np.empty_like(Vp)
    Kq[perm], Vq[perm] = Kp, Vp
    o2, _ = Pg.attend_paged(q, Kq, Vq, perm[table], S, 0.3, variant, 16, 2)
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    o3, _ = Pg.attend_paged(q, Kq, Vq, table, S, 0.3, variant, 16, 2)
    assert np.abs(o3 - o1).max() > 1e-3


@pytest.mark.parametrize("variant", ["full", "windowed"])
def test_spread_option_over_binary_pool(variant):
    rng = np.random.default_rng(4)
    P, S, Hkv, d = 200, 90, 2, 8
    q = rng.standard_normal((4, d))
    Kp = rng.standard_normal((P, Hkv, d))
    Vp = (rng.random((P, Hkv, d)) < 0.6).astype(np.float64)
    table = rng.permutation(P)[:S]
    o, lse, s = Pg.attend_paged(q, Kp, Vp, table, S, 0.3, variant, 16, 2, spread=True)
    o2, lse2 = Pg.attend_paged(q, Kp, Vp, table, S, 0.3, variant, 16, 2)
    assert np.array_equal(o, o2) and np.array_equal(lse, lse2)
    np.testing.assert_allclose(s, 2 * o * (1 - o), atol=1e-13)
