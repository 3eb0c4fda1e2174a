"""GPU parity on the five draft-attention workloads at their full sizes.

  decode_s8k        B=1 Hq=16 Hkv=2 d=128 S=8192, full and windowed (W=512, sink=4)
  draft_loop_s128k  B=1 Hq=16 Hkv=2 d=256 S=131072, 3 draft steps (append, attend)
  draft_loop_s1m    B=1 Hq=32 Hkv=2 d=256 S=1048576, K rows 0..3 scaled x4, 7 draft steps
  batch32_varlen    B=32 Hq=32 Hkv=2 d=256 S ~ U[65536, 1048576]
(the ring workload is tests/test_ring_sim_gpu.py)

Every windowed output is compared with the oracle; the full variant is
compared in full at 8K and 128K, at the first and last draft step at 1M, and
on every one of the 32 sequences of the batch.  The
oracle reads the inputs (the generated cache plus the appended rows written
by torch), never the HIP path's own cache.
"""

import numpy as np
import pytest
import torch

from paper_2607_21535_amd import inputs as I
from paper_2607_21535_amd import wmtp as W

from . import _gpu as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    return G.device()


def _both(q, k, v, lt, wl, dev):
    B, Hq = q.shape[0], q.shape[1]
    lse_f = torch.empty(B, Hq, dtype=torch.float32, device=dev)
    lse_w = torch.empty_like(lse_f)
    err = G.err_word(dev)
    of = W.draft_attn_full(q, k, v, lt, lse=lse_f, scale=wl.scale, err=err)
    ow = W.draft_attn_windowed(q, k, v, lt, wl.W, wl.sink, lse=lse_w, scale=wl.scale, err=err)
    torch.cuda.synchronize()
    assert err.item() == 0
    return of, lse_f, ow, lse_w


def test_decode_s8k(dev):
    wl = I.WORKLOADS["decode_s8k"]
    G.say("decode_s8k: generating")
    case = I.decode_case(wl, dev, steps=1)
    q = case["q"][0]
    lt = G.lens_tensor(case["lens"], dev)
    of, lse_f, ow, lse_w = _both(q, case["k"], case["v"], lt, wl, dev)
    qb = I.bf16_bits(q)
    S = int(case["lens"][0])
    of_ref, lf_ref = G.oracle_seq(qb[0], case["k"][0], case["v"][0], S, wl.scale, "full")
    ow_ref, lw_ref = G.oracle_seq(qb[0], case["k"][0], case["v"][0], S, wl.scale, "windowed", wl.W, wl.sink)
    G.say(f"decode_s8k full err {G.assert_attn_close(of, of_ref[None], lse_f, lf_ref, 'full')}")
    G.say(f"decode_s8k windowed err {G.assert_attn_close(ow, ow_ref[None], lse_w, lw_ref, 'windowed')}")
    # distinguishable: past the threshold the window changes the result
    assert np.linalg.norm(of_ref - ow_ref) > 50 * G.NREL * np.linalg.norm(of_ref)


def _draft_loop(dev, wl, full_steps):
    G.say(f"{wl.name}: generating S={wl.S}")
    case = I.decode_case(wl, dev)
    k, v = case["k"], case["v"]
    ref_k, ref_v = k.clone(), v.clone()  # torch-built reference cache
    lt = G.lens_tensor(case["lens"], dev)
    ones = torch.ones(wl.B, dtype=torch.int32, device=dev)
    S0 = wl.S
    for j in range(wl.gamma):
        W.cache_append(k, v, case["k_new"][j], case["v_new"][j], ones, lt)
        ref_k[:, S0 + j] = case["k_new"][j][:, 0]
        ref_v[:, S0 + j] = case["v_new"][j][:, 0]
        q = case["q"][j]
        of, lse_f, ow, lse_w = _both(q, k, v, lt, wl, dev)
        S = S0 + j + 1
        assert lt.cpu().tolist() == [S] * wl.B
        qb = I.bf16_bits(q)
        ow_ref, lw_ref = G.oracle_seq(qb[0], ref_k[0], ref_v[0], S, wl.scale, "windowed", wl.W, wl.sink)
        e = G.assert_attn_close(ow, ow_ref[None], lse_w, lw_ref, f"{wl.name} step {j + 1} windowed")
        G.say(f"{wl.name} step {j + 1} windowed err {e}")
        if j in full_steps:
            of_ref, lf_ref = G.oracle_seq(qb[0], ref_k[0], ref_v[0], S, wl.scale, "full")
            e = G.assert_attn_close(of, of_ref[None], lse_f, lf_ref, f"{wl.name} step {j + 1} full")
            G.say(f"{wl.name} step {j + 1} full err {e}")
            assert np.linalg.norm(of_ref - ow_ref) > 10 * G.NREL * np.linalg.norm(of_ref)
    assert torch.equal(k, ref_k) and torch.equal(v, ref_v)  # appends are exact


def test_draft_loop_s128k(dev):
    wl = I.WORKLOADS["draft_loop_s128k"]
    _draft_loop(dev, wl, full_steps=range(wl.gamma))


def test_draft_loop_s1m(dev):
    wl = I.WORKLOADS["draft_loop_s1m"]
    _draft_loop(dev, wl, full_steps=(0, wl.gamma - 1))


@pytest.fixture(scope="module")
def batch32(dev):
    """The 32-sequence batch (about 35 GB of live KV in a 64 GiB cache), with
    its full-context and windowed outputs from one call each."""
    wl = I.WORKLOADS["batch32_varlen"]
    G.say("batch32_varlen: generating (about 64 GiB of cache)")
    case = I.decode_case(wl, dev, steps=1)
    lens = case["lens"]
    q = case["q"][0]
    lt = G.lens_tensor(lens, dev)
    of, lse_f, ow, lse_w = _both(q, case["k"], case["v"], lt, wl, dev)
    yield wl, case, I.bf16_bits(q), of, lse_f, ow, lse_w
    del case, of, lse_f, ow, lse_w
    torch.cuda.empty_cache()


def test_batch32_varlen_windowed(batch32):
    wl, case, qb, of, lse_f, ow, lse_w = batch32
    lens = case["lens"]
    refs = [G.oracle_seq(qb[b], case["k"][b], case["v"][b], int(lens[b]), wl.scale, "windowed",
                         wl.W, wl.sink) for b in range(wl.B)]
    e = G.assert_attn_close(ow, np.stack([r[0] for r in refs]), lse_w, np.stack([r[1] for r in refs]),
                            "batch32 windowed")
    G.say(f"batch32 windowed err {e}")


@pytest.mark.parametrize("b", range(32))
def test_batch32_varlen_full(batch32, b):
    """Every sequence's full-context output (its work items placed by the
    device-side prefix sum over the lengths) against the oracle."""
    wl, case, qb, of, lse_f, ow, lse_w = batch32
    S = int(case["lens"][b])
    o_ref, l_ref = G.oracle_seq(qb[b], case["k"][b], case["v"][b], S, wl.scale, "full")
    e = G.assert_attn_close(of[b:b + 1], o_ref[None], lse_f[b:b + 1], l_ref, f"batch32 full b={b}")
    G.say(f"batch32 full b={b} S={S} err {e}")
