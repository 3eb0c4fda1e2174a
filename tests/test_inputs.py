"""The seeded input generators: determinism, shapes and recipe."""

import numpy as np
import torch

from paper_2607_21535_amd import inputs as I


def test_normal_bf16_is_deterministic_and_standard():
    a = I.normal_bf16((1000, 64), 123)
    b = I.normal_bf16((1000, 64), 123)
    c = I.normal_bf16((1000, 64), 124)
    assert a.dtype == torch.bfloat16
    assert torch.equal(a, b) and not torch.equal(a, c)
    x = a.float()
    assert abs(x.mean().item()) < 0.02 and abs(x.std().item() - 1.0) < 0.02


def test_bits_round_trip():
    a = I.normal_bf16((7, 5), 1)
    assert torch.equal(I.from_bits(I.bf16_bits(a)), a)


def test_lengths_and_accepts_in_range():
    lens = I.uniform_lengths(32, 65536, 1048576, I.stream_seed(1003, I.STREAM_LENS))
    assert lens.dtype == np.int32 and lens.min() >= 65536 and lens.max() <= 1048576
    acc = I.accept_counts(1000, 8, 8, I.stream_seed(1004, I.STREAM_ACCEPT))
    assert acc.shape == (1000, 8) and acc.min() == 1 and acc.max() == 8


def test_decode_case_shapes():
    wl = I.WORKLOADS["draft_loop_s128k"]
    c = I.decode_case(wl, "cpu", S=300)
    assert c["q"].shape == (3, 1, 16, 256)
    assert c["k"].shape == (1, 303, 2, 256) and c["S_max"] == 303
    assert c["k_new"].shape == (3, 1, 1, 2, 256)
    assert np.all(c["lens"] == 300)
    assert torch.count_nonzero(c["k"][0, 300:]) == 0


def test_varlen_case_lengths():
    wl = I.WORKLOADS["batch32_varlen"]
    c = I.decode_case(wl, "cpu", S=500, B=6)
    assert c["lens"].min() >= 1 and c["lens"].max() <= 500
    for b in range(6):
        L = int(c["lens"][b])
        assert torch.count_nonzero(c["k"][b, L:]) == 0
        assert torch.count_nonzero(c["k"][b, :L]) > 0
