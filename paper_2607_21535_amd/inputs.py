"""Seeded synthetic inputs for the draft-attention workloads.

This module is shared by the tests, the benchmark and the smoke check: it
draws queries, KV caches, appended rows, sequence lengths and accept counts,
and holds none of the attention arithmetic (no selection, no slot map, no
softmax).  The oracle never imports it; callers hand the generated arrays to
both sides.

Recipe (stands in for the paper's 1.04M-token RULER / LongBench-v2 /
BABILong prompts, which are not available; the draft attention's cost does not
depend on the KV contents, Section 3 of the Windowed-MTP paper):
  * values are float32 standard normal, rounded to bfloat16 (round to nearest
    even, torch's conversion);
  * every tensor comes from its own torch.Generator seeded from the workload
    seed and a fixed stream id, so any one of them can be regenerated alone
    (per sequence for the batched cache);
  * integer draws (lengths, accept counts) always use a CPU generator, so they
    are the same whichever device holds the tensors;
  * fp8 caches hold E4M3 codes (uint8) of float32 draws, rounded by torch's
    float8_e4m3fn conversion (the draws stay far inside its range).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

__all__ = [
    "Workload",
    "WORKLOADS",
    "stream_seed",
    "normal_bf16",
    "normal_fp8",
    "fp8_codes",
    "uniform_lengths",
    "accept_counts",
    "bf16_bits",
    "from_bits",
    "decode_case",
]

# Stream ids: one generator per tensor role.
STREAM_Q, STREAM_K, STREAM_V, STREAM_KNEW, STREAM_VNEW, STREAM_LENS, STREAM_ACCEPT = range(1, 8)


@dataclass(frozen=True)
class Workload:
    """One synthetic draft-attention workload (shapes and seeds only)."""

    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    S: int                 # cache length before the loop (max length if varlen)
    W: int
    sink: int
    gamma: int = 1         # draft steps per decode iteration (rows appended)
    seed: int = 0
    S_lo: int = 0          # varlen: lengths uniform in [S_lo, S]
    sink_bias: float = 1.0  # factor applied to K rows [0, bias_rows)
    bias_rows: int = 0
    R_w: int = 0           # ring: window slots
    iterations: int = 0    # ring: speculative iterations
    max_accept: int = 0    # ring: accept counts uniform in [1, max_accept]
    notes: str = field(default="", compare=False)

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.d))


WORKLOADS = {
    w.name: w
    for w in [
        Workload("decode_s8k", B=1, Hq=16, Hkv=2, d=128, S=8192, W=512, sink=4,
                 gamma=1, seed=1000,
                 notes="single-token GQA decode, full and windowed"),
        Workload("draft_loop_s128k", B=1, Hq=16, Hkv=2, d=256, S=131072, W=2048,
                 sink=4, gamma=3, seed=1001,
                 notes="3 draft steps, each appending one K/V row before attending"),
        Workload("draft_loop_s1m", B=1, Hq=32, Hkv=2, d=256, S=1048576, W=2048,
                 sink=4, gamma=7, seed=1002, sink_bias=4.0, bias_rows=4,
                 notes="1M-token draft KV (2 GiB bf16), first 4 keys scaled x4"),
        Workload("batch32_varlen", B=32, Hq=32, Hkv=2, d=256, S=1048576,
                 S_lo=65536, W=2048, sink=4, gamma=1, seed=1003,
                 notes="32 sequences, lengths uniform in [65536, 1048576]"),
        Workload("ring_b8", B=8, Hq=32, Hkv=2, d=256, S=0, W=2048, sink=4,
                 R_w=2048, iterations=1000, max_accept=8, seed=1004,
                 notes="ring of 4 + 2048 slots, 1000 iterations of 1..8 appended rows"),
    ]
}


def stream_seed(seed: int, stream: int, sub: int = 0) -> int:
    """Seed of one named sub-stream of a workload (a fixed integer map)."""
    return (int(seed) * 1_000_003 + int(stream) * 10_007 + int(sub)) % (2**63 - 1)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(seed)
    return g


def normal_bf16(shape, seed: int, device="cpu") -> torch.Tensor:
    """Standard-normal float32 draws rounded to bfloat16."""
    g = _gen(seed, device)
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def fp8_codes(x: torch.Tensor) -> torch.Tensor:
    """E4M3 codes (uint8) of a float tensor, by torch's float8_e4m3fn
    conversion (round to nearest even)."""
    return x.float().to(torch.float8_e4m3fn).view(torch.uint8)


def normal_fp8(shape, seed: int, device="cpu", spread: float = 1.0) -> torch.Tensor:
    """E4M3 codes (uint8) of standard-normal float32 draws times `spread`."""
    g = _gen(seed, device)
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    return fp8_codes(x * spread)


def uniform_lengths(B: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """B integers uniform in [lo, hi] inclusive (CPU generator)."""
    g = _gen(seed, "cpu")
    return torch.randint(int(lo), int(hi) + 1, (int(B),), generator=g).numpy().astype(np.int32)


def accept_counts(iterations: int, B: int, hi: int, seed: int) -> np.ndarray:
    """[iterations, B] integers uniform in [1, hi] inclusive (CPU generator)."""
    g = _gen(seed, "cpu")
    return torch.randint(1, int(hi) + 1, (int(iterations), int(B)), generator=g).numpy().astype(np.int32)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Host copy of a bfloat16 tensor as its uint16 bit patterns."""
    if t.dtype != torch.bfloat16:
        raise TypeError("expected a bfloat16 tensor")
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def from_bits(bits: np.ndarray, device="cpu") -> torch.Tensor:
    """bfloat16 tensor holding the given uint16 bit patterns."""
    a = np.ascontiguousarray(bits).view(np.int16)
    return torch.from_numpy(a.copy()).view(torch.bfloat16).to(device)


def decode_case(wl: Workload, device="cpu", S: int | None = None, B: int | None = None,
                steps: int | None = None, extra_capacity: int = 0):
    """Inputs of a draft decode workload.

    Returns a dict with
      q      bf16 [steps, B, Hq, d]     one query per draft step
      k, v   bf16 [B, S_max, Hkv, d]    cache; rows [0, lens[b]) drawn, others 0
      lens   int32 [B] (CPU numpy)      lengths before the first step
      k_new, v_new bf16 [steps, B, 1, Hkv, d]  the row each step appends
      S_max  capacity = max(lens) + steps + extra_capacity
    S / B override the workload's length / batch (smaller parity cases keep
    the same head shapes and seeds).
    """
    B = wl.B if B is None else int(B)
    steps = wl.gamma if steps is None else int(steps)
    S0 = wl.S if S is None else int(S)
    if wl.S_lo:
        lo = min(wl.S_lo, S0)
        lens = uniform_lengths(B, lo, S0, stream_seed(wl.seed, STREAM_LENS))
    else:
        lens = np.full(B, S0, dtype=np.int32)
    S_max = int(lens.max()) + steps + int(extra_capacity)
    k = torch.zeros((B, S_max, wl.Hkv, wl.d), dtype=torch.bfloat16, device=device)
    v = torch.zeros_like(k)
    for b in range(B):
        L = int(lens[b])
        if L == 0:
            continue
        k[b, :L] = normal_bf16((L, wl.Hkv, wl.d), stream_seed(wl.seed, STREAM_K, b), device)
        v[b, :L] = normal_bf16((L, wl.Hkv, wl.d), stream_seed(wl.seed, STREAM_V, b), device)
    if wl.bias_rows and wl.sink_bias != 1.0:
        k[:, :wl.bias_rows] *= wl.sink_bias
    q = normal_bf16((steps, B, wl.Hq, wl.d), stream_seed(wl.seed, STREAM_Q), device)
    k_new = normal_bf16((steps, B, 1, wl.Hkv, wl.d), stream_seed(wl.seed, STREAM_KNEW), device)
    v_new = normal_bf16((steps, B, 1, wl.Hkv, wl.d), stream_seed(wl.seed, STREAM_VNEW), device)
    return dict(q=q, k=k, v=v, lens=lens, k_new=k_new, v_new=v_new, S_max=S_max)
