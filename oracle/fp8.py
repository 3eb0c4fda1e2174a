"""FP8 (E4M3) draft KV cache -- the oracle's statement of it.

TEST INFRASTRUCTURE ONLY (see the package docstring): nothing on the product
path imports this module.

What the paper fixes (Windowed-MTP, Section 7 "Robustness to KV-cache
quantization"): the draft may read an fp8 KV cache; windowing changes which
entries are read, the KV dtype only the bytes per entry, and the attention
result is the same masked-softmax attention over the dequantized entries.
The paper does not spell out the format.  Readings:

  * Format: OCP 8-bit floating point, E4M3 variant ("e4m3fn"): 1 sign bit,
    4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 encodes
    subnormals m/8 * 2^-6; no infinities; S.1111.111 is NaN; largest finite
    magnitude 448.  (OCP OFP8 specification, rev. 1.0, E4M3 column.)
  * Scaling: one float32 scale per tensor (k_scale for keys, v_scale for
    values), as serving stacks attach to an fp8 KV cache: the stored code c
    stands for decode(c) * scale.
  * Quantization on append: y = x / scale computed in float32 (x is the bf16
    row value), clamped to [-448, 448] (saturation, never NaN), then rounded
    to the nearest E4M3 value, ties to the even code (round-to-nearest-even).
    The sign of a value that rounds to zero is kept (code 0x80 is -0).
  * Non-finite inputs (inf, NaN in x) are outside the contract.

The attention itself is the float64 definition of oracle.attention applied to
K = decode(k_codes) * k_scale and V = decode(v_codes) * v_scale (every such
product of an E4M3 value and a float32 scale is exact in float64).
"""

from __future__ import annotations

import numpy as np

from . import attention as A
from . import ring as R

__all__ = [
    "E4M3_MAX",
    "decode_code",
    "decode",
    "encode",
    "quantize",
    "dequantize",
    "DequantizedRows",
    "attend_sequence_fp8",
    "attend_ring_fp8",
]

E4M3_MAX = 448.0


def decode_code(c: int) -> float:
    """Value of one E4M3 code, from the field definition."""
    c = int(c) & 0xFF
    sign = -1.0 if c & 0x80 else 1.0
    e = (c >> 3) & 0xF
    m = c & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return sign * (m / 8.0) * 2.0 ** (1 - 7)
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


# Value of every code, computed once from the definition.
_TABLE = np.array([decode_code(c) for c in range(256)], dtype=np.float64)
# Non-negative finite codes 0x00 .. 0x7E have strictly increasing values.
_POS_CODES = np.arange(0x7F, dtype=np.int64)
_POS_VALUES = _TABLE[:0x7F]


def decode(codes) -> np.ndarray:
    """E4M3 codes (uint8 array) -> float64 values."""
    return _TABLE[np.asarray(codes, dtype=np.uint8).astype(np.int64)]


def encode(y) -> np.ndarray:
    """Round float32 values to E4M3 codes: clamp to [-448, 448], then the
    nearest representable magnitude, ties to the even code; sign kept."""
    y = np.asarray(y, dtype=np.float32).astype(np.float64)
    neg = np.signbit(y)
    a = np.minimum(np.abs(y), E4M3_MAX)
    # neighbours lo <= a <= hi among the non-negative finite values
    hi_i = np.searchsorted(_POS_VALUES, a, side="left")
    hi_i = np.minimum(hi_i, len(_POS_VALUES) - 1)
    lo_i = np.where(_POS_VALUES[hi_i] == a, hi_i, np.maximum(hi_i - 1, 0))
    lo_v, hi_v = _POS_VALUES[lo_i], _POS_VALUES[hi_i]
    d_lo, d_hi = a - lo_v, hi_v - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (_POS_CODES[hi_i] % 2 == 0) & (hi_i != lo_i))
    mag = np.where(pick_hi, _POS_CODES[hi_i], _POS_CODES[lo_i])
    return (mag | np.where(neg, 0x80, 0)).astype(np.uint8)


def quantize(x_bf16_bits, scale: float) -> np.ndarray:
    """Codes of bf16 values x stored with per-tensor `scale`: encode(x / scale)
    with the division in float32."""
    x = A.bf16_to_f64(x_bf16_bits).astype(np.float32)
    with np.errstate(over="ignore"):  # a quotient past float32's range saturates like any other
        y = x / np.float32(scale)
    return encode(y)


def dequantize(codes, scale: float) -> np.ndarray:
    """Value each code stands for: decode(c) * scale, exact in float64."""
    return decode(codes) * np.float64(np.float32(scale))


class DequantizedRows:
    """Row view of an fp8 cache [rows, Hkv, d] for oracle.attention:
    view[idx] = dequantize(codes[idx], scale).  `codes` is anything indexable
    by an array of row numbers that yields uint8 codes (a numpy array, or a
    host view of a device cache)."""

    def __init__(self, codes, scale: float):
        self.codes = codes
        self.scale = scale
        self.shape = tuple(codes.shape)

    def __getitem__(self, rows):
        return dequantize(np.asarray(self.codes[rows]), self.scale)


def attend_sequence_fp8(q, k_codes, v_codes, S, scale, k_scale, v_scale, variant="full", W=1, sink=0,
                        spread=False):
    """Single-token GQA decode attention of one sequence over an fp8 cache.

    q [Hq, d] (bf16 bits or floats); k_codes, v_codes [rows >= S, Hkv, d]
    uint8 (or row views, see DequantizedRows).  The key set is the variant's
    (oracle.attention.window_mask); the softmax and the value sum are
    oracle.attention.attend_sequence over the dequantized rows.  Returns
    (o [Hq, d], lse [Hq]) in float64, and with spread=True also
    oracle.attention.value_spread over the same rows.
    """
    mask = None if variant == "full" else A.window_mask(S, W, sink)
    K, V = DequantizedRows(k_codes, k_scale), DequantizedRows(v_codes, v_scale)
    o, lse = A.attend_sequence(q, K, V, S, scale, mask)
    if not spread:
        return o, lse
    return o, lse, A.value_spread(q, K, V, S, scale, mask)


def attend_ring_fp8(q, ring_k, ring_v, S, scale, k_scale, v_scale, W, sink, R_w, spread=False):
    """Windowed attention read through the compact ring's slot map
    (oracle.ring.ring_slot) from an fp8 ring [sink + R_w, Hkv, d]
    (spread as for attend_sequence_fp8)."""
    slots = R.ring_slots(A.selected_positions(S, W, sink), sink, R_w)
    K = dequantize(np.asarray(ring_k)[slots], k_scale)
    V = dequantize(np.asarray(ring_v)[slots], v_scale)
    o, lse = A.attend_sequence(q, K, V, len(slots), scale, None)
    if not spread:
        return o, lse
    return o, lse, A.value_spread(q, K, V, len(slots), scale, None)
