"""Pins of the fp8 (E4M3) oracle.

* code values against the OCP E4M3 field layout written out by hand
  (tests/golden/e4m3_values.txt) and against a library routine (torch's
  float8_e4m3fn -> float32 conversion) for all 256 codes;
* rounding against torch's float32 -> float8_e4m3fn cast (round to nearest
  even) on every bf16 value within range and on exact midpoints;
  saturation beyond 448 (a reading: torch's cast gives NaN there);
* round trip, monotonicity;
* quantize-on-append (division by the scale in float32) against torch;
* attention over codes equals the pinned bf16 oracle over the same values
  (every E4M3 value is a bf16 value), the scales fold as the definition
  says, and the ring read through its slot map equals the windowed read.
"""

from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import fp8 as F
from oracle import ring as R

from .conftest import read_golden


def _torch_decode_all():
    return torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).float().double().numpy()


def test_golden_code_values():
    rows = read_golden("e4m3_values.txt")
    assert len(rows) >= 12
    for code, val, _ in rows:
        got = F.decode_code(int(code, 16))
        if val == "nan":
            assert np.isnan(got), code
        else:
            exp = float(Fraction(val)) if val != "-0" else -0.0
            assert got == exp, code
            assert np.signbit(got) == np.signbit(exp), code


def test_all_codes_match_library():
    mine = F.decode(np.arange(256, dtype=np.uint8))
    ref = _torch_decode_all()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert np.array_equal(np.signbit(mine[ok]), np.signbit(ref[ok]))
    assert np.flatnonzero(np.isnan(mine)).tolist() == [0x7F, 0xFF]
    assert np.nanmax(mine) == F.E4M3_MAX == 448.0


def _finite_bf16_bits():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    return bits[(bits & 0x7F80) != 0x7F80]  # exponent field all ones: inf / NaN


def test_encode_matches_library_on_every_bf16_in_range():
    x = A.bf16_to_f64(_finite_bf16_bits()).astype(np.float32)
    x = x[np.abs(x) <= 448]
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.encode(x), ref)


def test_encode_midpoints_round_to_even():
    vals = F.decode(np.arange(0x7F, dtype=np.uint8))
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    assert np.array_equal(mids.astype(np.float64), (vals[:-1] + vals[1:]) / 2)  # exact in float32
    codes = F.encode(mids)
    lo = np.arange(0x7E)
    exp = np.where(lo % 2 == 0, lo, lo + 1)
    assert np.array_equal(codes, exp.astype(np.uint8))
    ref = torch.from_numpy(mids).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, ref)
    assert np.array_equal(F.encode(-mids), (exp | 0x80).astype(np.uint8))


def test_encode_random_floats_match_library():
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(200_000) * s for s in (1e-3, 0.05, 1.0, 30.0, 150.0)])
    x = np.clip(x, -448, 448).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.encode(x), ref)


def test_saturation_and_signed_zero():
    x = np.array([448.0, 449.0, 464.0, 480.0, 1e6, 3.4e38, -500.0, -1e30, 0.0, -0.0, 1e-30, -1e-30],
                 dtype=np.float32)
    assert F.encode(x).tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0x7E, 0xFE, 0xFE, 0x00, 0x80, 0x00, 0x80]


def test_round_trip_and_monotone():
    finite = [c for c in range(256) if c not in (0x7F, 0xFF)]
    assert F.encode(F.decode(np.array(finite, dtype=np.uint8)).astype(np.float32)).tolist() == finite
    xs = np.linspace(-460, 460, 400_001).astype(np.float32)
    v = F.decode(F.encode(xs))
    assert np.all(np.diff(v) >= 0)
    # nearest: no representable value is closer than the chosen one
    vals = F.decode(np.array(finite, dtype=np.uint8))
    sub = xs[np.abs(xs) <= 448][::97]
    best = np.min(np.abs(vals[None, :] - sub[:, None].astype(np.float64)), axis=1)
    assert np.array_equal(np.abs(F.decode(F.encode(sub)) - sub), best)


@pytest.mark.parametrize("scale", [1.0, 0.5, 0.0625, 0.7, 3.0])
def test_quantize_divides_in_float32(scale):
    bits = _finite_bf16_bits()
    x = A.bf16_to_f64(bits).astype(np.float32)
    y = (torch.from_numpy(x) / torch.tensor(scale, dtype=torch.float32)).clamp(-448, 448)
    ref = y.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.quantize(bits, scale), ref)


def _codes(rng, shape, spread=1.0):
    x = (rng.standard_normal(shape) * spread).astype(np.float32)
    return torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _bf16_bits_of(values):
    f32 = values.astype(np.float32)
    assert np.array_equal(f32.astype(np.float64), values)  # E4M3 values are exact in float32 / bf16
    u = f32.view(np.uint32)
    assert np.all(u & 0xFFFF == 0)
    return (u >> 16).astype(np.uint16)


@pytest.mark.parametrize("variant", ["full", "windowed"])
def test_attention_equals_bf16_oracle_on_same_values(variant):
    rng = np.random.default_rng(5)
    Hq, Hkv, d, S, W, sink = 8, 2, 32, 300, 40, 3
    q = rng.standard_normal((Hq, d))
    kc, vc = _codes(rng, (S, Hkv, d)), _codes(rng, (S, Hkv, d), 3.0)
    o8, l8 = F.attend_sequence_fp8(q, kc, vc, S, 0.2, 1.0, 1.0, variant, W, sink)
    mask = None if variant == "full" else A.window_mask(S, W, sink)
    ob, lb = A.attend_sequence(q, _bf16_bits_of(F.decode(kc)), _bf16_bits_of(F.decode(vc)), S, 0.2, mask)
    assert np.array_equal(o8, ob) and np.array_equal(l8, lb)


def test_scales_fold_as_defined():
    rng = np.random.default_rng(6)
    Hq, Hkv, d, S = 4, 1, 16, 97
    q = rng.standard_normal((Hq, d))
    kc, vc = _codes(rng, (S, Hkv, d)), _codes(rng, (S, Hkv, d))
    o1, l1 = F.attend_sequence_fp8(q, kc, vc, S, 0.25, 1.0, 1.0)
    # k_scale multiplies every logit: the same as scaling the softmax scale
    o2, l2 = F.attend_sequence_fp8(q, kc, vc, S, 0.125, 2.0, 1.0)
    assert np.allclose(o1, o2, atol=1e-13) and np.allclose(l1, l2, atol=1e-13)
    # v_scale multiplies the output and leaves the log-sum-exp alone
    o3, l3 = F.attend_sequence_fp8(q, kc, vc, S, 0.25, 1.0, 0.375)
    assert np.allclose(o3, 0.375 * o1, atol=1e-13) and np.array_equal(l3, l1)
    # dequantized values are code value times scale, exactly
    assert np.array_equal(F.dequantize(kc, 0.3), F.decode(kc) * np.float64(np.float32(0.3)))


def test_ring_read_equals_windowed_read():
    rng = np.random.default_rng(7)
    Hq, Hkv, d, W, sink = 4, 2, 16, 24, 3
    for S, R_w in ((10, 24), (27, 24), (28, 30), (200, 24), (501, 37)):
        kc, vc = _codes(rng, (S, Hkv, d)), _codes(rng, (S, Hkv, d))
        ring_k = np.zeros((sink + R_w, Hkv, d), dtype=np.uint8)
        ring_v = np.zeros_like(ring_k)
        for p in range(S):  # appends in order: a slot keeps its last writer
            s = R.ring_slot(p, sink, R_w)
            ring_k[s], ring_v[s] = kc[p], vc[p]
        q = rng.standard_normal((Hq, d))
        o_r, l_r = F.attend_ring_fp8(q, ring_k, ring_v, S, 0.3, 0.5, 2.0, W, sink, R_w)
        o_w, l_w = F.attend_sequence_fp8(q, kc, vc, S, 0.3, 0.5, 2.0, "windowed", W, sink)
        assert np.array_equal(o_r, o_w) and np.array_equal(l_r, l_w), (S, R_w)


# ------------------------------------------------------------------ mutants
# Each plants one plausible mistake in the fp8 oracle (on the CPU) and checks
# that at least one pin above then fails.
_PINS = [test_golden_code_values, test_all_codes_match_library,
         test_encode_matches_library_on_every_bf16_in_range, test_encode_midpoints_round_to_even,
         test_saturation_and_signed_zero, test_round_trip_and_monotone,
         lambda: test_quantize_divides_in_float32(0.7), test_scales_fold_as_defined,
         lambda: test_attention_equals_bf16_oracle_on_same_values("full")]


def _some_pin_fails():
    for pin in _PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except AssertionError:
            return True
    return False


def _decode_bias8(c):
    c = int(c) & 0xFF
    s, e, m = (-1.0 if c & 0x80 else 1.0), (c >> 3) & 0xF, c & 7
    if e == 15 and m == 7:
        return float("nan")
    return s * (m / 8.0) * 2.0 ** -7 if e == 0 else s * (1 + m / 8.0) * 2.0 ** (e - 8)


def _decode_no_subnormals(c):
    c = int(c) & 0xFF
    s, e, m = (-1.0 if c & 0x80 else 1.0), (c >> 3) & 0xF, c & 7
    if e == 15 and m == 7:
        return float("nan")
    return s * (1 + m / 8.0) * 2.0 ** (max(e, 1) - 7) if (e or m) else 0.0 * s


def _table_mutant(monkeypatch, fn):
    table = np.array([fn(c) for c in range(256)])
    monkeypatch.setattr(F, "decode_code", fn)
    monkeypatch.setattr(F, "_TABLE", table)
    monkeypatch.setattr(F, "_POS_VALUES", table[:0x7F])


def test_mutant_wrong_bias(monkeypatch):
    _table_mutant(monkeypatch, _decode_bias8)
    assert _some_pin_fails()


def test_mutant_subnormals_with_hidden_one(monkeypatch):
    _table_mutant(monkeypatch, _decode_no_subnormals)
    assert _some_pin_fails()


def test_mutant_ties_away_from_zero(monkeypatch):
    orig = F.encode

    def enc(y):
        y = np.asarray(y, dtype=np.float32)
        c = orig(y)
        up = np.minimum((c & 0x7F).astype(np.int64) + 1, 0x7E)
        mid = (F._TABLE[c & 0x7F] + F._TABLE[up]) / 2
        return np.where(np.abs(y.astype(np.float64)) == mid, up | (c & 0x80), c).astype(np.uint8)

    monkeypatch.setattr(F, "encode", enc)
    assert _some_pin_fails()


def test_mutant_no_saturation(monkeypatch):
    orig = F.encode
    monkeypatch.setattr(F, "encode", lambda y: np.where(np.abs(np.asarray(y, dtype=np.float32)) > 448,
                                                        np.uint8(0x7F), orig(y)).astype(np.uint8))
    assert _some_pin_fails()


def test_mutant_multiply_by_scale_on_append(monkeypatch):
    monkeypatch.setattr(F, "quantize", lambda bits, scale: F.encode(
        A.bf16_to_f64(bits).astype(np.float32) * np.float32(scale)))
    assert _some_pin_fails()


def test_mutant_v_scale_on_keys(monkeypatch):
    orig = F.attend_sequence_fp8

    def swapped(q, kc, vc, S, scale, k_scale, v_scale, variant="full", W=1, sink=0):
        return orig(q, kc, vc, S, scale, v_scale, k_scale, variant, W, sink)

    monkeypatch.setattr(F, "attend_sequence_fp8", swapped)
    assert _some_pin_fails()


def test_spread_option_over_binary_codes():
    # codes of 0.0 and 1.0 (0x38) with v_scale 1: Bernoulli values, spread 2 o (1 - o)
    rng = np.random.default_rng(9)
    S, Hkv, d = 60, 2, 16
    q = rng.standard_normal((4, d))
    kc = F.encode(rng.standard_normal((S, Hkv, d)).astype(np.float32))
    vc = np.where(rng.random((S, Hkv, d)) < 0.3, 0x38, 0x00).astype(np.uint8)
    for variant in ("full", "windowed"):
        o, lse, s = F.attend_sequence_fp8(q, kc, vc, S, 0.3, 0.5, 1.0, variant, 20, 2, spread=True)
        o2, lse2 = F.attend_sequence_fp8(q, kc, vc, S, 0.3, 0.5, 1.0, variant, 20, 2)
        assert np.array_equal(o, o2) and np.array_equal(lse, lse2)
        np.testing.assert_allclose(s, 2 * o * (1 - o), atol=1e-13)
    R_w = 24
    slots = R.ring_slots(A.selected_positions(S, 20, 2), 2, R_w)
    rk = np.zeros((2 + R_w, Hkv, d), np.uint8)
    rv = np.zeros_like(rk)
    rk[slots], rv[slots] = kc[A.selected_positions(S, 20, 2)], vc[A.selected_positions(S, 20, 2)]
    o, _, s = F.attend_ring_fp8(q, rk, rv, S, 0.3, 0.5, 1.0, 20, 2, R_w, spread=True)
    np.testing.assert_allclose(s, 2 * o * (1 - o), atol=1e-13)
