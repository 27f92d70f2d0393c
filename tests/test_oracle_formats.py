"""Pins for the oracle's number formats.

Each codec is checked against something other than itself: torch's own fp8
and fp16 conversions (an independent implementation), the published value
lists of the OCP formats, and a brute-force nearest-even search over every
finite code.
"""
import itertools
import math

import numpy as np
import pytest
import torch

from oracle import formats as F


def _brute_nearest_even(x: float, values, sign_bit: int, vmax: float) -> int:
    """Nearest finite code by exhaustive search; ties to the even code."""
    a = min(abs(x), vmax)
    best, best_d = None, None
    for c, v in enumerate(values):
        if math.isnan(v) or v < 0 or (c & sign_bit):
            continue
        d = abs(v - a)
        if best is None or d < best_d or (d == best_d and c % 2 == 0 and best % 2 == 1):
            best, best_d = c, d
    if math.copysign(1.0, x) < 0:
        best |= sign_bit
    return best


# ------------------------------------------------------------------ E4M3FN
def test_e4m3_table_matches_torch():
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy()
    ours = F.E4M3_TABLE.astype(np.float32)
    assert np.array_equal(np.isnan(ref), np.isnan(ours))
    ok = ~np.isnan(ref)
    assert np.array_equal(ref[ok], ours[ok])
    # NaN codes are exactly S.1111.111
    assert [c for c in range(256) if math.isnan(F.E4M3_TABLE[c])] == [0x7F, 0xFF]
    assert F.E4M3_TABLE[0x7E] == 448.0 and F.E4M3_TABLE[0x01] == 2.0 ** -9


def _e4m3_probe_values():
    pos = F.E4M3_TABLE[:0x7F]
    mids = (pos[1:] + pos[:-1]) / 2
    vals = [0.0, -0.0, 448.0, -448.0, 1e-30, -1e-30, 2.0 ** -10, 3 * 2.0 ** -11]
    for m in mids:  # every rounding boundary, and one fp32 ulp either side
        m32 = np.float32(m)
        vals += [float(m32), float(np.nextafter(m32, np.float32(0))),
                 float(np.nextafter(m32, np.float32(1e9)))]
    rng = np.random.default_rng(7)
    vals += list(rng.uniform(-448, 448, 3000).astype(np.float32).astype(float))
    vals += list((rng.standard_normal(3000) * 2.0 ** rng.integers(-12, 9, 3000))
                 .astype(np.float32).astype(float))
    v = np.array(vals, dtype=np.float32)
    return np.concatenate([v, -v])


def test_e4m3_encoder_matches_torch_in_range():
    v = _e4m3_probe_values()
    v = v[np.abs(v) <= 448]
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(F.e4m3_encode(v), ref)


def test_e4m3_encoder_matches_brute_force():
    v = _e4m3_probe_values()[::7]
    got = F.e4m3_encode(v)
    table = list(F.E4M3_TABLE)
    for x, c in zip(v.astype(float), got):
        assert c == _brute_nearest_even(x, table, 0x80, 448.0), x


def test_e4m3_roundtrip_and_saturation():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(F.e4m3_encode(F.e4m3_decode(codes)), codes)
    assert list(F.e4m3_encode(np.array([449.0, 1e6, -1e6, 464.0]))) == [0x7E, 0x7E, 0xFE, 0x7E]


def test_e4m3_relative_error_bound():
    # normals: |x - q| <= 2^-4 |x| (half an ulp of a 3-bit mantissa)
    rng = np.random.default_rng(1)
    x = rng.uniform(2.0 ** -6, 448, 20000)
    q = F.e4m3_decode(F.e4m3_encode(x))
    assert (np.abs(x - q) <= 2.0 ** -4 * np.abs(x)).all()


# ------------------------------------------------------------------ E2M1
def test_e2m1_values_are_the_ocp_list():
    assert list(F.E2M1_TABLE[:8]) == [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    assert list(F.E2M1_TABLE[8:]) == [-0.0, -0.5, -1.0, -1.5, -2.0, -3.0, -4.0, -6.0]


def test_e2m1_encoder_brute_force_and_roundtrip():
    rng = np.random.default_rng(2)
    pos = F.E2M1_TABLE[:8]
    mids = list((pos[1:] + pos[:-1]) / 2)
    v = np.array(mids + [0.0, 6.0, 7.0, 100.0, 0.2] + list(rng.uniform(-7, 7, 2000)))
    v = np.concatenate([v, -v])
    got = F.e2m1_encode(v)
    table = list(F.E2M1_TABLE)
    for x, c in zip(v, got):
        assert c == _brute_nearest_even(float(x), table, 0x8, 6.0), x
    # ties go to the even code: 0.25 -> 0, 0.75 -> 1.0, 1.25 -> 1.0, 2.5 -> 2, 3.5 -> 4, 5 -> 4
    assert [F.E2M1_TABLE[c] for c in F.e2m1_encode(np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]))] \
        == [0.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0]
    codes = np.arange(16, dtype=np.uint8)
    assert np.array_equal(F.e2m1_encode(F.e2m1_decode(codes)), codes)


# ------------------------------------------------------------------ E8M0, log2
def test_e8m0():
    assert F.e8m0_value(127) == 1.0
    assert F.e8m0_value(0) == 2.0 ** -127
    assert F.e8m0_value(254) == 2.0 ** 127
    assert math.isnan(F.e8m0_value(255))


@pytest.mark.parametrize("k", list(range(-140, 128, 3)))
def test_floor_log2_at_powers_of_two(k):
    p = np.float32(2.0 ** k) if k >= -149 else None
    assert F.floor_log2(np.array([float(p)]))[0] == k
    below = np.nextafter(p, np.float32(0))
    if below > 0:
        assert F.floor_log2(np.array([float(below)]))[0] == k - 1


# ------------------------------------------------------------------ ints, fp16
def test_int_rne_clamp_ties_to_even():
    x = np.array([0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 126.5, 127.4, 200.0, -300.0])
    assert list(F.int_rne_clamp(x, 127)) == [0, 2, 2, 0, -2, -2, 126, 127, 127, -127]
    assert list(F.int_rne_clamp(np.array([6.5, 7.5, -7.5, 3.5]), 7)) == [6, 7, -7, 4]


def test_f16_round_matches_torch():
    rng = np.random.default_rng(3)
    x = (rng.standard_normal(50000) * 2.0 ** rng.integers(-30, 16, 50000)).astype(np.float32)
    ref = torch.from_numpy(x).half().numpy()
    assert np.array_equal(F.f16_round(x).view(np.uint16), ref.view(np.uint16))


def test_every_fp16_value_is_exact_in_fp32():
    # The product path reads fp16 scales into fp32 exactly.
    h = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16)
    assert np.array_equal(h.astype(np.float32).astype(np.float16).view(np.uint16), h.view(np.uint16))


def test_formats_exact_in_fp16():
    # int8 and every finite e4m3 / e2m1 value are exact fp16 numbers.
    ints = np.arange(-127, 128).astype(np.float16).astype(np.float64)
    assert np.array_equal(ints, np.arange(-127, 128))
    fin = F.E4M3_TABLE[~np.isnan(F.E4M3_TABLE)]
    assert np.array_equal(fin.astype(np.float16).astype(np.float64), fin)
    assert np.array_equal(F.E2M1_TABLE.astype(np.float16).astype(np.float64), F.E2M1_TABLE)
