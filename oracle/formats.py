"""Number formats, written out from their definitions.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The paper uses int8, int4, fp8-e4m3 and fp4-e2m1 for weights and activations
(Section 5.1 and Table 2/3 labels) and per-vector scale factors (Section 3.3,
VS-Quant).  The exact encodings follow the public format definitions:

* fp8 E4M3FN (OCP 8-bit floating point): 1 sign, 4 exponent bits (bias 7),
  3 mantissa bits; exponent field 0 encodes subnormals m * 2^-9; the only
  NaN is S.1111.111; there is no infinity; the largest finite value is 448.
* fp4 E2M1 (OCP MX): 1 sign, 2 exponent bits (bias 1), 1 mantissa bit;
  values 0, 0.5, 1, 1.5, 2, 3, 4, 6.
* E8M0 (OCP MX shared scale): an unsigned biased exponent, value 2^(c-127);
  code 255 is NaN.
* ufp8 E6M2 (the unsigned scale format of the paper's quantization study,
  Section 6.4): 6 exponent bits with bias 31, 2 mantissa bits, no sign;
  exponent field 0 encodes subnormals m/4 * 2^-30; every code is finite
  (the largest is 1.75 * 2^32).
* fp16: IEEE binary16 (numpy's float16 cast is round-to-nearest-even).
* integers: round-to-nearest-even (``numpy.rint``) followed by a clamp.

Encoders return the code whose value is nearest to the input; ties go to the
code with an even mantissa (its lowest bit is 0).  Inputs beyond the largest
finite value saturate to it.  The sign is kept, so a negative input that
rounds to zero encodes negative zero (as an IEEE conversion would).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0
E2M1_MAX = 6.0


# --------------------------------------------------------------------------
# fp8 E4M3FN
# --------------------------------------------------------------------------
def e4m3_value(code: int) -> float:
    """Value of one E4M3FN code (NaN for the NaN codes)."""
    code = int(code) & 0xFF
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return s * m * 2.0 ** -9
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3_TABLE = np.array([e4m3_value(c) for c in range(256)], dtype=np.float64)


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    return E4M3_TABLE[np.asarray(codes, dtype=np.uint8)]


def _encode_nearest_even(x: np.ndarray, pos_values: np.ndarray, sign_bit: int,
                         vmax: float) -> np.ndarray:
    """Nearest-even encoder for a sign-magnitude format.

    ``pos_values[c]`` is the value of the non-negative code ``c`` and is
    strictly increasing in ``c``.  Magnitudes above ``vmax`` saturate.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), vmax)
    hi = np.searchsorted(pos_values, a, side="left")  # first code with value >= a
    hi = np.clip(hi, 0, len(pos_values) - 1)
    lo = np.clip(hi - 1, 0, len(pos_values) - 1)
    d_hi = pos_values[hi] - a
    d_lo = a - pos_values[lo]
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(pick_lo, lo, hi).astype(np.uint8)
    # Rounding keeps the sign: a negative input that rounds to zero gives -0.
    return np.where(np.signbit(x), code | sign_bit, code).astype(np.uint8)


_E4M3_POS = E4M3_TABLE[:0x7F]  # codes 0..126 (0x7F is NaN)


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """fp32/fp64 -> E4M3FN code, nearest-even, saturating to +-448."""
    return _encode_nearest_even(x, _E4M3_POS, 0x80, E4M3_MAX)


# --------------------------------------------------------------------------
# fp4 E2M1
# --------------------------------------------------------------------------
def e2m1_value(code: int) -> float:
    code = int(code) & 0xF
    s = -1.0 if code & 0x8 else 1.0
    e = (code >> 1) & 0x3
    m = code & 0x1
    if e == 0:
        return s * m * 0.5
    return s * (1.0 + m / 2.0) * 2.0 ** (e - 1)


E2M1_TABLE = np.array([e2m1_value(c) for c in range(16)], dtype=np.float64)
_E2M1_POS = E2M1_TABLE[:8]


def e2m1_decode(codes: np.ndarray) -> np.ndarray:
    return E2M1_TABLE[np.asarray(codes, dtype=np.uint8) & 0xF]


def e2m1_encode(x: np.ndarray) -> np.ndarray:
    """fp32/fp64 -> E2M1 code (low nibble), nearest-even, saturating to +-6."""
    return _encode_nearest_even(x, _E2M1_POS, 0x8, E2M1_MAX)


# --------------------------------------------------------------------------
# ufp8 E6M2 (unsigned)
# --------------------------------------------------------------------------
def ue6m2_value(code: int) -> float:
    code = int(code) & 0xFF
    e, m = code >> 2, code & 0x3
    if e == 0:
        return (m / 4.0) * 2.0 ** -30
    return (1.0 + m / 4.0) * 2.0 ** (e - 31)


UE6M2_TABLE = np.array([ue6m2_value(c) for c in range(256)], dtype=np.float64)
UE6M2_MAX = float(UE6M2_TABLE[255])


def ue6m2_decode(codes: np.ndarray) -> np.ndarray:
    return UE6M2_TABLE[np.asarray(codes, dtype=np.uint8)]


def ue6m2_encode(x: np.ndarray) -> np.ndarray:
    """Non-negative fp32/fp64 -> ufp8 E6M2 code, nearest-even, saturating."""
    assert not np.signbit(np.asarray(x, dtype=np.float64)).any(), "E6M2 is unsigned"
    return _encode_nearest_even(x, UE6M2_TABLE, 0, UE6M2_MAX)


# --------------------------------------------------------------------------
# E8M0 shared exponent
# --------------------------------------------------------------------------
def e8m0_value(code: np.ndarray) -> np.ndarray:
    c = np.asarray(code, dtype=np.int64)
    v = np.ldexp(1.0, c - 127)
    return np.where(c == 255, np.nan, v)


def floor_log2(a: np.ndarray) -> np.ndarray:
    """floor(log2(a)) for positive finite a, exactly (via the binary exponent)."""
    _, e = np.frexp(np.asarray(a, dtype=np.float64))
    return e.astype(np.int64) - 1


# --------------------------------------------------------------------------
# integers
# --------------------------------------------------------------------------
def int_rne_clamp(x: np.ndarray, qmax: int) -> np.ndarray:
    """Round to nearest integer, ties to even, then clamp to [-qmax, qmax]."""
    return np.clip(np.rint(np.asarray(x, dtype=np.float64)), -qmax, qmax).astype(np.int64)


# --------------------------------------------------------------------------
# fp16 / bf16
# --------------------------------------------------------------------------
def f16_round(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to IEEE binary16 (nearest-even); returns float16."""
    with np.errstate(over="ignore"):
        return np.asarray(x, dtype=np.float32).astype(np.float16)
