"""An 8-bit floating-point KV cache (E4M3), in plain numpy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper names its model and states no KV-cache precision; an 8-bit cache
is a model-serving option, offered by the store as an opt-in (the scope
table lists it with the other model variants).  Readings:

* Format: the OCP 8-bit E4M3 format (the MI355X's native FP8): 1 sign bit,
  4 exponent bits with bias 7, 3 mantissa bits.  Exponent field 0 holds the
  subnormals m/8 * 2^-6; codes 0x7F and 0xFF are NaN; there are no
  infinities; the largest finite magnitude is 448 (code 0x7E).
* Scales: one float32 scale per layer for K and one for V.  A stored value
  is decode(code) * scale.
* Quantisation of a bf16 input x: y = float32(float32(x) * inv), where
  inv = float32(1 / scale) (the division in double, then rounded to
  float32); code = the E4M3 value nearest to y, ties to the even code;
  magnitudes at or beyond 448 saturate to 448 (never NaN); the sign of y
  is kept (so -0 and tiny negatives give code 0x80).
"""

from __future__ import annotations

import numpy as np

MAX_FINITE = 448.0


def decode(codes):
    """E4M3 codes (uint8 array) -> float64 values, by the format's definition."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    normal = np.ldexp(1.0 + m / 8.0, e - 7)
    sub = np.ldexp(m / 8.0, -6)
    out = sign * np.where(e == 0, sub, normal)
    out = np.where((c & 0x7F) == 0x7F, np.nan, out)
    return out


# the non-negative finite magnitudes, indexed by code 0 .. 0x7E (increasing)
_MAGS = decode(np.arange(0x7F))


def encode(y):
    """float32 values -> E4M3 codes (uint8): nearest magnitude, ties to the
    even code, saturating at 448."""
    y = np.asarray(y, dtype=np.float32).astype(np.float64)
    if np.any(np.isnan(y)):
        raise ValueError("NaN input")
    a = np.abs(y)
    # candidates: the largest magnitude <= a and the next one
    lo = np.clip(np.searchsorted(_MAGS, a, side="right") - 1, 0, 0x7E)
    hi = np.minimum(lo + 1, 0x7E)
    d_lo = a - _MAGS[lo]
    d_hi = _MAGS[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0) & (hi != lo))
    code = np.where(pick_hi, hi, lo)
    code = np.where(a >= MAX_FINITE, 0x7E, code)
    code = code | np.where(np.signbit(y), 0x80, 0)
    return code.astype(np.uint8)


def inv_scale(scale):
    """float32(1 / scale), the division taken in double."""
    return np.float32(1.0 / np.float64(np.float32(scale)))


def quantize(x, scale):
    """bf16-valued x (any float array) -> codes, with the layer's scale."""
    y = np.asarray(x, dtype=np.float32) * inv_scale(scale)  # float32 product
    return encode(y.astype(np.float32))


def dequantize(codes, scale):
    return decode(codes) * np.float64(np.float32(scale))


def roundtrip(x, scale):
    """What the store holds for x: dequantize(quantize(x))."""
    return dequantize(quantize(x, scale), scale)
