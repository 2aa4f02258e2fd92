"""Number formats of the oracle, written from their definitions.

Test infrastructure (see the package docstring): not used by the library.

bf16: the upper 16 bits of an IEEE-754 binary32; widening is exact.
OCP FP8 E4M3FN: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; no
infinities; S.1111.111 is NaN; largest finite magnitude 1.75 * 2^8 = 448;
exponent field 0 encodes subnormals m/8 * 2^-6.
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bf16 bit patterns (uint16) as float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):  # signalling-NaN patterns widen to NaN
        return u.view(np.float32).astype(np.float64)


def _e4m3fn_table() -> np.ndarray:
    """Value of every one of the 256 codes, from the field definition."""
    vals = np.empty(256, dtype=np.float64)
    for c in range(256):
        sign = -1.0 if (c >> 7) & 1 else 1.0
        e = (c >> 3) & 0xF
        m = c & 0x7
        if e == 0xF and m == 0x7:
            vals[c] = np.nan
        elif e == 0:
            vals[c] = sign * (m / 8.0) * 2.0 ** (1 - 7)
        else:
            vals[c] = sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)
    return vals


E4M3FN_VALUES = _e4m3fn_table()
E4M3FN_MAX = 448.0


def e4m3fn_decode(codes: np.ndarray) -> np.ndarray:
    """Exact float64 value of fp8 codes (uint8)."""
    return E4M3FN_VALUES[np.asarray(codes, dtype=np.uint8)]


def e4m3fn_encode_rne(x: np.ndarray) -> np.ndarray:
    """Nearest E4M3FN code to each (already clamped, |x| <= 448) value; ties to even.

    NaN maps to 0x7F.  Values beyond +-448 are rejected: quantise-on-write
    clamps before encoding, so such a value is a caller error here.
    """
    x = np.asarray(x, dtype=np.float64)
    if np.any(np.abs(x[~np.isnan(x)]) > E4M3FN_MAX):
        raise ValueError("e4m3fn_encode_rne expects |x| <= 448")
    mags = E4M3FN_VALUES[:0x7F]  # codes 0x00..0x7E: 0 .. 448, increasing
    a = np.abs(x)
    a_safe = np.where(np.isnan(a), 0.0, a)
    hi = np.searchsorted(mags, a_safe, side="left")  # first code with value >= a
    hi = np.clip(hi, 0, 0x7E)
    lo = np.clip(hi - 1, 0, 0x7E)
    d_hi = mags[hi] - a_safe
    d_lo = a_safe - mags[lo]
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (lo % 2 == 0))
    code = np.where(pick_lo, lo, hi).astype(np.uint8)
    code = np.where(np.signbit(x), code | np.uint8(0x80), code).astype(np.uint8)
    return np.where(np.isnan(x), np.uint8(0x7F), code).astype(np.uint8)
