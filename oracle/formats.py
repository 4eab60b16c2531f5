"""Number formats used by the paged KV pool, written from their definitions.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this.

* bfloat16: the upper 16 bits of an IEEE-754 binary32, rounded to nearest,
  ties to even.
* fp8 E4M3FN (OCP 8-bit floating point specification, "E4M3"): 1 sign bit,
  4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 encodes the
  subnormals m/8 * 2^-6; no infinities; S.1111.111 is NaN, so the largest
  finite magnitude is 1.75 * 2^8 = 448.

The fp8 pool stores codes plus a per-(page, head) fp32 scale s; a new-turn
value x is encoded as RNE_E4M3(clamp(fl32(x / s), -448, 448)) and decoded as
e4m3_value(code) * s (the scale policy is the caller's; the encoder and the
decoder are fixed here).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


# ----------------------------------------------------------------- bfloat16

def bf16_bits_from_f32(x) -> np.ndarray:
    """Round binary32 values to bfloat16 (RNE); return the 16-bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    r = np.where(nan, ((u >> 16) & 0x8000) | 0x7FC0, r)
    return r.astype(np.uint16)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact value of bfloat16 bit patterns, as float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def bf16_bits_to_f32(bits) -> np.ndarray:
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32)


# ------------------------------------------------------------- fp8 E4M3FN

def _e4m3_value(code: int) -> float:
    s = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return float("nan")
    if e == 0:
        return s * (m / 8.0) * 2.0 ** -6
    return s * (1.0 + m / 8.0) * 2.0 ** (e - 7)


E4M3_TABLE = np.array([_e4m3_value(c) for c in range(256)], dtype=np.float64)
# non-negative finite codes 0x00..0x7E in increasing value order
_POS_VALUES = E4M3_TABLE[:0x7F].copy()


def e4m3_to_f64(codes) -> np.ndarray:
    """Exact value of E4M3FN codes (NaN for 0x7F / 0xFF)."""
    return E4M3_TABLE[np.asarray(codes, dtype=np.uint8)]


def e4m3_encode(r) -> np.ndarray:
    """Round finite values with |r| <= 448 to the nearest E4M3FN code, ties
    to the even code (even mantissa).  The sign is kept, so -0 -> 0x80.
    NaN inputs give 0x7F | sign.  |r| > 448 is rejected: saturation is the
    caller's explicit clamp, not part of rounding."""
    r = np.asarray(r, dtype=np.float64)
    nan = np.isnan(r)
    a = np.abs(np.where(nan, 0.0, r))
    if np.any(a > E4M3_MAX):
        raise ValueError("e4m3_encode: |r| > 448 must be clamped first")
    hi = np.searchsorted(_POS_VALUES, a, side="left")  # first value >= a
    hi = np.minimum(hi, 0x7E)
    lo = np.maximum(hi - 1, 0)
    d_hi = _POS_VALUES[hi] - a
    d_lo = a - _POS_VALUES[lo]
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo)
    code = np.where(_POS_VALUES[hi] == a, hi, code)
    sign = np.signbit(r)
    code = np.where(sign, code | 0x80, code)
    code = np.where(nan, np.where(sign, 0xFF, 0x7F), code)
    return code.astype(np.uint8)


def fp8_quantize(x_f32, scale_f32) -> np.ndarray:
    """Pool encoding of value x with scale s: binary32 division x / s
    (round to nearest even), clamp to [-448, 448], then RNE to E4M3FN."""
    x = np.asarray(x_f32, dtype=np.float32)
    s = np.asarray(scale_f32, dtype=np.float32)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        q = np.divide(x, s, dtype=np.float32)
    nan = np.isnan(q)
    q = np.clip(np.where(nan, 0, q), -E4M3_MAX, E4M3_MAX).astype(np.float32)
    q = np.where(nan, np.float32("nan"), q)
    return e4m3_encode(q)
