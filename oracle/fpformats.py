"""Floating-point storage formats of the certified cache, written out exactly.

* ``f32``          round a float64 value to the nearest fp32 (ties to even).  Used to
                   emulate each fp32 operation of the quantizer: for +, -, * and /
                   of fp32 operands the float64 result rounded once more to fp32 is
                   the correctly rounded fp32 result (53 >= 2*24 + 2, Figueroa 1995).
* ``f16_round_up`` round toward +inf to fp16.  The paper stores scales and
                   witnesses in fp16 but names no rounding mode; rounding up keeps
                   "amax/s <= 126.5" (no clipping, Sec. 4.2) and keeps the stored
                   witness an upper bound of the residual norm (Theorem black-box
                   logit bound needs w >= ||r_b||).
* ``f16_round_down`` round toward 0 to fp16, for the stored value norm, which the
                   value meter divides by (a lower bound keeps the meter an upper
                   bound).
* ``e4m3_*``       OCP fp8 E4M3 ("fn": no infinities, one NaN pattern), round to
                   nearest even, saturating at +-448 (the raw fp8 cast, a
                   black-box scheme of Sec. 4.1; saturation is our reading).
"""
from __future__ import annotations

import numpy as np


def f32(x) -> np.ndarray:
    """Nearest fp32 value (as float64) of float64 x."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def f16_round_up(x) -> np.ndarray:
    """Smallest fp16 value >= x (as float64); x must be finite and >= 0."""
    x = np.asarray(x, dtype=np.float64)
    h = x.astype(np.float16)                     # nearest even
    low = h.astype(np.float64) < x
    with np.errstate(over="ignore"):
        up = np.nextafter(h, np.float16(np.inf))
    h = np.where(low, up, h)
    return h.astype(np.float64)


def f16_round_down(x) -> np.ndarray:
    """Largest fp16 value <= x (as float64); x must be finite and >= 0 (values
    above 65504 give 65504)."""
    x = np.asarray(x, dtype=np.float64)
    h = np.minimum(x, 65504.0).astype(np.float16)   # nearest even
    high = h.astype(np.float64) > x
    down = np.nextafter(h, np.float16(0.0))
    h = np.where(high, down, h)
    return h.astype(np.float64)


def f16_bits(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def bf16_bits_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


E4M3_MAX = 448.0


def e4m3_round(x) -> np.ndarray:
    """Value of x after the raw cast to fp8 E4M3 (RNE, saturating), float64.

    Format: sign, 4 exponent bits (bias 7), 3 mantissa bits.  Normals are
    (1 + m/8) * 2^(e-7) for e = 1..15 (e=15, m=7 is NaN), so the largest finite
    value is 1.75 * 2^8 = 448; subnormals are m * 2^-9.  Rounding to nearest
    even is done on the magnitude with the quantum of its binade.
    """
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    e = np.maximum(e, -6.0)                       # subnormal binade shares 2^-6's quantum
    q = np.exp2(e - 3.0)                          # quantum: 3 mantissa bits
    r = np.rint(a / q) * q                        # exact scaling by a power of two, RNE
    r = np.minimum(r, E4M3_MAX)                   # saturate
    r = np.where(a >= E4M3_MAX, E4M3_MAX, r)
    return np.copysign(r, x)


def e4m3_encode(x) -> np.ndarray:
    """uint8 E4M3 bit patterns of e4m3_round(x) (sign kept, also for zero)."""
    v = e4m3_round(x)
    a = np.abs(v)
    sign = (np.signbit(v)).astype(np.uint8) << 7
    out = np.zeros(v.shape, dtype=np.uint8)
    sub = a < 2.0 ** -6
    m_sub = np.rint(a / 2.0 ** -9).astype(np.int64)              # 0..7
    with np.errstate(divide="ignore"):
        e = np.floor(np.log2(np.where(a > 0, a, 1.0))).astype(np.int64)
    m_nrm = np.rint((a / np.exp2(e) - 1.0) * 8.0).astype(np.int64)
    code_n = ((e + 7) << 3) | m_nrm
    out = np.where(sub, m_sub, code_n).astype(np.uint8)
    return out | sign


def e4m3_decode(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    s = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = b & 0x7
    val = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    val = np.where((e == 15) & (m == 7), np.nan, val)
    return s * val
