"""Exact OCP FP8 E4M3FN codec (test infrastructure only).

Format: 1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; no
infinities; S.1111.111 is NaN, so the largest finite magnitude is
1.75 * 2^8 = 448 = R_max (Sec. 1, "Problem formulation").  Subnormals are
m * 2^-9, m = 1..7.  Rounding is to nearest, ties to even.

The paper's overflow criterion is |S| > s * R_max, i.e. |S / s| > 448.
Round-to-nearest would still map magnitudes in (448, 464] onto 448; the
predicate ``overflows`` follows the paper, ``encode`` the number format.
"""

from __future__ import annotations

import numpy as np

R_MAX = 448.0
NAN_CODE = 0x7F


def decode(codes) -> np.ndarray:
    c = np.asarray(codes, dtype=np.int64) & 0xFF
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = c & 0x7
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return sign * mag


def encode(x, saturate: bool = False) -> np.ndarray:
    """float64 -> uint8 code, round to nearest even.  Magnitudes above 464
    (the midpoint past 448) are NaN, or 448 with ``saturate``."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    sign = np.where(np.signbit(x), 0x80, 0x00)
    code = np.zeros(x.shape, dtype=np.int64)

    sub = a < 2.0 ** -6
    # subnormal range (and the first normal, reached by rounding up): code = m
    code = np.where(sub, np.rint(a / 2.0 ** -9).astype(np.int64), code)

    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.floor(np.log2(np.where(sub | ~np.isfinite(a), 1.0, a)))
    q = np.exp2(e - 3.0)
    m = np.rint(np.where(sub, 8.0, a) / q)             # 8..16
    bump = m >= 16.0
    e = np.where(bump, e + 1.0, e)
    m = np.where(bump, 8.0, m)
    normal_code = ((e + 7.0).astype(np.int64) << 3) | (m.astype(np.int64) - 8)
    code = np.where(sub, code, normal_code)

    over = a > 464.0
    code = np.where(~sub & (a > 448.0) & ~over, 0x7E, code)   # (448, 464] rounds to 448
    code = np.where(over, 0x7E if saturate else NAN_CODE, code)
    code = np.where(np.isnan(x), NAN_CODE, code)
    return (code | sign).astype(np.uint8)


def overflows(x, r_max: float = R_MAX) -> np.ndarray:
    """The paper's overflow predicate |x| > R_max for an already-scaled value.
    A value that is not finite (NaN, inf: e.g. logits scaled by a NaN or zero
    scale) is not representable either and counts as an overflow, the outcome
    the predicate exists to flag (Sec. 1: an overflow yields NaN or inf)."""
    return ~(np.abs(np.asarray(x, dtype=np.float64)) <= r_max)
