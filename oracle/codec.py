"""OCP FP8 E4M3 codec and bfloat16 rounding (oracle; test infrastructure only).

E4M3 byte layout (paper section 3.1, the FP8 encoding of a row-wise quantized
value): sign bit SN (bit 7), exponent E (bits 6..3, bias 7), mantissa M (bits
2..0).  A normal code (E >= 1) has the value (-1)^SN * 2^(E-7) * (1 + M/8); the
largest finite magnitude is 448 (section 3.1, scale definition).  The paper does
not spell out the rest of the OCP E4M3FN format; this oracle follows it:
E = 0 codes are subnormals (-1)^SN * M * 2^-9, codes 0x7F and 0xFF are NaN, there
is no infinity.

Encoding (paper section 3.1: "round", a deterministic round-to-nearest) is read
as round-to-nearest-even onto the 127 finite non-negative magnitudes, saturating
at 448, with the sign bit kept (so -0.0 and tiny negatives encode to 0x80) and
NaN encoded as 0x7F.
"""

import numpy as np

E4M3_MAX = 448.0


def e4m3_decode(b):
    """Decode e4m3 bytes to float64 values (NaN for 0x7F/0xFF)."""
    b = np.asarray(b, dtype=np.uint8).astype(np.int64)
    sign = (b >> 7) & 1
    e = (b >> 3) & 0xF
    m = b & 0x7
    normal = np.ldexp(1.0 + m / 8.0, e - 7)
    subnormal = np.ldexp(m.astype(np.float64), -9)
    mag = np.where(e == 0, subnormal, normal)
    mag = np.where((b & 0x7F) == 0x7F, np.nan, mag)
    return np.where(sign == 1, -mag, mag)


# Magnitudes of codes 0x00..0x7E, strictly increasing with the code.
_MAGNITUDES = e4m3_decode(np.arange(127, dtype=np.uint8))


def e4m3_encode(v):
    """Saturating round-to-nearest-even encode of float values to e4m3 bytes.

    For a = min(|v|, 448): take the two neighbouring finite magnitudes
    lo <= a <= hi; choose the nearer one, and on an exact tie the one with the
    even code.  Comparisons are against the exact midpoint (lo + hi) / 2, which
    float64 represents exactly.
    """
    v = np.asarray(v, dtype=np.float64)
    a = np.minimum(np.abs(v), E4M3_MAX)
    nan = np.isnan(v)
    a = np.where(nan, 0.0, a)
    hi = np.searchsorted(_MAGNITUDES, a, side="left")  # _MAGNITUDES[hi] >= a
    hi = np.clip(hi, 0, 126)
    lo = np.maximum(hi - 1, 0)
    mid = (_MAGNITUDES[lo] + _MAGNITUDES[hi]) / 2.0
    exact_hi = _MAGNITUDES[hi] == a
    take_hi = exact_hi | (a > mid) | ((a == mid) & (hi % 2 == 0))
    code = np.where(take_hi, hi, lo).astype(np.int64)
    code = np.where(np.signbit(v), code | 0x80, code)
    code = np.where(nan, 0x7F, code)
    return code.astype(np.uint8)


def bf16_round(v):
    """Round float64 values to the nearest bfloat16 value (ties to even).

    bfloat16 keeps 8 significant bits and the float32 exponent range; values
    below 2^-126 use the subnormal spacing 2^-133.  Returned as float64 values
    that are exactly representable in bfloat16.  Overflow is not handled (the
    oracle never produces values near 2^128).
    """
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros_like(v)
    nz = v != 0
    _, e = np.frexp(v[nz])  # |v| in [2^(e-1), 2^e)
    ulp_exp = np.maximum(e - 1, -126) - 7
    out[nz] = np.ldexp(np.rint(np.ldexp(v[nz], -ulp_exp)), ulp_exp)
    out = np.where(np.signbit(v) & (out == 0), -0.0, out)
    return out


def bf16_bits(v):
    """Bit patterns (uint16) of float64 values that are exactly bfloat16."""
    f32 = np.asarray(v, dtype=np.float64).astype(np.float32)
    return (f32.view(np.uint32) >> 16).astype(np.uint16)
