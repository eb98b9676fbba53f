"""Fine-grained FP8 quantization with power-of-two scales (oracle; test infrastructure only).

Paper section 3.1:
  * scale definition: a tile of 128 contiguous elements gets s = max|x_i| / 448;
  * quantize: Q(x_i) = round(x_i / s); dequantize: D(Q(x_i)) = round(x_i / s) * s;
  * power-of-two constraint: s = 2^T, so rescaling between layouts only touches
    exponent bits.

Reading of the two together (the paper gives s = amax/448 and then requires
s = 2^T without saying how to round): T is the smallest integer with
amax <= 448 * 2^T, i.e. s is amax/448 rounded up to a power of two, so no
element overflows.  T is an integer of either sign (the text says natural
number, but N(0,1) tiles need T near -7), clamped to [-126, 127] so that s is a
normal float32.  An all-zero tile gets T = -126 (smallest scale), so that a zero
tile never dominates a block maximum in the scaling-aware transpose.

Layouts:
  * row-wise 1x128: q [rows, cols] uint8, s [rows, cols/128] float32;
  * block 128x128 (weights): q [rows, cols] uint8, s [rows/128, cols/128] float32.
"""

import numpy as np

from .codec import e4m3_decode, e4m3_encode, E4M3_MAX

TILE = 128
T_MIN = -126
T_MAX = 127


def scale_exponent(amax):
    """Smallest integer T with amax <= 448 * 2^T, clamped to [-126, 127]; amax == 0 gives -126.

    A float estimate of ceil(log2(amax/448)) is corrected with exact comparisons
    against 448 * 2^T (ldexp is exact), so the result is the exact integer.
    """
    amax = np.asarray(amax, dtype=np.float64)
    pos = amax > 0
    safe = np.where(pos, amax, 1.0)
    t = np.ceil(np.log2(safe / E4M3_MAX)).astype(np.int64)
    for _ in range(2):
        t = np.where(safe > np.ldexp(E4M3_MAX, t), t + 1, t)
        t = np.where(safe <= np.ldexp(E4M3_MAX, t - 1), t - 1, t)
    t = np.where(pos, t, T_MIN)
    return np.clip(t, T_MIN, T_MAX)


def scale_from_exponent(t):
    """fp32 scale 2^T."""
    return np.ldexp(np.float32(1.0), np.asarray(t, dtype=np.int64)).astype(np.float32)


def scale_to_e8m0(s):
    """UE8M0 byte of power-of-two scales 2^T (section 2.1 names UE8M0 as the recipe's scale
    format; the power-of-two constraint of section 3.1 makes every scale one): T + 127."""
    return (exponent_of_scale(s) + 127).astype(np.uint8)


def e8m0_to_scale(b):
    """Value of UE8M0 bytes as float32: 2^(b - 127)."""
    return scale_from_exponent(np.asarray(b, dtype=np.int64) - 127)


def exponent_of_scale(s):
    """Exact integer log2 of power-of-two scales (raises if a scale is not a power of two)."""
    s = np.asarray(s, dtype=np.float64)
    m, e = np.frexp(s)
    if not np.all(m == 0.5):
        raise ValueError("scale is not a power of two")
    return (e - 1).astype(np.int64)


def quant_rowwise(x):
    """1x128 row-wise quantization of a [rows, cols] array (cols % 128 == 0).

    Per tile: amax over the exact values, T = scale_exponent(amax),
    q = encode(x * 2^-T) (exact scaling).  Returns (q uint8, s float32).
    """
    x = np.asarray(x, dtype=np.float64)
    rows, cols = x.shape
    assert cols % TILE == 0
    tiles = x.reshape(rows, cols // TILE, TILE)
    t = scale_exponent(np.abs(tiles).max(axis=2))
    q = e4m3_encode(tiles * np.ldexp(1.0, -t)[:, :, None]).reshape(rows, cols)
    return q, scale_from_exponent(t)


def quant_block128(w):
    """128x128 block quantization of a [rows, cols] array (both multiples of 128)."""
    w = np.asarray(w, dtype=np.float64)
    rows, cols = w.shape
    assert rows % TILE == 0 and cols % TILE == 0
    blocks = w.reshape(rows // TILE, TILE, cols // TILE, TILE)
    t = scale_exponent(np.abs(blocks).max(axis=(1, 3)))
    q = e4m3_encode(blocks * np.ldexp(1.0, -t)[:, None, :, None]).reshape(rows, cols)
    return q, scale_from_exponent(t)


def dequant_rowwise(q, s):
    """D(q) = q * s with 1x128 row-wise scales (exact in float64)."""
    q = np.asarray(q)
    rows, cols = q.shape
    v = e4m3_decode(q).reshape(rows, cols // TILE, TILE)
    return (v * np.asarray(s, dtype=np.float64)[:, :, None]).reshape(rows, cols)


def dequant_block128(q, s):
    """D(q) = q * s with 128x128 block scales (exact in float64)."""
    q = np.asarray(q)
    rows, cols = q.shape
    v = e4m3_decode(q).reshape(rows // TILE, TILE, cols // TILE, TILE)
    return (v * np.asarray(s, dtype=np.float64)[:, None, :, None]).reshape(rows, cols)
