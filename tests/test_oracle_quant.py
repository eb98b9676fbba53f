"""Pins of the oracle's power-of-two scale rule and 1x128 / 128x128 quantization (CPU only).

Independent references: brute-force search for the scale exponent, the
per-element rounding bound of e4m3, the idempotence argument of section 3.1
(re-quantizing with the same tiles leaves the values unchanged), and torch's
e4m3 cast for the element encoding.
"""

import math

import numpy as np
import torch

from oracle.codec import e4m3_decode
from oracle.quant import (scale_exponent, quant_rowwise, quant_block128, dequant_rowwise,
                          dequant_block128, exponent_of_scale)


def test_scale_exponent_brute_force_all_bf16():
    bits = (np.arange(1, 0x7F80, dtype=np.uint32) << 16)  # all positive finite bf16 patterns
    amax = bits.view(np.float32).astype(np.float64)
    got = scale_exponent(amax)
    ts = np.arange(-126, 128)
    ok = amax[:, None] <= 448.0 * np.power(2.0, ts)[None, :]
    first = np.where(ok.any(axis=1), ts[np.argmax(ok, axis=1)], 127)
    assert np.array_equal(got, first)
    assert scale_exponent(np.array([0.0]))[0] == -126


def test_scale_exponent_boundaries():
    for t in range(-120, 120, 7):
        edge = 448.0 * 2.0 ** t
        assert scale_exponent(np.array([edge]))[0] == t
        assert scale_exponent(np.array([np.nextafter(edge, np.inf)]))[0] == t + 1
        assert scale_exponent(np.array([np.nextafter(edge, 0)]))[0] == t


def _rand_tiles(rows, cols, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((rows, cols))
    x[rng.random((rows, cols)) < 0.01] *= 100.0
    x[0, :128] = 0.0                      # an all-zero tile
    x[1, 128:256] *= 1e-30                # a tiny tile
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()


def test_rowwise_round_trip_bound_and_amax_range():
    x = _rand_tiles(64, 512, 0)
    q, s = quant_rowwise(x)
    assert q.dtype == np.uint8 and s.dtype == np.float32 and s.shape == (64, 4)
    d = dequant_rowwise(q, s)
    sc = np.repeat(s.astype(np.float64), 128, axis=1)
    y = np.abs(x) / sc                                 # scaled magnitude, <= 448
    assert np.all(y <= 448.0)
    # half an e4m3 ulp: normal range 2^(e-4) for y in [2^e, 2^(e+1)), subnormal 2^-10
    e = np.floor(np.log2(np.maximum(y, 2.0 ** -6)))
    half_ulp = np.where(y >= 2.0 ** -6, 2.0 ** (e - 4), 2.0 ** -10) * sc
    assert np.all(np.abs(d - x) <= half_ulp)
    t = exponent_of_scale(s)
    amax = np.abs(x).reshape(64, 4, 128).max(axis=2)
    nz = amax > 0
    r = amax[nz] / np.ldexp(1.0, t[nz])
    assert np.all((r > 224.0) | (t[nz] == -126)) and np.all(r <= 448.0)
    assert s[0, 0] == np.float32(2.0 ** -126) and np.all(q[0, :128] == 0)


def test_rowwise_encoding_matches_torch_cast_of_scaled_values():
    x = _rand_tiles(32, 256, 1)
    q, s = quant_rowwise(x)
    scaled = (x / np.repeat(s.astype(np.float64), 128, axis=1)).astype(np.float32)
    ref = torch.from_numpy(scaled).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(q, ref)


def test_value_idempotence_and_byte_band():
    """Section 3.1: Q_row(D(Q_row(x))) has the same values as Q_row(x).

    Bytes also repeat except for tiles whose amax/s lies in (224, 232]: such a tile
    rounds its maximum to 224 (232 is the midpoint of 224 and 240 and ties to the even
    code of 224), so the second pass halves s and every exponent moves by one.
    """
    x = _rand_tiles(256, 1024, 2)
    q1, s1 = quant_rowwise(x)
    d1 = dequant_rowwise(q1, s1)
    q2, s2 = quant_rowwise(d1)
    assert np.array_equal(dequant_rowwise(q2, s2), d1)
    amax = np.abs(x).reshape(256, 8, 128).max(axis=2) / s1
    band = (amax > 224.0) & (amax <= 232.0)
    same = np.all(q1.reshape(256, 8, 128) == q2.reshape(256, 8, 128), axis=2)
    assert np.array_equal(same, ~band)
    # a constructed tile in the band
    t = np.zeros((1, 128))
    t[0, 0] = 228.0 * 2.0 ** -5
    t[0, 1:] = 0.3 * 2.0 ** -5
    qa, sa = quant_rowwise(t)
    qb, sb = quant_rowwise(dequant_rowwise(qa, sa))
    assert sb[0, 0] == sa[0, 0] / 2 and not np.array_equal(qa, qb)
    assert np.array_equal(dequant_rowwise(qa, sa), dequant_rowwise(qb, sb))


def test_block128_brute_force():
    rng = np.random.default_rng(4)
    w = torch.from_numpy(rng.standard_normal((256, 384)) * 0.02).to(torch.bfloat16).to(torch.float64).numpy()
    q, s = quant_block128(w)
    assert s.shape == (2, 3)
    mags = e4m3_decode(np.arange(127, dtype=np.uint8))
    for bi in range(2):
        for bj in range(3):
            blk = w[bi * 128:(bi + 1) * 128, bj * 128:(bj + 1) * 128]
            amax = np.abs(blk).max()
            t = next(t for t in range(-126, 128) if amax <= 448.0 * 2.0 ** t)
            assert s[bi, bj] == np.float32(2.0 ** t)
            # spot-check elements by nearest-magnitude search
            for (i, j) in [(0, 0), (5, 77), (127, 127), (64, 3)]:
                v = blk[i, j] / 2.0 ** t
                d = np.abs(mags - abs(v))
                c = np.nonzero(d == d.min())[0]
                c = c[0] if len(c) == 1 else [x for x in c if x % 2 == 0][0]
                c = c | (0x80 if v < 0 else 0)
                assert q[bi * 128 + i, bj * 128 + j] == c
    d = dequant_block128(q, s)
    assert np.max(np.abs(d - w) / np.repeat(np.repeat(s, 128, 0), 128, 1)) <= 16.0  # half ulp at 448 is 16


def test_e8m0_scale_bytes():
    """UE8M0 storage of the power-of-two scales: for every T in [-126, 127] the byte is T + 127,
    which is the exponent field of the float32 scale (IEEE 754 binary32, bias 127), and the byte
    decodes back to exactly 2^T; the scales a quantizer produces are always bytes 1..254 (never
    0, and never 255, the format's NaN)."""
    from oracle.quant import scale_to_e8m0, e8m0_to_scale, quant_rowwise

    T = np.arange(-126, 128)
    s = np.array([2.0 ** int(t) for t in T], dtype=np.float32)  # exact powers of two
    b = scale_to_e8m0(s)
    assert b.dtype == np.uint8 and np.array_equal(b.astype(np.int64), T + 127)
    assert np.array_equal(b.astype(np.uint32), s.view(np.uint32) >> 23)      # the exponent field
    assert np.array_equal(s.view(np.uint32) & 0x7FFFFF, np.zeros_like(T))    # no mantissa bits
    assert np.array_equal(e8m0_to_scale(b), s)
    for t, v in zip(T, e8m0_to_scale(b)):
        assert float(v) == math.ldexp(1.0, int(t))
    rng = np.random.default_rng(3)
    x = rng.standard_normal((64, 512)) * np.exp2(rng.integers(-120, 120, size=(64, 1)))
    x[0] = 0.0  # all-zero tiles: T = -126, byte 1
    _, sx = quant_rowwise(x)
    bx = scale_to_e8m0(sx)
    assert bx.min() >= 1 and bx.max() <= 254 and np.all(bx[0] == 1)
    assert np.array_equal(e8m0_to_scale(bx), sx)
