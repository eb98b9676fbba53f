"""Pins of the oracle's e4m3 codec and bf16 rounding (CPU only).

Independent references: hand-derived codes from the paper's E4M3 definition
(tests/golden), torch's float8_e4m3fn / bfloat16 conversions (library routines),
and brute-force nearest-value search over all codes.
"""

import os

import numpy as np
import pytest
import torch

from oracle.codec import e4m3_decode, e4m3_encode, bf16_round


def _torch_encode(v):
    t = torch.from_numpy(np.asarray(v, dtype=np.float32)).clamp(-448.0, 448.0)
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def _golden(golden_dir, name):
    rows = []
    with open(os.path.join(golden_dir, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def test_golden_anchor_codes(golden_dir):
    rows = _golden(golden_dir, "e4m3_anchors.txt")
    assert len(rows) >= 15
    for r in rows:
        v, code = float(r[0]), int(r[1], 16)
        assert int(e4m3_encode(np.array([v]))[0]) == code, r
        if code not in (0x80,) and abs(v) <= 448.0 and float(e4m3_decode(np.array([code]))[0]) == v:
            pass  # exactly representable anchors round-trip
    assert float(e4m3_decode(np.array([0x7E]))[0]) == 448.0
    assert float(e4m3_decode(np.array([0x01]))[0]) == 2.0 ** -9


def test_decode_all_codes_vs_torch():
    codes = np.arange(256, dtype=np.uint8)
    ours = e4m3_decode(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan)
    assert np.array_equal(ours[~nan], ref[~nan])
    assert np.array_equal(np.signbit(ours[~nan]), np.signbit(ref[~nan]))
    assert set(np.nonzero(nan)[0].tolist()) == {0x7F, 0xFF}


def _boundary_probes():
    mags = e4m3_decode(np.arange(127, dtype=np.uint8))
    mids = (mags[:-1] + mags[1:]) / 2.0
    pts = np.concatenate([mags, mids, [448.0, 456.0, 464.0, 480.0, 1e4, 2.0 ** -10, 2.0 ** -11]]).astype(np.float32)
    ups = np.nextafter(pts, np.float32(np.inf))
    downs = np.nextafter(pts, np.float32(0))
    allp = np.concatenate([pts, ups, downs])
    return np.concatenate([allp, -allp]).astype(np.float32)


def test_encode_vs_torch_all_bf16_patterns():
    bits = np.arange(65536, dtype=np.uint32) << 16
    v = bits.view(np.float32)
    v = v[np.isfinite(v)]
    assert np.array_equal(e4m3_encode(v), _torch_encode(v))


def test_encode_vs_torch_boundaries_and_random():
    v = _boundary_probes()
    assert np.array_equal(e4m3_encode(v), _torch_encode(v))
    rng = np.random.default_rng(123)
    bits = rng.integers(0, 2 ** 32, size=1 << 20, dtype=np.uint64).astype(np.uint32)
    r = bits.view(np.float32)
    r = r[np.isfinite(r)]
    assert np.array_equal(e4m3_encode(r), _torch_encode(r))
    # scaled-range values as produced by quantization: |v| <= 448
    s = rng.uniform(-448, 448, size=1 << 18).astype(np.float32)
    assert np.array_equal(e4m3_encode(s), _torch_encode(s))


def test_encode_brute_force_nearest_even():
    """Nearest finite code by exhaustive search; ties go to the even code (of the magnitude)."""
    rng = np.random.default_rng(7)
    v = np.concatenate([rng.standard_normal(3000) * 10, rng.standard_normal(2000) * 0.003,
                        _boundary_probes()[:1500]]).astype(np.float64)
    codes = np.arange(127)
    mags = e4m3_decode(codes.astype(np.uint8))
    for x in v:
        a = min(abs(x), 448.0)
        d = np.abs(mags - a)
        best = np.nonzero(d == d.min())[0]
        c = best[0] if len(best) == 1 else [b for b in best if b % 2 == 0][0]
        if np.signbit(x):
            c |= 0x80
        assert int(e4m3_encode(np.array([x]))[0]) == int(c), x


def test_encode_nan_and_sign():
    out = e4m3_encode(np.array([np.nan, -0.0, 0.0, -1e-300, 1e300, -1e300]))
    assert out.tolist() == [0x7F, 0x80, 0x00, 0x80, 0x7E, 0xFE]


def test_bf16_round_vs_torch():
    rng = np.random.default_rng(3)
    bits = rng.integers(0, 2 ** 32, size=1 << 18, dtype=np.uint64).astype(np.uint32)
    v = bits.view(np.float32)
    v = v[np.isfinite(v) & (np.abs(v) < 1e38)]
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_round(v.astype(np.float64)), ref)


def test_bf16_round_brute_force_float64():
    """float64 inputs (not float32-representable) round directly, not via float32."""
    rng = np.random.default_rng(5)
    v = rng.standard_normal(2000) * 3.0
    out = bf16_round(v)
    for x, y in zip(v, out):
        m, e = np.frexp(x)
        ulp = 2.0 ** (e - 1 - 7)
        lo = np.floor(x / ulp) * ulp
        hi = lo + ulp
        if x - lo < hi - x:
            want = lo
        elif x - lo > hi - x:
            want = hi
        else:
            want = lo if int(round(lo / ulp)) % 2 == 0 else hi
        assert y == want
    # a float64 value just above a bf16 midpoint must round up (double rounding through float32 would not)
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert bf16_round(np.array([x]))[0] == 1.0 + 2.0 ** -7
