"""Pins of the oracle's scaling-aware transpose (CPU only).

Independent references: hand-worked elements (tests/golden), the exponent-shift
identity of section 3.1 done on the bit fields, integer round-to-nearest-even on
the subnormal grid for underflow, re-quantization of the exact dequantized
values at the forced block scale, and brute force on tiny tensors.
"""

import os

import numpy as np
import torch

from oracle.codec import e4m3_decode
from oracle.quant import quant_rowwise, dequant_rowwise, exponent_of_scale
from oracle.sat import scaling_aware_transpose, requant_forced_scale, naive_pow2, naive_fp32


def _one_element_sat(byte, k):
    """Run the oracle transpose on a 128x128 block whose row 0 holds `byte` at scale 2^-k and row 1 sets S_max = 1."""
    q = np.zeros((128, 128), dtype=np.uint8)
    s = np.full((128, 1), np.float32(2.0 ** -126), dtype=np.float32)
    q[0, 0] = byte
    s[0, 0] = np.float32(2.0 ** -k) if k < 126 else s[0, 0]
    q[1, 0] = 0x38
    s[1, 0] = np.float32(1.0)
    qT, sT = scaling_aware_transpose(q, s)
    assert sT[0, 0] == 1.0
    return int(qT[0, 0])


def test_golden_hand_worked_elements(golden_dir):
    with open(os.path.join(golden_dir, "sat_exponent_shift.txt")) as f:
        rows = [l.split("#", 1)[0].split() for l in f]
    rows = [r for r in rows if r]
    assert len(rows) >= 15
    for r in rows:
        b, k, want = r[:3]
        assert _one_element_sat(int(b, 16), int(k)) == int(want, 16), (b, k)


def _integer_reference(byte, k):
    """Exponent-shift identity on the bit fields; integer RNE on the 2^-9 grid when the exponent underflows."""
    sign, e, m = byte & 0x80, (byte >> 3) & 0xF, byte & 7
    if e - k >= 1:
        return sign | ((e - k) << 3) | m
    units = (8 + m) << (e - 1) if e >= 1 else m       # value in units of 2^-9
    q, r = divmod(units, 1 << k)
    half = 1 << (k - 1) if k >= 1 else 0
    if k >= 1 and (r > half or (r == half and q % 2 == 1)):
        q += 1
    return sign | q                                   # q <= 8 and code 0x08 is 2^-6


def test_exhaustive_byte_k_table():
    n_underflow = 0
    for b in range(256):
        if (b & 0x7F) == 0x7F:
            continue
        for k in range(0, 17):
            want = _integer_reference(b, k)
            assert _one_element_sat(b, k) == want, (hex(b), k)
            n_underflow += ((b >> 3) & 0xF) - k < 1
    assert n_underflow > 2000


def _row_scaled_tensor(rows, cols, seed, kmax=12):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((rows, cols))
    x *= np.ldexp(1.0, rng.integers(-kmax, 1, size=(rows, 1)))   # per-row magnitudes spanning k = 0..kmax
    x[3, :] = 0.0                                                 # zero row (scale 2^-126)
    x = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    return x


def test_transpose_matches_forced_scale_requant_and_values():
    x = _row_scaled_tensor(256, 384, 0)
    q, s = quant_rowwise(x)
    qT, sT = scaling_aware_transpose(q, s)
    assert qT.shape == (384, 256) and sT.shape == (384, 2)
    d = dequant_rowwise(q, s)                                      # D(Q_row X), exact
    t_max = np.zeros((384, 256), dtype=np.int64)
    for b in range(2):
        for c in range(3):
            tm = exponent_of_scale(s[b * 128:(b + 1) * 128, c]).max()
            assert np.all(sT[c * 128:(c + 1) * 128, b] == np.float32(2.0 ** tm))
            t_max[c * 128:(c + 1) * 128, b * 128:(b + 1) * 128] = tm
    # bit-identical to re-quantizing the exact values at the forced scale S_max
    assert np.array_equal(qT, requant_forced_scale(d.T, t_max))
    # value-exact wherever the lowered exponent stays normal (no underflow)
    dT = e4m3_decode(qT) * np.ldexp(1.0, t_max)
    k = t_max.T - np.repeat(exponent_of_scale(s), 128, axis=1)
    e = (q.astype(np.int64) >> 3) & 0xF
    exact = (e - k >= 1) | ((q & 0x7F) == 0)
    assert exact.mean() > 0.5
    assert np.array_equal(dT.T[exact], d[exact])
    # underflowed elements stay within half a subnormal step of the exact value
    err = np.abs(dT.T - d)[~exact] / np.ldexp(1.0, t_max.T[~exact])
    assert np.all(err <= 2.0 ** -10)


def test_partial_rows_and_k_zero_blocks():
    x = _row_scaled_tensor(384, 128, 1, kmax=0)
    x[:, :] = np.abs(x) + 1.0    # every row amax in [1, ...): rows share scales often
    q, s = quant_rowwise(x)
    qT, sT = scaling_aware_transpose(q, s, n_rows=256)
    assert qT.shape == (128, 256) and sT.shape == (128, 2)
    same = (exponent_of_scale(s[:256]) == exponent_of_scale(s[:256]).max())[:, 0]
    assert np.array_equal(qT.T[same], q[:256][same])   # k = 0 rows keep their bytes


def test_double_quantization_error_ordering():
    """Section 3.1: dequant->transpose->requant with fp32 scales adds error of the order of a
    quantization step; the scaling-aware transpose adds (almost) none."""
    rng = np.random.default_rng(9)
    x = torch.from_numpy(rng.standard_normal((512, 512))).to(torch.bfloat16).to(torch.float64).numpy()
    q, s = quant_rowwise(x)
    d = dequant_rowwise(q, s)
    qT, sT = scaling_aware_transpose(q, s)
    sat_err = np.linalg.norm(dequant_rowwise(qT, sT).T - d) / np.linalg.norm(d)
    q1, s1, q2, s2 = naive_fp32(x)
    d1 = dequant_rowwise(q1, s1)
    n2_err = np.linalg.norm(dequant_rowwise(q2, s2).T - d1) / np.linalg.norm(d1)
    qn, sn = naive_pow2(q, s)
    n1_err = np.linalg.norm(dequant_rowwise(qn, sn).T - d) / np.linalg.norm(d)
    assert sat_err < 1e-5 and n1_err < 1e-5
    assert n2_err > 1e-2
    assert n2_err > 1000 * sat_err


def test_partial_last_block_equals_zero_padding():
    """A last block with fewer than 128 rows (groups padded to 16) transposes as if the missing
    rows were all-zero rows at scale 2^-126, which never raise S_max."""
    rng = np.random.default_rng(31)
    x = rng.standard_normal((176, 256)) * np.exp2(rng.integers(-6, 6, size=(176, 1)))
    q, s = quant_rowwise(x)
    qT, sT = scaling_aware_transpose(q, s, 176)
    assert qT.shape == (256, 176) and sT.shape == (256, 2)
    qp = np.concatenate([q, np.zeros((80, 256), dtype=np.uint8)])
    sp = np.concatenate([s, np.full((80, 2), np.float32(2.0 ** -126))])
    qT2, sT2 = scaling_aware_transpose(qp, sp)
    assert np.array_equal(qT, qT2[:, :176]) and np.array_equal(sT, sT2)
    # the partial block's scale is the max over its 48 rows only
    assert np.array_equal(exponent_of_scale(sT[::128, 1]), exponent_of_scale(s[128:176]).max(axis=0))
