"""Parity of every HIP kernel against the CPU oracle on the same seeded inputs (GPU).

Bars: e4m3 bytes, scales, routing maps and offsets bit-exact; GEMM outputs within
2e-3 relative Frobenius of the float64 oracle; SwiGLU outputs per the reading that
both sides quantize the same activation (bytes may differ by one code only where
the exact value sits at a rounding midpoint, scales only at power-of-two edges).
"""

import numpy as np
import pytest
import torch

import workloads
from oracle import codec, quant, sat, moe
from layouts import from_kblock, to_kblock
from paper_2511_02302_amd import ff8

pytestmark = pytest.mark.gpu

POISON = 0xA5


def dev(t):
    return t.contiguous().cuda()


def host(t):
    return t.detach().cpu().numpy()


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_frob(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def poisoned(shape, dtype):
    t = torch.empty(shape, dtype=dtype, device="cuda")
    t.view(torch.uint8).fill_(POISON)
    return t


def untouched(t):
    return bool((t.view(torch.uint8) == POISON).all())


# ---------------------------------------------------------------- codec

def test_cast_f32_to_e4m3_rounding_classes():
    """Every rounding class: all upper-16-bit patterns x low-16-bit patterns
    {0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF} (the e4m3 round and sticky bits live above bit 16)."""
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    bits = (hi[:, None] | lows[None, :]).ravel()
    x = bits.view(np.float32)
    q = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    ff8.ff8_cast_f32_to_e4m3(dev(torch.from_numpy(x)), q)
    torch.cuda.synchronize()
    want = codec.e4m3_encode(x.astype(np.float64))
    got = host(q)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(bits[i])), float(x[i]), hex(got[i]), hex(want[i])) for i in bad[:10]]


def test_cast_e4m3_to_f32_all_codes():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    out = torch.empty(256, dtype=torch.float32, device="cuda")
    ff8.ff8_cast_e4m3_to_f32(dev(codes), out)
    got = host(out).astype(np.float64)
    want = codec.e4m3_decode(np.arange(256, dtype=np.uint8))
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], want[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(want[~nan]))


# ---------------------------------------------------------------- quantization

def _special_rows(x):
    x = x.clone()
    x[0, :128] = 0.0
    x[1, 128:256] *= 1e-30
    x[2, :] = -x[2, :].abs()
    x[3, 5] = 448.0
    x[4, 0] = -0.0
    return x


@pytest.mark.parametrize("rows,cols", [(1, 128), (37, 384), (300, 1024)])
def test_quant_rowwise_bit_exact(rows, cols):
    x = workloads.outlier_activation(rows, cols, seed=rows)
    if rows >= 5:
        x = _special_rows(x)
    q = poisoned((rows + 1, cols), torch.uint8)
    s = poisoned((rows + 1, cols // 128), torch.float32)
    ff8.ff8_quant_rowwise(dev(x), q[:rows], s[:rows])
    torch.cuda.synchronize()
    wq, ws = quant.quant_rowwise(f64(x))
    assert np.array_equal(host(q[:rows]), wq)
    assert np.array_equal(host(s[:rows]), ws)
    assert untouched(q[rows:]) and untouched(s[rows:])


def test_quant_rowwise_full_size_sampled():
    rows, cols = workloads.CAST_X
    x = workloads.outlier_activation(rows, cols, seed=0, device="cuda")
    q = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows, cols // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_rowwise(x, q, s)
    torch.cuda.synchronize()
    idx = torch.from_numpy(np.random.default_rng(0).choice(rows, 96, replace=False)).cuda()
    wq, ws = quant.quant_rowwise(f64(x[idx]))
    assert np.array_equal(host(q[idx]), wq)
    assert np.array_equal(host(s[idx]), ws)


@pytest.mark.parametrize("rows,cols", [(128, 128), (256, 384), (2048, 7168)])
def test_quant_block128_bit_exact(rows, cols):
    w = workloads.randn_bf16((rows, cols), 0.02, seed=cols)
    w[:128, :128] = 0
    q = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows // 128, cols // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_block128(dev(w), q, s)
    torch.cuda.synchronize()
    wq, ws = quant.quant_block128(f64(w))
    assert np.array_equal(host(q), wq)
    assert np.array_equal(host(s), ws)


# ---------------------------------------------------------------- scaling-aware transpose

def _row_scaled_fp8(rows, cols, seed, kmax=12):
    g = torch.Generator().manual_seed(seed)
    x = torch.randn((rows, cols), generator=g)
    x *= torch.pow(2.0, -torch.randint(0, kmax + 1, (rows, 1), generator=g).float())
    x[3] = 0.0
    x = x.to(torch.bfloat16)
    q, s = quant.quant_rowwise(f64(x))
    return q, s


@pytest.mark.parametrize("rows,cols,n_rows", [(128, 128, 128), (640, 384, 640), (1024, 256, 512), (896, 128, 384),
                                         (16384, 256, 12800), (384, 256, 272)])  # odd block count; 16-row end
def test_sat_bit_exact(rows, cols, n_rows):
    q, s = _row_scaled_fp8(rows, cols, seed=rows + cols)
    qT = poisoned((rows // 128, cols, 128), torch.uint8)  # K-blocked transpose
    sT = poisoned((rows // 128, cols), torch.float32)
    offsets = None
    if n_rows != rows:
        offsets = dev(torch.tensor([0, n_rows // 2, n_rows], dtype=torch.int32))
    ff8.ff8_scaling_aware_transpose(dev(torch.from_numpy(q)), dev(torch.from_numpy(s)), qT, sT, offsets,
                                    2 if offsets is not None else 0)
    torch.cuda.synchronize()
    wqT, wsT = sat.scaling_aware_transpose(q, s, n_rows)
    nb = -(-n_rows // 128)
    assert np.array_equal(from_kblock(host(qT))[:, :n_rows], wqT)
    assert np.array_equal(host(sT[:nb]).T, wsT)  # block-major on the device
    assert untouched(qT[nb:]) and untouched(sT[nb:])
    if n_rows % 128:  # the rows of the last slab past the active rows stay untouched
        assert untouched(qT[nb - 1, :, n_rows % 128:].contiguous())


@pytest.mark.parametrize("fmt,n_rows,n", [("f32", 1024, 4), ("f32", 912, 4), ("e8m0", 1024, 4), ("e8m0", 912, 4),
                                          ("f32", 912, 1), ("f32", 912, 3), ("f32", None, 2)])
def test_sat_batch_bit_exact(fmt, n_rows, n):
    """One launch over up to four tensors of one row count (7, 1, 5 and 2 column tiles: odd and
    even tile counts, a single tile) writes, for each, the oracle's transpose and block scales,
    and nothing past the active rows (912: a last block cut after 16 of its rows; None: no
    offsets, every row)."""
    rows, cols_list = 1024, [896, 128, 640, 256][:n]
    qs, ss, want, qTs, sTs = [], [], [], [], []
    n_active = rows if n_rows is None else n_rows
    for i, cols in enumerate(cols_list):
        q, s = _row_scaled_fp8(rows, cols, seed=40 + i, kmax=20 + 10 * i)
        want.append(sat.scaling_aware_transpose(q, s, n_active))
        qs.append(dev(torch.from_numpy(q)))
        ss.append(dev(torch.from_numpy(s if fmt == "f32" else quant.scale_to_e8m0(s))))
        qTs.append(poisoned((rows // 128, cols, 128), torch.uint8))
        sTs.append(poisoned((rows // 128, cols), torch.float32 if fmt == "f32" else torch.uint8))
    offsets = None if n_rows is None else dev(torch.tensor([0, 400, n_rows], dtype=torch.int32))
    ff8.ff8_scaling_aware_transpose_batch(qs, ss, qTs, sTs, offsets, 0 if offsets is None else 2)
    torch.cuda.synchronize()
    nb = -(-n_active // 128)
    for i, (wqT, wsT) in enumerate(want):
        assert np.array_equal(from_kblock(host(qTs[i]))[:, :n_active], wqT), i
        ws = wsT.T if fmt == "f32" else quant.scale_to_e8m0(wsT.T)
        assert np.array_equal(host(sTs[i][:nb]), ws), i
        assert untouched(qTs[i][nb:]) and untouched(sTs[i][nb:]), i
        if n_active % 128:
            assert untouched(qTs[i][nb - 1, :, n_active % 128:].contiguous()), i


def test_sat_extreme_row_range():
    """Rows of one block whose scales differ by up to 2^139: shifts of 18, 19 and >= 128
    (underflow to the nearest subnormal, to signed zero, and far beyond the float range of
    2^-k) must all match the oracle's exact enc(dec(b) * 2^-k)."""
    g = torch.Generator().manual_seed(7)
    x = torch.randn((256, 256), generator=g)
    octaves = [20, -118, 2, 1, 0, -50, -100, 12, -126, 20 - 17, 20 - 18]
    for r, o in enumerate(octaves):
        x[r] *= 2.0 ** o
        x[128 + r] *= -(2.0 ** o)
    x = x.to(torch.bfloat16)
    q, s = quant.quant_rowwise(f64(x))
    qT = poisoned((2, 256, 128), torch.uint8)
    sT = poisoned((2, 256), torch.float32)
    ff8.ff8_scaling_aware_transpose(dev(torch.from_numpy(q)), dev(torch.from_numpy(s)), qT, sT)
    torch.cuda.synchronize()
    wqT, wsT = sat.scaling_aware_transpose(q, s)
    assert np.array_equal(from_kblock(host(qT)), wqT)
    assert np.array_equal(host(sT).T, wsT)


def test_sat_full_size_sampled_blocks():
    rows, cols = workloads.CAST_X
    x = workloads.outlier_activation(rows, cols, seed=0, device="cuda")
    q = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows, cols // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_rowwise(x, q, s)
    qT = torch.empty((rows // 128, cols, 128), dtype=torch.uint8, device="cuda")
    sT = torch.empty((rows // 128, cols), dtype=torch.float32, device="cuda")
    ff8.ff8_scaling_aware_transpose(q, s, qT, sT)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    for _ in range(24):
        rb, cb = int(rng.integers(rows // 128)), int(rng.integers(cols // 128))
        qb = host(q[rb * 128:(rb + 1) * 128, cb * 128:(cb + 1) * 128])
        sb = host(s[rb * 128:(rb + 1) * 128, cb:cb + 1])
        wqT, wsT = sat.scaling_aware_transpose(qb, sb)
        assert np.array_equal(host(qT[rb, cb * 128:(cb + 1) * 128]), wqT)  # the block's slab rows
        assert np.array_equal(host(sT[rb:rb + 1, cb * 128:(cb + 1) * 128]).T, wsT)


def test_naive_baseline_chain_matches_oracle():
    """dequantize -> bf16 transpose -> 1x128 requantize (the naive conversion) on the GPU."""
    rows, cols = 512, 384
    x = workloads.outlier_activation(rows, cols, seed=3)
    q = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows, cols // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_rowwise(dev(x), q, s)
    d = torch.empty((rows, cols), dtype=torch.bfloat16, device="cuda")
    ff8.ff8_baseline_dequant_rowwise(q, s, d)
    dT = torch.empty((cols, rows), dtype=torch.bfloat16, device="cuda")
    ff8.ff8_baseline_transpose_bf16(d, dT)
    qn = torch.empty((cols, rows), dtype=torch.uint8, device="cuda")
    sn = torch.empty((cols, rows // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_rowwise(dT, qn, sn)
    torch.cuda.synchronize()
    assert np.array_equal(f64(d), quant.dequant_rowwise(host(q), host(s)))
    wq, ws = sat.naive_pow2(host(q), host(s))
    assert np.array_equal(host(qn), wq) and np.array_equal(host(sn), ws)


def test_copy_probe():
    a = torch.randint(0, 255, (1 << 20,), dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    ff8.ff8_baseline_copy(a, b)
    assert torch.equal(a, b)
