"""The grouped GEMMs and the scaling-aware transpose at their largest operands (GPU).

The GEMM kernels address every operand with 32-bit byte offsets, and the host accepts an
operand up to just under 4 GiB.  Here each large operand is 599040 x 7168 e4m3 bytes
(4 293 918 720 < 2^32), the last expert holds almost all rows, so that its tiles read the
highest offsets, and sampled outputs -- among them the rows where the byte offset passes
2^31 and the very last rows -- are checked against the oracle's definitions.  The
operands are random e4m3 codes (every finite code) with random power-of-two scales.
"""

import numpy as np
import pytest
import torch

from oracle import codec, quant, sat
from paper_2511_02302_amd import ff8

from test_gpu_kernels import host
from test_gpu_fullsize import _check_gemm_samples, _dequant_weight, _kblock_rows

pytestmark = pytest.mark.gpu

K_BIG = 7168
M_MAX = ((1 << 32) - 1) // K_BIG // 128 * 128   # 599040 rows
N_SMALL = 256
OFFSETS = [0, 2048, 4096, M_MAX]                 # three experts, the last with 594944 rows
E = len(OFFSETS) - 1


def _rand_e4m3(shape, gen):
    """Uniform over the 254 finite e4m3 codes (0x7F and 0xFF, the NaNs, skipped)."""
    v = torch.randint(0, 254, shape, dtype=torch.uint8, device="cuda", generator=gen)
    return v.add_((v >= 127).to(torch.uint8))


def _rand_pow2(shape, lo, hi, gen):
    e = torch.randint(lo, hi, shape, dtype=torch.int32, device="cuda", generator=gen)
    return torch.exp2(e.float())


def _offsets():
    return torch.tensor(OFFSETS, dtype=torch.int32, device="cuda")


def _sample_rows(rng, n):
    """Rows of every expert: the first and last of each, those around the 2^31-byte mark
    of a 7168-byte row stride, the last rows of the operand, and random rows."""
    mark = (1 << 31) // K_BIG
    fixed = [0, 2047, 2048, 4095, 4096, mark - 1, mark, mark + 1, M_MAX - 129, M_MAX - 128, M_MAX - 2, M_MAX - 1]
    m = np.unique(np.concatenate([fixed, rng.integers(M_MAX, size=n - len(fixed))]))
    return m, np.searchsorted(np.array(OFFSETS), m, side="right") - 1


def _idx(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int64)).cuda()


@pytest.fixture
def gen():
    yield torch.Generator(device="cuda").manual_seed(2024)
    torch.cuda.empty_cache()


def test_fprop_largest_activation_operand(gen):
    a = _rand_e4m3((M_MAX, K_BIG), gen)
    a_s = _rand_pow2((M_MAX, K_BIG // 128), -6, 3, gen)
    w = _rand_e4m3((E, N_SMALL, K_BIG), gen)
    w_s = _rand_pow2((E, N_SMALL // 128, K_BIG // 128), -10, -6, gen)
    out = torch.empty((M_MAX, N_SMALL), dtype=torch.bfloat16, device="cuda")
    print(f"\nfprop M_cap {M_MAX} N {N_SMALL} K {K_BIG} offsets {OFFSETS}", flush=True)
    ff8.ff8_grouped_gemm_fprop(a, a_s, w, w_s, _offsets(), out)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    m, e = _sample_rows(rng, 256)
    n = rng.integers(N_SMALL, size=m.size)
    x = quant.dequant_rowwise(host(a.index_select(0, _idx(m))), host(a_s.index_select(0, _idx(m))))
    wt = _dequant_weight(host(w[_idx(e), _idx(n)]), host(w_s[_idx(e), _idx(n // 128)]))
    got = host(out[_idx(m), _idx(n)].float())
    _check_gemm_samples(got, np.sum(x * wt, axis=1), np.sum(np.abs(x * wt), axis=1), True, K_BIG)


def test_dgrad_largest_gradient_operand(gen):
    g = _rand_e4m3((M_MAX, K_BIG), gen)                       # contraction over 7168
    g_s = _rand_pow2((M_MAX, K_BIG // 128), -6, 3, gen)
    w = _rand_e4m3((E, K_BIG, N_SMALL), gen)                  # W_e [N = 7168][K = 256]
    w_s = _rand_pow2((E, K_BIG // 128, N_SMALL // 128), -10, -6, gen)
    out = torch.empty((M_MAX, N_SMALL), dtype=torch.bfloat16, device="cuda")
    print(f"\ndgrad M_cap {M_MAX} N {K_BIG} K {N_SMALL} offsets {OFFSETS}", flush=True)
    ff8.ff8_grouped_gemm_dgrad(g, g_s, w, w_s, _offsets(), out)
    torch.cuda.synchronize()
    rng = np.random.default_rng(12)
    m, e = _sample_rows(rng, 256)
    c = rng.integers(N_SMALL, size=m.size)
    gd = quant.dequant_rowwise(host(g.index_select(0, _idx(m))), host(g_s.index_select(0, _idx(m))))
    wt = _dequant_weight(host(w[_idx(e), :, _idx(c)]), host(w_s[_idx(e), :, _idx(c // 128)]))
    got = host(out[_idx(m), _idx(c)].float())
    _check_gemm_samples(got, np.sum(gd * wt, axis=1), np.sum(np.abs(gd * wt), axis=1), True, K_BIG)


def test_wgrad_largest_column_wise_operand(gen):
    """dW[e, n, c] = sum over expert e's tokens of GT[n, m] XT[c, m]: XT is 7168 x 599040
    (K-blocked, [4680, 7168, 128]), and the last expert contracts over 594944 tokens (4648 K
    blocks)."""
    xT = _rand_e4m3((M_MAX // 128, K_BIG, 128), gen)
    xT_s = _rand_pow2((M_MAX // 128, K_BIG), -6, 3, gen)
    gT = _rand_e4m3((M_MAX // 128, N_SMALL, 128), gen)
    gT_s = _rand_pow2((M_MAX // 128, N_SMALL), -10, -6, gen)
    dw = torch.full((E, N_SMALL, K_BIG), 7.0, dtype=torch.float32, device="cuda")
    print(f"\nwgrad M_cap {M_MAX} N {N_SMALL} K {K_BIG} offsets {OFFSETS}", flush=True)
    ff8.ff8_grouped_gemm_wgrad(gT, gT_s, xT, xT_s, _offsets(), dw, accumulate=False)
    torch.cuda.synchronize()
    rng = np.random.default_rng(13)
    got, want, terms_abs, k = [], [], [], []
    for e in range(E):
        lo, hi = OFFSETS[e], OFFSETS[e + 1]
        scale_rows = _idx(np.arange(lo, hi, 128) // 128)
        ns = np.concatenate([[0, N_SMALL - 1], rng.integers(N_SMALL, size=10)])
        cs = np.concatenate([[0, K_BIG - 1], rng.integers(K_BIG, size=10)])
        for n, c in zip(ns, cs):
            gv = codec.e4m3_decode(_kblock_rows(gT, [int(n)], lo, hi)[0]) * \
                np.repeat(host(gT_s.index_select(0, scale_rows)[:, int(n)]).astype(np.float64), 128)
            xv = codec.e4m3_decode(_kblock_rows(xT, [int(c)], lo, hi)[0]) * \
                np.repeat(host(xT_s.index_select(0, scale_rows)[:, int(c)]).astype(np.float64), 128)
            t = gv * xv
            got.append(float(dw[e, int(n), int(c)]))
            want.append(float(np.sum(t)))
            terms_abs.append(float(np.sum(np.abs(t))))
            k.append(hi - lo)
    _check_gemm_samples(np.array(got), np.array(want), np.array(terms_abs), False, np.array(k))


def test_sat_largest_operand(gen):
    """The scaling-aware transpose of the same 599040 x 7168 row-scaled tensor (64-bit
    indexing; 4680 row blocks), checked block by block, the last row and column blocks
    included."""
    q = _rand_e4m3((M_MAX, K_BIG), gen)
    s = _rand_pow2((M_MAX, K_BIG // 128), -6, 3, gen)
    qT = torch.empty((M_MAX // 128, K_BIG, 128), dtype=torch.uint8, device="cuda")
    sT = torch.empty((M_MAX // 128, K_BIG), dtype=torch.float32, device="cuda")
    print(f"\nSAT rows {M_MAX} cols {K_BIG}", flush=True)
    ff8.ff8_scaling_aware_transpose(q, s, qT, sT)
    torch.cuda.synchronize()
    rng = np.random.default_rng(14)
    blocks = [(0, 0), (M_MAX // 128 - 1, K_BIG // 128 - 1), ((1 << 31) // K_BIG // 128, 3)]
    blocks += [(int(rng.integers(M_MAX // 128)), int(rng.integers(K_BIG // 128))) for _ in range(13)]
    for rb, cb in blocks:
        qb = host(q[rb * 128:(rb + 1) * 128, cb * 128:(cb + 1) * 128])
        sb = host(s[rb * 128:(rb + 1) * 128, cb:cb + 1])
        wqT, wsT = sat.scaling_aware_transpose(qb, sb)
        assert np.array_equal(host(qT[rb, cb * 128:(cb + 1) * 128]), wqT), (rb, cb)
        assert np.array_equal(host(sT[rb:rb + 1, cb * 128:(cb + 1) * 128]).T, wsT), (rb, cb)
