"""Pins of the oracle's permute / GEMM / SwiGLU / unpermute steps (CPU only).

Independent references: pure-Python loops on tiny inputs (routing, GEMM
elements via math.fsum, unpermute), torch autograd and torch's SiLU for the
SwiGLU forward and backward, algebraic identities (transposing a 128x128-block
scaled weight is exact, so dgrad equals fprop against the transposed weight;
wgrad of all experts together is one product over the concatenated rows).
"""

import math

import numpy as np
import pytest
import torch

from oracle.codec import e4m3_decode
from oracle.quant import quant_rowwise, quant_block128, dequant_rowwise, TILE
from oracle import moe


def _routing(T, k, E, seed, drop=0.0):
    rng = np.random.default_rng(seed)
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    if drop:
        idx[rng.random((T, k)) < drop] = -1
    return idx


@pytest.mark.parametrize("align", [128, 16])
def test_route_brute_force(align):
    for (T, k, E, seed, drop) in [(37, 2, 5, 0, 0.0), (300, 4, 6, 1, 0.1), (5, 1, 9, 2, 0.0)]:
        idx = _routing(T, k, E, seed, drop)
        counts, offsets, row_map, src_row = moe.route(idx, E, align)
        # pure-Python reference: walk experts in order, tokens ascending
        row = 0
        ref_map = {}
        ref_off = [0]
        for e in range(E):
            start = row
            for t in range(T):
                for j in range(k):
                    if idx[t, j] == e:
                        ref_map[(t, j)] = row
                        row += 1
            n = row - start
            row = start + ((n + align - 1) // align) * align
            ref_off.append(row)
        assert offsets.tolist() == ref_off
        for t in range(T):
            for j in range(k):
                assert row_map[t, j] == ref_map.get((t, j), -1)
        real = src_row >= 0
        assert real.sum() == sum(1 for v in idx.ravel() if v >= 0)
        assert np.array_equal(np.sort(src_row[real]), np.sort(np.nonzero(idx.ravel() >= 0)[0]))
        assert all(o % align == 0 for o in ref_off)
        assert offsets[-1] <= moe.rows_bound(T, k, E, align) and moe.rows_bound(T, k, E, align) % 128 == 0
        assert np.array_equal(counts, np.bincount(idx[idx >= 0].ravel(), minlength=E))


def test_route_zero_token_experts():
    idx = np.array([[0, 3], [3, 0], [0, 3]])
    counts, offsets, row_map, src_row = moe.route(idx, 5)
    assert counts.tolist() == [3, 0, 0, 3, 0]
    assert offsets.tolist() == [0, 128, 128, 128, 256, 256]
    assert row_map.tolist() == [[0, 128], [129, 1], [2, 130]]


def test_permute_quant_rows_loop():
    T, k, E, H = 40, 3, 4, 256
    idx = _routing(T, k, E, 3, drop=0.05)
    rng = np.random.default_rng(0)
    x = torch.from_numpy(rng.standard_normal((T, H))).to(torch.bfloat16).float().numpy()
    w = rng.random((T, k)).astype(np.float32)
    _, offsets, row_map, src_row = moe.route(idx, E)
    for row_w in (None, w):
        q, s = moe.permute_quant_rows(x, src_row, k, row_w)
        assert q.shape == (offsets[-1], H)
        for r in range(offsets[-1]):
            if src_row[r] < 0:
                assert np.all(q[r] == 0) and np.all(s[r] == np.float32(2.0 ** -126))
                continue
            t, j = divmod(int(src_row[r]), k)
            v = x[t] if row_w is None else np.float32(w[t, j]) * x[t]
            qr, sr = quant_rowwise(v[None, :].astype(np.float32))
            assert np.array_equal(q[r], qr[0]) and np.array_equal(s[r], sr[0])
            assert row_map[t, j] == r


def _quant_expert_weights(E, N, K, seed):
    rng = np.random.default_rng(seed)
    w = rng.standard_normal((E, N, K)) * 0.02
    qs = [quant_block128(w[e]) for e in range(E)]
    return np.stack([q for q, _ in qs]), np.stack([s for _, s in qs])


def _dec_block(q, s):
    return e4m3_decode(q) * np.repeat(np.repeat(s.astype(np.float64), TILE, 0), TILE, 1)


def test_gemms_brute_force_elements():
    E, N, K = 3, 256, 384
    offsets = np.array([0, 128, 128, 384])   # expert 1 has no rows
    rng = np.random.default_rng(1)
    a = rng.standard_normal((offsets[-1], K))
    aq, as_ = quant_rowwise(a)
    wq, ws = _quant_expert_weights(E, N, K, 2)
    out = moe.grouped_gemm_fprop(aq, as_, wq, ws, offsets)
    A = e4m3_decode(aq) * np.repeat(as_.astype(np.float64), TILE, 1)
    for (m, n) in [(0, 0), (127, 255), (128, 17), (383, 100), (200, 128)]:
        e = 0 if m < 128 else 2
        W = _dec_block(wq[e], ws[e])
        assert out[m, n] == pytest.approx(math.fsum(A[m, kk] * W[n, kk] for kk in range(K)), rel=1e-13, abs=1e-300)
    # dgrad: out[m, k] = sum_n G[m, n] W_e[n, k]
    g = rng.standard_normal((offsets[-1], N))
    gq, gs = quant_rowwise(g)
    dg = moe.grouped_gemm_dgrad(gq, gs, wq, ws, offsets)
    G = e4m3_decode(gq) * np.repeat(gs.astype(np.float64), TILE, 1)
    for (m, kk) in [(0, 0), (127, 383), (300, 5)]:
        e = 0 if m < 128 else 2
        W = _dec_block(wq[e], ws[e])
        assert dg[m, kk] == pytest.approx(math.fsum(G[m, n] * W[n, kk] for n in range(N)), rel=1e-13, abs=1e-300)
    # dgrad == fprop against the transposed weight (transpose of a 128x128-block scaled tensor is exact)
    wqT = np.ascontiguousarray(np.transpose(wq, (0, 2, 1)))
    wsT = np.ascontiguousarray(np.transpose(ws, (0, 2, 1)))
    assert np.allclose(dg, moe.grouped_gemm_fprop(gq, gs, wqT, wsT, offsets), rtol=1e-12, atol=1e-14)


def test_wgrad_brute_force_and_zero_expert():
    N, K = 256, 128
    offsets = np.array([0, 256, 256, 384])
    rng = np.random.default_rng(5)
    gT = rng.standard_normal((N, 384))
    xT = rng.standard_normal((K, 384))
    gq, gs = quant_rowwise(gT)
    xq, xs = quant_rowwise(xT)
    dw = moe.grouped_gemm_wgrad(gq, gs, xq, xs, offsets)
    assert dw.shape == (3, N, K)
    assert np.all(dw[1] == 0)
    GT = dequant_rowwise(gq, gs)
    XT = dequant_rowwise(xq, xs)
    for (e, n, kk) in [(0, 0, 0), (0, 255, 127), (2, 3, 64)]:
        r0, r1 = offsets[e], offsets[e + 1]
        assert dw[e, n, kk] == pytest.approx(math.fsum(GT[n, m] * XT[kk, m] for m in range(r0, r1)), rel=1e-13)
    # all experts together: sum_e dW[e] = GT @ XT^T
    assert np.allclose(dw.sum(axis=0), GT @ XT.T, rtol=1e-12, atol=1e-12)


def test_swiglu_vs_torch_autograd():
    rng = np.random.default_rng(6)
    a = rng.standard_normal((16, 256)) * 3.0
    dh = rng.standard_normal((16, 128))
    at = torch.from_numpy(a).requires_grad_(True)
    h = torch.nn.functional.silu(at[:, :128]) * at[:, 128:]
    h.backward(torch.from_numpy(dh))
    assert np.allclose(moe.swiglu(a), h.detach().numpy(), rtol=1e-14, atol=1e-14)
    assert np.allclose(moe.swiglu_bwd(a, dh), at.grad.numpy(), rtol=1e-12, atol=1e-13)
    hq, hs = moe.swiglu_quant(a)
    q2, s2 = quant_rowwise(h.detach().numpy())
    assert np.array_equal(hq, q2) and np.array_equal(hs, s2)


def test_fp8_checkpoint_of_a():
    """The FP8 checkpoint of A is the plain 1x128 quantization of A, gate tiles and up tiles
    each with their own scale: when A is exactly representable (every tile holds a +-448 code
    times a power of two) it is lossless, and the backward from it equals the backward from A."""
    rng = np.random.default_rng(8)
    rows, I = 24, 256
    codes = rng.integers(0, 256, size=(rows, 2 * I), dtype=np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x00  # no NaN codes
    codes[:, ::TILE] = 0x7E  # every tile's amax is 448 (code 0x7E)
    t = rng.integers(-20, 6, size=(rows, 2 * I // TILE))
    t[:, : I // TILE] = -3  # gate tiles and up tiles on different scales
    s = np.power(2.0, t)
    a = e4m3_decode(codes) * np.repeat(s, TILE, axis=1)
    hq, hs, aq, a_s = moe.swiglu_quant_keep(a)
    assert np.array_equal(aq, codes) and np.array_equal(a_s, s.astype(np.float32))
    hq2, hs2 = moe.swiglu_quant(a)
    assert np.array_equal(hq, hq2) and np.array_equal(hs, hs2)
    dh = rng.standard_normal((rows, I))
    dq, ds = moe.swiglu_bwd_quant_from_checkpoint(aq, a_s, dh)
    dq2, ds2 = moe.swiglu_bwd_quant(a, dh)
    assert np.array_equal(dq, dq2) and np.array_equal(ds, ds2)
    # a general A: the gradient from the checkpoint stays within the e4m3 rounding of g and u
    a = rng.standard_normal((rows, 2 * I)) * 3.0
    _, _, aq, a_s = moe.swiglu_quant_keep(a)
    ad = dequant_rowwise(aq, a_s)
    assert np.all(np.abs(ad - a) <= np.abs(a) * 2.0 ** -4 + 2.0 ** -9 * np.repeat(a_s, TILE, axis=1))
    g_ref, g_ck = moe.swiglu_bwd(a, dh), moe.swiglu_bwd(ad, dh)
    assert np.linalg.norm(g_ck - g_ref) / np.linalg.norm(g_ref) < 0.05


def test_router_grad_loop_and_directional_derivative():
    """dprobs is the derivative of <dY, combine(w)> with respect to each routing weight: the
    combine is linear in w, so a unit step in w[t, j] changes the loss by exactly dprobs[t, j]."""
    rng = np.random.default_rng(9)
    T, k, H, M = 12, 3, 40, 50
    row_map = np.stack([rng.choice(M, size=k, replace=False) for _ in range(T)]).astype(np.int64)
    row_map[2, 1] = -1
    row_map[7, 0] = -1
    y_perm = rng.standard_normal((M, H))
    dy = rng.standard_normal((T, H))
    w = rng.random((T, k))
    dp = moe.router_grad(dy, y_perm, row_map)
    for t in range(T):
        for j in range(k):
            r = row_map[t, j]
            want = 0.0 if r < 0 else math.fsum(dy[t, h] * y_perm[r, h] for h in range(H))
            assert dp[t, j] == pytest.approx(want, rel=1e-12, abs=1e-12)

    def loss(wt):
        y = np.zeros((T, H))
        for j in range(k):
            ok = row_map[:, j] >= 0
            y[ok] += wt[ok, j][:, None] * y_perm[row_map[ok, j]]
        return float(np.sum(dy * y))

    base = loss(w)
    for t, j in [(0, 0), (2, 1), (5, 2), (11, 1)]:
        w2 = w.copy()
        w2[t, j] += 1.0
        assert loss(w2) - base == pytest.approx(dp[t, j], rel=1e-9, abs=1e-9)


def test_unpermute_loop_and_gather():
    T, k, E, H = 30, 3, 5, 128
    idx = _routing(T, k, E, 8, drop=0.1)
    _, offsets, row_map, _ = moe.route(idx, E)
    rng = np.random.default_rng(2)
    yp = torch.from_numpy(rng.standard_normal((offsets[-1], H))).to(torch.bfloat16).double().numpy()
    w = rng.random((T, k)).astype(np.float32)
    y = moe.unpermute(yp, row_map, w)
    for t in range(T):
        for hh in (0, 77, 127):
            acc = math.fsum(float(w[t, j]) * yp[row_map[t, j], hh] for j in range(k) if row_map[t, j] >= 0)
            assert abs(y[t, hh] - acc) <= abs(acc) * 2.0 ** -8
    # k = 1 with unit weight is a pure gather (exact)
    idx1 = _routing(T, 1, E, 9)
    _, off1, rm1, _ = moe.route(idx1, E)
    yp1 = torch.from_numpy(rng.standard_normal((off1[-1], H))).to(torch.bfloat16).double().numpy()
    assert np.array_equal(moe.unpermute(yp1, rm1, None), yp1[rm1[:, 0]])


def test_wgrad_groups_ending_inside_128_token_blocks():
    """Groups padded to 16 rows (section 3.3.1): expert boundaries fall inside 128-token blocks,
    the last block is partial, and one column scale covers tokens of two experts.  Each
    element of dW[e] is the exactly-rounded sum over precisely expert e's token columns, each
    token scaled by the column scale of its own 128-token block."""
    N, K = 128, 256
    offsets = np.array([0, 176, 176, 272, 400])  # 176 = 128 + 48, 272 = 2*128 + 16, 400 = 3*128 + 16
    m_pad = int(offsets[-1])
    nb = -(-m_pad // TILE)  # 4 blocks, the last one holds 16 tokens
    rng = np.random.default_rng(11)
    codes_g = rng.integers(0, 256, size=(N, m_pad), dtype=np.uint8)
    codes_x = rng.integers(0, 256, size=(K, m_pad), dtype=np.uint8)
    for c in (codes_g, codes_x):
        c[(c & 0x7F) == 0x7F] = 0x00  # no NaN codes
    # random power-of-two column scales, per (column row, 128-token block); a caller's scale
    # buffer is wider than the blocks in use (M_cap/128 entries), the extra entries are never used
    sg = np.ldexp(1.0, rng.integers(-30, 10, size=(N, nb + 2))).astype(np.float32)
    sx = np.ldexp(1.0, rng.integers(-30, 10, size=(K, nb + 2))).astype(np.float32)
    sg[:, nb:] = np.float32(np.nan)
    sx[:, nb:] = np.float32(np.nan)
    dw = moe.grouped_gemm_wgrad(codes_g, sg, codes_x, sx, offsets)
    assert dw.shape == (4, N, K)
    assert np.all(dw[1] == 0)  # zero-token expert
    dec_g, dec_x = e4m3_decode(codes_g), e4m3_decode(codes_x)
    picks = [(0, 0, 0), (0, 127, 255), (0, 5, 130), (2, 64, 7), (2, 100, 200), (3, 1, 1), (3, 127, 128)]
    picks += [(e, int(rng.integers(N)), int(rng.integers(K))) for e in (0, 2, 3) for _ in range(6)]
    for (e, n, kk) in picks:
        terms = [float(dec_g[n, m]) * float(sg[n, m // TILE]) * float(dec_x[kk, m]) * float(sx[kk, m // TILE])
                 for m in range(int(offsets[e]), int(offsets[e + 1]))]
        assert dw[e, n, kk] == pytest.approx(math.fsum(terms), rel=1e-12, abs=1e-300), (e, n, kk)
    # shifting a token's bytes from one expert to its neighbour moves exactly its product
    kk, n, m = 3, 9, 175  # token 175: the last of expert 0, inside block 1 which expert 2 shares
    zero_g = codes_g.copy()
    zero_g[n, m] = 0x00
    dw2 = moe.grouped_gemm_wgrad(zero_g, sg, codes_x, sx, offsets)
    moved = float(dec_g[n, m]) * float(sg[n, 1]) * float(dec_x[kk, m]) * float(sx[kk, 1])
    assert dw[0, n, kk] - dw2[0, n, kk] == pytest.approx(moved, rel=1e-9, abs=1e-300)
    assert np.array_equal(dw[2], dw2[2]) and np.array_equal(dw[3], dw2[3])


@pytest.mark.parametrize("T,k,E,align", [(4, 1, 4, 16), (3, 1, 3, 128), (5, 2, 3, 16), (2, 2, 3, 16),
                                         (6, 1, 2, 4), (3, 2, 4, 32)])
def test_rows_bound_is_the_worst_case(T, k, E, align):
    """rows_bound against brute force over EVERY routing of a tiny batch (k distinct experts
    per token): never below the largest padded row count, and equal to it (rounded up to whole
    128-row blocks) whenever some routing makes every expert's count 1 more than a multiple of
    the alignment, the worst case the bound assumes."""
    import itertools

    choices = list(itertools.permutations(range(E), k))
    worst, attained = 0, False
    for pick in itertools.product(choices, repeat=T):
        idx = np.array(pick, dtype=np.int64).reshape(T, k)
        counts, offsets, _, _ = moe.route(idx, E, align)
        worst = max(worst, int(offsets[-1]))
        attained |= bool(np.all(counts % align == 1))
    bound = moe.rows_bound(T, k, E, align)
    assert bound % 128 == 0 and worst <= bound
    if attained:
        assert worst == T * k + (align - 1) * E
        assert bound == -(-worst // 128) * 128
    else:
        assert worst < T * k + (align - 1) * E
