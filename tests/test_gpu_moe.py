"""Parity of the expert-layer kernels (permute, grouped GEMMs, SwiGLU, unpermute) and of
the whole layer against the CPU oracle, stage by stage (GPU)."""

import numpy as np
import pytest
import torch

import workloads
from oracle import codec, quant, sat, moe
from oracle import layer as olayer
from paper_2511_02302_amd import ff8
from paper_2511_02302_amd.layer import ExpertLayerFP8

from test_gpu_kernels import dev, host, f64, rel_frob, poisoned, untouched
from layouts import from_kblock, to_kblock

pytestmark = pytest.mark.gpu

GEMM_TOL = 2e-3   # max relative Frobenius error of a GEMM output against the float64 oracle
MAX_H_DPROBS = 8192  # the router-gradient kernel keeps one row of dY in registers (16 columns per lane)


def _skewed_routing(T, k, E, seed):
    """Routing with zero-token experts, tiny experts and one dominant expert."""
    rng = np.random.default_rng(seed)
    p = np.array([0.5, 0.0, 0.3, 0.02] + [0.18 / max(1, E - 5)] * (E - 5) + [0.0])[:E]
    p = p / p.sum()
    idx = np.stack([rng.choice(E, size=k, replace=False, p=p) for _ in range(T)]).astype(np.int32)
    return torch.from_numpy(idx)


CASES = {
    "tiny": (workloads.TINY, None),
    "ragged": (workloads.LayerShape("ragged T300 H384 E6 k2 I384", 300, 384, 6, 2, 384, "iid"), 7),
    "one_expert": (workloads.LayerShape("one expert T200 H256 E1 k1 I256", 200, 256, 1, 1, 256, "iid"), None),
    # every token routed to every expert (k = E), and a single token
    "all_experts": (workloads.LayerShape("all experts T130 H256 E4 k4 I256", 130, 256, 4, 4, 256, "iid"), None),
    "one_token": (workloads.LayerShape("one token T1 H256 E4 k2 I256", 1, 256, 4, 2, 256, "iid"), None),
    # a hidden size past what one-pass row kernels cover (the permute and unpermute loop over
    # 16-column chunks; fc1 contracts over 128 K blocks); wider than the router gradient takes
    "wide_hidden": (workloads.LayerShape("wide hidden T64 H16384 E2 k2 I256", 64, 16384, 2, 2, 256, "iid"), None),
    # the widest top-k the router-gradient kernel takes (k = 64), every expert chosen by every token
    "widest_topk": (workloads.LayerShape("widest top-k T300 H256 E64 k64 I256", 300, 256, 64, 64, 256, "iid"), None),
    # the narrowest widths: H = I = 128, one K block in fc1 fprop, fc2 fprop and fc2 dgrad, and a
    # 128-column W_e in dgrad (half of a 256-wide output tile)
    "min_width": (workloads.LayerShape("min width T257 H128 E3 k2 I128", 257, 128, 3, 2, 128, "iid"), None),
    # the most experts the kernels take (per-expert tables of E + 1 entries): ~4 rows each, many empty
    "max_experts": (workloads.LayerShape("max experts T2048 H256 E1024 k2 I256", 2048, 256, 1024, 2, 256, "iid"),
                    None),
}


def _inputs(case):
    shape, skew_seed = CASES[case]
    inp = workloads.layer_inputs(shape, seed=11)
    if skew_seed is not None:
        inp["topk_idx"] = _skewed_routing(shape.T, shape.k, shape.E, skew_seed)
    return shape, inp


def _routing_device(shape, inp):
    M_cap = ff8.ff8_rows_bound(shape.T, shape.k, shape.E)
    row_map = poisoned((shape.T, shape.k), torch.int32)
    offsets = poisoned((shape.E + 1,), torch.int32)
    src_row = poisoned((M_cap,), torch.int32)
    ws = torch.empty(max(1, ff8.ff8_permute_workspace_bytes(shape.T, shape.k, shape.E)), dtype=torch.uint8,
                     device="cuda")
    return M_cap, row_map, offsets, src_row, ws


@pytest.mark.parametrize("case", list(CASES))
def test_permute_quant_build_and_reuse(case):
    shape, inp = _inputs(case)
    M_cap, row_map, offsets, src_row, ws = _routing_device(shape, inp)
    q = poisoned((M_cap, shape.H), torch.uint8)
    s = poisoned((M_cap, shape.H // 128), torch.float32)
    ff8.ff8_permute_quant(dev(inp["x"]), None, shape.k, shape.E, dev(inp["topk_idx"]), False, row_map, offsets,
                          src_row, q, s, ws)
    torch.cuda.synchronize()
    counts, w_off, w_map, w_src = moe.route(host(inp["topk_idx"]), shape.E)
    m_pad = int(w_off[-1])
    assert np.array_equal(host(offsets), w_off)
    assert np.array_equal(host(row_map), w_map)
    assert np.array_equal(host(src_row)[:m_pad], w_src)
    assert untouched(src_row[m_pad:])
    wq, ws_ = moe.permute_quant_rows(f64(inp["x"]), w_src, shape.k)
    assert np.array_equal(host(q[:m_pad]), wq)
    assert np.array_equal(host(s[:m_pad]), ws_)
    assert untouched(q[m_pad:]) and untouched(s[m_pad:])
    # reuse mode with routing weights (the backward's dY cast)
    dq = poisoned((M_cap, shape.H), torch.uint8)
    dsc = poisoned((M_cap, shape.H // 128), torch.float32)
    ff8.ff8_permute_quant(dev(inp["dy"]), dev(inp["probs"]), shape.k, shape.E, None, True, row_map, offsets,
                          src_row, dq, dsc)
    torch.cuda.synchronize()
    wq2, ws2 = moe.permute_quant_rows(f64(inp["dy"]), w_src, shape.k, row_w=host(inp["probs"]))
    assert np.array_equal(host(dq[:m_pad]), wq2)
    assert np.array_equal(host(dsc[:m_pad]), ws2)
    assert untouched(dq[m_pad:])


@pytest.mark.parametrize("align", [16, 32, 64])
@pytest.mark.parametrize("case", ["ragged", "max_experts"])
def test_permute_quant_aligned(case, align):
    """Every group alignment the API takes: offsets, maps and the quantized rows bit-exact,
    padding rows zero, rows past the padded total untouched."""
    shape, inp = _inputs(case)
    M_cap = ff8.ff8_rows_bound_aligned(shape.T, shape.k, shape.E, align)
    _, row_map, offsets, _, ws = _routing_device(shape, inp)
    src_row = poisoned((M_cap,), torch.int32)
    q = poisoned((M_cap, shape.H), torch.uint8)
    s = poisoned((M_cap, shape.H // 128), torch.float32)
    ff8.ff8_permute_quant(dev(inp["x"]), None, shape.k, shape.E, dev(inp["topk_idx"]), False, row_map, offsets,
                          src_row, q, s, ws, align=align)
    torch.cuda.synchronize()
    counts, w_off, w_map, w_src = moe.route(host(inp["topk_idx"]), shape.E, align)
    m_pad = int(w_off[-1])
    assert np.all(w_off % align == 0) and np.array_equal(host(offsets), w_off)
    assert np.array_equal(host(row_map), w_map) and np.array_equal(host(src_row)[:m_pad], w_src)
    wq, ws_ = moe.permute_quant_rows(f64(inp["x"]), w_src, shape.k)
    assert np.array_equal(host(q[:m_pad]), wq) and np.array_equal(host(s[:m_pad]), ws_)
    assert untouched(q[m_pad:]) and untouched(s[m_pad:]) and untouched(src_row[m_pad:])


def test_permute_padding_spans_block():
    """Groups whose padding covers most of a 128-row block (rows in both 64-row halves),
    written into poisoned buffers: every padding row must come out zero with scale 2^-126."""
    shape = workloads.LayerShape("pad", 200, 256, 3, 1, 256, "iid")
    inp = workloads.layer_inputs(shape, seed=5)
    idx = torch.full((200, 1), 1, dtype=torch.int32)
    idx[:5, 0] = 0      # 5 rows -> 123 padding rows
    idx[5:70, 0] = 2    # 65 rows -> 63 padding rows
    M_cap, row_map, offsets, src_row, ws = _routing_device(shape, inp)
    for dst_rows in range(2):  # twice into the same poisoned buffers: the second pass overwrites the first
        q = poisoned((M_cap, shape.H), torch.uint8) if dst_rows == 0 else q
        s = poisoned((M_cap, shape.H // 128), torch.float32) if dst_rows == 0 else s
        ff8.ff8_permute_quant(dev(inp["x"]), None, shape.k, shape.E, dev(idx), False, row_map, offsets, src_row,
                              q, s, ws)
        torch.cuda.synchronize()
        _, w_off, _, w_src = moe.route(host(idx), shape.E)
        m_pad = int(w_off[-1])
        wq, wsc = moe.permute_quant_rows(f64(inp["x"]), w_src, shape.k)
        assert np.array_equal(host(q[:m_pad]), wq) and np.array_equal(host(s[:m_pad]), wsc)
        assert untouched(q[m_pad:]) and untouched(s[m_pad:])


def test_permute_deterministic_and_dropped_slots():
    shape = workloads.LayerShape("drop", 700, 256, 5, 3, 256, "iid")
    inp = workloads.layer_inputs(shape, seed=3)
    idx = inp["topk_idx"].clone()
    idx[::7, 1] = -1
    M_cap, row_map, offsets, src_row, ws = _routing_device(shape, inp)
    outs = []
    for _ in range(2):
        q = torch.zeros((M_cap, shape.H), dtype=torch.uint8, device="cuda")
        s = torch.zeros((M_cap, shape.H // 128), dtype=torch.float32, device="cuda")
        ff8.ff8_permute_quant(dev(inp["x"]), None, shape.k, shape.E, dev(idx), False, row_map, offsets, src_row,
                              q, s, ws)
        outs.append((host(q).copy(), host(row_map).copy()))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
    _, w_off, w_map, w_src = moe.route(host(idx), shape.E)
    assert np.array_equal(host(row_map), w_map)
    assert np.array_equal(host(offsets), w_off)


def _quantized_weights(shape, inp):
    E, H, I = shape.E, shape.H, shape.I
    w1q = torch.empty((E, 2 * I, H), dtype=torch.uint8, device="cuda")
    w1s = torch.empty((E, 2 * I // 128, H // 128), dtype=torch.float32, device="cuda")
    w2q = torch.empty((E, H, I), dtype=torch.uint8, device="cuda")
    w2s = torch.empty((E, H // 128, I // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_quant_block128(dev(inp["w1"]), w1q, w1s)
    ff8.ff8_quant_block128(dev(inp["w2"]), w2q, w2s)
    return w1q, w1s, w2q, w2s


@pytest.mark.parametrize("case", list(CASES))
def test_grouped_gemms(case):
    shape, inp = _inputs(case)
    E, H, I, T, k = shape.E, shape.H, shape.I, shape.T, shape.k
    M_cap, row_map, offsets, src_row, ws = _routing_device(shape, inp)
    xq = torch.empty((M_cap, H), dtype=torch.uint8, device="cuda")
    xs = torch.empty((M_cap, H // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_permute_quant(dev(inp["x"]), None, k, E, dev(inp["topk_idx"]), False, row_map, offsets, src_row, xq, xs,
                          ws)
    w1q, w1s, w2q, w2s = _quantized_weights(shape, inp)
    off = host(offsets).astype(np.int64)
    m_pad = int(off[-1])
    # fprop: A = Xq . W1^T
    a = poisoned((M_cap, 2 * I), torch.bfloat16)
    ff8.ff8_grouped_gemm_fprop(xq, xs, w1q, w1s, offsets, a)
    torch.cuda.synchronize()
    want = moe.grouped_gemm_fprop(host(xq), host(xs), host(w1q), host(w1s), off)
    got = f64(a[:m_pad])
    assert rel_frob(got, want) < GEMM_TOL
    assert rel_frob(got, codec.bf16_round(want)) < 1e-3
    assert untouched(a[m_pad:])
    # dgrad: dX = G . W1 with a random row-wise quantized G of width 2I
    g = workloads.randn_bf16((M_cap, 2 * I), 1.0, seed=5)
    gq_np, gs_np = quant.quant_rowwise(f64(g))
    gq, gs = dev(torch.from_numpy(gq_np)), dev(torch.from_numpy(gs_np))
    dx = poisoned((M_cap, H), torch.bfloat16)
    ff8.ff8_grouped_gemm_dgrad(gq, gs, w1q, w1s, offsets, dx)
    torch.cuda.synchronize()
    want = moe.grouped_gemm_dgrad(gq_np, gs_np, host(w1q), host(w1s), off)
    assert rel_frob(f64(dx[:m_pad]), want) < GEMM_TOL
    assert untouched(dx[m_pad:])
    # dgrad on fc2's weight (contraction over H)
    g2 = workloads.randn_bf16((M_cap, H), 1.0, seed=6)
    g2q_np, g2s_np = quant.quant_rowwise(f64(g2))
    dh = poisoned((M_cap, I), torch.bfloat16)
    ff8.ff8_grouped_gemm_dgrad(dev(torch.from_numpy(g2q_np)), dev(torch.from_numpy(g2s_np)), w2q, w2s, offsets, dh)
    torch.cuda.synchronize()
    want = moe.grouped_gemm_dgrad(g2q_np, g2s_np, host(w2q), host(w2s), off)
    assert rel_frob(f64(dh[:m_pad]), want) < GEMM_TOL
    # wgrad: dW1[e] = G_e^T X_e from column-wise operands (scaling-aware transposes)
    gT = torch.empty((M_cap // 128, 2 * I, 128), dtype=torch.uint8, device="cuda")  # K-blocked
    gTs = torch.empty((M_cap // 128, 2 * I), dtype=torch.float32, device="cuda")  # block-major
    xT = torch.empty((M_cap // 128, H, 128), dtype=torch.uint8, device="cuda")
    xTs = torch.empty((M_cap // 128, H), dtype=torch.float32, device="cuda")
    ff8.ff8_scaling_aware_transpose(gq, gs, gT, gTs, offsets, E)
    ff8.ff8_scaling_aware_transpose(xq, xs, xT, xTs, offsets, E)
    dw = torch.full((E, 2 * I, H), 7.0, dtype=torch.float32, device="cuda")
    ff8.ff8_grouped_gemm_wgrad(gT, gTs, xT, xTs, offsets, dw, accumulate=False)
    torch.cuda.synchronize()
    want = moe.grouped_gemm_wgrad(from_kblock(host(gT)), host(gTs).T, from_kblock(host(xT)), host(xTs).T, off)
    assert rel_frob(host(dw), want) < GEMM_TOL
    for e in range(E):
        if off[e + 1] == off[e]:
            assert bool((dw[e] == 0).all()), e
    # accumulate = 1 adds (and leaves empty experts untouched)
    ff8.ff8_grouped_gemm_wgrad(gT, gTs, xT, xTs, offsets, dw, accumulate=True)
    torch.cuda.synchronize()
    assert rel_frob(host(dw), 2 * want) < GEMM_TOL


def _swiglu_check(got_q, got_s, want_q, want_s, exact_vals, err_bound):
    """Both sides quantize the same activation; the device evaluates it in float32.

    err_bound[i] bounds |device value - exact value| for element i (float32 evaluation
    error, taken against the magnitude of the terms before any cancellation).  Then:
    a scale may differ only where the tile amax is within the tile's bound of a
    power-of-two edge 448 * 2^T; a byte may differ only by one code and only where the
    exact scaled value is within its bound of a rounding midpoint; and the dequantized
    tensors agree within 2e-3 relative Frobenius.
    """
    gq, gs = np.asarray(got_q), np.asarray(got_s)
    assert rel_frob(quant.dequant_rowwise(gq, gs), quant.dequant_rowwise(want_q, want_s)) < 2e-3
    rows, cols = gq.shape
    amax = np.abs(exact_vals).reshape(rows, cols // 128, 128).max(axis=2)
    tile_bound = err_bound.reshape(rows, cols // 128, 128).max(axis=2)
    t = quant.exponent_of_scale(want_s)
    edge = np.abs(amax - 448.0 * np.ldexp(1.0, t)) <= tile_bound
    edge |= np.abs(amax - 448.0 * np.ldexp(1.0, t - 1)) <= tile_bound
    sdiff = gs != want_s
    assert not np.any(sdiff & ~edge), np.argwhere(sdiff & ~edge)[:5]
    same_scale = np.repeat(~sdiff, 128, axis=1)
    bdiff = (gq != want_q) & same_scale
    assert bdiff.mean() < 1e-3, bdiff.mean()
    if bdiff.any():
        sc = np.repeat(want_s.astype(np.float64), 128, axis=1)[bdiff]
        a = np.abs(exact_vals[bdiff]) / sc
        mags = codec.e4m3_decode(np.arange(127, dtype=np.uint8))
        hi = np.clip(np.searchsorted(mags, a), 1, 126)
        mid = (mags[hi - 1] + mags[hi]) / 2
        near = np.abs(a - mid) <= err_bound[bdiff] / sc
        assert near.all(), (a[~near][:5], mid[~near][:5], (err_bound[bdiff] / sc)[~near][:5])
        steps = (gq[bdiff].astype(np.int64) & 0x7F) - (want_q[bdiff].astype(np.int64) & 0x7F)
        assert np.all(np.abs(steps) <= 1)


# float32 evaluation of exp, reciprocal and a few products: well under 64 ulp of the
# pre-cancellation magnitude for |g| <= 16 (exp's error grows like |g| ulp).
F32_EVAL = 64 * 2.0 ** -24


def _swiglu_bounds(a64, dh64):
    I = a64.shape[1] // 2
    g, u = a64[:, :I], a64[:, I:]
    sig = 1.0 / (1.0 + np.exp(-g))
    fwd = F32_EVAL * np.abs(g * sig * u) + 1e-30
    dg = F32_EVAL * np.abs(dh64 * u * sig) * (1.0 + np.abs(g) * (1.0 - sig)) + 1e-30
    du = F32_EVAL * np.abs(dh64 * g * sig) + 1e-30
    return fwd, np.concatenate([dg, du], axis=1)


@pytest.mark.parametrize("case", list(CASES))
def test_swiglu_fwd_bwd(case):
    shape, inp = _inputs(case)
    I, E = shape.I, shape.E
    M_cap = 1024
    a = workloads.randn_bf16((M_cap, 2 * I), 2.0, seed=8)
    dh = workloads.randn_bf16((M_cap, I), 1.0, seed=9)
    off_list = [0, 256, 256, 640, 896][: min(5, E + 1)] + [896] * max(0, E + 1 - 5)
    offsets = dev(torch.tensor(off_list, dtype=torch.int32))
    m_pad = off_list[-1]
    hq = poisoned((M_cap, I), torch.uint8)
    hs = poisoned((M_cap, I // 128), torch.float32)
    ff8.ff8_swiglu_quant(dev(a), hq, hs, offsets, E)
    daq = poisoned((M_cap, 2 * I), torch.uint8)
    das = poisoned((M_cap, 2 * I // 128), torch.float32)
    ff8.ff8_swiglu_bwd_quant(dev(a), dev(dh), daq, das, offsets, E)
    torch.cuda.synchronize()
    a64, dh64 = f64(a)[:m_pad], f64(dh)[:m_pad]
    h = moe.swiglu(a64)
    b_fwd, b_bwd = _swiglu_bounds(a64, dh64)
    wq, ws = quant.quant_rowwise(h)
    _swiglu_check(host(hq[:m_pad]), host(hs[:m_pad]), wq, ws, h, b_fwd)
    assert untouched(hq[m_pad:]) and untouched(hs[m_pad:])
    da = moe.swiglu_bwd(a64, dh64)
    wq2, ws2 = quant.quant_rowwise(da)
    _swiglu_check(host(daq[:m_pad]), host(das[:m_pad]), wq2, ws2, da, b_bwd)
    assert untouched(daq[m_pad:])


@pytest.mark.parametrize("case", list(CASES))
def test_permute_quant_dprobs(case):
    """B1 fused with the router gradient: the quantized copies bit-identical to the oracle's
    (and to the unfused entry point's), dprobs[t, j] = <dY[t], Y_perm[row]> within the fp32
    summation bound, 0 for dropped slots."""
    shape, inp = _inputs(case)
    T, H, E, k = shape.T, shape.H, shape.E, shape.k
    if H > MAX_H_DPROBS:  # rejected on the host, before any launch
        M_cap, row_map, offsets, src_row, _ = _routing_device(shape, inp)
        e = lambda *sh, dt=torch.float32: torch.empty(sh, dtype=dt, device="cuda")
        with pytest.raises(ff8.Ff8Error, match="bad shape"):
            ff8.ff8_permute_quant_dprobs(dev(inp["dy"]), dev(inp["probs"]), k, E, row_map, offsets, src_row,
                                         e(M_cap, H, dt=torch.uint8), e(M_cap, H // 128),
                                         e(M_cap, H, dt=torch.bfloat16), e(T, k))
        return
    idx = inp["topk_idx"].clone()
    idx[::7, 0] = -1  # dropped slots
    M_cap, row_map, offsets, src_row, ws = _routing_device(shape, inp)
    xq = torch.empty((M_cap, H), dtype=torch.uint8, device="cuda")
    xs = torch.empty((M_cap, H // 128), dtype=torch.float32, device="cuda")
    ff8.ff8_permute_quant(dev(inp["x"]), None, k, E, dev(idx), False, row_map, offsets, src_row, xq, xs, ws)
    y_perm = dev(workloads.randn_bf16((M_cap, H), 1.0, seed=21))
    dy, probs = dev(inp["dy"]), dev(inp["probs"])
    q = poisoned((M_cap, H), torch.uint8)
    s = poisoned((M_cap, H // 128), torch.float32)
    dprobs = poisoned((T, k), torch.float32)
    ff8.ff8_permute_quant_dprobs(dy, probs, k, E, row_map, offsets, src_row, q, s, y_perm, dprobs)
    q2 = torch.empty_like(q)
    s2 = torch.empty_like(s)
    ff8.ff8_permute_quant(dy, probs, k, E, None, True, row_map, offsets, src_row, q2, s2)
    torch.cuda.synchronize()
    _, w_off, w_map, w_src = moe.route(host(idx), E)
    m_pad = int(w_off[-1])
    assert np.array_equal(host(row_map), w_map)
    wq, wsc = moe.permute_quant_rows(f64(inp["dy"]), w_src, k, row_w=host(inp["probs"]))
    assert np.array_equal(host(q[:m_pad]), wq) and np.array_equal(host(s[:m_pad]), wsc)
    assert torch.equal(q[:m_pad], q2[:m_pad]) and torch.equal(s[:m_pad], s2[:m_pad])
    assert untouched(q[m_pad:]) and untouched(s[m_pad:])
    yp64, dy64 = f64(y_perm), f64(inp["dy"])
    want = moe.router_grad(dy64, yp64, w_map)
    mag = moe.router_grad(np.abs(dy64), np.abs(yp64), w_map)  # sum of |terms|
    got = host(dprobs).astype(np.float64)
    assert np.all(np.abs(got - want) <= mag * 2.0 ** -16 + 1e-30), np.max(np.abs(got - want) / (mag + 1e-30))
    assert np.all(got[w_map < 0] == 0.0) and (w_map < 0).any()


@pytest.mark.parametrize("case", list(CASES))
def test_swiglu_fp8_checkpoint(case):
    """F3 keeping A as an FP8 checkpoint, and B3 reading A back from it (section 4.2):
    the checkpoint bit-exact, H and dA against the oracle on the same operands."""
    shape, inp = _inputs(case)
    I, E = shape.I, shape.E
    M_cap = 1024
    a = workloads.randn_bf16((M_cap, 2 * I), 2.0, seed=8)
    dh = workloads.randn_bf16((M_cap, I), 1.0, seed=9)
    off_list = [0, 256, 256, 640, 896][: min(5, E + 1)] + [896] * max(0, E + 1 - 5)
    offsets = dev(torch.tensor(off_list, dtype=torch.int32))
    m_pad = off_list[-1]
    hq = poisoned((M_cap, I), torch.uint8)
    hs = poisoned((M_cap, I // 128), torch.float32)
    aq = poisoned((M_cap, 2 * I), torch.uint8)
    a_s = poisoned((M_cap, 2 * I // 128), torch.float32)
    ff8.ff8_swiglu_quant_keep_fp8(dev(a), hq, hs, aq, a_s, offsets, E)
    daq = poisoned((M_cap, 2 * I), torch.uint8)
    das = poisoned((M_cap, 2 * I // 128), torch.float32)
    ff8.ff8_swiglu_bwd_quant_fp8a(aq, a_s, dev(dh), daq, das, offsets, E)
    torch.cuda.synchronize()
    a64, dh64 = f64(a)[:m_pad], f64(dh)[:m_pad]
    want_hq, want_hs, want_aq, want_as = moe.swiglu_quant_keep(a64)
    assert np.array_equal(host(aq[:m_pad]), want_aq) and np.array_equal(host(a_s[:m_pad]), want_as)
    assert untouched(aq[m_pad:]) and untouched(a_s[m_pad:]) and untouched(hq[m_pad:])
    b_fwd, _ = _swiglu_bounds(a64, dh64)
    _swiglu_check(host(hq[:m_pad]), host(hs[:m_pad]), want_hq, want_hs, moe.swiglu(a64), b_fwd)
    ad = quant.dequant_rowwise(want_aq, want_as)
    _, b_bwd = _swiglu_bounds(ad, dh64)
    da = moe.swiglu_bwd(ad, dh64)
    wq, ws = moe.swiglu_bwd_quant_from_checkpoint(want_aq, want_as, dh64)
    _swiglu_check(host(daq[:m_pad]), host(das[:m_pad]), wq, ws, da, b_bwd)
    assert untouched(daq[m_pad:]) and untouched(das[m_pad:])


@pytest.mark.parametrize("k", [1, 2, 8])
def test_unpermute(k):
    T, H, E = 500, 256, 8
    shape = workloads.LayerShape("u", T, H, E, k, 128, "iid")
    idx, probs = workloads.routing(shape, seed=k)
    idx = idx.clone()
    if k > 1:
        idx[::5, 0] = -1
    _, off, row_map, _ = moe.route(host(idx), E)
    M_cap = ff8.ff8_rows_bound(T, k, E)
    yp = workloads.randn_bf16((M_cap, H), 1.0, seed=4)
    for w in (None, probs):
        y = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
        ff8.ff8_unpermute(dev(yp), dev(torch.from_numpy(row_map.astype(np.int32))), None if w is None else dev(w), y)
        torch.cuda.synchronize()
        want = moe.unpermute(f64(yp), row_map, None if w is None else host(w))
        got = f64(y)
        if k == 1 and w is None:
            assert np.array_equal(got, want)
        ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(want), 1e-30))[1] - 8)
        assert np.all(np.abs(got - want) <= ulp + 1e-6), np.max(np.abs(got - want) / ulp)


def test_layer_empty_batch():
    """T = 0: no routed rows; every kernel launches over empty groups, the weight gradients
    come out zero, and no row buffer is written."""
    shape = workloads.LayerShape("empty T0 H256 E4 k2 I256", 0, 256, 4, 2, 256, "iid")
    inp = workloads.layer_inputs(shape, seed=3)
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, fp8_checkpoint=True, router_grad=True)
    for n in ("xq", "a", "hq", "y_perm", "dyq", "dh", "daq", "dx_perm"):
        L.buf[n].view(torch.uint8).fill_(0xA5)
    d = {k: dev(v) for k, v in inp.items()}
    L.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    torch.cuda.synchronize()
    b = L.buf
    assert host(b["offsets"]).tolist() == [0] * (shape.E + 1)
    assert bool((b["dw1"] == 0).all()) and bool((b["dw2"] == 0).all())
    for n in ("xq", "a", "hq", "y_perm", "dyq", "dh", "daq", "dx_perm"):
        assert bool((b[n].view(torch.uint8) == 0xA5).all()), n
    assert b["y"].numel() == 0 and b["dx"].numel() == 0


@pytest.mark.parametrize("mode", ["paper_rows", "fp8_checkpoint_and_dprobs", "align16"])
@pytest.mark.parametrize("case", list(CASES))
def test_layer_stagewise(case, mode):
    """Whole forward+backward through ExpertLayerFP8; every stage is checked against the
    oracle applied to the GPU's own upstream outputs (no error compounding).  With the FP8
    checkpoint, A's checkpoint is bit-exact and the SwiGLU backward reads A from it; the router
    gradient of the same run is checked within its fp32 summation bound.  align16 pads the
    groups to 16 rows (the paper's padding): 128-row blocks then straddle experts."""
    shape, inp = _inputs(case)
    ckpt = mode == "fp8_checkpoint_and_dprobs"
    align = 16 if mode == "align16" else 128
    rgrad = ckpt and shape.H <= MAX_H_DPROBS
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, fp8_checkpoint=ckpt, router_grad=rgrad,
                       align=align)
    d = {k: dev(v) for k, v in inp.items()}
    L.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    torch.cuda.synchronize()
    b = {k: v for k, v in L.buf.items()}
    off = host(b["offsets"]).astype(np.int64)
    m_pad = int(off[-1])
    w = olayer.quantize_weights(f64(inp["w1"]), f64(inp["w2"]))
    for n in ("w1q", "w1s", "w2q", "w2s"):
        assert np.array_equal(host(b[n]), w[n]), n
    counts, w_off, w_map, w_src = moe.route(host(inp["topk_idx"]), shape.E, align)
    assert np.array_equal(off, w_off) and np.array_equal(host(b["row_map"]), w_map)
    if align == 16:
        assert np.any(w_off % 128 != 0)  # some group boundary inside a 128-row block
    xq, xs = moe.permute_quant_rows(f64(inp["x"]), w_src, shape.k)
    assert np.array_equal(host(b["xq"][:m_pad]), xq) and np.array_equal(host(b["xs"][:m_pad]), xs)
    A = moe.grouped_gemm_fprop(xq, xs, w["w1q"], w["w1s"], off)
    assert rel_frob(f64(b["a"][:m_pad]), A) < GEMM_TOL
    a_gpu = f64(b["a"][:m_pad])
    h = moe.swiglu(a_gpu)
    hq, hs = quant.quant_rowwise(h)
    _swiglu_check(host(b["hq"][:m_pad]), host(b["hs"][:m_pad]), hq, hs, h, _swiglu_bounds(a_gpu, a_gpu[:, :1])[0])
    Y = moe.grouped_gemm_fprop(host(b["hq"]), host(b["hs"]), w["w2q"], w["w2s"], off)
    assert rel_frob(f64(b["y_perm"][:m_pad]), Y) < GEMM_TOL
    y = moe.unpermute(f64(b["y_perm"][:m_pad]), w_map, host(inp["probs"]))
    assert rel_frob(f64(b["y"]), y) < 1e-3
    dyq, dys = moe.permute_quant_rows(f64(inp["dy"]), w_src, shape.k, row_w=host(inp["probs"]))
    assert np.array_equal(host(b["dyq"][:m_pad]), dyq) and np.array_equal(host(b["dys"][:m_pad]), dys)
    if rgrad:
        yp64 = f64(b["y_perm"][:m_pad])
        want = moe.router_grad(f64(inp["dy"]), yp64, w_map)
        mag = moe.router_grad(np.abs(f64(inp["dy"])), np.abs(yp64), w_map)
        assert np.all(np.abs(host(b["dprobs"]) - want) <= mag * 2.0 ** -16 + 1e-30)
    dH = moe.grouped_gemm_dgrad(dyq, dys, w["w2q"], w["w2s"], off)
    assert rel_frob(f64(b["dh"][:m_pad]), dH) < GEMM_TOL
    dh_gpu = f64(b["dh"][:m_pad])
    a_bwd = a_gpu
    if ckpt:
        aq, a_s = quant.quant_rowwise(a_gpu)
        assert np.array_equal(host(b["aq"][:m_pad]), aq) and np.array_equal(host(b["as"][:m_pad]), a_s)
        a_bwd = quant.dequant_rowwise(aq, a_s)
    da = moe.swiglu_bwd(a_bwd, dh_gpu)
    daq, das = quant.quant_rowwise(da)
    _swiglu_check(host(b["daq"][:m_pad]), host(b["das"][:m_pad]), daq, das, da, _swiglu_bounds(a_bwd, dh_gpu)[1])
    dXp = moe.grouped_gemm_dgrad(host(b["daq"][:m_pad]), host(b["das"][:m_pad]), w["w1q"], w["w1s"], off)
    assert rel_frob(f64(b["dx_perm"][:m_pad]), dXp) < GEMM_TOL
    dx = moe.unpermute(f64(b["dx_perm"][:m_pad]), w_map, None)
    assert rel_frob(f64(b["dx"]), dx) < 1e-3
    for name in ("x", "h", "dy", "da"):
        qT, sT = sat.scaling_aware_transpose(host(b[name + "q"][:m_pad]), host(b[name + "s"][:m_pad]))
        assert np.array_equal(from_kblock(host(b[name + "Tq"]))[:, :m_pad], qT), name
        assert np.array_equal(host(b[name + "Ts"][: -(-m_pad // 128)]).T, sT), name
    dW2 = moe.grouped_gemm_wgrad(from_kblock(host(b["dyTq"])), host(b["dyTs"]).T, from_kblock(host(b["hTq"])),
                                 host(b["hTs"]).T, off)
    assert rel_frob(host(b["dw2"]), dW2) < GEMM_TOL
    dW1 = moe.grouped_gemm_wgrad(from_kblock(host(b["daTq"])), host(b["daTs"]).T, from_kblock(host(b["xTq"])),
                                 host(b["xTs"]).T, off)
    assert rel_frob(host(b["dw1"]), dW1) < GEMM_TOL


@pytest.mark.parametrize("ckpt", [False, True], ids=["bf16_a", "fp8_checkpoint"])
def test_layer_stack_shared_workspace_and_saved_memory(ckpt):
    """Three layers sharing one step-local workspace, run forward 0..2 then backward 2..0 (each
    backward's dX feeding the next as dY) with the saved state released after each backward:
    every output equals that of a layer with its own workspace run the same way, bit for bit;
    the memory held between the forwards and the backwards is exactly the layers' saved state
    (with the FP8 checkpoint, A's 1x128 FP8 form instead of BF16); it is all returned after the
    backwards."""
    from paper_2511_02302_amd.layer import Workspace

    shape, inp = _inputs("ragged")
    d = {k: dev(v) for k, v in inp.items()}
    args = (shape.T, shape.H, shape.E, shape.k, shape.I)
    ws = Workspace(ExpertLayerFP8(*args, fp8_checkpoint=ckpt).d, fp8_checkpoint=ckpt)
    stack = [ExpertLayerFP8(*args, fp8_checkpoint=ckpt, workspace=ws) for _ in range(3)]
    alone = [ExpertLayerFP8(*args, fp8_checkpoint=ckpt) for _ in range(3)]
    outs = []
    for layers in (stack, alone):
        for L in layers:
            L.quantize_weights(d["w1"], d["w2"])
            L.release_saved()
        torch.cuda.synchronize()
        requested = lambda: torch.cuda.memory_stats()["requested_bytes.all.current"]  # exact tensor bytes
        base = requested()
        x = d["x"]
        for L in layers:
            x = L.forward(x, d["topk_idx"], d["probs"])
        torch.cuda.synchronize()
        kept = requested() - base
        g = d["dy"]
        for L in reversed(layers):
            g, _, _ = L.backward(g, d["probs"], release=True)
        torch.cuda.synchronize()
        assert requested() == base
        per_layer = stack[0].saved_activation_bytes()
        maps = 4 * (shape.T * shape.k + shape.E + 1 + stack[0].M_cap)
        assert kept == 3 * (per_layer + maps), (kept, per_layer, maps)
        outs.append([{n: L.own[n].clone() for n in ("y", "dx", "dw1", "dw2")} for L in layers])
    for i in range(3):
        for n in ("y", "dx", "dw1", "dw2"):
            assert torch.equal(outs[0][i][n].view(torch.uint8), outs[1][i][n].view(torch.uint8)), (i, n)
    M, I = stack[0].M_cap, shape.I
    fp8_xh = M * shape.H + M * shape.H // 32 + M * I + M * I // 32
    want = fp8_xh + (M * 2 * I + M * 2 * I // 32 if ckpt else M * 2 * I * 2)
    assert stack[0].saved_activation_bytes() == want


@pytest.mark.parametrize("mode", ["paper_rows", "fp8_checkpoint_and_dprobs"])
def test_layer_step_as_one_hip_graph(mode):
    """The step makes no host synchronization, allocation or memset, so it can be captured
    as one HIP graph.  Three replays, with eager work and synchronizations between them and
    the outputs poisoned before each, reproduce the eager step bit for bit (every kernel is
    deterministic)."""
    shape, inp = _inputs("ragged")
    ckpt = mode == "fp8_checkpoint_and_dprobs"
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, fp8_checkpoint=ckpt, router_grad=ckpt)
    d = {k: dev(v) for k, v in inp.items()}
    names = ["w1q", "w1s", "w2q", "w2s", "row_map", "offsets", "y", "dx", "dw1", "dw2"] + (["dprobs"] if ckpt else [])
    step = lambda: L.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager = {n: L.buf[n].clone() for n in names}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    other = torch.randn(1 << 20, device="cuda")
    for replay in range(3):
        for n in names:
            L.buf[n].view(torch.uint8).fill_(0xA5)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(L.buf[n].view(torch.uint8), eager[n].view(torch.uint8)), (replay, n)
        other.mul_(1.5).add_(1.0)  # the program's own eager work between replays
        torch.cuda.synchronize()


@pytest.mark.parametrize("rows", [[2048, 128, 0, 256], [2000, 128, 0, 272], [512, 512, 512, 512]],
                         ids=["skewed", "skewed_align16", "uniform"])
def test_wgrad_tile_schedules(rows):
    """dW of four experts with 4096 x 4096 weights (16 x 16 tiles each).  When the largest
    expert has more than twice the mean rows, the kernel splits every expert's tiles over
    the 8 XCDs in equal 8 x 4-tile rectangles; otherwise it walks XCD blocks.  Both orders,
    with 128- and 16-row groups, against the oracle over the whole output; operands are
    random e4m3 codes with random power-of-two column-wise scales (rows outside the groups
    hold data too, which the kernel must not add)."""
    E, N, K = len(rows), 4096, 4096
    off = np.concatenate([[0], np.cumsum(rows)]).astype(np.int64)
    M_cap = int(-(-(off[-1] + 128) // 128) * 128)
    rng = np.random.default_rng(sum(rows))
    code = lambda shape: rng.choice(np.r_[0:127, 128:255].astype(np.uint8), size=shape)
    gT, xT = code((N, M_cap)), code((K, M_cap))
    gTs = np.exp2(rng.integers(-8, 0, size=(M_cap // 128, N))).astype(np.float32)
    xTs = np.exp2(rng.integers(-4, 4, size=(M_cap // 128, K))).astype(np.float32)
    dw = torch.full((E, N, K), 7.0, dtype=torch.float32, device="cuda")
    ff8.ff8_grouped_gemm_wgrad(dev(torch.from_numpy(to_kblock(gT))), dev(torch.from_numpy(gTs)),
                               dev(torch.from_numpy(to_kblock(xT))), dev(torch.from_numpy(xTs)),
                               dev(torch.from_numpy(off.astype(np.int32))), dw)
    torch.cuda.synchronize()
    want = moe.grouped_gemm_wgrad(gT, gTs.T, xT, xTs.T, off)
    got = host(dw)
    for e in range(E):
        if rows[e] == 0:
            assert not got[e].any(), e
        else:
            assert rel_frob(got[e], want[e]) < GEMM_TOL, e
    # accumulating into the same gradient doubles it (experts without rows keep their zeros)
    args = [dev(torch.from_numpy(a)) for a in (to_kblock(gT), gTs, to_kblock(xT), xTs, off.astype(np.int32))]
    ff8.ff8_grouped_gemm_wgrad(*args, dw, accumulate=True)
    torch.cuda.synchronize()
    got = host(dw)
    for e in range(E):
        if rows[e] == 0:
            assert not got[e].any(), e
        else:
            assert rel_frob(got[e], 2 * want[e]) < GEMM_TOL, e
