"""Parity at full size: the DeepSeek-V3 expert-parallel share (T16384 H7168 E32 k8 I2048)
and the Zipf-skewed layer (T8192, same widths), in the launch configuration bench.py
times.  One whole forward+backward step runs on the GPU; sampled outputs of every stage
are then checked against the oracle, element by element, each computed from the GPU's
own upstream tensors (so no error compounds across stages) (GPU)."""

import zlib

import numpy as np
import pytest
import torch

import workloads
from oracle import codec, quant, sat, moe
from paper_2511_02302_amd import ff8
from paper_2511_02302_amd.layer import ExpertLayerFP8

from test_gpu_kernels import f64, host, rel_frob
from test_gpu_moe import GEMM_TOL, _swiglu_bounds, _swiglu_check

pytestmark = pytest.mark.gpu

# (shape, row alignment of the expert groups): 128, and the paper's 16 on the DeepSeek-V3 share
SHAPES = {"dsv3": (workloads.DSV3, 128), "skew": (workloads.SKEW, 128), "dsv3_align16": (workloads.DSV3, 16)}
N_GEMM = 256  # sampled elements per GEMM output


def _cuda_idx(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int64)).cuda()


def _rows(t, idx):
    """Rows idx of a device tensor, on the host."""
    return host(t.index_select(0, _cuda_idx(idx)))


@pytest.fixture(scope="module", params=list(SHAPES))
def run(request):
    shape, align = SHAPES[request.param]
    print(f"\nfull-size layer step: {shape.name}, groups padded to {align}", flush=True)
    d = workloads.layer_inputs(shape, seed=0, device="cuda")
    if shape.routing == "zipf":  # the stress case's populations, on the very routing the GPU runs
        print(f"expert populations: {workloads.check_skew(d['topk_idx'], shape.E)}", flush=True)
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, align=align)
    L.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    torch.cuda.synchronize()
    _, off, row_map, src_row = moe.route(host(d["topk_idx"]), shape.E, align)
    yield {"shape": shape, "d": d, "b": L.buf, "L": L, "off": off.astype(np.int64), "row_map": row_map,
           "src_row": src_row, "rng": np.random.default_rng(zlib.crc32(request.param.encode()))}
    del L, d
    torch.cuda.empty_cache()


def _kblock_rows(t, idx, lo, hi):
    """Rows idx (transposed-operand rows: columns of the original) over tokens [lo, hi) of a
    K-blocked transpose t [M_cap/128, rows, 128], on the host as [len(idx), hi - lo]."""
    kb0, kb1 = lo // 128, -(-hi // 128)
    slabs = t[kb0:kb1].index_select(1, _cuda_idx(idx))            # [blocks, len(idx), 128]
    return host(slabs.permute(1, 0, 2).reshape(len(idx), -1))[:, lo - 128 * kb0:hi - 128 * kb0]


def _sample_rows(r, n):
    """n distinct routed rows (padding excluded), sorted, and the expert of each."""
    real = np.nonzero(r["src_row"] >= 0)[0]
    m = np.sort(r["rng"].choice(real, size=min(n, real.size), replace=False))
    return m, np.searchsorted(r["off"], m, side="right") - 1


def test_routing_full(run):
    b = run["b"]
    m_pad = int(run["off"][-1])
    assert np.array_equal(host(b["offsets"]).astype(np.int64), run["off"])
    assert np.array_equal(host(b["row_map"]), run["row_map"])
    assert np.array_equal(host(b["src_row"])[:m_pad], run["src_row"])


def test_padding_rows_full(run):
    """Every padding row of the four row-wise FP8 tensors (F1, B1, F3, B3): bytes 0x00 and
    scale 2^-126 (padding rows enter the weight-gradient sums, so none may hold stale data)."""
    b = run["b"]
    pad = _cuda_idx(np.nonzero(run["src_row"] < 0)[0])
    for qn, sn in (("xq", "xs"), ("dyq", "dys"), ("hq", "hs"), ("daq", "das")):
        assert not bool(b[qn].index_select(0, pad).any()), qn
        assert bool((b[sn].index_select(0, pad) == 2.0 ** -126).all()), sn


def test_weight_quant_sampled_blocks(run):
    d, b, rng = run["d"], run["b"], run["rng"]
    for wn in ("w1", "w2"):
        E, R, C = d[wn].shape
        for _ in range(8):
            e, rb, cb = int(rng.integers(E)), int(rng.integers(R // 128)), int(rng.integers(C // 128))
            sl = (e, slice(rb * 128, (rb + 1) * 128), slice(cb * 128, (cb + 1) * 128))
            wq, ws = quant.quant_block128(f64(d[wn][sl]))
            assert np.array_equal(host(b[wn + "q"][sl]), wq), (wn, e, rb, cb)
            assert host(b[wn + "s"][e, rb, cb]) == ws[0, 0], (wn, e, rb, cb)


def test_permute_quant_sampled_rows(run):
    """F1 (plain) and B1 (routing-weighted) rows: bytes and scales bit-exact on 2048 rows."""
    shape, d, b = run["shape"], run["d"], run["b"]
    m, _ = _sample_rows(run, 2048)
    src = run["src_row"][m]
    t, j = src // shape.k, src % shape.k
    local = np.arange(m.size) * shape.k + j  # sampled row i reads local token i
    probs = _rows(d["probs"], t)
    for src_t, qn, sn, w in (("x", "xq", "xs", None), ("dy", "dyq", "dys", probs)):
        wq, ws = moe.permute_quant_rows(f64(d[src_t].index_select(0, _cuda_idx(t))), local, shape.k, row_w=w)
        assert np.array_equal(_rows(b[qn], m), wq), qn
        assert np.array_equal(_rows(b[sn], m), ws), sn


def _check_gemm_samples(got, want, terms_abs, bf16_out, k):
    """Per-element bound.  The products of e4m3 values and power-of-two scales are exact, but
    the matrix core does not add the 64 products of one instruction exactly: on full-range
    e4m3 operands its error has reached several hundred units of 2^-24 of their sum of
    |terms| (more than the one or two roundings of an exact sum).  2^-13 of the sum of |terms|
    covers that with margin, and 2 ceil(k/64) units of 2^-24 the float32 accumulation over
    the k/64 instruction steps; a bf16 output adds half an ulp, at most 2^-8 relative.  On the
    whole sample: bf16 outputs within 1e-3 (relative Frobenius) of the bf16-rounded oracle,
    fp32 outputs within the GEMM tolerance of the oracle itself.  (The relative Frobenius
    error of a few hundred bf16 samples against the unrounded oracle is not used: bf16
    rounding alone puts it near 1.6e-3, at times above 2e-3.)"""
    got, want = np.asarray(got, dtype=np.float64), np.asarray(want, dtype=np.float64)
    steps = np.ceil(np.asarray(k, dtype=np.float64) / 64)
    bound = terms_abs * (2.0 ** -13 + 2 * steps * 2.0 ** -24) + \
        (np.abs(want) * 2.0 ** -8 if bf16_out else 0.0) + 1e-30
    bad = np.abs(got - want) > bound
    if not bf16_out:
        print(f"largest error: {np.max(np.abs(got - want) / (terms_abs * 2.0 ** -24 + 1e-300)):.0f} units of 2^-24 of "
              "the sum of |terms|", flush=True)
    assert not bad.any(), (np.nonzero(bad)[0][:4], got[bad][:4], want[bad][:4], bound[bad][:4])
    if bf16_out:
        assert rel_frob(got, codec.bf16_round(want)) < 1e-3
    else:
        assert rel_frob(got, want) < GEMM_TOL


def _dequant_weight(q, s):
    """Dequantize block-scaled weight rows or columns: q [..., n], s [..., n / 128] (float64)."""
    return codec.e4m3_decode(q) * np.repeat(s.astype(np.float64), 128, axis=-1)


def _fprop_samples(run, qa, sa, wn, out):
    """out[m, n] = sum_k A[m, k] W_e[n, k] at sampled (m, n)."""
    b, rng = run["b"], run["rng"]
    m, e = _sample_rows(run, N_GEMM)
    n = rng.integers(b[out].shape[1], size=m.size)
    a = quant.dequant_rowwise(_rows(b[qa], m), _rows(b[sa], m))
    got = host(b[out][_cuda_idx(m), _cuda_idx(n)].float())
    wq = host(b[wn + "q"][_cuda_idx(e), _cuda_idx(n)])           # [samples, K]
    ws = host(b[wn + "s"][_cuda_idx(e), _cuda_idx(n // 128)])    # [samples, K / 128]
    w = _dequant_weight(wq, ws)
    _check_gemm_samples(got, np.sum(a * w, axis=1), np.sum(np.abs(a * w), axis=1), True, a.shape[1])


def test_fc1_fc2_fprop_sampled(run):
    _fprop_samples(run, "xq", "xs", "w1", "a")
    _fprop_samples(run, "hq", "hs", "w2", "y_perm")


def _dgrad_samples(run, qg, sg, wn, out):
    """out[m, c] = sum_n G[m, n] W_e[n, c] at sampled (m, c): column c of the weight."""
    b, rng = run["b"], run["rng"]
    m, e = _sample_rows(run, N_GEMM)
    c = rng.integers(b[out].shape[1], size=m.size)
    g = quant.dequant_rowwise(_rows(b[qg], m), _rows(b[sg], m))
    got = host(b[out][_cuda_idx(m), _cuda_idx(c)].float())
    wq = host(b[wn + "q"][_cuda_idx(e), :, _cuda_idx(c)])          # [samples, N]
    ws = host(b[wn + "s"][_cuda_idx(e), :, _cuda_idx(c // 128)])   # [samples, N / 128]
    w = _dequant_weight(wq, ws)
    _check_gemm_samples(got, np.sum(g * w, axis=1), np.sum(np.abs(g * w), axis=1), True, g.shape[1])


def test_fc2_fc1_dgrad_sampled(run):
    _dgrad_samples(run, "dyq", "dys", "w2", "dh")
    _dgrad_samples(run, "daq", "das", "w1", "dx_perm")


def _wgrad_samples(run, gT, xT, out):
    """dW[e, n, c] = sum over expert e's rows m of GT[n, m] XT[c, m] (column-wise operands
    from the scaling-aware transpose) on a few busy experts; zeros for experts without rows."""
    b, off, rng = run["b"], run["off"], run["rng"]
    E, N, K = b[out].shape
    busy = np.nonzero(off[1:] > off[:-1])[0]
    for e in sorted(rng.choice(busy, size=min(4, busy.size), replace=False)):
        lo, hi = int(off[e]), int(off[e + 1])
        n = rng.integers(N, size=N_GEMM // 4)
        c = rng.integers(K, size=N_GEMM // 4)
        got = host(b[out][int(e)][_cuda_idx(n), _cuda_idx(c)])
        blk = _cuda_idx(np.arange(lo, hi) // 128)  # each token's 128-row block (groups may share one)
        g = codec.e4m3_decode(_kblock_rows(b[gT + "q"], n, lo, hi)) * \
            host(b[gT + "s"].index_select(0, blk)[:, _cuda_idx(n)]).T.astype(np.float64)
        x = codec.e4m3_decode(_kblock_rows(b[xT + "q"], c, lo, hi)) * \
            host(b[xT + "s"].index_select(0, blk)[:, _cuda_idx(c)]).T.astype(np.float64)
        _check_gemm_samples(got, np.sum(g * x, axis=1), np.sum(np.abs(g * x), axis=1), False, hi - lo)
    empty = np.nonzero(off[1:] == off[:-1])[0]
    if run["shape"].routing == "zipf":
        assert empty.size > 0, "the skewed layer must have experts without tokens"
    for e in empty:
        assert not bool(b[out][int(e)].any()), f"expert {e} has no rows but a nonzero gradient"


def test_fc2_fc1_wgrad_sampled(run):
    _wgrad_samples(run, "dyT", "hT", "dw2")
    _wgrad_samples(run, "daT", "xT", "dw1")


def _whole_tiles(run):
    """Two 256 x 256 output tiles per GEMM: the first row tile of the busiest expert with the
    first column tile, and the last (ragged) row tile of another busy expert with the last
    column tile.  Every lane, accumulator and epilogue position of the tile is compared."""
    off, rng = run["off"], run["rng"]
    rows = off[1:] - off[:-1]
    busy = np.nonzero(rows > 0)[0]
    e0 = int(np.argmax(rows))
    e1 = int(rng.choice(busy[busy != e0])) if busy.size > 1 else e0
    lo1, hi1 = int(off[e1]), int(off[e1 + 1])
    last = lo1 + (hi1 - lo1 - 1) // 256 * 256
    return [(e0, np.arange(int(off[e0]), min(int(off[e0]) + 256, int(off[e0 + 1]))), True),
            (e1, np.arange(last, hi1), False)]


def _cols(n, first):
    return np.arange(0, 256) if first else np.arange(n - 256, n)


def test_gemm_whole_tiles(run):
    b, off = run["b"], run["off"]
    for e, m, first in _whole_tiles(run):
        for qa, sa, wn, out in (("xq", "xs", "w1", "a"), ("hq", "hs", "w2", "y_perm")):  # fprop
            n = _cols(b[out].shape[1], first)
            a = quant.dequant_rowwise(_rows(b[qa], m), _rows(b[sa], m))
            w = _dequant_weight(host(b[wn + "q"][e].index_select(0, _cuda_idx(n))),
                                host(b[wn + "s"][e].index_select(0, _cuda_idx(n // 128))))
            got = host(b[out].index_select(0, _cuda_idx(m)).index_select(1, _cuda_idx(n)).float())
            _check_gemm_samples(got.ravel(), (a @ w.T).ravel(), (np.abs(a) @ np.abs(w).T).ravel(), True, a.shape[1])
        for qg, sg, wn, out in (("dyq", "dys", "w2", "dh"), ("daq", "das", "w1", "dx_perm")):  # dgrad
            c = _cols(b[out].shape[1], first)
            g = quant.dequant_rowwise(_rows(b[qg], m), _rows(b[sg], m))
            wq = host(b[wn + "q"][e].index_select(1, _cuda_idx(c))).T           # [256 c, N]
            ws = host(b[wn + "s"][e].index_select(1, _cuda_idx(c // 128))).T    # [256 c, N / 128]
            w = _dequant_weight(wq, ws)
            got = host(b[out].index_select(0, _cuda_idx(m)).index_select(1, _cuda_idx(c)).float())
            _check_gemm_samples(got.ravel(), (g @ w.T).ravel(), (np.abs(g) @ np.abs(w).T).ravel(), True, g.shape[1])
        lo, hi = int(off[e]), int(off[e + 1])
        blk = _cuda_idx(np.arange(lo, hi) // 128)
        for gT, xT, out in (("dyT", "hT", "dw2"), ("daT", "xT", "dw1")):  # wgrad
            N, K = b[out].shape[1:]
            n, c = _cols(N, first), _cols(K, first)
            g = codec.e4m3_decode(_kblock_rows(b[gT + "q"], n, lo, hi)) * \
                host(b[gT + "s"].index_select(0, blk)[:, _cuda_idx(n)]).T.astype(np.float64)
            x = codec.e4m3_decode(_kblock_rows(b[xT + "q"], c, lo, hi)) * \
                host(b[xT + "s"].index_select(0, blk)[:, _cuda_idx(c)]).T.astype(np.float64)
            got = host(b[out][e].index_select(0, _cuda_idx(n)).index_select(1, _cuda_idx(c)))
            _check_gemm_samples(got.ravel(), (g @ x.T).ravel(), (np.abs(g) @ np.abs(x).T).ravel(), False, hi - lo)


def test_swiglu_fwd_bwd_sampled_rows(run):
    b = run["b"]
    m, _ = _sample_rows(run, 48)
    a64, dh64 = f64(b["a"].index_select(0, _cuda_idx(m))), f64(b["dh"].index_select(0, _cuda_idx(m)))
    b_fwd, b_bwd = _swiglu_bounds(a64, dh64)
    h = moe.swiglu(a64)
    wq, ws = quant.quant_rowwise(h)
    _swiglu_check(_rows(b["hq"], m), _rows(b["hs"], m), wq, ws, h, b_fwd)
    da = moe.swiglu_bwd(a64, dh64)
    wq, ws = quant.quant_rowwise(da)
    _swiglu_check(_rows(b["daq"], m), _rows(b["das"], m), wq, ws, da, b_bwd)


def test_fp8_checkpoint_sampled_rows(run):
    """F3 with the FP8 checkpoint of A and B3 reading it, on the step's own A and dH: H equal
    to the step's, the checkpoint bit-exact and dA against the oracle at sampled rows."""
    shape, b = run["shape"], run["b"]
    M_cap, I2 = b["a"].shape
    m_pad = int(run["off"][-1])
    u8, f32 = torch.uint8, torch.float32
    hq, hs = torch.empty((M_cap, I2 // 2), dtype=u8, device="cuda"), torch.empty((M_cap, I2 // 256), dtype=f32,
                                                                                    device="cuda")
    aq, a_s = torch.empty((M_cap, I2), dtype=u8, device="cuda"), torch.empty((M_cap, I2 // 128), dtype=f32,
                                                                               device="cuda")
    daq, das = torch.empty_like(aq), torch.empty_like(a_s)
    ff8.ff8_swiglu_quant_keep_fp8(b["a"], hq, hs, aq, a_s, b["offsets"], shape.E)
    ff8.ff8_swiglu_bwd_quant_fp8a(aq, a_s, b["dh"], daq, das, b["offsets"], shape.E)
    torch.cuda.synchronize()
    assert torch.equal(hq[:m_pad], b["hq"][:m_pad]) and torch.equal(hs[:m_pad], b["hs"][:m_pad])
    m, _ = _sample_rows(run, 48)
    a64, dh64 = f64(b["a"].index_select(0, _cuda_idx(m))), f64(b["dh"].index_select(0, _cuda_idx(m)))
    want_aq, want_as = quant.quant_rowwise(a64)
    assert np.array_equal(_rows(aq, m), want_aq) and np.array_equal(_rows(a_s, m), want_as)
    ad = quant.dequant_rowwise(want_aq, want_as)
    _, b_bwd = _swiglu_bounds(ad, dh64)
    da = moe.swiglu_bwd(ad, dh64)
    wq, ws = quant.quant_rowwise(da)
    _swiglu_check(_rows(daq, m), _rows(das, m), wq, ws, da, b_bwd)
    del hq, hs, aq, a_s, daq, das


def test_router_grad_sampled_tokens(run):
    """B1 fused with the router gradient on the step's own dY and Y_perm: the quantized copies
    equal the step's B1 output, dprobs at sampled tokens within the fp32 summation bound."""
    shape, d, b, rng = run["shape"], run["d"], run["b"], run["rng"]
    m_pad = int(run["off"][-1])
    q, s = torch.empty_like(b["dyq"]), torch.empty_like(b["dys"])
    dprobs = torch.empty((shape.T, shape.k), dtype=torch.float32, device="cuda")
    ff8.ff8_permute_quant_dprobs(d["dy"], d["probs"], shape.k, shape.E, b["row_map"], b["offsets"], b["src_row"],
                                 q, s, b["y_perm"], dprobs)
    torch.cuda.synchronize()
    assert torch.equal(q[:m_pad], b["dyq"][:m_pad]) and torch.equal(s[:m_pad], b["dys"][:m_pad])
    t = np.sort(rng.choice(shape.T, size=64, replace=False))
    rows = run["row_map"][t]
    local = np.where(rows >= 0, np.arange(rows.size).reshape(rows.shape), -1)
    yp = f64(b["y_perm"].index_select(0, _cuda_idx(np.maximum(rows, 0).reshape(-1))))
    dy = f64(d["dy"].index_select(0, _cuda_idx(t)))
    want = moe.router_grad(dy, yp, local)
    mag = moe.router_grad(np.abs(dy), np.abs(yp), local)
    got = f64(dprobs.index_select(0, _cuda_idx(t)))
    assert np.all(np.abs(got - want) <= mag * 2.0 ** -16 + 1e-30), np.max(np.abs(got - want) / (mag + 1e-30))
    del q, s, dprobs


def test_unpermute_sampled_tokens(run):
    """F5 (routing-weighted) and B5 (plain) at sampled tokens: within one bf16 ulp of the
    float64 weighted sum of the GPU's own expert outputs."""
    shape, d, b, rng = run["shape"], run["d"], run["b"], run["rng"]
    t = np.sort(rng.choice(shape.T, size=64, replace=False))
    rows = run["row_map"][t]                                 # [64, k], -1 for dropped slots
    local = np.where(rows >= 0, np.arange(rows.size).reshape(rows.shape), -1)
    for src, out, w in (("y_perm", "y", _rows(d["probs"], t)), ("dx_perm", "dx", None)):
        yp = f64(b[src].index_select(0, _cuda_idx(np.maximum(rows, 0).reshape(-1))))
        want = moe.unpermute(yp, local, w)
        got = f64(b[out].index_select(0, _cuda_idx(t)))
        ulp = np.ldexp(1.0, np.frexp(np.maximum(np.abs(want), 1e-30))[1] - 8)
        assert np.all(np.abs(got - want) <= ulp + 1e-6), (out, np.max(np.abs(got - want) / ulp))


def test_sat_sampled_blocks(run):
    """B6: all four transposed tensors bit-exact, scales included, on 8 random whole 128-row
    stripes (every column tile) and the last stripe (partial with groups padded to 16)."""
    b, rng = run["b"], run["rng"]
    m_pad = int(run["off"][-1])
    n_rb = -(-m_pad // 128)
    stripes = sorted(set(rng.choice(n_rb, size=min(8, n_rb), replace=False).tolist()) | {n_rb - 1})
    for name in ("x", "h", "dy", "da"):
        q, s, qT, sT = b[name + "q"], b[name + "s"], b[name + "Tq"], b[name + "Ts"]
        for rb in stripes:
            r1 = min((rb + 1) * 128, m_pad)
            rs = slice(rb * 128, r1)
            wqT, wsT = sat.scaling_aware_transpose(host(q[rs]), host(s[rs]), r1 - rb * 128)
            assert np.array_equal(host(qT[rb])[:, :r1 - rb * 128], wqT), (name, rb)  # block rb's slab
            assert np.array_equal(host(sT[rb:rb + 1]).T, wsT), (name, rb)


def test_step_is_reproducible(run):
    """A second step on the same inputs writes bit-identical routing maps, FP8 tensors and
    outputs: every reduction (GEMM K order, tile amax, unpermute slot sum, routing ranks) has a
    fixed order.  Runs last in the module, since it re-runs the step in the buffers the other
    tests read (which it leaves identical when it passes)."""
    b, d, L = run["b"], run["d"], run["L"]
    names = ["row_map", "offsets", "xq", "xs", "a", "hq", "hs", "y_perm", "y", "dyq", "dh", "daq", "das", "dx",
             "dw1", "dw2"]
    first = {n: b[n].clone() for n in names}
    L.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    torch.cuda.synchronize()
    after = L.buf
    for n in names:
        assert torch.equal(first[n].view(torch.uint8), after[n].view(torch.uint8)), n

