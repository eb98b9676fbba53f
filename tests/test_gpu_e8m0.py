"""UE8M0 scale storage: the _e8m0 entry points against the float32-scale entry points and the
oracle's byte conversion.  The scale format changes only how the scale 2^T is stored (the byte
T + 127, paper section 2.1), so every FP8 byte, routing map and GEMM output must be bit-identical
to the float32 path, and every scale byte must be the oracle's conversion of the float32 scale
(GPU)."""

import numpy as np
import pytest
import torch

import workloads
from oracle import quant
from paper_2511_02302_amd import ff8
from paper_2511_02302_amd.layer import ExpertLayerFP8

from test_gpu_kernels import dev, host, poisoned

pytestmark = pytest.mark.gpu


def _bytes(s_f32):
    """The oracle's UE8M0 bytes of a float32 scale tensor (a device tensor)."""
    return quant.scale_to_e8m0(host(s_f32))


def test_quantizers_and_transpose_e8m0():
    """1x128 row quant (ragged row count), 128x128 block quant and the scaling-aware transpose
    (shifts over a wide exponent range, a last block cut at 16-row granularity): bytes equal the
    float32 path's, scale bytes equal the oracle's conversion of its scales."""
    x = workloads.outlier_activation(1000, 1024, seed=3, device="cuda")
    q, s = poisoned((1000, 1024), torch.uint8), poisoned((1000, 8), torch.float32)
    q8, s8 = poisoned((1000, 1024), torch.uint8), poisoned((1000, 8), torch.uint8)
    ff8.ff8_quant_rowwise(x, q, s)
    ff8.ff8_quant_rowwise(x, q8, s8)
    torch.cuda.synchronize()
    oq, os_ = quant.quant_rowwise(host(x.float()).astype(np.float64))
    assert np.array_equal(host(q8), oq) and np.array_equal(host(s8), quant.scale_to_e8m0(os_))
    assert torch.equal(q, q8) and np.array_equal(host(s8), _bytes(s))

    w = workloads.randn_bf16((3 * 128, 1024), 0.02, seed=4, device="cuda")
    wq, ws = poisoned((384, 1024), torch.uint8), poisoned((3, 8), torch.float32)
    wq8, ws8 = poisoned((384, 1024), torch.uint8), poisoned((3, 8), torch.uint8)
    ff8.ff8_quant_block128(w, wq, ws)
    ff8.ff8_quant_block128(w, wq8, ws8)
    torch.cuda.synchronize()
    assert torch.equal(wq, wq8) and np.array_equal(host(ws8), _bytes(ws))

    # transpose: row scales spread over 60 octaves, so many rows are shifted, some to zero
    R, C = 1024, 768
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 256, size=(R, C), dtype=np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0
    t = rng.integers(-40, 20, size=(R, C // 128))
    sf = torch.from_numpy(np.ldexp(np.float32(1), t).astype(np.float32)).cuda()
    sb = torch.from_numpy(quant.scale_to_e8m0(host(sf))).cuda()
    qd = dev(torch.from_numpy(codes))
    for rows_valid in (R, 1024 - 112):  # all rows; a last block cut after 16 of its rows
        off = torch.tensor([0, rows_valid], dtype=torch.int32, device="cuda")
        qT, sT = poisoned((R // 128, C, 128), torch.uint8), poisoned((R // 128, C), torch.float32)
        qT8, sT8 = poisoned((R // 128, C, 128), torch.uint8), poisoned((R // 128, C), torch.uint8)
        ff8.ff8_scaling_aware_transpose(qd, sf, qT, sT, off, 1)
        ff8.ff8_scaling_aware_transpose(qd, sb, qT8, sT8, off, 1)
        torch.cuda.synchronize()
        assert torch.equal(qT, qT8), rows_valid
        nb = -(-rows_valid // 128)
        assert np.array_equal(host(sT8[:nb]), _bytes(sT[:nb])), rows_valid


def test_gemms_e8m0_match_f32():
    """fprop, dgrad and wgrad with UE8M0 scales over a wide exponent range: outputs bit-identical
    to the float32-scale GEMMs (the MFMA receives the same E8M0 bytes either way).  The weight
    scales cover every byte position of the dgrad scale dwords."""
    E, N, K = 3, 1024, 1536
    rows = [512, 0, 300]
    off = np.concatenate([[0], np.cumsum([-(-r // 128) * 128 for r in rows])]).astype(np.int32)
    M_cap = int(off[-1]) + 256
    rng = np.random.default_rng(6)
    code = lambda shape: torch.from_numpy(rng.choice(np.r_[0:127, 128:255].astype(np.uint8), size=shape)).cuda()
    pow2 = lambda shape, lo, hi: torch.from_numpy(np.ldexp(np.float32(1), rng.integers(lo, hi, size=shape))
                                                  .astype(np.float32)).cuda()
    to8 = lambda s: torch.from_numpy(quant.scale_to_e8m0(host(s))).cuda()
    offd = dev(torch.from_numpy(off))
    a, a_s = code((M_cap, K)), pow2((M_cap, K // 128), -12, 4)
    w, w_s = code((E, N, K)), pow2((E, N // 128, K // 128), -14, 2)
    g, g_s = code((M_cap, N)), pow2((M_cap, N // 128), -12, 4)
    for fn, args, out_shape in (
            (ff8.ff8_grouped_gemm_fprop, (a, a_s, w, w_s), (M_cap, N)),
            (ff8.ff8_grouped_gemm_dgrad, (g, g_s, w, w_s), (M_cap, K))):
        o, o8 = poisoned(out_shape, torch.bfloat16), poisoned(out_shape, torch.bfloat16)
        fn(args[0], args[1], args[2], args[3], offd, o)
        fn(args[0], to8(args[1]), args[2], to8(args[3]), offd, o8)
        torch.cuda.synchronize()
        m_pad = int(off[-1])
        assert torch.equal(o[:m_pad].view(torch.int16), o8[:m_pad].view(torch.int16)), fn.__name__
    gT, gTs = code((M_cap // 128, N, 128)), pow2((M_cap // 128, N), -10, 6)  # K-blocked transposes
    xT, xTs = code((M_cap // 128, K, 128)), pow2((M_cap // 128, K), -10, 6)
    dw, dw8 = poisoned((E, N, K), torch.float32), poisoned((E, N, K), torch.float32)
    ff8.ff8_grouped_gemm_wgrad(gT, gTs, xT, xTs, offd, dw)
    ff8.ff8_grouped_gemm_wgrad(gT, to8(gTs), xT, to8(xTs), offd, dw8)
    torch.cuda.synchronize()
    assert torch.equal(dw.view(torch.int32), dw8.view(torch.int32))
    assert not bool(dw8[1].any())  # the expert without rows gets zeros


@pytest.mark.parametrize("case", ["uniform", "skewed_align16_fp8_checkpoint", "uniform_router_grad"])
def test_layer_step_e8m0_equals_f32(case):
    """The whole step (F0..B8) with every scale tensor in UE8M0 against the same step with
    float32 scales: every FP8 tensor, routing map and output (and the router gradient)
    bit-identical, every scale byte the oracle's conversion of the float32 scale."""
    rg = case == "uniform_router_grad"
    if case.startswith("uniform"):
        shape, align, ckpt = workloads.LayerShape("e8m0 T700 H1024 E8 k4 I512", 700, 1024, 8, 4, 512, "iid"), 128, False
    else:
        shape, align, ckpt = workloads.LayerShape("e8m0 skew T600 H512 E6 k2 I1024", 600, 512, 6, 2, 1024,
                                                  "zipf"), 16, True
    d = workloads.layer_inputs(shape, seed=7, device="cuda")
    args = (shape.T, shape.H, shape.E, shape.k, shape.I)
    L = ExpertLayerFP8(*args, align=align, fp8_checkpoint=ckpt, router_grad=rg)
    L8 = ExpertLayerFP8(*args, align=align, fp8_checkpoint=ckpt, router_grad=rg, scale_fmt="e8m0")
    for layer in (L, L8):
        layer.step(d["x"], d["topk_idx"], d["probs"], d["dy"], d["w1"], d["w2"])
    torch.cuda.synchronize()
    b, b8 = L.buf, L8.buf
    m_pad = int(b["offsets"][-1].item())
    nb = -(-m_pad // 128)
    same = ["row_map", "offsets", "w1q", "w2q", "y", "dx", "dw1", "dw2"] + (["dprobs"] if rg else [])
    rows = ["xq", "hq", "dyq", "daq", "a" if not ckpt else "aq", "dh", "dx_perm"]
    for n in same:
        assert torch.equal(b[n].view(torch.uint8), b8[n].view(torch.uint8)), n
    for n in rows:
        assert torch.equal(b[n][:m_pad].view(torch.uint8), b8[n][:m_pad].view(torch.uint8)), n
    for n in ("xT", "hT", "dyT", "daT"):
        kq, kq8 = b[n + "q"], b8[n + "q"]  # K-blocked: rows past m_pad in the last slab are untouched
        assert torch.equal(kq.permute(1, 0, 2).reshape(kq.shape[1], -1)[:, :m_pad],
                           kq8.permute(1, 0, 2).reshape(kq8.shape[1], -1)[:, :m_pad]), n
        assert np.array_equal(host(b8[n + "s"][:nb]), _bytes(b[n + "s"][:nb])), n
    for n in ("w1s", "w2s"):
        assert np.array_equal(host(b8[n]), _bytes(b[n])), n
    for n in ("xs", "hs", "dys", "das") + (("as",) if ckpt else ()):
        assert np.array_equal(host(b8[n][:m_pad]), _bytes(b[n][:m_pad])), n
    assert L8.saved_activation_bytes() < L.saved_activation_bytes()
