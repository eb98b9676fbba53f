"""The whole FP8-Flow-MoE expert layer, forward and backward, stage by stage (oracle; test infrastructure only).

Paper section 3.2: inputs and upstream gradients stay FP8 along the expert path;
BF16 is kept only (1) at the output of the first grouped linear, which feeds the
activation, and (2) at the output of the second grouped linear, which feeds the
combine (forward) and the dispatch (backward).  The only explicit casts are the
entry quantization of X (fused into the permute) and of the upstream gradient
dY; everything else is quantized inside the producing step.  Column-wise
operands for the weight gradients come from the scaling-aware transpose.

Steps (names used by the tests and the benchmark):
  F0 weight 128x128 quantization          F1 permute + quantize X
  F2 fc1 fprop -> A (bf16)                F3 SwiGLU + quantize -> Hq
  F4 fc2 fprop -> Y_perm (bf16)           F5 unpermute with routing weights -> Y (bf16)
  B1 permute + quantize w * dY            B2 fc2 dgrad -> dH (bf16)
  B3 SwiGLU backward + quantize -> dAq    B4 fc1 dgrad -> dX_perm (bf16)
  B5 unpermute without weights -> dX      B6 scaling-aware transpose of Xq, Hq, dYq, dAq
  B7 fc2 wgrad -> dW2 (fp32)              B8 fc1 wgrad -> dW1 (fp32)

GEMM outputs that the dataflow keeps in BF16 are rounded to bf16 here as well,
so that the next stage sees the same kind of operand as on the device.

fp8_checkpoint=True keeps A for the backward as its 1x128 FP8 quantization (the
activations saved for the backward stored in FP8, section 4.2): F3 also returns
aq, as, and B3 takes A = D(aq).  router_grad=True adds the routing weights' gradient
dprobs (the backward of the weighted combine) to the backward's outputs.
"""

import numpy as np

from .codec import bf16_round
from .quant import quant_block128
from .sat import scaling_aware_transpose
from . import moe


def quantize_weights(w1, w2):
    """F0: 128x128 block quantization of W1 [E, 2I, H] and W2 [E, H, I]."""
    E = w1.shape[0]
    out = {}
    for name, w in (("w1", w1), ("w2", w2)):
        qs = [quant_block128(w[e]) for e in range(E)]
        out[name + "q"] = np.stack([q for q, _ in qs])
        out[name + "s"] = np.stack([s for _, s in qs])
    return out


def forward(x, topk_idx, probs, w1q, w1s, w2q, w2s, E, fp8_checkpoint=False, align=moe.ALIGN):
    """F1..F5 (expert groups padded to `align` rows).  Returns a dict of every intermediate."""
    T, k = topk_idx.shape
    st = {}
    counts, offsets, row_map, src_row = moe.route(topk_idx, E, align)
    st.update(counts=counts, offsets=offsets, row_map=row_map, src_row=src_row)
    st["xq"], st["xs"] = moe.permute_quant_rows(x, src_row, k)
    st["a"] = bf16_round(moe.grouped_gemm_fprop(st["xq"], st["xs"], w1q, w1s, offsets))
    if fp8_checkpoint:
        st["hq"], st["hs"], st["aq"], st["as"] = moe.swiglu_quant_keep(st["a"])
    else:
        st["hq"], st["hs"] = moe.swiglu_quant(st["a"])
    st["y_perm"] = bf16_round(moe.grouped_gemm_fprop(st["hq"], st["hs"], w2q, w2s, offsets))
    st["y"] = moe.unpermute(st["y_perm"], row_map, probs)
    return st


def backward(st, dy, probs, w1q, w1s, w2q, w2s, router_grad=False):
    """B1..B8 given the forward state.  Returns a dict of every intermediate."""
    k = st["row_map"].shape[1]
    offsets = st["offsets"]
    bw = {}
    bw["dyq"], bw["dys"] = moe.permute_quant_rows(dy, st["src_row"], k, row_w=probs)
    if router_grad:
        bw["dprobs"] = moe.router_grad(dy, st["y_perm"], st["row_map"])
    bw["dh"] = bf16_round(moe.grouped_gemm_dgrad(bw["dyq"], bw["dys"], w2q, w2s, offsets))
    if "aq" in st:
        bw["daq"], bw["das"] = moe.swiglu_bwd_quant_from_checkpoint(st["aq"], st["as"], bw["dh"])
    else:
        bw["daq"], bw["das"] = moe.swiglu_bwd_quant(st["a"], bw["dh"])
    bw["dx_perm"] = bf16_round(moe.grouped_gemm_dgrad(bw["daq"], bw["das"], w1q, w1s, offsets))
    bw["dx"] = moe.unpermute(bw["dx_perm"], st["row_map"], None)
    for name, (q, s) in (("x", (st["xq"], st["xs"])), ("h", (st["hq"], st["hs"])),
                         ("dy", (bw["dyq"], bw["dys"])), ("da", (bw["daq"], bw["das"]))):
        bw[name + "Tq"], bw[name + "Ts"] = scaling_aware_transpose(q, s)
    bw["dw2"] = moe.grouped_gemm_wgrad(bw["dyTq"], bw["dyTs"], bw["hTq"], bw["hTs"], offsets)
    bw["dw1"] = moe.grouped_gemm_wgrad(bw["daTq"], bw["daTs"], bw["xTq"], bw["xTs"], offsets)
    return bw


def gemm_flops(counts, H, I):
    """Algorithmic GEMM FLOPs of forward+backward on the real (unpadded) rows: 6 GEMMs, 18*M*H*I in total."""
    M = int(np.sum(counts))
    fwd = 2 * M * H * (2 * I) + 2 * M * I * H
    return {"fwd": fwd, "bwd": 2 * fwd, "total": 3 * fwd}
