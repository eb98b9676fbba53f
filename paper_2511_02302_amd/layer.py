"""FP8-Flow-MoE expert layer, forward and backward, on one GPU.

The layer follows the casting-free dataflow of the paper (section 3.2): X and dY are
quantized once, inside the fused permute (the two explicit casts); the SwiGLU and its
backward twin emit FP8 directly; the weight-gradient GEMMs take column-wise operands
made by the scaling-aware transpose from the row-wise FP8 tensors already in memory.
BF16 stays only at the fc1 output (feeding the activation) and at the fc2 output
(feeding the combine in the forward and the dispatch in the backward).

Every step is one or more calls into libff8.so through the ctypes binding; torch
only provides device memory (all buffers are allocated once, in __init__) and the
stream.

With fp8_checkpoint=True the forward also keeps A, the fc1 output, as a 1x128 FP8
checkpoint, and the backward reads A from it: the BF16 A is then only needed between
fc1 and the activation (the paper stores the activations saved for the backward in
FP8, section 4.2).

With router_grad=True the backward permute of dY also computes the routing weights'
gradient, dprobs[t, j] = <dY[t], Y_perm[row_map[t, j]]> (the backward of the weighted
combine), in the same pass over dY.

align=16 pads the expert groups to 16 rows, the paper's padding (section 3.3.1), instead
of 128.
"""

from dataclasses import dataclass

import torch

from . import ff8


@dataclass
class Dims:
    T: int
    H: int
    E: int
    k: int
    I: int
    align: int = 128

    @property
    def m_cap(self):
        """Rows of the grouped buffers: the smallest admissible count, rounded up to a multiple
        of 2048.  M_cap is also the row stride of the transposed operands, and strides that
        are only a multiple of 512 bytes (131584 at the DeepSeek-V3 share with 16-row
        padding) measured 17% slower in the transpose than multiples of 2048."""
        need = ff8.ff8_rows_bound_aligned(self.T, self.k, self.E, self.align)
        return -(-need // 2048) * 2048


def _empty(shape, dtype, device):
    return torch.empty(shape, dtype=dtype, device=device)


class ExpertLayerFP8:
    """Buffers and step sequence of one expert layer (E local experts, top-k routing)."""

    def __init__(self, T, H, E, k, I, device="cuda", fp8_checkpoint=False, router_grad=False, align=128):
        self.d = d = Dims(T, H, E, k, I, align)
        self.fp8_checkpoint = fp8_checkpoint
        self.router_grad = router_grad
        self.device = dev = torch.device(device)
        M = self.M_cap = d.m_cap
        u8, f32, bf16, i32 = torch.uint8, torch.float32, torch.bfloat16, torch.int32
        b = self.buf = {}
        # weights (F0 outputs)
        b["w1q"] = _empty((E, 2 * I, H), u8, dev)
        b["w1s"] = _empty((E, 2 * I // 128, H // 128), f32, dev)
        b["w2q"] = _empty((E, H, I), u8, dev)
        b["w2s"] = _empty((E, H // 128, I // 128), f32, dev)
        # routing
        b["row_map"] = _empty((T, k), i32, dev)
        b["offsets"] = _empty((E + 1,), i32, dev)
        b["src_row"] = _empty((M,), i32, dev)
        b["ws"] = _empty((max(1, ff8.ff8_permute_workspace_bytes(T, k, E)),), u8, dev)
        # forward
        b["xq"] = _empty((M, H), u8, dev)
        b["xs"] = _empty((M, H // 128), f32, dev)
        b["a"] = _empty((M, 2 * I), bf16, dev)
        b["hq"] = _empty((M, I), u8, dev)
        b["hs"] = _empty((M, I // 128), f32, dev)
        if fp8_checkpoint:
            b["aq"] = _empty((M, 2 * I), u8, dev)
            b["as"] = _empty((M, 2 * I // 128), f32, dev)
        b["y_perm"] = _empty((M, H), bf16, dev)
        b["y"] = _empty((T, H), bf16, dev)
        # backward
        b["dyq"] = _empty((M, H), u8, dev)
        b["dys"] = _empty((M, H // 128), f32, dev)
        b["dh"] = _empty((M, I), bf16, dev)
        b["daq"] = _empty((M, 2 * I), u8, dev)
        b["das"] = _empty((M, 2 * I // 128), f32, dev)
        b["dx_perm"] = _empty((M, H), bf16, dev)
        b["dx"] = _empty((T, H), bf16, dev)
        if router_grad:
            b["dprobs"] = _empty((T, k), f32, dev)
        for name, cols in (("x", H), ("h", I), ("dy", H), ("da", 2 * I)):
            b[name + "Tq"] = _empty((cols, M), u8, dev)
            b[name + "Ts"] = _empty((M // 128, cols), f32, dev)  # block-major column scales
        b["dw1"] = _empty((E, 2 * I, H), f32, dev)
        b["dw2"] = _empty((E, H, I), f32, dev)

    # ---- F0 ----
    def quantize_weights(self, w1, w2):
        b = self.buf
        ff8.ff8_quant_block128(w1, b["w1q"], b["w1s"])
        ff8.ff8_quant_block128(w2, b["w2q"], b["w2s"])

    # ---- F1..F5 ----
    def forward(self, x, topk_idx, probs):
        b, d = self.buf, self.d
        ff8.ff8_permute_quant(x, None, d.k, d.E, topk_idx, False, b["row_map"], b["offsets"], b["src_row"],
                              b["xq"], b["xs"], b["ws"], align=None if d.align == 128 else d.align)
        ff8.ff8_grouped_gemm_fprop(b["xq"], b["xs"], b["w1q"], b["w1s"], b["offsets"], b["a"])
        if self.fp8_checkpoint:
            ff8.ff8_swiglu_quant_keep_fp8(b["a"], b["hq"], b["hs"], b["aq"], b["as"], b["offsets"], d.E)
        else:
            ff8.ff8_swiglu_quant(b["a"], b["hq"], b["hs"], b["offsets"], d.E)
        ff8.ff8_grouped_gemm_fprop(b["hq"], b["hs"], b["w2q"], b["w2s"], b["offsets"], b["y_perm"])
        ff8.ff8_unpermute(b["y_perm"], b["row_map"], probs, b["y"])
        return b["y"]

    # ---- B1..B8 ----
    def backward(self, dy, probs):
        b, d = self.buf, self.d
        off = b["offsets"]
        if self.router_grad:
            ff8.ff8_permute_quant_dprobs(dy, probs, d.k, d.E, b["row_map"], off, b["src_row"], b["dyq"], b["dys"],
                                         b["y_perm"], b["dprobs"])
        else:
            ff8.ff8_permute_quant(dy, probs, d.k, d.E, None, True, b["row_map"], off, b["src_row"], b["dyq"],
                                  b["dys"])
        ff8.ff8_grouped_gemm_dgrad(b["dyq"], b["dys"], b["w2q"], b["w2s"], off, b["dh"])
        if self.fp8_checkpoint:
            ff8.ff8_swiglu_bwd_quant_fp8a(b["aq"], b["as"], b["dh"], b["daq"], b["das"], off, d.E)
        else:
            ff8.ff8_swiglu_bwd_quant(b["a"], b["dh"], b["daq"], b["das"], off, d.E)
        ff8.ff8_grouped_gemm_dgrad(b["daq"], b["das"], b["w1q"], b["w1s"], off, b["dx_perm"])
        ff8.ff8_unpermute(b["dx_perm"], b["row_map"], None, b["dx"])
        for name in ("x", "h", "dy", "da"):
            ff8.ff8_scaling_aware_transpose(b[name + "q"], b[name + "s"], b[name + "Tq"], b[name + "Ts"], off, d.E)
        ff8.ff8_grouped_gemm_wgrad(b["dyTq"], b["dyTs"], b["hTq"], b["hTs"], off, b["dw2"])
        ff8.ff8_grouped_gemm_wgrad(b["daTq"], b["daTs"], b["xTq"], b["xTs"], off, b["dw1"])
        return b["dx"], b["dw1"], b["dw2"]

    def saved_activation_bytes(self):
        """Bytes of the expert-path activations the forward keeps for the backward: the
        row-wise FP8 X and H (inputs of the weight gradients) and A (the SwiGLU backward's
        input), as BF16 or as its FP8 checkpoint.  Routing maps are not counted."""
        b = self.buf
        names = ["xq", "xs", "hq", "hs"] + (["aq", "as"] if self.fp8_checkpoint else ["a"])
        return sum(b[n].numel() * b[n].element_size() for n in names)

    def step(self, x, topk_idx, probs, dy, w1, w2):
        """One pass of the whole hot path: F0, F1..F5, B1..B8."""
        self.quantize_weights(w1, w2)
        self.forward(x, topk_idx, probs)
        return self.backward(dy, probs)
