"""FP8-Flow-MoE expert layer, forward and backward, on one GPU.

The layer follows the casting-free dataflow of the paper (section 3.2): X and dY are
quantized once, inside the fused permute (the two explicit casts); the SwiGLU and its
backward twin emit FP8 directly; the weight-gradient GEMMs take column-wise operands
made by the scaling-aware transpose from the row-wise FP8 tensors already in memory.
BF16 stays only at the fc1 output (feeding the activation) and at the fc2 output
(feeding the combine in the forward and the dispatch in the backward).

Every step is one or more calls into libff8.so through the ctypes binding; torch
only provides device memory and the stream.

Memory is split the way a training step uses it:
  * per layer, for the whole step: the quantized weights, the weight gradients and the
    layer's outputs (Y, dX);
  * per layer, from its forward to its backward (`saved`): the routing maps and the
    activations the backward reads -- Xq and Hq (inputs of the weight gradients) and A,
    the fc1 output the SwiGLU backward reads;
  * step-local scratch (`Workspace`): buffers that live only inside one forward or one
    backward pass (dYq, dH, dAq, dX_perm, the transposed operands, ...), shared by every
    layer of a stack that runs its passes one layer at a time.
The saved state is allocated when the forward runs and, with backward(..., release=True),
released when the backward is done, so the memory a stack holds between its forward and
its backward is the sum of its layers' saved state.

With fp8_checkpoint=True A is kept as its 1x128 FP8 checkpoint, and the backward reads A
from it: the BF16 A then lives only between fc1 and the activation, in the shared scratch
(the paper stores the activations saved for the backward in FP8, section 4.2).

With router_grad=True the backward permute of dY also computes the routing weights'
gradient, dprobs[t, j] = <dY[t], Y_perm[row_map[t, j]]> (the backward of the weighted
combine), in the same pass over dY; Y_perm is then saved for the backward.

align=16 pads the expert groups to 16 rows, the paper's padding (section 3.3.1), instead
of 128.

scale_fmt="e8m0" stores every scale tensor as UE8M0 bytes (T + 127 for the scale 2^T; the
format section 2.1 names) instead of float32: a quarter of the scale bytes, and bit-identical
FP8 tensors and outputs.  It needs H and I to be multiples of 512.
"""

from dataclasses import dataclass

import torch

from . import ff8


@dataclass(frozen=True)
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
        of 2048."""
        need = ff8.ff8_rows_bound_aligned(self.T, self.k, self.E, self.align)
        return -(-need // 2048) * 2048


_u8, _f32, _bf16, _i32 = torch.uint8, torch.float32, torch.bfloat16, torch.int32
SCALE_DTYPES = {"f32": torch.float32, "e8m0": torch.uint8}


def _alloc(spec, device):
    return {n: torch.empty(shape, dtype=dt, device=device) for n, (shape, dt) in spec.items()}


def _nbytes(bufs):
    return sum(t.numel() * t.element_size() for t in bufs.values())


class Workspace:
    """Step-local scratch of one expert layer's forward and backward passes.  Any number of
    layers with the same dimensions and options may share one workspace, provided their
    passes run one at a time on one stream (a layer's pass leaves nothing in it that a
    later pass reads)."""

    def __init__(self, dims, device="cuda", fp8_checkpoint=False, router_grad=False, scale_fmt="f32"):
        self.d = d = dims
        self.fp8_checkpoint, self.router_grad, self.scale_fmt = fp8_checkpoint, router_grad, scale_fmt
        self.device = torch.device(device)
        M, H, I, T, k, E = d.m_cap, d.H, d.I, d.T, d.k, d.E
        sdt = SCALE_DTYPES[scale_fmt]
        spec = {"ws": ((max(1, ff8.ff8_permute_workspace_bytes(T, k, E)),), _u8)}
        if fp8_checkpoint:
            spec["a"] = ((M, 2 * I), _bf16)      # fc1 output, consumed by the activation only
        if not router_grad:
            spec["y_perm"] = ((M, H), _bf16)     # fc2 output, consumed by the combine only
        spec.update({
            "dyq": ((M, H), _u8), "dys": ((M, H // 128), sdt),
            "dh": ((M, I), _bf16),
            "daq": ((M, 2 * I), _u8), "das": ((M, 2 * I // 128), sdt),
            "dx_perm": ((M, H), _bf16),
        })
        for name, cols in (("x", H), ("h", I), ("dy", H), ("da", 2 * I)):
            spec[name + "Tq"] = ((M // 128, cols, 128), _u8)  # K-blocked transpose
            spec[name + "Ts"] = ((M // 128, cols), sdt)  # block-major column scales
        self.buf = _alloc(spec, self.device)

    def nbytes(self):
        return _nbytes(self.buf)


class ExpertLayerFP8:
    """Buffers and step sequence of one expert layer (E local experts, top-k routing)."""

    def __init__(self, T, H, E, k, I, device="cuda", fp8_checkpoint=False, router_grad=False, align=128,
                 workspace=None, scale_fmt="f32"):
        self.d = d = Dims(T, H, E, k, I, align)
        self.fp8_checkpoint = fp8_checkpoint
        self.router_grad = router_grad
        if scale_fmt not in SCALE_DTYPES:
            raise ValueError(f"scale_fmt must be one of {sorted(SCALE_DTYPES)}")
        if scale_fmt == "e8m0" and (H % 512 or I % 512):
            raise ValueError("UE8M0 scales need H and I multiples of 512")
        self.scale_fmt = scale_fmt
        sdt = SCALE_DTYPES[scale_fmt]
        self.device = dev = torch.device(device)
        self.M_cap = M = d.m_cap
        if workspace is None:
            workspace = Workspace(d, dev, fp8_checkpoint, router_grad, scale_fmt)
        elif (workspace.d != d or workspace.fp8_checkpoint != fp8_checkpoint
              or workspace.router_grad != router_grad or workspace.scale_fmt != scale_fmt):
            raise ValueError("the shared workspace was made for other dimensions or options")
        self.ws = workspace
        spec = {
            "w1q": ((E, 2 * I, H), _u8), "w1s": ((E, 2 * I // 128, H // 128), sdt),
            "w2q": ((E, H, I), _u8), "w2s": ((E, H // 128, I // 128), sdt),
            "y": ((T, H), _bf16), "dx": ((T, H), _bf16),
            "dw1": ((E, 2 * I, H), _f32), "dw2": ((E, H, I), _f32),
        }
        if router_grad:
            spec["dprobs"] = ((T, k), _f32)
        self.own = _alloc(spec, dev)
        self.saved = None
        saved = {
            "row_map": ((T, k), _i32), "offsets": ((E + 1,), _i32), "src_row": ((M,), _i32),
            "xq": ((M, H), _u8), "xs": ((M, H // 128), sdt),
            "hq": ((M, I), _u8), "hs": ((M, I // 128), sdt),
        }
        if fp8_checkpoint:
            saved.update({"aq": ((M, 2 * I), _u8), "as": ((M, 2 * I // 128), sdt)})
        else:
            saved["a"] = ((M, 2 * I), _bf16)
        if router_grad:
            saved["y_perm"] = ((M, H), _bf16)
        self._saved_spec = saved
        self.alloc_saved()

    # ---- buffers ----
    def alloc_saved(self):
        """Allocate the state the forward keeps for the backward (no-op if it exists)."""
        if self.saved is None:
            self.saved = _alloc(self._saved_spec, self.device)

    def release_saved(self):
        """Drop the state kept for the backward (its memory returns to torch's allocator)."""
        self.saved = None

    @property
    def buf(self):
        """Every buffer of the layer by name: its own, its saved state and the shared scratch."""
        out = dict(self.ws.buf)
        out.update(self.own)
        if self.saved is not None:
            out.update(self.saved)
        return out

    def saved_activation_bytes(self):
        """Bytes of the expert-path activations the forward keeps for the backward: the
        row-wise FP8 X and H (inputs of the weight gradients) and A (the SwiGLU backward's
        input), as BF16 or as its FP8 checkpoint.  Routing maps are not counted."""
        names = ["xq", "xs", "hq", "hs"] + (["aq", "as"] if self.fp8_checkpoint else ["a"])
        spec = self._saved_spec
        return sum(torch.Size(spec[n][0]).numel() * torch.empty((), dtype=spec[n][1]).element_size() for n in names)

    # ---- F0 ----
    def quantize_weights(self, w1, w2):
        b = self.own
        ff8.ff8_quant_block128(w1, b["w1q"], b["w1s"])
        ff8.ff8_quant_block128(w2, b["w2q"], b["w2s"])

    # ---- F1..F5 ----
    def forward(self, x, topk_idx, probs):
        self.alloc_saved()
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
    def backward(self, dy, probs, release=False):
        """B1..B8.  With release=True the saved state is dropped once the work is enqueued
        (torch's allocator keeps stream order, so the memory is reused only by later work)."""
        if self.saved is None:
            raise RuntimeError("backward without a forward: the saved state has been released")
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
        names = ("x", "h", "dy", "da")  # one launch for the four column-wise Wgrad operands
        ff8.ff8_scaling_aware_transpose_batch([b[n + "q"] for n in names], [b[n + "s"] for n in names],
                                              [b[n + "Tq"] for n in names], [b[n + "Ts"] for n in names], off, d.E)
        ff8.ff8_grouped_gemm_wgrad(b["dyTq"], b["dyTs"], b["hTq"], b["hTs"], off, b["dw2"])
        ff8.ff8_grouped_gemm_wgrad(b["daTq"], b["daTs"], b["xTq"], b["xTs"], off, b["dw1"])
        if release:
            self.release_saved()
        return b["dx"], b["dw1"], b["dw2"]

    def step(self, x, topk_idx, probs, dy, w1, w2):
        """One pass of the whole hot path: F0, F1..F5, B1..B8."""
        self.quantize_weights(w1, w2)
        self.forward(x, topk_idx, probs)
        return self.backward(dy, probs)
