"""The no-allocation permute entry point, ff8_permute_quant_noalloc, against the entry point it
varies, ff8_permute_quant_aligned with a caller-owned workspace: routing maps, offsets, padding
marks and quantized rows bit-exact, on two calls in a row, the second with a smaller input (the
library's own workspace still holds the first call's counts when the second runs) (GPU)."""

import pytest
import torch

import workloads
from paper_2511_02302_amd import ff8

pytestmark = pytest.mark.gpu

# (T, H, E, k, align, seed): a ragged token count spanning several 256-token routing chunks,
# then a smaller one with the paper's 16-row padding
CASES = [(3000, 512, 16, 4, 128, 0), (700, 256, 16, 2, 16, 1)]


def _buffers(T, H, E, k, M_cap):
    dev = "cuda"
    return {"row_map": torch.full((T, k), -7, dtype=torch.int32, device=dev),
            "offsets": torch.full((E + 1,), -7, dtype=torch.int32, device=dev),
            "src_row": torch.full((M_cap,), -7, dtype=torch.int32, device=dev),
            "q": torch.full((M_cap, H), 0xAB, dtype=torch.uint8, device=dev),
            "s": torch.full((M_cap, H // 128), -1.0, dtype=torch.float32, device=dev)}


def _compare(a, b, m_pad, what):
    for n in ("row_map", "offsets"):
        assert torch.equal(a[n], b[n]), (what, n)
    for n in ("src_row", "q", "s"):
        assert torch.equal(a[n][:m_pad], b[n][:m_pad]), (what, n)


def test_noalloc_permute_matches_workspace_permute_twice():
    for (T, H, E, k, align, seed) in CASES:
        print(f"noalloc permute: T={T} H={H} E={E} k={k} align={align}", flush=True)
        shape = workloads.LayerShape("noalloc case", T, H, E, k, 128, "iid")
        idx, probs = workloads.routing(shape, seed, device="cuda")
        x = workloads.randn_bf16((T, H), 1.0, seed + 2, device="cuda")
        dy = workloads.randn_bf16((T, H), 1.0, seed + 5, device="cuda")
        M_cap = ff8.ff8_rows_bound_aligned(T, k, E, align)
        ws = torch.empty(max(ff8.ff8_permute_workspace_bytes(T, k, E), 4), dtype=torch.uint8, device="cuda")
        ref, got = _buffers(T, H, E, k, M_cap), _buffers(T, H, E, k, M_cap)
        # forward: routing built from topk_idx
        ff8.ff8_permute_quant(x, None, k, E, idx, False, ref["row_map"], ref["offsets"], ref["src_row"], ref["q"],
                              ref["s"], ws, align=align)
        ff8.ff8_permute_quant_noalloc(x, None, k, E, idx, False, got["row_map"], got["offsets"], got["src_row"],
                                      got["q"], got["s"], align=align)
        torch.cuda.synchronize()
        m_pad = int(ref["offsets"][-1].item())
        assert m_pad >= T * k and m_pad % align == 0
        _compare(ref, got, m_pad, "forward")
        # backward: the forward's maps reused, routing-weighted copies of dY
        for b in (ref, got):
            b["q"].fill_(0xCD)
            b["s"].fill_(-2.0)
        ff8.ff8_permute_quant(dy, probs, k, E, None, True, ref["row_map"], ref["offsets"], ref["src_row"], ref["q"],
                              ref["s"])
        ff8.ff8_permute_quant_noalloc(dy, probs, k, E, None, True, got["row_map"], got["offsets"], got["src_row"],
                                      got["q"], got["s"], align=align)
        torch.cuda.synchronize()
        _compare(ref, got, m_pad, "backward")
        del ref, got, ws
