"""Pin of the oracle's whole-layer wiring (CPU only).

The FP8 layer must track an unquantized float64 layer computed by torch
autograd (a library): every output and gradient within a few per cent, the
size of e4m3 rounding.  A transposed operand, a wrong routing weight or a
swapped gate/up half would give errors of order one.
"""

import numpy as np
import torch

import workloads
from oracle import layer


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


def test_tiny_layer_against_unquantized_autograd():
    shape = workloads.LayerShape("t", 256, 256, 4, 2, 256, "iid")
    inp = workloads.layer_inputs(shape, seed=0)
    np_in = {k: v.float().numpy() if v.is_floating_point() else v.numpy() for k, v in inp.items()}
    wq = layer.quantize_weights(np_in["w1"], np_in["w2"])
    st = layer.forward(np_in["x"], np_in["topk_idx"], np_in["probs"], wq["w1q"], wq["w1s"], wq["w2q"], wq["w2s"], shape.E)
    bw = layer.backward(st, np_in["dy"], np_in["probs"], wq["w1q"], wq["w1s"], wq["w2q"], wq["w2s"])

    # unquantized float64 reference with autograd
    x = torch.from_numpy(np_in["x"]).double().requires_grad_(True)
    w1 = torch.from_numpy(np_in["w1"]).double().requires_grad_(True)
    w2 = torch.from_numpy(np_in["w2"]).double().requires_grad_(True)
    idx = torch.from_numpy(np_in["topk_idx"]).long()
    p = torch.from_numpy(np_in["probs"]).double()
    y = torch.zeros_like(x)
    I = shape.I
    for j in range(shape.k):
        for e in range(shape.E):
            sel = idx[:, j] == e
            if sel.any():
                a = x[sel] @ w1[e].T
                h = torch.nn.functional.silu(a[:, :I]) * a[:, I:]
                y = y.index_add(0, torch.nonzero(sel)[:, 0], p[sel, j:j + 1] * (h @ w2[e].T))
    y.backward(torch.from_numpy(np_in["dy"]).double())

    assert _rel(st["y"], y.detach().numpy()) < 0.08
    assert _rel(bw["dx"], x.grad.numpy()) < 0.08
    assert _rel(bw["dw1"], w1.grad.numpy()) < 0.08
    assert _rel(bw["dw2"], w2.grad.numpy()) < 0.08
    flops = layer.gemm_flops(st["counts"], shape.H, shape.I)
    assert flops["total"] == 18 * shape.T * shape.k * shape.H * shape.I
