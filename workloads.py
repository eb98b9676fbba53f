"""Seeded synthetic inputs for the FP8-Flow-MoE expert layer.

This module holds input generation only (random tensors, routing of random
logits); it holds none of the method's arithmetic.  Both the CPU oracle side
and the device side of the tests and of bench.py draw their inputs here, so
the two sides always see the same values.

Shapes follow the DeepSeek-V3 expert layer on one expert-parallel rank (32 of
256 experts) and a tiny layer for fast parity checks; the paper's own kernel
microbenchmarks also use simulated inputs at DeepSeek shapes (section 3.3).
Distributions: activations and upstream gradients N(0, 1), weights N(0, 0.02),
all rounded to bf16 (round-to-nearest-even, torch's conversion).

Routing recipes:
  * "iid"  : top-k of i.i.d. N(0, 1) logits over E experts; routing weights are
             the softmax over all E logits gathered at the chosen experts (not
             renormalized);
  * "zipf" : skewed popularity; expert e (at a seeded rank r_e in 1..E) gets logit
             ln(r_e^-1.2 / sum_r r^-1.2) + 0.4 * N(0, 1); top-k and weights as above.
"""

from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class LayerShape:
    name: str
    T: int        # tokens
    H: int        # hidden size
    E: int        # local experts
    k: int        # top-k
    I: int        # SwiGLU intermediate size
    routing: str  # "iid" or "zipf"


TINY = LayerShape("tiny T1024 H256 E8 k2 I512", 1024, 256, 8, 2, 512, "iid")
DSV3 = LayerShape("DeepSeek-V3 EP-share T16384 H7168 E32 k8 I2048", 16384, 7168, 32, 8, 2048, "iid")
SKEW = LayerShape("Zipf(1.2) skew T8192 H7168 E32 k8 I2048", 8192, 7168, 32, 8, 2048, "zipf")
# Standalone cast-op workload: one rank's 32768 x 7168 activation with outliers,
# and one 2048 x 7168 weight.
CAST_X = (32768, 7168)
CAST_W = (2048, 7168)


def _gen(seed, device):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def randn_bf16(shape, std=1.0, seed=0, device="cpu"):
    """N(0, std^2) rounded to bf16."""
    g = _gen(seed, device)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    return x.to(torch.bfloat16)


def outlier_activation(rows, cols, seed=0, device="cpu", frac=1e-3, factor=100.0):
    """N(0, 1) activation with a Bernoulli(frac) mask of entries multiplied by `factor`, in bf16."""
    g = _gen(seed, device)
    x = torch.randn((rows, cols), generator=g, device=device, dtype=torch.float32)
    mask = torch.rand((rows, cols), generator=g, device=device) < frac
    x = torch.where(mask, x * factor, x)
    return x.to(torch.bfloat16)


def routing(shape, seed=0, device="cpu"):
    """(topk_idx int32 [T, k], probs float32 [T, k]) for the shape's routing recipe.

    Always drawn on the CPU generator and then moved to `device`, so that the routing (and
    hence the expert populations a test or the benchmark relies on) is the same whichever
    device the other inputs are generated on."""
    g = _gen(seed + 1, "cpu")
    T, E, k = shape.T, shape.E, shape.k
    logits = torch.randn((T, E), generator=g, dtype=torch.float32)
    if shape.routing == "zipf":
        rank = torch.randperm(E, generator=g).to(torch.float32) + 1.0
        p = rank ** -1.2
        p = p / p.sum()
        logits = torch.log(p)[None, :] + 0.4 * logits
    probs_all = torch.softmax(logits, dim=1)
    _, idx = torch.topk(logits, k, dim=1)
    probs = torch.gather(probs_all, 1, idx)
    return idx.to(torch.int32).contiguous().to(device), probs.contiguous().to(device)


def layer_inputs(shape, seed=0, device="cpu", with_grad=True):
    """All inputs of one expert-layer forward+backward: X, routing, W1, W2, dY (bf16 / int32 / fp32)."""
    T, H, E, I = shape.T, shape.H, shape.E, shape.I
    idx, probs = routing(shape, seed, device)
    out = {
        "x": randn_bf16((T, H), 1.0, seed + 2, device),
        "topk_idx": idx,
        "probs": probs,
        "w1": randn_bf16((E, 2 * I, H), 0.02, seed + 3, device),
        "w2": randn_bf16((E, H, I), 0.02, seed + 4, device),
    }
    if with_grad:
        out["dy"] = randn_bf16((T, H), 1.0, seed + 5, device)
    return out


def expert_counts(topk_idx, E):
    """Tokens routed to each expert (for checking the skewed recipe's properties)."""
    idx = topk_idx.reshape(-1).to(torch.int64)
    idx = idx[idx >= 0]
    return torch.bincount(idx, minlength=E)


def skew_census(topk_idx, E):
    """Experts with no tokens, with 1..127 tokens (a partial 128-row tile) and with more than
    4000 tokens: the three populations the skewed-routing stress case must contain."""
    c = expert_counts(topk_idx, E).cpu()
    return {"zero": int((c == 0).sum()), "under_128": int(((c > 0) & (c < 128)).sum()),
            "over_4000": int((c > 4000).sum())}


def check_skew(topk_idx, E):
    """Raise unless the routing has every population of the skewed stress case (see skew_census)."""
    census = skew_census(topk_idx, E)
    missing = [k for k, v in census.items() if v < 1]
    if missing:
        raise AssertionError(f"skewed routing lacks experts of kind {missing}: {census}")
    return census
