"""Benchmark of the FP8-Flow-MoE expert layer on one MI355X.

One step = one pass of the whole hot path: 128x128 weight quantization (F0), the
forward (F1 permute+quant, F2 fc1 fprop, F3 SwiGLU+quant, F4 fc2 fprop, F5 unpermute)
and the backward (B1 dY permute+quant, B2 fc2 dgrad, B3 SwiGLU backward+quant, B4 fc1
dgrad, B5 unpermute, B6 four scaling-aware transposes in one launch, B7/B8 wgrad), on the
DeepSeek-V3 expert layer of one expert-parallel rank: 16384 tokens, hidden 7168,
32 local experts, top-8 softmax routing, SwiGLU intermediate 2048.  Inputs are
synthetic (seeded), resident in HBM before timing starts.

Prints ONE JSON line.  `value` is the step's algorithmic GEMM FLOPs (18 M H I on the
routed rows, padding excluded) divided by the step time.  `roofline` is the dominant
kernel measured with HIP events on its launch stream inside the timed region;
`cast_ops` is the standalone 1x128 quantization and scaling-aware transpose of a
32768 x 7168 bf16 activation; `cpu_baseline` is the float64 CPU oracle timed on a
bounded sample of the same layer.
"""

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0      # MI355X dense FP8 MFMA
HBM_PEAK_GBS = 8000.0         # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_expert_layer_dsv3.md")
CSRC = os.path.join(ROOT, "paper_2511_02302_amd", "csrc")
# Kernel source each stage runs; the measured traffic of a stage is only reported while
# the hash of its source (and the shared device header) still matches the measurement.
STAGE_SOURCE = {"F0_weight_quant": "quant.hip", "F1_permute_quant": "permute.hip", "F2_fc1_fprop": "gemm.hip",
                "F3_swiglu_quant": "swiglu.hip", "F4_fc2_fprop": "gemm.hip", "F5_unpermute": "permute.hip",
                "B1_permute_quant_dy": "permute.hip", "B2_fc2_dgrad": "gemm.hip", "B3_swiglu_bwd_quant": "swiglu.hip",
                "B4_fc1_dgrad": "gemm.hip", "B5_unpermute": "permute.hip", "B6_sat_x4": "sat.hip",
                "B7_fc2_wgrad": "gemm.hip", "B8_fc1_wgrad": "gemm.hip"}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", choices=["dsv3", "skew", "tiny"], default="dsv3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cast-ops", action="store_true")
    ap.add_argument("--no-fp8-checkpoint", action="store_true")
    ap.add_argument("--no-router-grad", action="store_true")
    ap.add_argument("--no-align16", action="store_true")
    ap.add_argument("--no-hip-graph", action="store_true")
    ap.add_argument("--no-skew", action="store_true")
    ap.add_argument("--no-cast-accuracy", action="store_true")
    ap.add_argument("--no-e8m0", action="store_true")
    return ap.parse_args()


def stage_costs(shape, M):
    """Algorithmic FLOPs (GEMMs) and bytes (memory-bound steps) per stage, on the M routed rows."""
    T, H, E, k, I = shape.T, shape.H, shape.E, shape.k, shape.I
    sc = lambda n: 4 * n // 128  # one fp32 scale per 128 elements
    wq = 2 * I * H + H * I       # weight elements per expert (W1 + W2)
    c = {
        "F0_weight_quant": ("hbm", E * wq * 3 + sc(E * wq)),
        "F1_permute_quant": ("hbm", T * H * 2 + M * H + sc(M * H) + T * k * 4 * 3),
        "F2_fc1_fprop": ("mfma", 2 * M * H * 2 * I),
        "F3_swiglu_quant": ("hbm", M * 2 * I * 2 + M * I + sc(M * I)),
        "F4_fc2_fprop": ("mfma", 2 * M * I * H),
        "F5_unpermute": ("hbm", M * H * 2 + T * k * 8 + T * H * 2),
        "B1_permute_quant_dy": ("hbm", T * H * 2 + T * k * 8 + M * H + sc(M * H)),
        "B2_fc2_dgrad": ("mfma", 2 * M * H * I),
        "B3_swiglu_bwd_quant": ("hbm", M * 2 * I * 2 + M * I * 2 + M * 2 * I + sc(M * 2 * I)),
        "B4_fc1_dgrad": ("mfma", 2 * M * 2 * I * H),
        "B5_unpermute": ("hbm", M * H * 2 + T * k * 4 + T * H * 2),
        "B6_sat_x4": ("hbm", 2 * (M * (H + I + H + 2 * I) + sc(M * (H + I + H + 2 * I)))),
        "B7_fc2_wgrad": ("mfma", 2 * M * H * I),
        "B8_fc1_wgrad": ("mfma", 2 * M * 2 * I * H),
    }
    return c


def forward_only(costs, st_ms, shape):
    """The forward alone (F1..F5: permute+quant, fc1, SwiGLU+quant, fc2, unpermute), from the per-stage
    event times of the same timed steps; the weight quantization F0 is reported beside it."""
    fwd = ["F1_permute_quant", "F2_fc1_fprop", "F3_swiglu_quant", "F4_fc2_fprop", "F5_unpermute"]
    ms = sum(st_ms[n] for n in fwd)
    flops = sum(costs[n][1] for n in fwd if costs[n][0] == "mfma")
    tf = flops / (ms * 1e-3) / 1e12
    return {"workload": f"{shape.name} expert-layer forward F1..F5", "ms": round(ms, 4), "TFLOP/s": round(tf, 1),
            "frac_mfma": round(tf / FP8_PEAK_TFLOPS, 4), "ms_with_weight_quant": round(ms + st_ms["F0_weight_quant"], 4)}


class StageTimer:
    """HIP events recorded on the launch stream between stages."""

    def __init__(self, torch, names, steps):
        self.torch = torch
        self.names = names
        self.ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in names]
                   for _ in range(steps)]

    def ms(self):
        out = {n: [] for n in self.names}
        for row in self.ev:
            for n, (a, b) in zip(self.names, row):
                out[n].append(a.elapsed_time(b))
        return {n: sum(v) / len(v) for n, v in out.items()}


def run_step(L, d, ev=None, ckpt=None, dprobs=None):
    """One full step; `ev` is a list of (start, end) event pairs, one per stage.  With `ckpt`
    (buffers "aq", "as"), F3 also writes the FP8 checkpoint of A and B3 reads A from it; with
    `dprobs` (a [T, k] float32 buffer), B1 also computes the router gradient."""
    from paper_2511_02302_amd import ff8

    b, dm = L.buf, L.d
    off = b["offsets"]
    if ckpt is None:
        f3 = lambda: ff8.ff8_swiglu_quant(b["a"], b["hq"], b["hs"], off, dm.E)
        b3 = lambda: ff8.ff8_swiglu_bwd_quant(b["a"], b["dh"], b["daq"], b["das"], off, dm.E)
    else:
        f3 = lambda: ff8.ff8_swiglu_quant_keep_fp8(b["a"], b["hq"], b["hs"], ckpt["aq"], ckpt["as"], off, dm.E)
        b3 = lambda: ff8.ff8_swiglu_bwd_quant_fp8a(ckpt["aq"], ckpt["as"], b["dh"], b["daq"], b["das"], off, dm.E)
    if dprobs is None:
        b1 = lambda: ff8.ff8_permute_quant(d["dy"], d["probs"], dm.k, dm.E, None, True, b["row_map"], off,
                                           b["src_row"], b["dyq"], b["dys"])
    else:
        b1 = lambda: ff8.ff8_permute_quant_dprobs(d["dy"], d["probs"], dm.k, dm.E, b["row_map"], off, b["src_row"],
                                                  b["dyq"], b["dys"], b["y_perm"], dprobs)
    stages = [
        lambda: L.quantize_weights(d["w1"], d["w2"]),
        lambda: ff8.ff8_permute_quant(d["x"], None, dm.k, dm.E, d["topk_idx"], False, b["row_map"], off,
                                      b["src_row"], b["xq"], b["xs"], b["ws"],
                                      align=None if dm.align == 128 else dm.align),
        lambda: ff8.ff8_grouped_gemm_fprop(b["xq"], b["xs"], b["w1q"], b["w1s"], off, b["a"]),
        f3,
        lambda: ff8.ff8_grouped_gemm_fprop(b["hq"], b["hs"], b["w2q"], b["w2s"], off, b["y_perm"]),
        lambda: ff8.ff8_unpermute(b["y_perm"], b["row_map"], d["probs"], b["y"]),
        b1,
        lambda: ff8.ff8_grouped_gemm_dgrad(b["dyq"], b["dys"], b["w2q"], b["w2s"], off, b["dh"]),
        b3,
        lambda: ff8.ff8_grouped_gemm_dgrad(b["daq"], b["das"], b["w1q"], b["w1s"], off, b["dx_perm"]),
        lambda: ff8.ff8_unpermute(b["dx_perm"], b["row_map"], None, b["dx"]),
        lambda: ff8.ff8_scaling_aware_transpose_batch(*[[b[n + sfx] for n in ("x", "h", "dy", "da")]
                                                        for sfx in ("q", "s", "Tq", "Ts")], off, dm.E),
        lambda: ff8.ff8_grouped_gemm_wgrad(b["dyTq"], b["dyTs"], b["hTq"], b["hTs"], off, b["dw2"]),
        lambda: ff8.ff8_grouped_gemm_wgrad(b["daTq"], b["daTs"], b["xTq"], b["xTs"], off, b["dw1"]),
    ]
    for i, fn in enumerate(stages):
        if ev is not None:
            ev[i][0].record()
        fn()
        if ev is not None:
            ev[i][1].record()


def fp8_checkpoint(torch, L, d, shape, M, steps, warmup, ms_bf16_a):
    """The step with A kept as an FP8 checkpoint (F3 writes it, B3 reads it), and the bytes of
    activations the forward keeps for the backward under three recipes (M_cap-row buffers):
    all BF16 (permuted X, A, H), FP8-Flow with BF16 A, FP8-Flow with the FP8 checkpoint."""
    Mc, H, I = L.M_cap, shape.H, shape.I
    ck = {"aq": torch.empty((Mc, 2 * I), dtype=torch.uint8, device="cuda"),
          "as": torch.empty((Mc, 2 * I // 128), dtype=torch.float32, device="cuda")}
    for _ in range(warmup):
        run_step(L, d, ckpt=ck)
    torch.cuda.synchronize()
    names = list(stage_costs(shape, M))
    timer = StageTimer(torch, names, steps)
    t0 = time.perf_counter()
    for i in range(steps):
        run_step(L, d, timer.ev[i], ckpt=ck)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    st = timer.ms()
    sc = lambda n: 4 * n // 128
    f3_bytes = M * 2 * I * 2 + M * I + sc(M * I) + M * 2 * I + sc(M * 2 * I)
    b3_bytes = M * 2 * I + sc(M * 2 * I) + M * I * 2 + M * 2 * I + sc(M * 2 * I)
    out = {}
    for name, stage, by in (("F3_swiglu_quant_keep_fp8", "F3_swiglu_quant", f3_bytes),
                            ("B3_swiglu_bwd_quant_fp8a", "B3_swiglu_bwd_quant", b3_bytes)):
        gbs = by / (st[stage] * 1e-3) / 1e9
        out[name] = {"ms": round(st[stage], 4), "GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 3)}
    fp8_xh = Mc * H + sc(Mc * H) + Mc * I + sc(Mc * I)
    saved = {"bf16_recipe": Mc * (H + 2 * I + I) * 2, "fp8_flow_bf16_a": fp8_xh + Mc * 2 * I * 2,
             "fp8_flow_fp8_checkpoint": fp8_xh + Mc * 2 * I + sc(Mc * 2 * I)}
    assert saved["fp8_flow_bf16_a"] == L.saved_activation_bytes()  # the layer's own buffers
    out.update({"ms_per_step": round(ms_step, 4), "ms_per_step_bf16_a": round(ms_bf16_a, 4),
                "saved_activation_bytes": saved,
                "saving_vs_bf16_a": round(1 - saved["fp8_flow_fp8_checkpoint"] / saved["fp8_flow_bf16_a"], 4),
                "saving_vs_bf16_recipe": round(1 - saved["fp8_flow_fp8_checkpoint"] / saved["bf16_recipe"], 4)})
    del ck
    return out


def checkpoint_memory(torch, shape, d, n_layers=2):
    """Measured memory of the activations a stack of n_layers expert layers keeps between its
    forwards and its backwards, with A kept in BF16 and as its FP8 checkpoint.  The layers
    share one step-local workspace; each layer's saved state is allocated by its forward and
    released by its backward.  `kept_per_layer` is torch's allocated bytes after the last
    forward minus before the first, over n_layers; `peak_above_base` is the allocator's peak
    over the whole forward+backward sequence (the workspace and the weights are allocated
    before, so they are not in it); `kept_requested_per_layer` counts the tensors' own bytes
    (the allocator's requested-bytes statistic, without its block rounding)."""
    from paper_2511_02302_amd.layer import ExpertLayerFP8, Workspace

    out = {"layers": n_layers}
    args = (shape.T, shape.H, shape.E, shape.k, shape.I)
    for key, ckpt in (("bf16_a", False), ("fp8_checkpoint", True)):
        ws = Workspace(ExpertLayerFP8(*args, fp8_checkpoint=ckpt).d, fp8_checkpoint=ckpt)
        layers = [ExpertLayerFP8(*args, fp8_checkpoint=ckpt, workspace=ws) for _ in range(n_layers)]
        for L in layers:
            L.quantize_weights(d["w1"], d["w2"])
            L.release_saved()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        stats = torch.cuda.memory_stats
        base, base_req = torch.cuda.memory_allocated(), stats()["requested_bytes.all.current"]
        torch.cuda.reset_peak_memory_stats()
        x = d["x"]
        for L in layers:
            x = L.forward(x, d["topk_idx"], d["probs"])
        torch.cuda.synchronize()
        kept, kept_req = torch.cuda.memory_allocated() - base, stats()["requested_bytes.all.current"] - base_req
        g = d["dy"]
        for L in reversed(layers):
            g, _, _ = L.backward(g, d["probs"], release=True)
        torch.cuda.synchronize()
        out[key] = {"kept_per_layer": kept // n_layers, "kept_requested_per_layer": kept_req // n_layers,
                    "peak_above_base": torch.cuda.max_memory_allocated() - base,
                    "accounted_per_layer": layers[0].saved_activation_bytes(), "workspace_bytes": ws.nbytes()}
        del layers, ws, x, g
        torch.cuda.empty_cache()
    out["measured_saving_per_layer"] = out["bf16_a"]["kept_per_layer"] - out["fp8_checkpoint"]["kept_per_layer"]
    out["measured_saving_frac"] = round(out["measured_saving_per_layer"] / out["bf16_a"]["kept_per_layer"], 4)
    return out


def router_grad(torch, L, d, shape, M, steps, warmup, ms_base, b1_base_ms):
    """The step with B1 fused with the router gradient dprobs[t, j] = <dY[t], Y_perm[row]>: its
    step time and B1's time and rate.  The fused B1 additionally reads the k rows of Y_perm of
    every token (the dot products) and writes dprobs."""
    T, H, k = shape.T, shape.H, shape.k
    dp = torch.empty((T, k), dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        run_step(L, d, dprobs=dp)
    torch.cuda.synchronize()
    names = list(stage_costs(shape, M))
    timer = StageTimer(torch, names, steps)
    t0 = time.perf_counter()
    for i in range(steps):
        run_step(L, d, timer.ev[i], dprobs=dp)
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    st = timer.ms()
    by = stage_costs(shape, M)["B1_permute_quant_dy"][1] + M * H * 2 + T * k * 4
    gbs = by / (st["B1_permute_quant_dy"] * 1e-3) / 1e9
    del dp
    return {"B1_permute_quant_dprobs": {"ms": round(st["B1_permute_quant_dy"], 4), "GB/s": round(gbs, 1),
                                        "frac_hbm": round(gbs / HBM_PEAK_GBS, 3), "bytes": by},
            "B1_without_dprobs_ms": round(b1_base_ms, 4),
            "ms_per_step": round(ms_step, 4), "ms_per_step_without": round(ms_base, 4)}


def align16(torch, d, shape, M, steps, warmup, ms_base):
    """The step with the expert groups padded to 16 rows (the paper's padding) instead of 128:
    fewer padding rows, 128-row blocks shared by neighbouring experts (partial K blocks in
    wgrad).  A separate layer object (its M_cap differs)."""
    from paper_2511_02302_amd.layer import ExpertLayerFP8

    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, align=16)
    for _ in range(warmup):
        run_step(L, d)
    torch.cuda.synchronize()
    names = list(stage_costs(shape, M))
    timer = StageTimer(torch, names, steps)
    t0 = time.perf_counter()
    for i in range(steps):
        run_step(L, d, timer.ev[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    st = timer.ms()
    m_pad = int(L.buf["offsets"][-1].item())
    costs = stage_costs(shape, M)
    gemm_flops = sum(v for kind, v in costs.values() if kind == "mfma")
    out = {"ms_per_step": round(ms_step, 4), "ms_per_step_align128": round(ms_base, 4),
           "value": round(gemm_flops / (ms_step * 1e-3) / 1e12, 2), "padded_rows": m_pad, "routed_rows": M,
           "stages_ms": {n: round(st[n], 4) for n in names}}
    del L
    torch.cuda.empty_cache()
    return out


def stage_table(costs, st_ms):
    """Per-stage time and rate against the stage's roofline (FP8 MFMA or HBM)."""
    out = {}
    for n, (kind, amount) in costs.items():
        t = st_ms[n]
        if kind == "mfma":
            ach = amount / (t * 1e-3) / 1e12
            out[n] = {"ms": round(t, 4), "TFLOP/s": round(ach, 1), "frac_mfma": round(ach / FP8_PEAK_TFLOPS, 3)}
        else:
            ach = amount / (t * 1e-3) / 1e9
            out[n] = {"ms": round(t, 4), "GB/s": round(ach, 1), "frac_hbm": round(ach / HBM_PEAK_GBS, 3)}
    return out


def timed_steps(torch, L, d, names, steps, warmup, **kw):
    """Warm-up steps, then `steps` timed steps: (wall ms per step, per-stage event ms)."""
    for _ in range(warmup):
        run_step(L, d, **kw)
    torch.cuda.synchronize()
    timer = StageTimer(torch, names, steps)
    t0 = time.perf_counter()
    for i in range(steps):
        run_step(L, d, timer.ev[i], **kw)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps, timer.ms()


def skew(torch, steps, warmup):
    """The Zipf(1.2)-skewed layer (8192 tokens, the DeepSeek-V3 widths): ragged groups with empty
    experts, experts under one 128-row tile and experts over 4000 tokens, asserted on the very
    routing the GPU runs.  Step time, GEMM rate on the real rows, and every stage's rate."""
    import workloads
    from paper_2511_02302_amd.layer import ExpertLayerFP8

    shape = workloads.SKEW
    d = workloads.layer_inputs(shape, seed=0, device="cuda")
    census = workloads.check_skew(d["topk_idx"], shape.E)
    counts = workloads.expert_counts(d["topk_idx"], shape.E).cpu()
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I)
    M = int(counts.sum())
    costs = stage_costs(shape, M)
    names = list(costs)
    ms_step, st = timed_steps(torch, L, d, names, steps, warmup)
    gemm_flops = sum(v for kind, v in costs.values() if kind == "mfma")
    gemm_ms = sum(st[n] for n in names if costs[n][0] == "mfma")
    out = {"workload": shape.name, "routed_rows": M, "padded_rows": int(L.buf["offsets"][-1].item()),
           "expert_tokens_min_max": [int(counts.min()), int(counts.max())], "populations": census,
           "ms_per_step": round(ms_step, 4), "value": round(gemm_flops / (ms_step * 1e-3) / 1e12, 2),
           "unit": "TFLOP/s", "frac_mfma_step": round(gemm_flops / (ms_step * 1e-3) / 1e12 / FP8_PEAK_TFLOPS, 4),
           "gemm_only": {"TFLOP/s": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 1),
                         "frac_mfma": round(gemm_flops / (gemm_ms * 1e-3) / 1e12 / FP8_PEAK_TFLOPS, 4),
                         "ms": round(gemm_ms, 3)},
           "stages": stage_table(costs, st)}
    del L, d
    torch.cuda.empty_cache()
    return out


def cast_accuracy(torch):
    """Conversion error on the cast-op activation (32768 x 7168 bf16 N(0,1), 0.1% x100 outliers),
    every FP8 tensor made by the library's kernels (section 3.1, Eq. 1 and the exponent-shift
    identity): relative to D(Q_row X), the extra error of the scaling-aware transpose, of the
    naive power-of-two chain N1 (dequantize -> bf16 transpose -> requantize, the library's
    baseline kernels), and of the naive fp32-scale chain N2 (s = amax/448 quantization applied
    twice through a bf16 intermediate, written here with plain torch ops since it is the
    comparison recipe, not part of the path), plus the single-quantization errors.  The error
    norms themselves are computed with torch reductions."""
    import workloads
    from paper_2511_02302_amd import ff8

    R, C = workloads.CAST_X
    x = workloads.outlier_activation(R, C, seed=0, device="cuda")
    f8 = torch.float8_e4m3fn
    dec = lambda q: q.view(f8).float()  # exact decode of e4m3 bytes
    rep = lambda s: s.repeat_interleave(128, dim=1)
    q, s = torch.empty((R, C), dtype=torch.uint8, device="cuda"), torch.empty((R, C // 128), device="cuda")
    ff8.ff8_quant_rowwise(x, q, s)
    d_row = dec(q) * rep(s)                                   # D(Q_row X), [R, C]
    d_rowT = d_row.t().contiguous()
    del d_row
    qK, sT = torch.empty((R // 128, C, 128), dtype=torch.uint8, device="cuda"), torch.empty((R // 128, C), device="cuda")
    ff8.ff8_scaling_aware_transpose(q, s, qK, sT)
    qT = qK.permute(1, 0, 2).reshape(C, R)                   # the K-blocked transpose as [C, R]
    del qK
    xT = x.float().t().contiguous()

    def rel(a, b):
        return float(torch.linalg.vector_norm(a - b) / torch.linalg.vector_norm(b))

    out = {"workload": f"bf16 activation {R}x{C} N(0,1) with 0.1% x100 outliers, seed 0"}
    d_sat = dec(qT) * rep(sT.t().contiguous())                # D(SAT(Q_row X)), [C, R]
    changed = d_sat != d_rowT
    out["sat_extra_rel_err"] = rel(d_sat, d_rowT)
    out["sat_elements_changed_frac"] = float(changed.float().mean())
    del d_sat, changed
    tmp = torch.empty((R, C), dtype=torch.bfloat16, device="cuda")
    tmpT = torch.empty((C, R), dtype=torch.bfloat16, device="cuda")
    qn, sn = torch.empty((C, R), dtype=torch.uint8, device="cuda"), torch.empty((C, R // 128), device="cuda")
    ff8.ff8_baseline_dequant_rowwise(q, s, tmp)
    ff8.ff8_baseline_transpose_bf16(tmp, tmpT)
    ff8.ff8_quant_rowwise(tmpT, qn, sn)
    out["naive_pow2_N1_extra_rel_err"] = rel(dec(qn) * rep(sn), d_rowT)
    del tmp, tmpT, qn, sn
    out["row_quant_rel_err_vs_x"] = rel(d_rowT, xT)
    # direct column-wise quantization of X (the error a column-wise operand should carry)
    xTb = x.t().contiguous()
    qc, sc = torch.empty((C, R), dtype=torch.uint8, device="cuda"), torch.empty((C, R // 128), device="cuda")
    ff8.ff8_quant_rowwise(xTb, qc, sc)
    out["col_quant_rel_err_vs_x"] = rel(dec(qc) * rep(sc), xT)
    del qc, sc, xTb, d_rowT

    def q_fp32(v):  # 1x128 tiles, s = amax / 448 in fp32, RNE, saturating
        t = v.reshape(v.shape[0], -1, 128)
        sc = t.abs().amax(dim=2, keepdim=True) / 448.0
        sc = torch.where(sc == 0, torch.ones_like(sc), sc)
        return ((t / sc).clamp(-448.0, 448.0).to(f8).float() * sc).reshape(v.shape)

    d1 = q_fp32(x.float()).to(torch.bfloat16).float()         # N2 step 1, through bf16
    d1T = d1.t().contiguous()
    del d1
    d2 = q_fp32(d1T)                                          # N2 step 2, column-wise
    out["naive_fp32_N2_extra_rel_err"] = rel(d2, d1T)
    out["naive_fp32_N2_total_rel_err_vs_x"] = rel(d2, xT)
    out["fp32_single_quant_rel_err_vs_x"] = rel(d1T, xT)
    del d1T, d2, xT, x, q, s, qT, sT
    torch.cuda.empty_cache()
    return out


def e8m0_scales(torch, d, shape, M, steps, warmup, ms_base, st_base):
    """The step with every scale tensor stored as UE8M0 bytes (T + 127) instead of float32: step
    time, each stage's time against the float32-scale step, and the scale bytes of the step's
    tensors in both formats (every FP8 byte and output is bit-identical; the GPU tests check)."""
    from paper_2511_02302_amd.layer import ExpertLayerFP8

    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I, scale_fmt="e8m0")
    names = list(stage_costs(shape, M))
    ms_step, st = timed_steps(torch, L, d, names, steps, warmup)
    scale_names = [n for n, t in L.buf.items() if n.endswith("s") and n not in ("ws",) and t.dtype == torch.uint8]
    bytes8 = sum(L.buf[n].numel() for n in scale_names)
    out = {"ms_per_step": round(ms_step, 4), "ms_per_step_f32_scales": round(ms_base, 4),
           "scale_tensors": sorted(scale_names), "scale_bytes": bytes8, "scale_bytes_f32": 4 * bytes8,
           "stage_ms": {n: round(st[n], 4) for n in names},
           "stage_change_vs_f32": {n: round(st[n] / st_base[n] - 1.0, 4) for n in names}}
    gemm = [n for n in names if stage_costs(shape, M)[n][0] == "mfma"]
    out["gemm_ms"] = round(sum(st[n] for n in gemm), 4)
    out["gemm_ms_f32_scales"] = round(sum(st_base[n] for n in gemm), 4)
    del L
    torch.cuda.empty_cache()
    return out


def hip_graph(torch, L, d, steps, warmup, ms_eager, gemm_flops):
    """The whole step captured once as a HIP graph and replayed.  The path makes no host
    synchronization, allocation or memset, so one replay launches every kernel of the step
    (the replays' outputs are checked against the eager step in the GPU tests)."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run_step(L, d)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run_step(L, d)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        graph.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    del graph
    return {"ms_per_step": round(ms, 4), "TFLOP/s": round(gemm_flops / (ms * 1e-3) / 1e12, 2),
            "ms_per_step_eager": round(ms_eager, 4)}


def cast_ops(torch, reps=20):
    """1x128 quantization and scaling-aware transpose of a 32768 x 7168 bf16 activation (0.1% x100 outliers),
    plus the naive dequantize -> bf16 transpose -> requantize chain and the 2048 x 7168 weight block quant.

    Every timed call takes the next of several input/output sets whose total exceeds twice the 256 MB
    MALL, so that the rates are HBM rates, not last-level-cache rates (the weight block quant, 44 MB, is
    the exception and says so)."""
    import workloads
    from paper_2511_02302_amd import ff8

    R, C = workloads.CAST_X
    n_sets = 3  # 3 x (470 MB bf16 + 235 MB fp8 + 235 MB transposed) per rotation
    x0 = workloads.outlier_activation(R, C, seed=0, device="cuda")
    xs = [x0] + [x0.clone() for _ in range(n_sets - 1)]
    qs = [torch.empty((R, C), dtype=torch.uint8, device="cuda") for _ in range(n_sets)]
    ss = [torch.empty((R, C // 128), dtype=torch.float32, device="cuda") for _ in range(n_sets)]
    qTs = [torch.empty((R // 128, C, 128), dtype=torch.uint8, device="cuda") for _ in range(n_sets)]
    sTs = [torch.empty((R // 128, C), dtype=torch.float32, device="cuda") for _ in range(n_sets)]
    for i in range(n_sets):
        ff8.ff8_quant_rowwise(xs[i], qs[i], ss[i])
    d = torch.empty((R, C), dtype=torch.bfloat16, device="cuda")
    dT = torch.empty((C, R), dtype=torch.bfloat16, device="cuda")
    qn = torch.empty((C, R), dtype=torch.uint8, device="cuda")
    sn = torch.empty((C, R // 128), dtype=torch.float32, device="cuda")
    wr, wc = workloads.CAST_W
    w = workloads.randn_bf16((wr, wc), 0.02, seed=1, device="cuda")
    wq = torch.empty((wr, wc), dtype=torch.uint8, device="cuda")
    ws = torch.empty((wr // 128, wc // 128), dtype=torch.float32, device="cuda")
    cp_src = [torch.empty(R * C * 2 // 16 * 16, dtype=torch.uint8, device="cuda") for _ in range(2)]
    cp_dst = [torch.empty_like(cp_src[0]) for _ in range(2)]
    rot = [0]

    def nxt(k):
        rot[0] += 1
        return rot[0] % k

    def timeit(fn):
        for _ in range(3):
            fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in evs:
            i = nxt(n_sets)
            a.record()
            fn(i)
            b.record()
        torch.cuda.synchronize()
        t = sorted(a.elapsed_time(b) for a, b in evs)
        return t[len(t) // 2]

    def warm(fn):
        return lambda i=0: fn(i)

    out = {}
    n = R * C
    quant_bytes = n * 2 + n + n // 128 * 4
    sat_bytes = 2 * (n + n // 128 * 4)
    t_q = timeit(warm(lambda i: ff8.ff8_quant_rowwise(xs[i], qs[i], ss[i])))
    t_sat = timeit(warm(lambda i: ff8.ff8_scaling_aware_transpose(qs[i], ss[i], qTs[i], sTs[i])))

    def naive(i):
        ff8.ff8_baseline_dequant_rowwise(qs[i], ss[i], d)
        ff8.ff8_baseline_transpose_bf16(d, dT)
        ff8.ff8_quant_rowwise(dT, qn, sn)

    t_naive = timeit(warm(naive))
    t_w = timeit(warm(lambda i: ff8.ff8_quant_block128(w, wq, ws)))
    t_cp = timeit(warm(lambda i: ff8.ff8_baseline_copy(cp_src[i % 2], cp_dst[i % 2])))
    cp_bytes = 2 * cp_src[0].numel()
    for name, t, by in (("quant_rowwise_1x128", t_q, quant_bytes), ("scaling_aware_transpose", t_sat, sat_bytes),
                        ("naive_dequant_transpose_requant", t_naive, sat_bytes),
                        ("weight_quant_128x128_cache_resident", t_w, wr * wc * 3 + wr * wc // 16384 * 4),
                        ("copy_reference", t_cp, cp_bytes)):
        gbs = by / (t * 1e-3) / 1e9
        out[name] = {"ms": round(t, 4), "GB/s": round(gbs, 1), "frac_hbm": round(gbs / HBM_PEAK_GBS, 3),
                     "bytes": by}
    out["sat_speedup_vs_naive"] = round(t_naive / t_sat, 2)
    out["workload"] = (f"bf16 activation {R}x{C} N(0,1) with 0.1% x100 outliers ({n_sets} rotating input/output "
                       f"sets, beyond the MALL); weight {wr}x{wc} N(0,0.02)")
    return out


def source_hash(stage):
    import hashlib
    h = hashlib.sha256()
    for f in (STAGE_SOURCE[stage], "ff8_device.hpp"):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(stage):
    """HBM bytes per launch of `stage` from the committed rocprofv3 counter summary.

    The summary lists, per stage, FETCH_SIZE and WRITE_SIZE already scaled by the
    copy-kernel calibration, and the source hash of the kernel when they were taken.
    Returns None when there is no measurement or the kernel source has changed since.
    """
    try:
        with open(TRAFFIC_FILE) as fh:
            text = fh.read()
    except OSError:
        return None
    for m in re.finditer(r"^traffic (\S+) (\S+) fetch_bytes=(\d+) write_bytes=(\d+)$", text, re.M):
        name, digest, fetch, write = m.group(1), m.group(2), int(m.group(3)), int(m.group(4))
        if name == stage:
            return fetch + write if digest == source_hash(stage) else None
    return None


def oracle_full_tiny(seed=0):
    """The float64 oracle on the whole tiny layer (1024 tokens, hidden 256, 8 experts, top-2,
    intermediate 512): F0 and every step of the forward and backward, timed per phase."""
    import numpy as np
    import workloads
    from oracle import layer as olayer

    shape = workloads.TINY
    inp = workloads.layer_inputs(shape, seed=seed)
    f = lambda t: t.float().numpy().astype(np.float64)
    t0 = time.perf_counter()
    w = olayer.quantize_weights(f(inp["w1"]), f(inp["w2"]))
    t1 = time.perf_counter()
    st = olayer.forward(f(inp["x"]), inp["topk_idx"].numpy(), inp["probs"].numpy(), w["w1q"], w["w1s"], w["w2q"],
                        w["w2s"], shape.E)
    t2 = time.perf_counter()
    olayer.backward(st, f(inp["dy"]), inp["probs"].numpy(), w["w1q"], w["w1s"], w["w2q"], w["w2s"])
    t3 = time.perf_counter()
    flops = olayer.gemm_flops(st["counts"], shape.H, shape.I)["total"]
    return {"workload": shape.name, "seconds": {"F0": round(t1 - t0, 3), "forward": round(t2 - t1, 3),
                                                "backward": round(t3 - t2, 3), "total": round(t3 - t0, 3)},
            "TFLOP/s": round(flops / (t3 - t0) / 1e12, 7)}


def cpu_baseline(shape, rows=2048, seed=0):
    """The float64 oracle, as it stands, on a bounded sample of the workload.

    Sample: expert 0 of the layer -- its 128x128 weight quantization (F0 for one
    expert) and `rows` routed tokens of it (six 128-row groups) through F1..B8.  The full step
    runs F0 once per expert and the row work once per 128 routed rows, so the oracle's
    time for the full step is E * t(F0 sample) + (M / rows) * t(rows sample); `value`
    is the step's GEMM FLOPs over that time (the same unit as the GPU figure).
    """
    import numpy as np
    import workloads
    from oracle import layer as olayer

    sample = workloads.LayerShape("one-expert sample", rows, shape.H, 1, 1, shape.I, "iid")
    inp = workloads.layer_inputs(sample, seed=seed)
    f = lambda t: t.float().numpy().astype(np.float64)
    t0 = time.perf_counter()
    w = olayer.quantize_weights(f(inp["w1"]), f(inp["w2"]))
    t1 = time.perf_counter()
    st = olayer.forward(f(inp["x"]), inp["topk_idx"].numpy(), inp["probs"].numpy(), w["w1q"], w["w1s"], w["w2q"],
                        w["w2s"], 1)
    olayer.backward(st, f(inp["dy"]), inp["probs"].numpy(), w["w1q"], w["w1s"], w["w2q"], w["w2s"])
    t2 = time.perf_counter()
    M = shape.T * shape.k
    full_s = shape.E * (t1 - t0) + (M / rows) * (t2 - t1)
    flops = 18 * M * shape.H * shape.I
    cores = len(os.sched_getaffinity(0))
    return {"value": round(flops / full_s / 1e12, 7), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "full_tiny_layer": oracle_full_tiny(seed),
            "sample": f"expert 0 only: F0 on its W1 [{2 * shape.I}x{shape.H}] and W2 [{shape.H}x{shape.I}] "
                      f"({t1 - t0:.1f} s), F1..B8 on {rows} of its routed rows ({t2 - t1:.1f} s); "
                      f"scaled to the full step as {shape.E} x F0 + {M / rows:.1f} x rows = {full_s:.0f} s",
            "sample_seconds": round(t2 - t0, 1)}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only (single-GPU build); "
                                   f"--gpus {args.gpus} is not supported"}))
        sys.exit(2)
    import torch
    import workloads
    from paper_2511_02302_amd.layer import ExpertLayerFP8

    shape = {"dsv3": workloads.DSV3, "skew": workloads.SKEW, "tiny": workloads.TINY}[args.workload]
    torch.cuda.set_device(0)
    d = workloads.layer_inputs(shape, seed=0, device="cuda")
    census = workloads.check_skew(d["topk_idx"], shape.E) if shape.routing == "zipf" else None
    L = ExpertLayerFP8(shape.T, shape.H, shape.E, shape.k, shape.I)
    counts = workloads.expert_counts(d["topk_idx"], shape.E)
    M = int(counts.sum())
    costs = stage_costs(shape, M)
    names = list(costs)

    for _ in range(args.warmup):
        run_step(L, d)
    torch.cuda.synchronize()
    timer = StageTimer(torch, names, args.steps)
    t0 = time.perf_counter()
    for i in range(args.steps):
        run_step(L, d, timer.ev[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    st_ms = timer.ms()

    gemm_flops = sum(v for kind, v in costs.values() if kind == "mfma")
    value = gemm_flops / (ms_step * 1e-3) / 1e12
    stages = {}
    for n in names:
        kind, amount = costs[n]
        t = st_ms[n]
        if kind == "mfma":
            ach = amount / (t * 1e-3) / 1e12
            stages[n] = {"ms": round(t, 4), "TFLOP/s": round(ach, 1), "frac_mfma": round(ach / FP8_PEAK_TFLOPS, 3)}
        else:
            ach = amount / (t * 1e-3) / 1e9
            stages[n] = {"ms": round(t, 4), "GB/s": round(ach, 1), "frac_hbm": round(ach / HBM_PEAK_GBS, 3)}
    gemm_ms = sum(st_ms[n] for n in names if costs[n][0] == "mfma")
    dom = max(names, key=lambda n: st_ms[n])
    kind, amount = costs[dom]
    if kind == "mfma":
        ach = amount / (st_ms[dom] * 1e-3) / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(ach, 1), "peak": FP8_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / FP8_PEAK_TFLOPS, 4), "traffic": measured_traffic(dom),
                "per_launch": {"flops": amount, "avg_ms": round(st_ms[dom], 4)}}
    else:
        ach = amount / (st_ms[dom] * 1e-3) / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": measured_traffic(dom),
                "per_launch": {"bytes": amount, "avg_ms": round(st_ms[dom], 4)}}

    rec = {
        "metric": "FP8 MoE expert fwd+bwd TFLOP/s (% MFMA peak); quant/transpose GB/s (% HBM)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3",
        "data": "synthetic",
        "config": {"workload": f"{shape.name} expert layer, fwd+bwd incl. 128x128 weight quant", "tokens": shape.T,
                   "hidden": shape.H, "experts": shape.E, "top_k": shape.k, "intermediate": shape.I,
                   "routed_rows": M, "routing": shape.routing, **({"populations": census} if census else {})},
        "frac_mfma_step": round(value / FP8_PEAK_TFLOPS, 4),
        "gemm_only": {"TFLOP/s": round(gemm_flops / (gemm_ms * 1e-3) / 1e12, 1),
                      "frac_mfma": round(gemm_flops / (gemm_ms * 1e-3) / 1e12 / FP8_PEAK_TFLOPS, 4),
                      "ms": round(gemm_ms, 3)},
        "roofline": roof,
        "stages": stages,
        "forward_only": forward_only(costs, st_ms, shape),
    }
    if not args.no_fp8_checkpoint:
        rec["fp8_checkpoint"] = fp8_checkpoint(torch, L, d, shape, M, args.steps, args.warmup, ms_step)
    if not args.no_router_grad:
        rec["router_grad"] = router_grad(torch, L, d, shape, M, args.steps, args.warmup, ms_step,
                                         st_ms["B1_permute_quant_dy"])
    if not args.no_align16:
        rec["align16"] = align16(torch, d, shape, M, args.steps, args.warmup, ms_step)
    if not args.no_hip_graph:
        rec["hip_graph"] = hip_graph(torch, L, d, args.steps, args.warmup, ms_step, gemm_flops)
    if not args.no_fp8_checkpoint:
        rec["fp8_checkpoint"]["measured_memory"] = checkpoint_memory(torch, shape, d)
    if not args.no_e8m0 and shape.H % 512 == 0 and shape.I % 512 == 0:
        rec["e8m0_scales"] = e8m0_scales(torch, d, shape, M, args.steps, args.warmup, ms_step, st_ms)
    if not args.no_cast_ops or not args.no_skew or not args.no_cast_accuracy:
        del L, d
        torch.cuda.empty_cache()
    if not args.no_skew and args.workload != "skew":
        rec["skew"] = skew(torch, args.steps, args.warmup)
    if not args.no_cast_ops:
        rec["cast_ops"] = cast_ops(torch)
    if not args.no_cast_accuracy:
        rec["cast_accuracy"] = cast_accuracy(torch)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(shape)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
