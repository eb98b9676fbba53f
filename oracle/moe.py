"""Expert-layer steps of the FP8-Flow-MoE dataflow (oracle; test infrastructure only).

Paper section 3.2 (casting-free FP8 dataflow: permute -> grouped linear ->
activation -> grouped linear -> unpermute, with BF16 kept only at the output of
the first grouped linear and between the second grouped linear and the
combine) and section 3.3 (fused permute+padding, fused unpermute+unpadding,
fused SwiGLU+quantization).

Readings where the paper is silent:
  * padding multiple: by default every expert group is padded to a multiple of
    128 rows, which keeps every 128-row transpose block and every 128-token
    wgrad scale block inside one expert; `align` = 16 is the paper's padding
    (section 3.3.1), and then a 128-token block may hold tokens of two experts
    (wgrad sums each expert over exactly its own tokens, each scaled by the
    column scale of its 128-token block);
  * order inside a group: ascending token index (stable), one row per routed
    (token, slot) pair; a slot with expert id -1 is dropped (row_map = -1);
  * padding rows: bytes 0x00 with scale 2^-126 (an all-zero tile);
  * routing weights: multiplied in the unpermute (forward, float64 sum in slot
    order, one bf16 rounding) and into each copy of the upstream gradient
    before it is quantized (backward, float32 product as in the kernel); the
    gradient unpermute sums without weights;
  * fc1 output layout [gate | up]: the first I columns go through SiLU.

Row/column conventions (weights in [out, in] layout):
  fprop  out[m, n] = sum_k A[m, k] * W_e[n, k]
  dgrad  out[m, k] = sum_n G[m, n] * W_e[n, k]
  wgrad  dW[e, n, k] = sum_{m in group e} G[m, n] * X[m, k]
"""

import numpy as np

from .codec import bf16_round, e4m3_decode
from .quant import TILE, T_MIN, quant_rowwise, dequant_rowwise, dequant_block128, scale_from_exponent

ALIGN = 128


def rows_bound(T, k, E, align=ALIGN):
    """Upper bound on the padded row count, as a multiple of 128: every expert pads at
    most align - 1 rows."""
    return -(-(T * k + (align - 1) * E) // ALIGN) * ALIGN


def route(topk_idx, E, align=ALIGN):
    """Group the routed (token, slot) pairs by expert and pad each group to a multiple of
    `align` rows (128, or the paper's 16).

    Returns counts [E], offsets [E+1] (exclusive scan of the padded counts in
    expert order), row_map [T, k] (row of each pair, -1 if dropped) and
    src_row [offsets[E]] (t * k + j of each row, -1 for padding rows).
    """
    topk_idx = np.asarray(topk_idx, dtype=np.int64)
    T, k = topk_idx.shape
    counts = np.array([np.count_nonzero(topk_idx == e) for e in range(E)], dtype=np.int64)
    padded = -(-counts // align) * align
    offsets = np.concatenate([[0], np.cumsum(padded)]).astype(np.int64)
    row_map = np.full((T, k), -1, dtype=np.int64)
    src_row = np.full(int(offsets[-1]), -1, dtype=np.int64)
    for e in range(E):
        tt, jj = np.nonzero(topk_idx == e)  # row-major order: ascending t
        rows = offsets[e] + np.arange(tt.size)
        row_map[tt, jj] = rows
        src_row[rows] = tt * k + jj
    return counts, offsets, row_map, src_row


def permute_quant_rows(x, src_row, k, row_w=None):
    """Rows of the permuted, padded, 1x128-quantized tensor (fused permute+padding+quant).

    Row r with src_row[r] = t*k + j holds quant(X[t]) or, with routing weights,
    quant(w[t, j] * X[t]) where the product is taken in float32.  Padding rows
    are bytes 0x00 with scale 2^-126.
    """
    x = np.asarray(x, dtype=np.float32)
    src_row = np.asarray(src_row, dtype=np.int64)
    m_pad = src_row.size
    H = x.shape[1]
    q = np.zeros((m_pad, H), dtype=np.uint8)
    s = np.full((m_pad, H // TILE), scale_from_exponent(T_MIN), dtype=np.float32)
    real = np.nonzero(src_row >= 0)[0]
    t = src_row[real] // k
    j = src_row[real] % k
    vals = x[t]
    if row_w is not None:
        w = np.asarray(row_w, dtype=np.float32)[t, j]
        vals = (w[:, None] * vals).astype(np.float32)
    q[real], s[real] = quant_rowwise(vals)
    return q, s


def grouped_gemm_fprop(aq, a_s, wq, w_s, offsets):
    """out[m, n] = sum_k D(A)[m, k] * D(W_e)[n, k] for each expert group (float64)."""
    E = len(offsets) - 1
    A = dequant_rowwise(aq[: offsets[-1]], a_s[: offsets[-1]])
    out = np.zeros((offsets[-1], wq.shape[1]), dtype=np.float64)
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            out[r0:r1] = A[r0:r1] @ dequant_block128(wq[e], w_s[e]).T
    return out


def grouped_gemm_dgrad(gq, g_s, wq, w_s, offsets):
    """out[m, k] = sum_n D(G)[m, n] * D(W_e)[n, k] for each expert group (float64)."""
    E = len(offsets) - 1
    G = dequant_rowwise(gq[: offsets[-1]], g_s[: offsets[-1]])
    out = np.zeros((offsets[-1], wq.shape[2]), dtype=np.float64)
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            out[r0:r1] = G[r0:r1] @ dequant_block128(wq[e], w_s[e])
    return out


def grouped_gemm_wgrad(gTq, gT_s, xTq, xT_s, offsets):
    """dW[e, n, k] = sum_{m in group e} D(GT)[n, m] * D(XT)[k, m] (float64).

    gTq [N, rows] and xTq [K, rows] are column-wise scaled (stored transposed,
    scales [N, rows/128] and [K, rows/128]).  Experts without rows get zeros.
    """
    E = len(offsets) - 1
    m_pad = int(offsets[-1])
    nb = -(-m_pad // TILE)  # groups padded to 16 may end inside a 128-token block

    def dequant_cols(q, sc):
        return e4m3_decode(q[:, :m_pad]) * np.repeat(np.asarray(sc)[:, :nb].astype(np.float64), TILE, axis=1)[:, :m_pad]

    GT = dequant_cols(gTq, gT_s)
    XT = dequant_cols(xTq, xT_s)
    dw = np.zeros((E, gTq.shape[0], xTq.shape[0]), dtype=np.float64)
    for e in range(E):
        r0, r1 = offsets[e], offsets[e + 1]
        if r1 > r0:
            dw[e] = GT[:, r0:r1] @ XT[:, r0:r1].T
    return dw


def swiglu(a):
    """h = silu(g) * u with g = a[:, :I], u = a[:, I:] and silu(g) = g / (1 + exp(-g)) (float64)."""
    a = np.asarray(a, dtype=np.float64)
    I = a.shape[1] // 2
    g, u = a[:, :I], a[:, I:]
    return g / (1.0 + np.exp(-g)) * u


def swiglu_quant(a):
    """Fused SwiGLU + 1x128 quantization: the activation output goes straight to FP8 (section 3.3.2)."""
    return quant_rowwise(swiglu(a))


def swiglu_bwd(a, dh):
    """Gradient of h = silu(g) * u: with sig = 1/(1+exp(-g)),
    dg = dh * u * sig * (1 + g * (1 - sig)), du = dh * g * sig.  Returns [dg | du] (float64)."""
    a = np.asarray(a, dtype=np.float64)
    dh = np.asarray(dh, dtype=np.float64)
    I = a.shape[1] // 2
    g, u = a[:, :I], a[:, I:]
    sig = 1.0 / (1.0 + np.exp(-g))
    dg = dh * u * sig * (1.0 + g * (1.0 - sig))
    du = dh * g * sig
    return np.concatenate([dg, du], axis=1)


def swiglu_bwd_quant(a, dh):
    """Backward twin of the fused kernel: [dg | du] quantized 1x128."""
    return quant_rowwise(swiglu_bwd(a, dh))


def swiglu_quant_keep(a):
    """Fused SwiGLU + quantization that also keeps A, the fc1 output, as an FP8 checkpoint for
    the backward (section 4.2: activations saved for the backward are stored in FP8 rather
    than BF16).  Returns hq, hs and the 1x128 quantization aq, as of A itself."""
    hq, hs = swiglu_quant(a)
    aq, a_s = quant_rowwise(a)
    return hq, hs, aq, a_s


def swiglu_bwd_quant_from_checkpoint(aq, a_s, dh):
    """SwiGLU backward + quantization with A taken from its FP8 checkpoint: A = D(aq), exact."""
    return swiglu_bwd_quant(dequant_rowwise(aq, a_s), dh)


def router_grad(dy, y_perm, row_map):
    """Gradient of the routing weights through the weighted combine y[t] = sum_j w[t, j] *
    y_perm[row_map[t, j]]: dprobs[t, j] = <dy[t], y_perm[row_map[t, j]]> (float64), 0 for a
    dropped slot.  The combine's final bf16 rounding is taken as the identity."""
    dy = np.asarray(dy, dtype=np.float64)
    y_perm = np.asarray(y_perm, dtype=np.float64)
    row_map = np.asarray(row_map, dtype=np.int64)
    T, k = row_map.shape
    out = np.zeros((T, k), dtype=np.float64)
    for j in range(k):
        r = row_map[:, j]
        ok = r >= 0
        out[ok, j] = np.einsum("th,th->t", dy[ok], y_perm[r[ok]])
    return out


def unpermute(y_perm, row_map, row_w=None):
    """y[t] = sum_j w[t, j] * y_perm[row_map[t, j]] (float64, dropped slots skipped), then bf16 rounding."""
    y_perm = np.asarray(y_perm, dtype=np.float64)
    row_map = np.asarray(row_map, dtype=np.int64)
    T, k = row_map.shape
    y = np.zeros((T, y_perm.shape[1]), dtype=np.float64)
    for j in range(k):
        r = row_map[:, j]
        ok = r >= 0
        w = 1.0 if row_w is None else np.asarray(row_w, dtype=np.float64)[ok, j][:, None]
        y[ok] += w * y_perm[r[ok]]
    return bf16_round(y)
