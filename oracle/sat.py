"""Scaling-aware FP8 transpose and the naive conversion it replaces (oracle; test infrastructure only).

Paper section 3.1, Algorithm 1 (scaling-aware FP8 transpose), read together with
the exponent-shift identity that precedes it and the commented draft of the
algorithm that follows it in the source:

  for every block of 128 rows x 128 columns of a row-wise (1x128) scaled tensor,
    S_max = the largest of the 128 row scales of the block;
    every element of row i is re-expressed at scale S_max by lowering its
    exponent by k_i = log2(S_max / S_row[i]) (an integer >= 0, because all
    scales are powers of two);
    the output is stored transposed, and every output row (an input column)
    of the block gets the scale S_max for that 128-row segment.

The printed line "k = log2(S_max)/S" is read as k = log2(S_max / S_row[i]), as in
the draft.  The identity only holds while the lowered exponent stays >= 1; the
paper excludes underflow without saying what happens there.  Reading: the
element is re-encoded exactly as the value dec(b) * 2^-k, rounded to nearest
even into the e4m3 subnormals (or zero), sign kept.  Overflow cannot happen
because k >= 0.

Layout: input q [rows, cols] with s [rows, cols/128]; output qT [cols, rows]
with sT [cols, rows/128] (column-wise 128x1 scaling of the original tensor).
"""

import numpy as np

from .codec import e4m3_decode, e4m3_encode, bf16_round
from .quant import TILE, exponent_of_scale, scale_from_exponent, quant_rowwise, dequant_rowwise


def scaling_aware_transpose(q, s, n_rows=None):
    """Algorithm 1 on the first n_rows rows (default all rows).

    Blocks are 128 consecutive rows.  When n_rows is not a multiple of 128 the last block
    is partial: its S_max is taken over the rows it has (a group padded to 16 rows ends
    inside a block).  Returns (qT uint8 [cols, n_rows], sT float32 [cols, ceil(n_rows/128)]).
    """
    q = np.asarray(q)
    rows, cols = q.shape
    n = rows if n_rows is None else int(n_rows)
    assert cols % TILE == 0 and n <= rows
    nb = -(-n // TILE)
    t_row = np.full((nb * TILE, cols // TILE), np.iinfo(np.int64).min // 2, dtype=np.int64)
    t_row[:n] = exponent_of_scale(np.asarray(s)[:n])        # [n, cols/128]; missing rows never win the max
    blocks = t_row.reshape(nb, TILE, cols // TILE)
    t_max = blocks.max(axis=1)                               # [nb, cols/128]: log2 S_max
    k = (t_max[:, None, :] - blocks).reshape(nb * TILE, cols // TILE)[:n]  # k_i >= 0 per row and column tile
    k_elem = np.repeat(k, TILE, axis=1)                      # [n, cols]
    shifted = e4m3_encode(e4m3_decode(q[:n]) * np.ldexp(1.0, -k_elem))
    qT = np.ascontiguousarray(shifted.T)
    sT = np.repeat(scale_from_exponent(t_max).T, TILE, axis=0)  # [cols, nb]
    return qT, np.ascontiguousarray(sT)


def requant_forced_scale(values, t_forced):
    """Quantize exact values at a given (forced) exponent: encode(values * 2^-t).

    Used as an independent cross-check of Algorithm 1: re-quantizing the exact
    dequantized values at the block scale S_max must give the same bytes.
    """
    return e4m3_encode(np.asarray(values, dtype=np.float64) * np.ldexp(1.0, -np.asarray(t_forced)))


def naive_pow2(q, s):
    """Naive conversion, power-of-two scales: dequantize -> bf16 -> transpose -> 1x128 requantize.

    The bf16 intermediate is exact here (an e4m3 value times a power of two has
    4 significant bits), so this path is itself free of double quantization
    error but computes its own (tighter) column scales.
    """
    x_bf16 = bf16_round(dequant_rowwise(q, s))
    return quant_rowwise(x_bf16.T)


def _quant_rowwise_fp32_scale(x):
    """1x128 quantization with non-power-of-two fp32 scales s = amax/448 (IEEE division).

    This is the scale of section 3.1 taken literally, without the power-of-two
    constraint; used only to reproduce the double quantization error.
    """
    x = np.asarray(x, dtype=np.float32)
    rows, cols = x.shape
    tiles = x.reshape(rows, cols // TILE, TILE)
    amax = np.abs(tiles).max(axis=2)
    s = (amax / np.float32(448.0)).astype(np.float32)
    s = np.where(s == 0, np.float32(1.0), s).astype(np.float32)
    scaled = (tiles / s[:, :, None]).astype(np.float32)
    return e4m3_encode(np.clip(scaled, -448.0, 448.0)).reshape(rows, cols), s


def naive_fp32(x):
    """Naive conversion with fp32 scales (the double-quantization path of section 3.1).

    Q_row with s = amax/448, dequantize in fp32, round to bf16, transpose,
    Q_col with fresh s' = amax'/448.  Returns (Q_row bytes, row scales,
    Q_col bytes, column scales) so that both D(Q_row(X)) and D(Q_col(D(Q_row(X))))
    can be formed.
    """
    q1, s1 = _quant_rowwise_fp32_scale(x)
    rows, cols = q1.shape
    d1 = (e4m3_decode(q1).reshape(rows, cols // TILE, TILE).astype(np.float32) * s1[:, :, None]).astype(np.float32)
    d1 = bf16_round(d1.reshape(rows, cols)).astype(np.float32)
    q2, s2 = _quant_rowwise_fp32_scale(d1.T)
    return q1, s1, q2, s2
