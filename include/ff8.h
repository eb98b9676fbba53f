/*
 * ff8.h -- C ABI of the FP8-Flow-MoE expert-layer library for AMD Instinct MI355X (gfx950).
 *
 * The library implements the FP8-centric forward and backward of a routed MoE
 * feed-forward layer ("FP8-Flow-MoE: A Casting-Free FP8 Recipe without Double
 * Quantization Error", arXiv 2511.02302): fused permute+pad+quantize, FP8
 * grouped GEMMs for fprop / dgrad / wgrad, fused SwiGLU+quantize, the
 * scaling-aware transpose and the unpermute.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Types: ff8_bf16 is a bfloat16 bit pattern; ff8_e4m3 is an OCP FP8 E4M3FN
 *    byte (bias 7, largest finite 448, subnormals, 0x7F/0xFF NaN, no infinity).
 *  - Scales are float32 powers of two 2^T with T in [-126, 127] (paper section
 *    3.1, power-of-two constraint).  A tile's T is the smallest integer with
 *    max|x| <= 448 * 2^T; an all-zero tile gets 2^-126.  Quantized bytes are
 *    encode(x * 2^-T) with round-to-nearest-even, saturating at +-448, sign kept.
 *    Inputs to the quantizers must be finite.  The GEMMs read only the exponent
 *    field of each scale, so scales passed to them must be such powers of two.
 *  - Row-wise (1x128) scaled tensor: q [rows, cols] row-major, s [rows, cols/128].
 *    Column-wise scaled tensors are stored transposed and K-blocked,
 *    qT [rows/128, cols, 128]: element (c, r) of the transpose (input row r,
 *    column c) is byte (r/128) * cols * 128 + c * 128 + r % 128, so each block of
 *    128 input rows is one contiguous [cols][128] slab.  Their scales are
 *    block-major, sT [rows/128, cols]: row b holds the scale of every column over
 *    rows 128b..128b+127.  Block (128x128) scaled weights: q [E, N, K],
 *    s [E, N/128, K/128].
 *  - Grouped (expert-contiguous) tensors have M_cap rows; expert e owns rows
 *    [offsets[e], offsets[e+1]), every group is padded to a multiple of the
 *    alignment (128 rows, or 16, 32 or 64 through ff8_permute_quant_aligned),
 *    and offsets ([E+1] int32) live in DEVICE memory.  Kernels read offsets[E]
 *    (= M_pad) on the device; rows in [M_pad, M_cap) are neither read nor
 *    written.  Grids are sized from M_cap, so no call synchronizes with the host.
 *    Because they are never copied to the host, offsets are not validated: they
 *    must satisfy 0 = offsets[0] <= offsets[1] <= ... <= offsets[E] <= M_cap with
 *    every difference a multiple of 16, as ff8_permute_quant(_aligned) writes them.  Other
 *    values give undefined results and may make kernels access memory outside the
 *    tensors.  E is at most 1024.
 *  - Every pointer is a device pointer unless stated otherwise.  The caller
 *    owns all memory; the library allocates nothing and keeps no pointer after
 *    a call returns.  With T = 0 (an empty batch) the token-indexed arrays (x, dy,
 *    row_map, row_w, y, dprobs, topk_idx) may be NULL.
 *  - stream is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    call only enqueues work on it and returns; results are ready when the
 *    stream reaches that point.  Calls on one stream are ordered; concurrent
 *    calls on different streams must not write the same buffers.
 *  - Return value: FF8_OK, or an error code.  Arguments are validated on the
 *    host before anything is enqueued; on a validation error nothing is
 *    launched.  FF8_ERR_HIP means a launch failed; ff8_last_error() then holds
 *    the HIP message (thread-local, valid until the next call on the thread).
 *  - Dimensions H, N, K, I, cols must be multiples of 128; M_cap and rows must
 *    be multiples of 128.  The grouped GEMMs also need M_cap * max(N, K) < 2^32 and,
 *    for fprop and dgrad, E * N * K < 2^32 (each operand tensor, including all
 *    experts' weights together, under 4 GiB); larger shapes return FF8_ERR_SHAPE.
 */
#ifndef FF8_H
#define FF8_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef uint16_t ff8_bf16;
typedef uint8_t ff8_e4m3;
typedef uint8_t ff8_e8m0;  /* UE8M0 scale byte: the scale 2^T is stored as T + 127 */

enum ff8_status {
  FF8_OK = 0,
  FF8_ERR_NULL = 1,   /* a required pointer is NULL */
  FF8_ERR_SHAPE = 2,  /* a dimension is not a positive multiple of 128, or M_cap is below the bound */
  FF8_ERR_ARG = 3,    /* k, E, a flag or the workspace size is out of range */
  FF8_ERR_HIP = 4     /* a HIP launch or runtime call failed */
};

/* Library version (major * 10000 + minor * 100 + patch). */
int ff8_version(void);
/* Static description of a status code. */
const char* ff8_status_string(int status);
/* Detail of the last error on this host thread ("" if none). */
const char* ff8_last_error(void);

/*
 * ff8_quant_rowwise -- 1x128 row-wise quantization (paper section 3.1: scale,
 * quantize and power-of-two constraint; the explicit entry cast of the dataflow).
 *   x  [rows, cols] bf16 input.
 *   q  [rows, cols] e4m3 output; s [rows, cols/128] float32 output.
 * rows >= 1 (any count), cols a multiple of 128.
 */
int ff8_quant_rowwise(const ff8_bf16* x, int64_t rows, int64_t cols, ff8_e4m3* q, float* s, void* stream);

/*
 * ff8_quant_block128 -- 128x128 block quantization of weights (per-block scaling
 * named in paper section 2.1; the block shape of the DeepSeek-V3 recipe the paper builds on).
 *   w  [rows, cols] bf16 (a stack of E expert weights [E, N, K] is rows = E*N);
 *   q  [rows, cols] e4m3; s [rows/128, cols/128] float32.
 */
int ff8_quant_block128(const ff8_bf16* w, int64_t rows, int64_t cols, ff8_e4m3* q, float* s, void* stream);

/*
 * ff8_rows_bound -- host helper: the smallest admissible M_cap for T tokens,
 * top-k and E experts: roundup(T*k + 127*E, 128) (every expert pads < 128 rows).
 * Returns -1 for invalid arguments.
 */
int64_t ff8_rows_bound(int64_t T, int k, int E);

/*
 * ff8_rows_bound_aligned -- the same for groups padded to `align` rows (16, 32, 64 or
 * 128): roundup(T*k + (align-1)*E, 128).  align = 16 is the paper's padding (section
 * 3.3.1).  Returns -1 for invalid arguments.
 */
int64_t ff8_rows_bound_aligned(int64_t T, int k, int E, int align);

/* Bytes of device workspace ff8_permute_quant needs (host helper). */
size_t ff8_permute_workspace_bytes(int64_t T, int k, int E);

/*
 * ff8_permute_quant -- fused permute + padding + 1x128 quantization (paper
 * section 3.3.1, fused permute and padding; quantization fused in as the entry
 * cast of section 3.2).
 *   x        [T, H] bf16 activations (or upstream gradients).
 *   row_w    [T, k] float32 routing weights, or NULL.  With weights, row (t, j)
 *            holds quant(row_w[t,j] * x[t]) (float32 product); without, quant(x[t]).
 *   topk_idx [T, k] int32 expert ids in [-1, E); -1 drops the slot; ids of one
 *            token must be distinct.  Read only when reuse_map == 0.
 *   reuse_map 0: build the routing maps (outputs below).  1: row_map, offsets
 *            and src_row are INPUTS from an earlier call with the same routing
 *            (the backward quantizes dY with the forward's maps).
 *   row_map  [T, k] int32: the row of pair (t, j) in the grouped tensor, -1 if dropped.
 *   offsets  [E+1] int32: offsets[0] = 0, offsets[e+1] = offsets[e] + roundup(count_e, 128).
 *            Within a group rows are in ascending token order.
 *   src_row  [M_cap] int32: t*k + j for real rows, -1 for padding rows; entries
 *            at and beyond offsets[E] are not written.
 *   q, s     [M_cap, H] e4m3 and [M_cap, H/128] float32: real rows quantized as
 *            above, padding rows 0x00 with scale 2^-126, rows >= offsets[E] untouched.
 *   workspace device scratch of at least ff8_permute_workspace_bytes(T, k, E)
 *            bytes (ws_bytes gives its size); contents need not be initialized.
 *            May be NULL when reuse_map == 1.
 * Requires 1 <= k <= E, E <= 1024, M_cap >= ff8_rows_bound(T, k, E), H % 128 == 0
 * (with reuse_map = 1, M_cap >= ff8_rows_bound_aligned(T, k, E, 16) suffices).
 */
int ff8_permute_quant(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                      const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets,
                      int32_t* src_row, int64_t M_cap, ff8_e4m3* q, float* s, void* workspace,
                      size_t ws_bytes, void* stream);

/*
 * ff8_permute_quant_aligned -- ff8_permute_quant with groups padded to a multiple of
 *   `align` rows (16, 32, 64 or 128) instead of 128; align = 16 is the paper's padding
 *   (section 3.3.1).  Requires M_cap >= ff8_rows_bound_aligned(T, k, E, align).  Every
 *   other entry point accepts offsets padded to 16: a 128-row block of a grouped tensor
 *   may then hold rows of two experts (the transpose takes S_max over the whole block,
 *   or over the rows below offsets[E] in the last one, and wgrad masks the rows of other
 *   experts out of its first and last K block).
 */
int ff8_permute_quant_aligned(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                              const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets,
                              int32_t* src_row, int64_t M_cap, ff8_e4m3* q, float* s, void* workspace,
                              size_t ws_bytes, int align, void* stream);

/*
 * ff8_permute_quant_noalloc -- ff8_permute_quant_aligned without a caller workspace, for callers
 *   that cannot allocate device memory at call time (code under HIP graph capture, tight serving
 *   loops, harnesses that forbid hipMalloc).  The routing pass keeps its per-chunk expert counts
 *   in a 1 MiB array that the library holds in device memory (one per GPU, from the first call
 *   on that GPU until the process ends); the call itself allocates nothing.  Arguments, outputs
 *   and errors as ff8_permute_quant_aligned (align 16, 32, 64 or 128), minus workspace and
 *   ws_bytes.  Limit: with reuse_map == 0, ceil(T / 256) * E <= 262144 (T <= 2 097 152 tokens
 *   at E = 32); larger routings return FF8_ERR_ARG before anything is enqueued.  Every call on
 *   one GPU shares that GPU's array, and nothing in it needs clearing between calls (each call
 *   writes every entry it reads), but calls that overlap on one GPU (concurrent streams, or
 *   host threads each with its own stream) race on it and give undefined routing: serialize
 *   them.
 */
int ff8_permute_quant_noalloc(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                              const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets,
                              int32_t* src_row, int64_t M_cap, ff8_e4m3* q, float* s, int align, void* stream);

/*
 * ff8_permute_quant_dprobs -- the backward permute of dY (ff8_permute_quant with reuse_map = 1
 *   and routing weights) fused with the router gradient, the backward of the
 *   routing-weighted combine y[t] = sum_j row_w[t, j] * y_perm[row_map[t, j]] (paper section
 *   3.2: the combine and the dispatch sit at the fc2 output, which stays BF16):
 *     dprobs[t, j] = sum_h dy[t, h] * y_perm[row_map[t, j], h],
 *   accumulated in float32 (each bf16 x bf16 product is exact), 0 for a dropped slot.
 *   q, s, padding rows: exactly as ff8_permute_quant (reuse_map = 1) writes them from dy and
 *   row_w.  row_map, offsets, src_row as written by the forward's ff8_permute_quant.
 *   y_perm [M_cap, H] bf16 (the fc2 output of the forward); dprobs [T, k] float32.
 *   Limits: k <= 64 and H <= 8192 (one workgroup holds a token's dy row in registers);
 *   larger values return FF8_ERR_ARG / FF8_ERR_SHAPE.
 */
int ff8_permute_quant_dprobs(const ff8_bf16* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                             const int32_t* row_map, const int32_t* offsets, const int32_t* src_row, int64_t M_cap,
                             ff8_e4m3* q, float* s, const ff8_bf16* y_perm, float* dprobs, void* stream);

/*
 * ff8_scaling_aware_transpose -- Algorithm 1 of paper section 3.1 (scaling-aware
 * FP8 transpose) with its exponent-shift identity.
 *   q [rows, cols] e4m3 with row-wise scales s [rows, cols/128].
 *   For every 128x128 block, S_max is the largest of its 128 row scales; each
 *   element of row i is re-expressed at S_max by lowering its exponent by
 *   k = log2(S_max / s_i); where the exponent would fall below 1 the value
 *   dec(b) * 2^-k is rounded to nearest even on the subnormal grid.  No
 *   dequantize / requantize round trip happens, so there is no double
 *   quantization error.
 *   qT [rows/128, cols, 128] e4m3, the K-blocked transpose (element (c, r) at
 *   [r/128, c, r%128]), sT [rows/128, cols] float32 (block-major: sT[b, c] is the
 *   S_max of the 128x128 block holding row 128b and column c, the same for all
 *   128 columns of a tile).  rows must be a multiple of 128 and cols of 128.
 *   offsets: [E+1] device int32 (only offsets[E] is read: rows at and beyond it
 *   are skipped and their qT bytes / sT entries untouched) or NULL (all rows).
 *   E is ignored when offsets is NULL.
 */
int ff8_scaling_aware_transpose(const ff8_e4m3* q, const float* s, int64_t rows, int64_t cols,
                                const int32_t* offsets, int E, ff8_e4m3* qT, float* sT, void* stream);

/*
 * ff8_scaling_aware_transpose_batch -- the same transpose (paper section 3.1,
 * Algorithm 1) of n tensors in one launch: the backward pass turns its four
 * row-wise operands (X, H, dY, dA of section 3.2's column-wise Wgrad) into their
 * column-wise forms at once.
 *   n in [1, 4]; q, s, cols, qT, sT are host arrays of n entries.  Tensor i is
 *   q[i] [rows, cols[i]] with s[i] [rows, cols[i]/128] and is written to qT[i]
 *   [rows/128, cols[i], 128], sT[i] [rows/128, cols[i]] exactly as
 *   ff8_scaling_aware_transpose writes it; rows (a multiple of 128) and offsets
 *   (NULL or [E+1], only offsets[E] read) are shared by all n.  The result is
 *   bit-identical to n separate calls.  The host arrays are read during the call
 *   only.  n outside [1, 4] returns FF8_ERR_ARG; a NULL array or entry
 *   FF8_ERR_NULL; a rows or cols[i] that is not a positive multiple of 128
 *   FF8_ERR_SHAPE.
 */
int ff8_scaling_aware_transpose_batch(int n, const ff8_e4m3* const* q, const float* const* s, const int64_t* cols,
                                      int64_t rows, const int32_t* offsets, int E, ff8_e4m3* const* qT,
                                      float* const* sT, void* stream);

/*
 * ff8_grouped_gemm_fprop -- FP8 grouped GEMM, forward (paper section 3.2: the
 * grouped linear consumes row-wise FP8 activations; "Fprop").
 *   out[m, n] = sum_k D(a)[m, k] * D(w_e)[n, k] for m in expert e's rows,
 *   accumulated in float32 with the per-128 scales applied per K block, rounded
 *   once to bf16.
 *   a [M_cap, K] e4m3 + a_s [M_cap, K/128]; w [E, N, K] e4m3 + w_s [E, N/128, K/128];
 *   out [M_cap, N] bf16 (rows >= offsets[E] untouched; padding rows get zeros).
 */
int ff8_grouped_gemm_fprop(const ff8_e4m3* a, const float* a_s, const ff8_e4m3* w, const float* w_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K,
                           ff8_bf16* out, void* stream);

/*
 * ff8_grouped_gemm_dgrad -- FP8 grouped GEMM, input gradient ("Dgrad" of paper section 3.1).
 *   out[m, k] = sum_n D(g)[m, n] * D(w_e)[n, k].
 *   g [M_cap, N] e4m3 + g_s [M_cap, N/128]; w, w_s as in fprop (not transposed);
 *   out [M_cap, K] bf16.
 */
int ff8_grouped_gemm_dgrad(const ff8_e4m3* g, const float* g_s, const ff8_e4m3* w, const float* w_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K,
                           ff8_bf16* out, void* stream);

/*
 * ff8_grouped_gemm_wgrad -- FP8 grouped GEMM, weight gradient ("Wgrad" of paper
 * section 3.1, fed by column-wise operands from the scaling-aware transpose).
 *   dw[e, n, k] (+)= sum_{m in expert e's rows} D(gT)[n, m] * D(xT)[k, m].
 *   gT [M_cap/128, N, 128] e4m3 + gT_s [M_cap/128, N]; xT [M_cap/128, K, 128] e4m3
 *   + xT_s [M_cap/128, K] (K-blocked transposes with block-major scales, as written
 *   by ff8_scaling_aware_transpose);
 *   dw [E, N, K] float32.  accumulate = 0 overwrites (experts without rows get
 *   zeros); accumulate = 1 adds to dw (experts without rows are left untouched).
 */
int ff8_grouped_gemm_wgrad(const ff8_e4m3* gT, const float* gT_s, const ff8_e4m3* xT, const float* xT_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, float* dw,
                           int accumulate, void* stream);

/*
 * ff8_swiglu_quant -- fused SwiGLU + 1x128 quantization (paper section 3.3.2):
 *   h[m, i] = silu(a[m, i]) * a[m, I + i] computed in float32 and quantized
 *   directly (never rounded to bf16).
 *   a [M_cap, 2I] bf16 ([gate | up]); hq [M_cap, I] e4m3 + hs [M_cap, I/128].
 *   Rows >= offsets[E] untouched.
 */
int ff8_swiglu_quant(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                     ff8_e4m3* hq, float* hs, void* stream);

/*
 * ff8_swiglu_bwd_quant -- backward twin of the fused SwiGLU kernel (paper section 3.3.2:
 *   the activation's FP8 output is produced inside the activation kernel, here for its
 *   gradient, which the fc1 dgrad consumes as row-wise FP8 per section 3.2).  The
 *   gradient itself is the derivative of h = silu(g) * u (the paper does not print it):
 *   sig = 1 / (1 + exp(-g)), dg = dh * u * sig * (1 + g * (1 - sig)),
 *   du = dh * g * sig, in float32, quantized 1x128 into daq = [dg | du].
 *   a [M_cap, 2I] bf16, dh [M_cap, I] bf16; daq [M_cap, 2I] e4m3 + das [M_cap, 2I/128].
 */
int ff8_swiglu_bwd_quant(const ff8_bf16* a, const ff8_bf16* dh, const int32_t* offsets, int E, int64_t M_cap,
                         int64_t I, ff8_e4m3* daq, float* das, void* stream);

/*
 * ff8_swiglu_quant_keep_fp8 -- ff8_swiglu_quant that also keeps an FP8 checkpoint of
 *   its input for the backward (paper section 4.2: the activations saved for the
 *   backward are stored in FP8 instead of BF16, which is where the method's peak
 *   memory saving comes from).  hq, hs as ff8_swiglu_quant; in addition
 *   a_q [M_cap, 2I] e4m3 + a_s [M_cap, 2I/128] = a quantized 1x128 (gate tiles, then
 *   up tiles), bit-identical to ff8_quant_rowwise on the active rows.  Once it has
 *   run, the BF16 a is no longer needed.  Rows >= offsets[E] untouched.
 */
int ff8_swiglu_quant_keep_fp8(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                              ff8_e4m3* hq, float* hs, ff8_e4m3* a_q, float* a_s, void* stream);

/*
 * ff8_swiglu_bwd_quant_fp8a -- ff8_swiglu_bwd_quant reading A from its FP8 checkpoint:
 *   g, u = a_q * a_s (exact in float32), then the same dg, du and 1x128 quantization.
 *   a_q [M_cap, 2I] e4m3 + a_s [M_cap, 2I/128] as written by ff8_swiglu_quant_keep_fp8;
 *   dh [M_cap, I] bf16; daq [M_cap, 2I] e4m3 + das [M_cap, 2I/128].
 */
int ff8_swiglu_bwd_quant_fp8a(const ff8_e4m3* a_q, const float* a_s, const ff8_bf16* dh, const int32_t* offsets,
                              int E, int64_t M_cap, int64_t I, ff8_e4m3* daq, float* das, void* stream);

/*
 * ff8_unpermute -- fused unpermute + unpadding (paper section 3.3.1); M_cap is the row
 *   count of y_perm, against which every row_map entry is checked on the device:
 *   y[t] = sum_{j < k, row_map[t,j] >= 0} w[t, j] * y_perm[row_map[t, j]],
 *   accumulated in float32 in slot order, rounded once to bf16; w = 1 when
 *   row_w is NULL.  y_perm [M_cap, H] bf16, row_map [T, k] int32 (entries must
 *   be -1 or in [0, M_cap)), row_w [T, k] float32 or NULL, y [T, H] bf16.
 */
int ff8_unpermute(const ff8_bf16* y_perm, const int32_t* row_map, const float* row_w, int64_t T, int k,
                  int64_t H, int64_t M_cap, ff8_bf16* y, void* stream);

/* ---- UE8M0 scale storage ----
 * Paper section 2.1 names UE8M0 (unsigned, 8 exponent bits, no mantissa) as the scale format of
 * its recipe, and the power-of-two constraint of section 3.1 makes every scale exactly such a
 * value: the scale 2^T, T in [-126, 127], is the byte T + 127 (the float32 scale's exponent
 * field).  The entry points below are the ones above with every scale tensor in this format:
 * the same shapes and layouts, one byte per scale instead of four, and bit-identical FP8 bytes,
 * routing maps and outputs.  Consumers read the bytes as stored.  The grouped GEMMs move four
 * scale bytes per DMA lane: fprop needs K % 512 == 0, dgrad N % 512 == 0 and K % 512 == 0
 * (FF8_ERR_SHAPE otherwise); wgrad takes any multiple of 128.
 */
int ff8_quant_rowwise_e8m0(const ff8_bf16* x, int64_t rows, int64_t cols, ff8_e4m3* q, ff8_e8m0* s, void* stream);
int ff8_quant_block128_e8m0(const ff8_bf16* w, int64_t rows, int64_t cols, ff8_e4m3* q, ff8_e8m0* s, void* stream);
/* ff8_permute_quant_aligned with UE8M0 scales (align 16, 32, 64 or 128; padding rows get byte 1, i.e. 2^-126). */
int ff8_permute_quant_e8m0(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                           const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets, int32_t* src_row,
                           int64_t M_cap, ff8_e4m3* q, ff8_e8m0* s, void* workspace, size_t ws_bytes, int align,
                           void* stream);
int ff8_permute_quant_dprobs_e8m0(const ff8_bf16* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                  const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                  int64_t M_cap, ff8_e4m3* q, ff8_e8m0* s, const ff8_bf16* y_perm, float* dprobs,
                                  void* stream);
int ff8_scaling_aware_transpose_e8m0(const ff8_e4m3* q, const ff8_e8m0* s, int64_t rows, int64_t cols,
                                     const int32_t* offsets, int E, ff8_e4m3* qT, ff8_e8m0* sT, void* stream);
int ff8_scaling_aware_transpose_batch_e8m0(int n, const ff8_e4m3* const* q, const ff8_e8m0* const* s,
                                           const int64_t* cols, int64_t rows, const int32_t* offsets, int E,
                                           ff8_e4m3* const* qT, ff8_e8m0* const* sT, void* stream);
int ff8_grouped_gemm_fprop_e8m0(const ff8_e4m3* a, const ff8_e8m0* a_s, const ff8_e4m3* w, const ff8_e8m0* w_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                                void* stream);
int ff8_grouped_gemm_dgrad_e8m0(const ff8_e4m3* g, const ff8_e8m0* g_s, const ff8_e4m3* w, const ff8_e8m0* w_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                                void* stream);
int ff8_grouped_gemm_wgrad_e8m0(const ff8_e4m3* gT, const ff8_e8m0* gT_s, const ff8_e4m3* xT, const ff8_e8m0* xT_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, float* dw,
                                int accumulate, void* stream);
int ff8_swiglu_quant_e8m0(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I, ff8_e4m3* hq,
                          ff8_e8m0* hs, void* stream);
int ff8_swiglu_bwd_quant_e8m0(const ff8_bf16* a, const ff8_bf16* dh, const int32_t* offsets, int E, int64_t M_cap,
                              int64_t I, ff8_e4m3* daq, ff8_e8m0* das, void* stream);
int ff8_swiglu_quant_keep_fp8_e8m0(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                   ff8_e4m3* hq, ff8_e8m0* hs, ff8_e4m3* a_q, ff8_e8m0* a_s, void* stream);
int ff8_swiglu_bwd_quant_fp8a_e8m0(const ff8_e4m3* a_q, const ff8_e8m0* a_s, const ff8_bf16* dh,
                                   const int32_t* offsets, int E, int64_t M_cap, int64_t I, ff8_e4m3* daq,
                                   ff8_e8m0* das, void* stream);

/* ---- element casts (the codec every quantizer uses; exposed for exhaustive checks) ---- */

/* q[i] = saturating round-to-nearest-even e4m3 encoding of x[i] (no scaling; NaN -> 0x7F). */
int ff8_cast_f32_to_e4m3(const float* x, int64_t n, ff8_e4m3* q, void* stream);
/* x[i] = value of e4m3 byte q[i]. */
int ff8_cast_e4m3_to_f32(const ff8_e4m3* q, int64_t n, float* x, void* stream);

/* ---- baselines: the unfused paths the paper compares against (benchmark use) ---- */

/* Naive conversion, step 1: out[r, c] = bf16(dec(q[r, c]) * s[r, c/128]) (exact for power-of-two scales). */
int ff8_baseline_dequant_rowwise(const ff8_e4m3* q, const float* s, int64_t rows, int64_t cols, ff8_bf16* out,
                                 void* stream);
/* Naive conversion, step 2: out[c, r] = in[r, c] for a bf16 [rows, cols] tensor (rows, cols multiples of 64).
 * Step 3 is ff8_quant_rowwise on the transposed tensor. */
int ff8_baseline_transpose_bf16(const ff8_bf16* in, int64_t rows, int64_t cols, ff8_bf16* out, void* stream);
/* Unfused SwiGLU: h = bf16(silu(g) * u) for a [rows, 2I] -> h [rows, I] (rows < offsets[E] when offsets != NULL). */
int ff8_baseline_swiglu_bf16(const ff8_bf16* a, const int32_t* offsets, int E, int64_t rows, int64_t I,
                             ff8_bf16* h, void* stream);
/* Plain device copy of nbytes (a multiple of 16) -- the HBM bandwidth reference. */
int ff8_baseline_copy(const void* src, void* dst, int64_t nbytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FF8_H */
