"""ctypes binding of libff8.so: one Python function per C entry point, same names.

Argument marshalling only: each function checks dtypes, devices and contiguity of
the torch tensors it is given, and that every tensor's shape matches the extents the
C ABI takes from the first operand (the C side receives plain pointers and cannot see
an undersized buffer), passes raw device pointers and the current HIP stream to the
C ABI, and raises Ff8Error on a non-zero status.  No
function allocates, computes or falls back to anything: if libff8.so is missing
the first call raises.
"""

import ctypes
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libff8.so")
_lib = None

_c_i64 = ctypes.c_int64
_c_int = ctypes.c_int
_c_vp = ctypes.c_void_p
_c_size = ctypes.c_size_t

_SIGNATURES = {
    "ff8_version": (_c_int, []),
    "ff8_status_string": (ctypes.c_char_p, [_c_int]),
    "ff8_last_error": (ctypes.c_char_p, []),
    "ff8_quant_rowwise": (_c_int, [_c_vp, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_quant_block128": (_c_int, [_c_vp, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_rows_bound": (_c_i64, [_c_i64, _c_int, _c_int]),
    "ff8_rows_bound_aligned": (_c_i64, [_c_i64, _c_int, _c_int, _c_int]),
    "ff8_permute_workspace_bytes": (_c_size, [_c_i64, _c_int, _c_int]),
    "ff8_permute_quant": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_int, _c_vp, _c_vp,
                                   _c_vp, _c_i64, _c_vp, _c_vp, _c_vp, _c_size, _c_vp]),
    "ff8_permute_quant_aligned": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_int, _c_vp,
                                           _c_vp, _c_vp, _c_i64, _c_vp, _c_vp, _c_vp, _c_size, _c_int, _c_vp]),
    "ff8_permute_quant_noalloc": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_int, _c_vp,
                                           _c_vp, _c_vp, _c_i64, _c_vp, _c_vp, _c_int, _c_vp]),
    "ff8_scaling_aware_transpose": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_vp, _c_int, _c_vp, _c_vp, _c_vp]),
    "ff8_scaling_aware_transpose_batch": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_vp, _c_int, _c_vp, _c_vp,
                                                   _c_vp]),
    "ff8_grouped_gemm_fprop": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64, _c_vp,
                                        _c_vp]),
    "ff8_grouped_gemm_dgrad": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64, _c_vp,
                                        _c_vp]),
    "ff8_grouped_gemm_wgrad": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64, _c_vp,
                                        _c_int, _c_vp]),
    "ff8_swiglu_quant": (_c_int, [_c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_swiglu_bwd_quant": (_c_int, [_c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_permute_quant_dprobs": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_vp, _c_vp, _c_i64,
                                          _c_vp, _c_vp, _c_vp, _c_vp, _c_vp]),
    "ff8_swiglu_quant_keep_fp8": (_c_int, [_c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp, _c_vp,
                                           _c_vp]),
    "ff8_swiglu_bwd_quant_fp8a": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp,
                                           _c_vp]),
    "ff8_unpermute": (_c_int, [_c_vp, _c_vp, _c_vp, _c_i64, _c_int, _c_i64, _c_i64, _c_vp, _c_vp]),
    "ff8_quant_rowwise_e8m0": (_c_int, [_c_vp, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_quant_block128_e8m0": (_c_int, [_c_vp, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_permute_quant_e8m0": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_int, _c_vp, _c_vp,
                                        _c_vp, _c_i64, _c_vp, _c_vp, _c_vp, _c_size, _c_int, _c_vp]),
    "ff8_permute_quant_dprobs_e8m0": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_int, _c_int, _c_vp, _c_vp, _c_vp,
                                               _c_i64, _c_vp, _c_vp, _c_vp, _c_vp, _c_vp]),
    "ff8_scaling_aware_transpose_e8m0": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_vp, _c_int, _c_vp, _c_vp, _c_vp]),
    "ff8_scaling_aware_transpose_batch_e8m0": (_c_int, [_c_int, _c_vp, _c_vp, _c_vp, _c_i64, _c_vp, _c_int, _c_vp,
                                                        _c_vp, _c_vp]),
    "ff8_grouped_gemm_fprop_e8m0": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64,
                                             _c_vp, _c_vp]),
    "ff8_grouped_gemm_dgrad_e8m0": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64,
                                             _c_vp, _c_vp]),
    "ff8_grouped_gemm_wgrad_e8m0": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_i64,
                                             _c_vp, _c_int, _c_vp]),
    "ff8_swiglu_quant_e8m0": (_c_int, [_c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_swiglu_bwd_quant_e8m0": (_c_int, [_c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp]),
    "ff8_swiglu_quant_keep_fp8_e8m0": (_c_int, [_c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp, _c_vp, _c_vp,
                                                _c_vp]),
    "ff8_swiglu_bwd_quant_fp8a_e8m0": (_c_int, [_c_vp, _c_vp, _c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp,
                                                _c_vp]),
    "ff8_cast_f32_to_e4m3": (_c_int, [_c_vp, _c_i64, _c_vp, _c_vp]),
    "ff8_cast_e4m3_to_f32": (_c_int, [_c_vp, _c_i64, _c_vp, _c_vp]),
    "ff8_baseline_dequant_rowwise": (_c_int, [_c_vp, _c_vp, _c_i64, _c_i64, _c_vp, _c_vp]),
    "ff8_baseline_transpose_bf16": (_c_int, [_c_vp, _c_i64, _c_i64, _c_vp, _c_vp]),
    "ff8_baseline_swiglu_bf16": (_c_int, [_c_vp, _c_vp, _c_int, _c_i64, _c_i64, _c_vp, _c_vp]),
    "ff8_baseline_copy": (_c_int, [_c_vp, _c_vp, _c_i64, _c_vp]),
}

EXPORTS = tuple(_SIGNATURES)


class Ff8Error(RuntimeError):
    pass


def library_path():
    return _LIB_PATH


def load():
    """Load libff8.so (once) and declare every entry point's signature."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2511_02302_amd.build`")
        lib = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(status, name):
    if status != 0:
        lib = load()
        raise Ff8Error(f"{name}: {lib.ff8_status_string(status).decode()} ({lib.ff8_last_error().decode()})")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t, dtype, name, ndim=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions, got {t.dim()}")
    return ctypes.c_void_p(t.data_ptr())


def _shape(t, shape, name):
    """t is None or has exactly this shape."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _numel(t, n, name):
    """t is None or holds exactly n elements (any shape)."""
    if t is not None and t.numel() != n:
        raise ValueError(f"{name} must hold {n} elements, got {t.numel()}")


_bf16, _u8, _f32, _i32 = torch.bfloat16, torch.uint8, torch.float32, torch.int32


def _scale_kind(*scales):
    """Scale storage of a call: float32 tensors (powers of two) or uint8 tensors (UE8M0 bytes,
    T + 127), the same for every scale tensor of the call.  Returns (dtype, C-symbol suffix)."""
    kinds = {t.dtype for t in scales if t is not None}
    if kinds == {_f32}:
        return _f32, ""
    if kinds == {_u8}:
        return _u8, "_e8m0"
    raise TypeError(f"scale tensors must all be float32 or all uint8 (UE8M0), got {sorted(map(str, kinds))}")


def ff8_version():
    return load().ff8_version()


def ff8_rows_bound_aligned(T, k, E, align):
    return int(load().ff8_rows_bound_aligned(T, k, E, align))


def ff8_rows_bound(T, k, E):
    return int(load().ff8_rows_bound(T, k, E))


def ff8_permute_workspace_bytes(T, k, E):
    return int(load().ff8_permute_workspace_bytes(T, k, E))


def ff8_quant_rowwise(x, q, s, stream=None):
    rows, cols = x.shape
    _shape(q, (rows, cols), "q"); _shape(s, (rows, cols // 128), "s")
    sd, sfx = _scale_kind(s)
    name = "ff8_quant_rowwise" + sfx
    _check(getattr(load(), name)(_ptr(x, _bf16, "x", 2), rows, cols, _ptr(q, _u8, "q"), _ptr(s, sd, "s"),
                                 _stream(stream)), name)


def ff8_quant_block128(w, q, s, stream=None):
    rows, cols = w.reshape(-1, w.shape[-1]).shape
    _shape(q, w.shape, "q"); _numel(s, (rows // 128) * (cols // 128), "s")
    sd, sfx = _scale_kind(s)
    name = "ff8_quant_block128" + sfx
    _check(getattr(load(), name)(_ptr(w, _bf16, "w"), rows, cols, _ptr(q, _u8, "q"), _ptr(s, sd, "s"),
                                 _stream(stream)), name)


def ff8_permute_quant(x, row_w, k, E, topk_idx, reuse_map, row_map, offsets, src_row, q, s, workspace=None,
                      stream=None, align=None):
    """align None calls ff8_permute_quant (groups padded to 128 rows); 16/32/64/128 calls
    ff8_permute_quant_aligned; a uint8 (UE8M0) scale tensor calls ff8_permute_quant_e8m0."""
    T, H = x.shape
    M_cap = q.shape[0]
    _numel(row_w, T * k, "row_w"); _numel(topk_idx, T * k, "topk_idx"); _numel(row_map, T * k, "row_map")
    _numel(offsets, E + 1, "offsets"); _numel(src_row, M_cap, "src_row")
    _shape(q, (M_cap, H), "q"); _shape(s, (M_cap, H // 128), "s")
    ws = 0 if workspace is None else workspace.numel() * workspace.element_size()
    sd, sfx = _scale_kind(s)
    args = [_ptr(x, _bf16, "x", 2), _ptr(row_w, _f32, "row_w"), T, H, k, E, _ptr(topk_idx, _i32, "topk_idx"),
            int(reuse_map), _ptr(row_map, _i32, "row_map"), _ptr(offsets, _i32, "offsets"),
            _ptr(src_row, _i32, "src_row"), M_cap, _ptr(q, _u8, "q", 2), _ptr(s, sd, "s", 2),
            None if workspace is None else ctypes.c_void_p(workspace.data_ptr()), ws]
    if sfx:
        _check(load().ff8_permute_quant_e8m0(*args, int(align or 128), _stream(stream)), "ff8_permute_quant_e8m0")
    elif align is None:
        _check(load().ff8_permute_quant(*args, _stream(stream)), "ff8_permute_quant")
    else:
        _check(load().ff8_permute_quant_aligned(*args, int(align), _stream(stream)), "ff8_permute_quant_aligned")


def ff8_permute_quant_noalloc(x, row_w, k, E, topk_idx, reuse_map, row_map, offsets, src_row, q, s, align=128,
                              stream=None):
    """ff8_permute_quant_aligned with the library's own routing workspace (no caller buffer)."""
    T, H = x.shape
    M_cap = q.shape[0]
    _numel(row_w, T * k, "row_w"); _numel(topk_idx, T * k, "topk_idx"); _numel(row_map, T * k, "row_map")
    _numel(offsets, E + 1, "offsets"); _numel(src_row, M_cap, "src_row")
    _shape(q, (M_cap, H), "q"); _shape(s, (M_cap, H // 128), "s")
    _check(load().ff8_permute_quant_noalloc(
        _ptr(x, _bf16, "x", 2), _ptr(row_w, _f32, "row_w"), T, H, k, E, _ptr(topk_idx, _i32, "topk_idx"),
        int(reuse_map), _ptr(row_map, _i32, "row_map"), _ptr(offsets, _i32, "offsets"), _ptr(src_row, _i32, "src_row"),
        M_cap, _ptr(q, _u8, "q", 2), _ptr(s, _f32, "s", 2), int(align), _stream(stream)), "ff8_permute_quant_noalloc")


def ff8_permute_quant_dprobs(dy, row_w, k, E, row_map, offsets, src_row, q, s, y_perm, dprobs, stream=None):
    T, H = dy.shape
    M_cap = q.shape[0]
    _numel(row_w, T * k, "row_w"); _numel(row_map, T * k, "row_map"); _numel(dprobs, T * k, "dprobs")
    _numel(offsets, E + 1, "offsets"); _numel(src_row, M_cap, "src_row")
    _shape(q, (M_cap, H), "q"); _shape(s, (M_cap, H // 128), "s"); _shape(y_perm, (M_cap, H), "y_perm")
    sd, sfx = _scale_kind(s)
    name = "ff8_permute_quant_dprobs" + sfx
    _check(getattr(load(), name)(_ptr(dy, _bf16, "dy", 2), _ptr(row_w, _f32, "row_w"), T, H, k, E,
                                 _ptr(row_map, _i32, "row_map"), _ptr(offsets, _i32, "offsets"),
                                 _ptr(src_row, _i32, "src_row"), M_cap, _ptr(q, _u8, "q", 2), _ptr(s, sd, "s", 2),
                                 _ptr(y_perm, _bf16, "y_perm", 2), _ptr(dprobs, _f32, "dprobs"), _stream(stream)),
           name)


def ff8_scaling_aware_transpose(q, s, qT, sT, offsets=None, E=0, stream=None):
    """qT is K-blocked: [rows // 128, cols, 128], element (c, r) of the transpose at [r // 128, c, r % 128]."""
    rows, cols = q.shape
    _shape(s, (rows, cols // 128), "s"); _shape(qT, (rows // 128, cols, 128), "qT")
    _shape(sT, (rows // 128, cols), "sT")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    sd, sfx = _scale_kind(s, sT)
    name = "ff8_scaling_aware_transpose" + sfx
    _check(getattr(load(), name)(
        _ptr(q, _u8, "q", 2), _ptr(s, sd, "s", 2), rows, cols, _ptr(offsets, _i32, "offsets"), E,
        _ptr(qT, _u8, "qT", 3), _ptr(sT, sd, "sT", 2), _stream(stream)), name)


def ff8_scaling_aware_transpose_batch(qs, ss, qTs, sTs, offsets=None, E=0, stream=None):
    """Transposes of up to four tensors with the same rows in one launch; each tensor's
    arguments are those of ff8_scaling_aware_transpose."""
    n = len(qs)
    if not (len(ss) == len(qTs) == len(sTs) == n):
        raise ValueError("qs, ss, qTs and sTs must have the same length")
    if n == 0:
        raise ValueError("at least one tensor is required")
    rows = qs[0].shape[0]
    for i in range(n):
        r, cols = qs[i].shape
        if r != rows:
            raise ValueError(f"qs[{i}] must have shape ({rows}, cols): every tensor has the same rows")
        _shape(ss[i], (rows, cols // 128), f"ss[{i}]"); _shape(qTs[i], (rows // 128, cols, 128), f"qTs[{i}]")
        _shape(sTs[i], (rows // 128, cols), f"sTs[{i}]")
    sd, sfx = _scale_kind(*ss, *sTs)
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    arr = lambda vals: (ctypes.c_void_p * n)(*[v.value for v in vals])
    q_a = arr([_ptr(q, _u8, f"qs[{i}]", 2) for i, q in enumerate(qs)])
    s_a = arr([_ptr(x, sd, f"ss[{i}]", 2) for i, x in enumerate(ss)])
    qT_a = arr([_ptr(x, _u8, f"qTs[{i}]", 3) for i, x in enumerate(qTs)])
    sT_a = arr([_ptr(x, sd, f"sTs[{i}]", 2) for i, x in enumerate(sTs)])
    cols_a = (ctypes.c_int64 * n)(*[q.shape[1] for q in qs])
    name = "ff8_scaling_aware_transpose_batch" + sfx
    _check(getattr(load(), name)(n, q_a, s_a, cols_a, rows, _ptr(offsets, _i32, "offsets"), E, qT_a, sT_a,
                                 _stream(stream)), name)


def ff8_grouped_gemm_fprop(a, a_s, w, w_s, offsets, out, stream=None):
    M_cap, K = a.shape
    E, N, _ = w.shape
    _shape(a_s, (M_cap, K // 128), "a_s"); _shape(w, (E, N, K), "w"); _numel(w_s, E * (N // 128) * (K // 128), "w_s")
    _numel(offsets, E + 1, "offsets"); _shape(out, (M_cap, N), "out")
    sd, sfx = _scale_kind(a_s, w_s)
    name = "ff8_grouped_gemm_fprop" + sfx
    _check(getattr(load(), name)(
        _ptr(a, _u8, "a", 2), _ptr(a_s, sd, "a_s"), _ptr(w, _u8, "w", 3), _ptr(w_s, sd, "w_s"),
        _ptr(offsets, _i32, "offsets"), E, M_cap, N, K, _ptr(out, _bf16, "out", 2), _stream(stream)), name)


def ff8_grouped_gemm_dgrad(g, g_s, w, w_s, offsets, out, stream=None):
    M_cap, N = g.shape
    E, _, K = w.shape
    _shape(g_s, (M_cap, N // 128), "g_s"); _shape(w, (E, N, K), "w"); _numel(w_s, E * (N // 128) * (K // 128), "w_s")
    _numel(offsets, E + 1, "offsets"); _shape(out, (M_cap, K), "out")
    sd, sfx = _scale_kind(g_s, w_s)
    name = "ff8_grouped_gemm_dgrad" + sfx
    _check(getattr(load(), name)(
        _ptr(g, _u8, "g", 2), _ptr(g_s, sd, "g_s"), _ptr(w, _u8, "w", 3), _ptr(w_s, sd, "w_s"),
        _ptr(offsets, _i32, "offsets"), E, M_cap, N, K, _ptr(out, _bf16, "out", 2), _stream(stream)), name)


def ff8_grouped_gemm_wgrad(gT, gT_s, xT, xT_s, offsets, dw, accumulate=False, stream=None):
    """gT [M_cap // 128, N, 128] and xT [M_cap // 128, K, 128]: K-blocked transposes (as
    ff8_scaling_aware_transpose writes them)."""
    n_kb, N, _ = gT.shape
    M_cap = 128 * n_kb
    K = xT.shape[1]
    E = dw.shape[0]
    _shape(gT, (n_kb, N, 128), "gT"); _shape(gT_s, (n_kb, N), "gT_s"); _shape(xT, (n_kb, K, 128), "xT")
    _shape(xT_s, (n_kb, K), "xT_s")
    _numel(offsets, E + 1, "offsets"); _shape(dw, (E, N, K), "dw")
    sd, sfx = _scale_kind(gT_s, xT_s)
    name = "ff8_grouped_gemm_wgrad" + sfx
    _check(getattr(load(), name)(
        _ptr(gT, _u8, "gT", 3), _ptr(gT_s, sd, "gT_s"), _ptr(xT, _u8, "xT", 3), _ptr(xT_s, sd, "xT_s"),
        _ptr(offsets, _i32, "offsets"), E, M_cap, N, K, _ptr(dw, _f32, "dw", 3), int(bool(accumulate)),
        _stream(stream)), name)


def ff8_swiglu_quant(a, hq, hs, offsets=None, E=0, stream=None):
    M_cap, I2 = a.shape
    _shape(hq, (M_cap, I2 // 2), "hq"); _shape(hs, (M_cap, I2 // 256), "hs")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    sd, sfx = _scale_kind(hs)
    name = "ff8_swiglu_quant" + sfx
    _check(getattr(load(), name)(_ptr(a, _bf16, "a", 2), _ptr(offsets, _i32, "offsets"), E, M_cap, I2 // 2,
                                 _ptr(hq, _u8, "hq", 2), _ptr(hs, sd, "hs", 2), _stream(stream)), name)


def ff8_swiglu_bwd_quant(a, dh, daq, das, offsets=None, E=0, stream=None):
    M_cap, I2 = a.shape
    _shape(dh, (M_cap, I2 // 2), "dh"); _shape(daq, (M_cap, I2), "daq"); _shape(das, (M_cap, I2 // 128), "das")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    sd, sfx = _scale_kind(das)
    name = "ff8_swiglu_bwd_quant" + sfx
    _check(getattr(load(), name)(_ptr(a, _bf16, "a", 2), _ptr(dh, _bf16, "dh", 2),
                                 _ptr(offsets, _i32, "offsets"), E, M_cap, I2 // 2, _ptr(daq, _u8, "daq", 2),
                                 _ptr(das, sd, "das", 2), _stream(stream)), name)


def ff8_swiglu_quant_keep_fp8(a, hq, hs, a_q, a_s, offsets=None, E=0, stream=None):
    M_cap, I2 = a.shape
    _shape(hq, (M_cap, I2 // 2), "hq"); _shape(hs, (M_cap, I2 // 256), "hs")
    _shape(a_q, (M_cap, I2), "a_q"); _shape(a_s, (M_cap, I2 // 128), "a_s")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    sd, sfx = _scale_kind(hs, a_s)
    name = "ff8_swiglu_quant_keep_fp8" + sfx
    _check(getattr(load(), name)(_ptr(a, _bf16, "a", 2), _ptr(offsets, _i32, "offsets"), E, M_cap, I2 // 2,
                                 _ptr(hq, _u8, "hq", 2), _ptr(hs, sd, "hs", 2), _ptr(a_q, _u8, "a_q", 2),
                                 _ptr(a_s, sd, "a_s", 2), _stream(stream)), name)


def ff8_swiglu_bwd_quant_fp8a(a_q, a_s, dh, daq, das, offsets=None, E=0, stream=None):
    M_cap, I2 = a_q.shape
    _shape(a_s, (M_cap, I2 // 128), "a_s"); _shape(dh, (M_cap, I2 // 2), "dh")
    _shape(daq, (M_cap, I2), "daq"); _shape(das, (M_cap, I2 // 128), "das")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    sd, sfx = _scale_kind(a_s, das)
    name = "ff8_swiglu_bwd_quant_fp8a" + sfx
    _check(getattr(load(), name)(_ptr(a_q, _u8, "a_q", 2), _ptr(a_s, sd, "a_s", 2),
                                 _ptr(dh, _bf16, "dh", 2), _ptr(offsets, _i32, "offsets"), E, M_cap,
                                 I2 // 2, _ptr(daq, _u8, "daq", 2), _ptr(das, sd, "das", 2),
                                 _stream(stream)), name)


def ff8_unpermute(y_perm, row_map, row_w, y, stream=None):
    M_cap, H = y_perm.shape
    T, k = row_map.shape
    _numel(row_w, T * k, "row_w"); _shape(y, (T, H), "y")
    _check(load().ff8_unpermute(_ptr(y_perm, _bf16, "y_perm", 2), _ptr(row_map, _i32, "row_map", 2),
                                _ptr(row_w, _f32, "row_w"), T, k, H, M_cap, _ptr(y, _bf16, "y", 2),
                                _stream(stream)), "ff8_unpermute")


def ff8_cast_f32_to_e4m3(x, q, stream=None):
    _numel(q, x.numel(), "q")
    _check(load().ff8_cast_f32_to_e4m3(_ptr(x, _f32, "x"), x.numel(), _ptr(q, _u8, "q"), _stream(stream)),
           "ff8_cast_f32_to_e4m3")


def ff8_cast_e4m3_to_f32(q, x, stream=None):
    _numel(x, q.numel(), "x")
    _check(load().ff8_cast_e4m3_to_f32(_ptr(q, _u8, "q"), q.numel(), _ptr(x, _f32, "x"), _stream(stream)),
           "ff8_cast_e4m3_to_f32")


def ff8_baseline_dequant_rowwise(q, s, out, stream=None):
    rows, cols = q.shape
    _shape(s, (rows, cols // 128), "s"); _shape(out, (rows, cols), "out")
    _check(load().ff8_baseline_dequant_rowwise(_ptr(q, _u8, "q", 2), _ptr(s, _f32, "s", 2), rows, cols,
                                               _ptr(out, _bf16, "out", 2), _stream(stream)),
           "ff8_baseline_dequant_rowwise")


def ff8_baseline_transpose_bf16(x, out, stream=None):
    rows, cols = x.shape
    _shape(out, (cols, rows), "out")
    _check(load().ff8_baseline_transpose_bf16(_ptr(x, _bf16, "x", 2), rows, cols, _ptr(out, _bf16, "out", 2),
                                              _stream(stream)), "ff8_baseline_transpose_bf16")


def ff8_baseline_swiglu_bf16(a, h, offsets=None, E=0, stream=None):
    rows, I2 = a.shape
    _shape(h, (rows, I2 // 2), "h")
    if offsets is not None:
        _numel(offsets, E + 1, "offsets")
    _check(load().ff8_baseline_swiglu_bf16(_ptr(a, _bf16, "a", 2), _ptr(offsets, _i32, "offsets"), E, rows,
                                           I2 // 2, _ptr(h, _bf16, "h", 2), _stream(stream)),
           "ff8_baseline_swiglu_bf16")


def ff8_baseline_copy(src, dst, stream=None):
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < n:
        raise ValueError("dst is smaller than src")
    _check(load().ff8_baseline_copy(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()), n,
                                    _stream(stream)), "ff8_baseline_copy")
