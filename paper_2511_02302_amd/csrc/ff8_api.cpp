// C ABI of the FP8-Flow-MoE expert-layer library: host-side argument validation,
// error reporting, and dispatch to the gfx950 launchers.  Validation happens before
// anything is enqueued; the library allocates no memory and keeps no state apart
// from a thread-local error string and a per-device CU count.

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/ff8.h"
#include "ff8_launch.hpp"

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

int hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) {
    g_err[0] = '\0';
    return FF8_OK;
  }
  return fail(FF8_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool mult128(int64_t v) { return v > 0 && v % 128 == 0; }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

#define REQUIRE_PTR(p) \
  if ((p) == nullptr) return fail(FF8_ERR_NULL, "%s: argument '%s' is NULL", __func__, #p)
#define REQUIRE_SHAPE(cond) \
  if (!(cond)) return fail(FF8_ERR_SHAPE, "%s: shape check failed: %s", __func__, #cond)
#define REQUIRE_ARG(cond) \
  if (!(cond)) return fail(FF8_ERR_ARG, "%s: argument check failed: %s", __func__, #cond)

}  // namespace

namespace ff8 {

int device_cu_count() {
  static std::mutex mu;
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  std::lock_guard<std::mutex> lock(mu);
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

}  // namespace ff8

template <typename S>
static int sat_batch(const char* fn, int n, const ff8_e4m3* const* q, const S* const* s, const int64_t* cols,
                     int64_t rows, const int32_t* offsets, int E, ff8_e4m3* const* qT, S* const* sT, void* stream) {
  if (n < 1 || n > ff8::kSatMaxJobs) return fail(FF8_ERR_ARG, "%s: n must be in [1, %d]", fn, ff8::kSatMaxJobs);
  if (!q || !s || !cols || !qT || !sT) return fail(FF8_ERR_NULL, "%s: a required array is NULL", fn);
  for (int i = 0; i < n; ++i) {
    if (!q[i] || !s[i] || !qT[i] || !sT[i]) return fail(FF8_ERR_NULL, "%s: a pointer of tensor %d is NULL", fn, i);
    if (!mult128(cols[i])) return fail(FF8_ERR_SHAPE, "%s: cols[%d] must be a positive multiple of 128", fn, i);
  }
  if (!mult128(rows)) return fail(FF8_ERR_SHAPE, "%s: rows must be a positive multiple of 128", fn);
  if (offsets && E < 1) return fail(FF8_ERR_ARG, "%s: E must be >= 1 with offsets", fn);
  return hip_status(ff8::launch_sat_batch(n, q, s, cols, rows, offsets, E, qT, sT, as_stream(stream)), fn);
}

template <typename S>
static int permute_quant_dprobs_common(const char* fn, const ff8_bf16* dy, const float* row_w, int64_t T, int64_t H,
                                       int k, int E, const int32_t* row_map, const int32_t* offsets,
                                       const int32_t* src_row, int64_t M_cap, ff8_e4m3* q, S* s,
                                       const ff8_bf16* y_perm, float* dprobs, void* stream) {
  if (!(k >= 1 && E >= 1 && k <= E && E <= 1024 && k <= ff8::max_k_dprobs()))
    return fail(FF8_ERR_ARG, "%s: need 1 <= k <= E <= 1024 and k <= %d", fn, ff8::max_k_dprobs());
  if (!(T >= 0 && mult128(H) && H <= ff8::max_h_dprobs() && M_cap % 128 == 0))
    return fail(FF8_ERR_SHAPE, "%s: H must be a multiple of 128 up to %lld and M_cap a multiple of 128", fn,
                (long long)ff8::max_h_dprobs());
  if (M_cap < ff8_rows_bound_aligned(T, k, E, 16))  // the map may come from any alignment
    return fail(FF8_ERR_SHAPE, "%s: M_cap is below the row bound", fn);
  if (!(T * (int64_t)k < (int64_t)1 << 31 && M_cap < (int64_t)1 << 31))
    return fail(FF8_ERR_SHAPE, "%s: T*k and M_cap must be below 2^31", fn);
  if (T > 0 && (!dy || !row_w || !y_perm || !dprobs || !row_map))  // an empty batch may pass NULL for these
    return fail(FF8_ERR_NULL, "%s: dy, row_w, y_perm, dprobs or row_map is NULL", fn);
  if (!offsets || !src_row || !q || !s) return fail(FF8_ERR_NULL, "%s: offsets, src_row, q or s is NULL", fn);
  return hip_status(ff8::launch_permute_quant_dprobs(dy, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s,
                                                     y_perm, dprobs, as_stream(stream)),
                    fn);
}

extern "C" {

int ff8_version(void) { return 100; }

const char* ff8_status_string(int status) {
  switch (status) {
    case FF8_OK: return "ok";
    case FF8_ERR_NULL: return "null pointer";
    case FF8_ERR_SHAPE: return "bad shape";
    case FF8_ERR_ARG: return "bad argument";
    case FF8_ERR_HIP: return "HIP error";
    default: return "unknown status";
  }
}

const char* ff8_last_error(void) { return g_err; }

int ff8_quant_rowwise(const ff8_bf16* x, int64_t rows, int64_t cols, ff8_e4m3* q, float* s, void* stream) {
  REQUIRE_PTR(x); REQUIRE_PTR(q); REQUIRE_PTR(s);
  REQUIRE_SHAPE(rows >= 1 && mult128(cols));
  return hip_status(ff8::launch_quant_rowwise(x, rows, cols, q, s, as_stream(stream)), __func__);
}

int ff8_quant_block128(const ff8_bf16* w, int64_t rows, int64_t cols, ff8_e4m3* q, float* s, void* stream) {
  REQUIRE_PTR(w); REQUIRE_PTR(q); REQUIRE_PTR(s);
  REQUIRE_SHAPE(mult128(rows) && mult128(cols));
  return hip_status(ff8::launch_quant_block128(w, rows, cols, q, s, as_stream(stream)), __func__);
}

int64_t ff8_rows_bound_aligned(int64_t T, int k, int E, int align) {
  if (T < 0 || k < 1 || E < 1 || k > E || !(align == 16 || align == 32 || align == 64 || align == 128)) return -1;
  const int64_t need = T * k + (int64_t)(align - 1) * E;
  return (need + 127) / 128 * 128;
}

int64_t ff8_rows_bound(int64_t T, int k, int E) { return ff8_rows_bound_aligned(T, k, E, 128); }

size_t ff8_permute_workspace_bytes(int64_t T, int k, int E) {
  if (T < 0 || k < 1 || E < 1) return 0;
  return ff8::permute_workspace_bytes(T, k, E);
}

}  // extern "C"

// Host-side checks of a permute call; `ws_need_check` is false for the no-allocation entry
// point, whose workspace is the library's own.
static int permute_validate(const char* fn, const void* x, int64_t T, int64_t H, int k, int E, const void* topk_idx,
                            int reuse_map, const void* row_map, const void* offsets, const void* src_row, int64_t M_cap,
                            const void* q, const void* s, const void* workspace, size_t ws_bytes, int align,
                            bool ws_need_check) {
  if (!(reuse_map == 0 || reuse_map == 1)) return fail(FF8_ERR_ARG, "%s: reuse_map must be 0 or 1", fn);
  if (!(k >= 1 && E >= 1 && k <= E && E <= 1024)) return fail(FF8_ERR_ARG, "%s: need 1 <= k <= E <= 1024", fn);
  if (!(align == 16 || align == 32 || align == 64 || align == 128))
    return fail(FF8_ERR_ARG, "%s: align must be 16, 32, 64 or 128", fn);
  if (!(T >= 0 && mult128(H) && M_cap % 128 == 0))
    return fail(FF8_ERR_SHAPE, "%s: need T >= 0, H and M_cap multiples of 128", fn);
  // a reused map may come from any alignment: only the smallest bound is known here
  if (M_cap < ff8_rows_bound_aligned(T, k, E, reuse_map ? 16 : align))
    return fail(FF8_ERR_SHAPE, "%s: M_cap is below the row bound", fn);
  if (!(T * (int64_t)k < (int64_t)1 << 31 && M_cap < (int64_t)1 << 31))
    return fail(FF8_ERR_SHAPE, "%s: T*k and M_cap must be below 2^31", fn);
  if (T > 0 && (!x || !row_map)) return fail(FF8_ERR_NULL, "%s: x or row_map is NULL", fn);
  if (!offsets || !src_row || !q || !s) return fail(FF8_ERR_NULL, "%s: offsets, src_row, q or s is NULL", fn);
  if (!reuse_map) {
    if (T > 0 && !topk_idx) return fail(FF8_ERR_NULL, "%s: topk_idx is NULL", fn);
    if (ws_need_check) {
      const size_t need = ff8::permute_workspace_bytes(T, k, E);
      if (need > 0 && !workspace) return fail(FF8_ERR_NULL, "%s: workspace is NULL", fn);
      if (ws_bytes < need) return fail(FF8_ERR_ARG, "%s: workspace of %zu bytes, %zu needed", fn, ws_bytes, need);
    }
  }
  return FF8_OK;
}

template <typename SC>
static int permute_launch(const char* fn, const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                          const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets, int32_t* src_row,
                          int64_t M_cap, ff8_e4m3* q, SC* s, void* workspace, int align, hipStream_t st) {
  if (!reuse_map) {
    const int rc = hip_status(
        ff8::launch_route(topk_idx, T, k, E, align, row_map, offsets, src_row, M_cap, workspace, st), fn);
    if (rc != FF8_OK) return rc;
  }
  return hip_status(ff8::launch_permute_quant(x, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, st), fn);
}

extern "C" {

int ff8_permute_quant_aligned(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                              const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets,
                              int32_t* src_row, int64_t M_cap, ff8_e4m3* q, float* s, void* workspace,
                              size_t ws_bytes, int align, void* stream) {
  const int rc = permute_validate(__func__, x, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                                  workspace, ws_bytes, align, true);
  if (rc != FF8_OK) return rc;
  return permute_launch(__func__, x, row_w, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                        workspace, align, as_stream(stream));
}

int ff8_permute_quant(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                      const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets, int32_t* src_row,
                      int64_t M_cap, ff8_e4m3* q, float* s, void* workspace, size_t ws_bytes, void* stream) {
  return ff8_permute_quant_aligned(x, row_w, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                                   workspace, ws_bytes, 128, stream);
}

int ff8_permute_quant_noalloc(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                              const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets,
                              int32_t* src_row, int64_t M_cap, ff8_e4m3* q, float* s, int align, void* stream) {
  int rc = permute_validate(__func__, x, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                            nullptr, 0, align, false);
  if (rc != FF8_OK) return rc;
  const size_t need = ff8::permute_workspace_bytes(T, k, E);
  if (!reuse_map && need > (size_t)ff8::kRouteScratchInts * sizeof(int32_t))
    return fail(FF8_ERR_ARG,
                "%s: the routing of T = %lld tokens over E = %d experts needs %zu bytes of workspace, more than the "
                "%lld bytes the library holds (ceil(T / %d) * E must not exceed %lld); use ff8_permute_quant_aligned "
                "with a caller-owned workspace",
                __func__, (long long)T, E, need, (long long)(ff8::kRouteScratchInts * 4), ff8::kRouteChunk,
                (long long)ff8::kRouteScratchInts);
  int32_t* ws = nullptr;
  if (!reuse_map) {
    rc = hip_status(ff8::route_scratch(&ws), __func__);
    if (rc != FF8_OK) return rc;
  }
  return permute_launch(__func__, x, row_w, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s, ws,
                        align, as_stream(stream));
}

int ff8_permute_quant_dprobs(const ff8_bf16* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                             const int32_t* row_map, const int32_t* offsets, const int32_t* src_row, int64_t M_cap,
                             ff8_e4m3* q, float* s, const ff8_bf16* y_perm, float* dprobs, void* stream) {
  return permute_quant_dprobs_common(__func__, dy, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, y_perm,
                                     dprobs, stream);
}

int ff8_permute_quant_dprobs_e8m0(const ff8_bf16* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                  const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                  int64_t M_cap, ff8_e4m3* q, ff8_e8m0* s, const ff8_bf16* y_perm, float* dprobs,
                                  void* stream) {
  return permute_quant_dprobs_common(__func__, dy, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, y_perm,
                                     dprobs, stream);
}

int ff8_scaling_aware_transpose(const ff8_e4m3* q, const float* s, int64_t rows, int64_t cols,
                                const int32_t* offsets, int E, ff8_e4m3* qT, float* sT, void* stream) {
  REQUIRE_PTR(q); REQUIRE_PTR(s); REQUIRE_PTR(qT); REQUIRE_PTR(sT);
  REQUIRE_SHAPE(mult128(rows) && mult128(cols));
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_sat(q, s, rows, cols, offsets, E, qT, sT, as_stream(stream)), __func__);
}

int ff8_scaling_aware_transpose_batch(int n, const ff8_e4m3* const* q, const float* const* s, const int64_t* cols,
                                      int64_t rows, const int32_t* offsets, int E, ff8_e4m3* const* qT,
                                      float* const* sT, void* stream) {
  return sat_batch(__func__, n, q, s, cols, rows, offsets, E, qT, sT, stream);
}

int ff8_scaling_aware_transpose_batch_e8m0(int n, const ff8_e4m3* const* q, const ff8_e8m0* const* s,
                                           const int64_t* cols, int64_t rows, const int32_t* offsets, int E,
                                           ff8_e4m3* const* qT, ff8_e8m0* const* sT, void* stream) {
  return sat_batch(__func__, n, q, s, cols, rows, offsets, E, qT, sT, stream);
}

static int gemm_common(const char* fn, const void* a, const void* as, const void* b, const void* bs,
                       const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, const void* out,
                       bool expert_weights) {
  if (!a || !as || !b || !bs || !offsets || !out) return fail(FF8_ERR_NULL, "%s: a required pointer is NULL", fn);
  // fprop and dgrad keep per-expert tile counts and row offsets in LDS tables of 1025 entries
  if (E < 1 || E > 1024) return fail(FF8_ERR_ARG, "%s: E must be in [1, 1024]", fn);
  if (!mult128(M_cap) || !mult128(N) || !mult128(K))
    return fail(FF8_ERR_SHAPE, "%s: M_cap, N and K must be positive multiples of 128", fn);
  // the kernels address each operand tensor (the token-major activations, all experts'
  // weights) with 32-bit byte offsets
  const int64_t lim = (int64_t)1 << 32;
  if (M_cap * (N > K ? N : K) >= lim || (expert_weights ? (int64_t)E * N * K : N * K) >= lim)
    return fail(FF8_ERR_SHAPE, "%s: an operand exceeds 4 GiB (M_cap*max(N,K) and E*N*K must be < 2^32)", fn);
  return FF8_OK;
}

int ff8_grouped_gemm_fprop(const ff8_e4m3* a, const float* a_s, const ff8_e4m3* w, const float* w_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                           void* stream) {
  const int rc = gemm_common(__func__, a, a_s, w, w_s, offsets, E, M_cap, N, K, out, true);
  if (rc != FF8_OK) return rc;
  return hip_status(ff8::launch_grouped_gemm(ff8::kFprop, a, a_s, w, w_s, offsets, E, M_cap, N, K, out, 0,
                                             as_stream(stream)),
                    __func__);
}

int ff8_grouped_gemm_dgrad(const ff8_e4m3* g, const float* g_s, const ff8_e4m3* w, const float* w_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                           void* stream) {
  const int rc = gemm_common(__func__, g, g_s, w, w_s, offsets, E, M_cap, N, K, out, true);
  if (rc != FF8_OK) return rc;
  return hip_status(ff8::launch_grouped_gemm(ff8::kDgrad, g, g_s, w, w_s, offsets, E, M_cap, N, K, out, 0,
                                             as_stream(stream)),
                    __func__);
}

int ff8_grouped_gemm_wgrad(const ff8_e4m3* gT, const float* gT_s, const ff8_e4m3* xT, const float* xT_s,
                           const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, float* dw,
                           int accumulate, void* stream) {
  const int rc = gemm_common(__func__, gT, gT_s, xT, xT_s, offsets, E, M_cap, N, K, dw, false);
  if (rc != FF8_OK) return rc;
  REQUIRE_ARG(accumulate == 0 || accumulate == 1);
  return hip_status(ff8::launch_grouped_gemm(ff8::kWgrad, gT, gT_s, xT, xT_s, offsets, E, M_cap, N, K, dw,
                                             accumulate, as_stream(stream)),
                    __func__);
}

int ff8_swiglu_quant(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I, ff8_e4m3* hq,
                     float* hs, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(hq); REQUIRE_PTR(hs);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_quant(a, offsets, E, M_cap, I, hq, hs, as_stream(stream)), __func__);
}

int ff8_swiglu_bwd_quant(const ff8_bf16* a, const ff8_bf16* dh, const int32_t* offsets, int E, int64_t M_cap,
                         int64_t I, ff8_e4m3* daq, float* das, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(dh); REQUIRE_PTR(daq); REQUIRE_PTR(das);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_bwd_quant(a, dh, offsets, E, M_cap, I, daq, das, as_stream(stream)),
                    __func__);
}

int ff8_swiglu_quant_keep_fp8(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                              ff8_e4m3* hq, float* hs, ff8_e4m3* a_q, float* a_s, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(hq); REQUIRE_PTR(hs); REQUIRE_PTR(a_q); REQUIRE_PTR(a_s);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_quant_keep_fp8(a, offsets, E, M_cap, I, hq, hs, a_q, a_s, as_stream(stream)),
                    __func__);
}

int ff8_swiglu_bwd_quant_fp8a(const ff8_e4m3* a_q, const float* a_s, const ff8_bf16* dh, const int32_t* offsets,
                              int E, int64_t M_cap, int64_t I, ff8_e4m3* daq, float* das, void* stream) {
  REQUIRE_PTR(a_q); REQUIRE_PTR(a_s); REQUIRE_PTR(dh); REQUIRE_PTR(daq); REQUIRE_PTR(das);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(
      ff8::launch_swiglu_bwd_quant_fp8a(a_q, a_s, dh, offsets, E, M_cap, I, daq, das, as_stream(stream)), __func__);
}

int ff8_unpermute(const ff8_bf16* y_perm, const int32_t* row_map, const float* row_w, int64_t T, int k, int64_t H,
                  int64_t M_cap, ff8_bf16* y, void* stream) {
  REQUIRE_ARG(k >= 1);
  REQUIRE_SHAPE(T >= 0 && mult128(H) && M_cap >= 1);
  if (T > 0) {
    REQUIRE_PTR(y_perm); REQUIRE_PTR(row_map); REQUIRE_PTR(y);
  }
  return hip_status(ff8::launch_unpermute(y_perm, row_map, row_w, T, k, H, M_cap, y, as_stream(stream)), __func__);
}

/* ---- UE8M0 scale storage: the same operations with one scale byte T + 127 ---- */

int ff8_quant_rowwise_e8m0(const ff8_bf16* x, int64_t rows, int64_t cols, ff8_e4m3* q, ff8_e8m0* s, void* stream) {
  REQUIRE_PTR(x); REQUIRE_PTR(q); REQUIRE_PTR(s);
  REQUIRE_SHAPE(rows >= 1 && mult128(cols));
  return hip_status(ff8::launch_quant_rowwise(x, rows, cols, q, s, as_stream(stream)), __func__);
}

int ff8_quant_block128_e8m0(const ff8_bf16* w, int64_t rows, int64_t cols, ff8_e4m3* q, ff8_e8m0* s, void* stream) {
  REQUIRE_PTR(w); REQUIRE_PTR(q); REQUIRE_PTR(s);
  REQUIRE_SHAPE(mult128(rows) && mult128(cols));
  return hip_status(ff8::launch_quant_block128(w, rows, cols, q, s, as_stream(stream)), __func__);
}

int ff8_permute_quant_e8m0(const ff8_bf16* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                           const int32_t* topk_idx, int reuse_map, int32_t* row_map, int32_t* offsets, int32_t* src_row,
                           int64_t M_cap, ff8_e4m3* q, ff8_e8m0* s, void* workspace, size_t ws_bytes, int align,
                           void* stream) {
  const int rc = permute_validate(__func__, x, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                                  workspace, ws_bytes, align, true);
  if (rc != FF8_OK) return rc;
  return permute_launch(__func__, x, row_w, T, H, k, E, topk_idx, reuse_map, row_map, offsets, src_row, M_cap, q, s,
                        workspace, align, as_stream(stream));
}

int ff8_scaling_aware_transpose_e8m0(const ff8_e4m3* q, const ff8_e8m0* s, int64_t rows, int64_t cols,
                                     const int32_t* offsets, int E, ff8_e4m3* qT, ff8_e8m0* sT, void* stream) {
  REQUIRE_PTR(q); REQUIRE_PTR(s); REQUIRE_PTR(qT); REQUIRE_PTR(sT);
  REQUIRE_SHAPE(mult128(rows) && mult128(cols));
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_sat(q, s, rows, cols, offsets, E, qT, sT, as_stream(stream)), __func__);
}

int ff8_grouped_gemm_fprop_e8m0(const ff8_e4m3* a, const ff8_e8m0* a_s, const ff8_e4m3* w, const ff8_e8m0* w_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                                void* stream) {
  const int rc = gemm_common(__func__, a, a_s, w, w_s, offsets, E, M_cap, N, K, out, true);
  if (rc != FF8_OK) return rc;
  REQUIRE_SHAPE(K % 512 == 0);  // the scale DMAs move dwords of four K-block bytes
  return hip_status(ff8::launch_grouped_gemm(ff8::kFprop, a, a_s, w, w_s, offsets, E, M_cap, N, K, out, 0,
                                             as_stream(stream)),
                    __func__);
}

int ff8_grouped_gemm_dgrad_e8m0(const ff8_e4m3* g, const ff8_e8m0* g_s, const ff8_e4m3* w, const ff8_e8m0* w_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, ff8_bf16* out,
                                void* stream) {
  const int rc = gemm_common(__func__, g, g_s, w, w_s, offsets, E, M_cap, N, K, out, true);
  if (rc != FF8_OK) return rc;
  REQUIRE_SHAPE(N % 512 == 0 && K % 512 == 0);  // the scale DMAs move dwords of four scale bytes
  return hip_status(ff8::launch_grouped_gemm(ff8::kDgrad, g, g_s, w, w_s, offsets, E, M_cap, N, K, out, 0,
                                             as_stream(stream)),
                    __func__);
}

int ff8_grouped_gemm_wgrad_e8m0(const ff8_e4m3* gT, const ff8_e8m0* gT_s, const ff8_e4m3* xT, const ff8_e8m0* xT_s,
                                const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, float* dw,
                                int accumulate, void* stream) {
  const int rc = gemm_common(__func__, gT, gT_s, xT, xT_s, offsets, E, M_cap, N, K, dw, false);
  if (rc != FF8_OK) return rc;
  REQUIRE_ARG(accumulate == 0 || accumulate == 1);
  return hip_status(ff8::launch_grouped_gemm(ff8::kWgrad, gT, gT_s, xT, xT_s, offsets, E, M_cap, N, K, dw,
                                             accumulate, as_stream(stream)),
                    __func__);
}

int ff8_swiglu_quant_e8m0(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I, ff8_e4m3* hq,
                          ff8_e8m0* hs, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(hq); REQUIRE_PTR(hs);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_quant(a, offsets, E, M_cap, I, hq, hs, as_stream(stream)), __func__);
}

int ff8_swiglu_bwd_quant_e8m0(const ff8_bf16* a, const ff8_bf16* dh, const int32_t* offsets, int E, int64_t M_cap,
                              int64_t I, ff8_e4m3* daq, ff8_e8m0* das, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(dh); REQUIRE_PTR(daq); REQUIRE_PTR(das);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_bwd_quant(a, dh, offsets, E, M_cap, I, daq, das, as_stream(stream)), __func__);
}

int ff8_swiglu_quant_keep_fp8_e8m0(const ff8_bf16* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                   ff8_e4m3* hq, ff8_e8m0* hs, ff8_e4m3* a_q, ff8_e8m0* a_s, void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(hq); REQUIRE_PTR(hs); REQUIRE_PTR(a_q); REQUIRE_PTR(a_s);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_quant_keep_fp8(a, offsets, E, M_cap, I, hq, hs, a_q, a_s, as_stream(stream)),
                    __func__);
}

int ff8_swiglu_bwd_quant_fp8a_e8m0(const ff8_e4m3* a_q, const ff8_e8m0* a_s, const ff8_bf16* dh,
                                   const int32_t* offsets, int E, int64_t M_cap, int64_t I, ff8_e4m3* daq,
                                   ff8_e8m0* das, void* stream) {
  REQUIRE_PTR(a_q); REQUIRE_PTR(a_s); REQUIRE_PTR(dh); REQUIRE_PTR(daq); REQUIRE_PTR(das);
  REQUIRE_SHAPE(M_cap >= 1 && mult128(I));
  REQUIRE_SHAPE(M_cap * (I / 8) / 256 < ((int64_t)1 << 31));  // grid size
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(
      ff8::launch_swiglu_bwd_quant_fp8a(a_q, a_s, dh, offsets, E, M_cap, I, daq, das, as_stream(stream)), __func__);
}

int ff8_cast_f32_to_e4m3(const float* x, int64_t n, ff8_e4m3* q, void* stream) {
  REQUIRE_SHAPE(n >= 0);
  if (n == 0) return FF8_OK;
  REQUIRE_PTR(x); REQUIRE_PTR(q);
  REQUIRE_ARG(((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 3) == 0);
  return hip_status(ff8::launch_cast_f32_e4m3(x, n, q, as_stream(stream)), __func__);
}

int ff8_cast_e4m3_to_f32(const ff8_e4m3* q, int64_t n, float* x, void* stream) {
  REQUIRE_SHAPE(n >= 0);
  if (n == 0) return FF8_OK;
  REQUIRE_PTR(x); REQUIRE_PTR(q);
  REQUIRE_ARG(((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 3) == 0);
  return hip_status(ff8::launch_cast_e4m3_f32(q, n, x, as_stream(stream)), __func__);
}

int ff8_baseline_dequant_rowwise(const ff8_e4m3* q, const float* s, int64_t rows, int64_t cols, ff8_bf16* out,
                                 void* stream) {
  REQUIRE_PTR(q); REQUIRE_PTR(s); REQUIRE_PTR(out);
  REQUIRE_SHAPE(rows >= 1 && mult128(cols));
  return hip_status(ff8::launch_dequant_rowwise(q, s, rows, cols, out, as_stream(stream)), __func__);
}

int ff8_baseline_transpose_bf16(const ff8_bf16* in, int64_t rows, int64_t cols, ff8_bf16* out, void* stream) {
  REQUIRE_PTR(in); REQUIRE_PTR(out);
  REQUIRE_SHAPE(rows > 0 && cols > 0 && rows % 64 == 0 && cols % 64 == 0);
  return hip_status(ff8::launch_transpose_bf16(in, rows, cols, out, as_stream(stream)), __func__);
}

int ff8_baseline_swiglu_bf16(const ff8_bf16* a, const int32_t* offsets, int E, int64_t rows, int64_t I, ff8_bf16* h,
                             void* stream) {
  REQUIRE_PTR(a); REQUIRE_PTR(h);
  REQUIRE_SHAPE(rows >= 1 && mult128(I));
  if (offsets) REQUIRE_ARG(E >= 1);
  return hip_status(ff8::launch_swiglu_bf16(a, offsets, E, rows, I, h, as_stream(stream)), __func__);
}

int ff8_baseline_copy(const void* src, void* dst, int64_t nbytes, void* stream) {
  REQUIRE_PTR(src); REQUIRE_PTR(dst);
  REQUIRE_SHAPE(nbytes > 0 && nbytes % 16 == 0);
  return hip_status(ff8::launch_copy(src, dst, nbytes, as_stream(stream)), __func__);
}

}  // extern "C"
