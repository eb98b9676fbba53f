// Host-side launchers of the gfx950 kernels.  Arguments are already validated by
// the C ABI layer (ff8_api.cpp); each launcher only enqueues work on `stream`.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ff8 {

// UE8M0 scale byte (T + 127 for the scale 2^T)
typedef uint8_t e8m0_t;

hipError_t launch_quant_rowwise(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, float* s,
                                hipStream_t st);
hipError_t launch_quant_block128(const uint16_t* w, int64_t rows, int64_t cols, uint8_t* q, float* s,
                                 hipStream_t st);
hipError_t launch_quant_rowwise(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, e8m0_t* s, hipStream_t st);
hipError_t launch_quant_block128(const uint16_t* w, int64_t rows, int64_t cols, uint8_t* q, e8m0_t* s,
                                 hipStream_t st);
hipError_t launch_cast_f32_e4m3(const float* x, int64_t n, uint8_t* q, hipStream_t st);
hipError_t launch_cast_e4m3_f32(const uint8_t* q, int64_t n, float* x, hipStream_t st);
hipError_t launch_dequant_rowwise(const uint8_t* q, const float* s, int64_t rows, int64_t cols, uint16_t* out,
                                  hipStream_t st);
hipError_t launch_dequant_rowwise(const uint8_t* q, const e8m0_t* s, int64_t rows, int64_t cols, uint16_t* out,
                                  hipStream_t st);
hipError_t launch_transpose_bf16(const uint16_t* in, int64_t rows, int64_t cols, uint16_t* out, hipStream_t st);
hipError_t launch_copy(const void* src, void* dst, int64_t nbytes, hipStream_t st);

hipError_t launch_sat(const uint8_t* q, const float* s, int64_t rows, int64_t cols, const int32_t* offsets, int E,
                      uint8_t* qT, float* sT, hipStream_t st);
hipError_t launch_sat(const uint8_t* q, const e8m0_t* s, int64_t rows, int64_t cols, const int32_t* offsets, int E,
                      uint8_t* qT, e8m0_t* sT, hipStream_t st);
// Up to kSatMaxJobs tensors with the same rows (and active rows) in one launch.
constexpr int kSatMaxJobs = 4;
hipError_t launch_sat_batch(int n, const uint8_t* const* q, const float* const* s, const int64_t* cols, int64_t rows,
                            const int32_t* offsets, int E, uint8_t* const* qT, float* const* sT, hipStream_t st);
hipError_t launch_sat_batch(int n, const uint8_t* const* q, const e8m0_t* const* s, const int64_t* cols, int64_t rows,
                            const int32_t* offsets, int E, uint8_t* const* qT, e8m0_t* const* sT, hipStream_t st);

constexpr int kRouteChunk = 256;  // tokens per routing chunk: the workspace holds ceil(T / 256) x E counts
size_t permute_workspace_bytes(int64_t T, int k, int E);
// Capacity (int32 entries) of the routing workspace the library keeps in device memory for the
// no-allocation entry point, and its device address on the current device (looked up once per
// device; the array is resident until the process ends).
constexpr int64_t kRouteScratchInts = (int64_t)1 << 18;
hipError_t route_scratch(int32_t** out);
hipError_t launch_route(const int32_t* topk_idx, int64_t T, int k, int E, int align, int32_t* row_map,
                        int32_t* offsets, int32_t* src_row, int64_t M_cap, void* workspace, hipStream_t st);
hipError_t launch_permute_quant(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                int64_t M_cap, uint8_t* q, float* s, hipStream_t st);
hipError_t launch_permute_quant(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                int64_t M_cap, uint8_t* q, e8m0_t* s, hipStream_t st);
hipError_t launch_permute_quant_dprobs(const uint16_t* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                       const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                       int64_t M_cap, uint8_t* q, float* s, const uint16_t* y_perm, float* dprobs,
                                       hipStream_t st);
hipError_t launch_permute_quant_dprobs(const uint16_t* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                       const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                       int64_t M_cap, uint8_t* q, e8m0_t* s, const uint16_t* y_perm, float* dprobs,
                                       hipStream_t st);
int max_k_dprobs();
int64_t max_h_dprobs();
hipError_t launch_unpermute(const uint16_t* y_perm, const int32_t* row_map, const float* row_w, int64_t T, int k,
                            int64_t H, int64_t M_cap, uint16_t* y, hipStream_t st);

hipError_t launch_swiglu_quant(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                               uint8_t* hq, float* hs, hipStream_t st);
hipError_t launch_swiglu_quant(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                               uint8_t* hq, e8m0_t* hs, hipStream_t st);
hipError_t launch_swiglu_bwd_quant(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E,
                                   int64_t M_cap, int64_t I, uint8_t* daq, float* das, hipStream_t st);
hipError_t launch_swiglu_bwd_quant(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E,
                                   int64_t M_cap, int64_t I, uint8_t* daq, e8m0_t* das, hipStream_t st);
hipError_t launch_swiglu_quant_keep_fp8(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                        uint8_t* hq, float* hs, uint8_t* aq, float* as_, hipStream_t st);
hipError_t launch_swiglu_quant_keep_fp8(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                        uint8_t* hq, e8m0_t* hs, uint8_t* aq, e8m0_t* as_, hipStream_t st);
hipError_t launch_swiglu_bwd_quant_fp8a(const uint8_t* aq, const float* as_, const uint16_t* dh, const int32_t* offsets,
                                        int E, int64_t M_cap, int64_t I, uint8_t* daq, float* das, hipStream_t st);
hipError_t launch_swiglu_bwd_quant_fp8a(const uint8_t* aq, const e8m0_t* as_, const uint16_t* dh,
                                        const int32_t* offsets, int E, int64_t M_cap, int64_t I, uint8_t* daq,
                                        e8m0_t* das, hipStream_t st);
hipError_t launch_swiglu_bf16(const uint16_t* a, const int32_t* offsets, int E, int64_t rows, int64_t I,
                              uint16_t* h, hipStream_t st);

enum GemmMode { kFprop = 0, kDgrad = 1, kWgrad = 2 };
hipError_t launch_grouped_gemm(GemmMode mode, const uint8_t* a, const float* a_s, const uint8_t* b,
                               const float* b_s, const int32_t* offsets, int E, int64_t M_cap, int64_t N,
                               int64_t K, void* out, int accumulate, hipStream_t st);
// UE8M0 scales: fprop needs K % 512 == 0, dgrad N % 512 == 0 and K % 512 == 0 (the scale
// DMAs move dwords of four scale bytes)
hipError_t launch_grouped_gemm(GemmMode mode, const uint8_t* a, const e8m0_t* a_s, const uint8_t* b,
                               const e8m0_t* b_s, const int32_t* offsets, int E, int64_t M_cap, int64_t N,
                               int64_t K, void* out, int accumulate, hipStream_t st);

// Number of workgroups that fill the device (CU count x `per_cu`), cached per device.
int device_cu_count();

}  // namespace ff8
