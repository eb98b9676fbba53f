// Fused SwiGLU + quantization (paper section 3.3.2) and its backward twin, for gfx950.
//
// The fc1 output A [rows, 2I] is [gate | up].  Work item (m, c) covers 8 output
// columns of row m; 16 consecutive items form one 1x128 output tile, so the tile amax
// is a 16-lane DPP reduction and the activation goes from float32 registers straight
// to e4m3 without a bf16 round trip.  Rows at and beyond offsets[E] are skipped.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ float sigmoid(float g) { return __frcp_rn(1.0f + __expf(-g)); }

// One item per thread, no grid-stride loop.  Holding several items per thread issues
// more loads up front but measured slower inside the layer step, where A was just
// written by the fc1 GEMM.
__global__ __launch_bounds__(kThreads) void swiglu_quant_kernel(const uint16_t* __restrict__ a,
                                                                const int32_t* __restrict__ offsets, int E,
                                                                int64_t M_cap, int64_t I, uint8_t* __restrict__ hq,
                                                                float* __restrict__ hs) {
  const int64_t rows = active_rows(offsets, E, M_cap);
  const int64_t cpr = I / 8, n_items = rows * cpr, sh = I / kTile;
  const int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (it >= n_items) return;  // whole 16-lane tiles (cpr is a multiple of 16)
  const int64_t m = it / cpr, c = it - m * cpr;
  const uint16_t* row = a + m * 2 * I + c * 8;
  float g[8], u[8], h[8];
  unpack_bf16x8(ldnt16(row), g);
  unpack_bf16x8(ldnt16(row + I), u);
#pragma unroll
  for (int i = 0; i < 8; ++i) h[i] = g[i] * sigmoid(g[i]) * u[i];
  int t;
  const u32x2 r = quant8_tile16(h, t);
  stnt8(hq + m * I + c * 8, r);
  if ((threadIdx.x & 15) == 0) hs[m * sh + (c >> 4)] = exp2i(t);
}

// Backward: the same layout, three 16-byte loads per lane.
__global__ __launch_bounds__(kThreads) void swiglu_bwd_quant_kernel(const uint16_t* __restrict__ a,
                                                                    const uint16_t* __restrict__ dh,
                                                                    const int32_t* __restrict__ offsets, int E,
                                                                    int64_t M_cap, int64_t I,
                                                                    uint8_t* __restrict__ daq,
                                                                    float* __restrict__ das) {
  const int64_t rows = active_rows(offsets, E, M_cap);
  const int64_t cpr = I / 8, n_items = rows * cpr, sh = 2 * I / kTile;
  const int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (it >= n_items) return;  // whole 16-lane tiles (cpr is a multiple of 16)
  const int64_t m = it / cpr, c = it - m * cpr;
  const uint16_t* row = a + m * 2 * I + c * 8;
  float g[8], u[8], d[8], dg[8], du[8];
  unpack_bf16x8(ldnt16(row), g);
  unpack_bf16x8(ldnt16(row + I), u);
  unpack_bf16x8(ldnt16(dh + m * I + c * 8), d);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float sg = sigmoid(g[i]);
    const float gs = g[i] * sg;  // silu(g)
    du[i] = d[i] * gs;
    dg[i] = d[i] * u[i] * sg * (1.0f + g[i] * (1.0f - sg));
  }
  int tg, tu;
  const u32x2 rg = quant8_tile16(dg, tg);
  const u32x2 ru = quant8_tile16(du, tu);
  uint8_t* out = daq + m * 2 * I + c * 8;
  stnt8(out, rg);
  stnt8(out + I, ru);
  if ((threadIdx.x & 15) == 0) {
    das[m * sh + (c >> 4)] = exp2i(tg);
    das[m * sh + I / kTile + (c >> 4)] = exp2i(tu);
  }
}

__global__ __launch_bounds__(kThreads) void swiglu_bf16_kernel(const uint16_t* __restrict__ a,
                                                               const int32_t* __restrict__ offsets, int E,
                                                               int64_t n_rows, int64_t I, uint16_t* __restrict__ h) {
  const int64_t rows = active_rows(offsets, E, n_rows);
  const int64_t cpr = I / 8, n_items = rows * cpr;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x; it < n_items; it += stride) {
    const int64_t m = it / cpr, c = it - m * cpr;
    const uint16_t* row = a + m * 2 * I + c * 8;
    float g[8], u[8];
    unpack_bf16x8(ldnt16(row), g);
    unpack_bf16x8(ldnt16(row + I), u);
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = pack_bf16x2(g[2 * i] * sigmoid(g[2 * i]) * u[2 * i], g[2 * i + 1] * sigmoid(g[2 * i + 1]) * u[2 * i + 1]);
    stnt16(h + m * I + c * 8, o);
  }
}

constexpr int kStreamBlocksPerCU = 1 << 20;  // grid cap of the SwiGLU kernels (none: one pass)

int grid_for(int64_t items) {
  int64_t need = (items + kThreads - 1) / kThreads;
  const int64_t cap = (int64_t)device_cu_count() * kStreamBlocksPerCU;
  if (need < 1) need = 1;
  return (int)(need < cap ? need : cap);
}

}  // namespace

hipError_t launch_swiglu_quant(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                               uint8_t* hq, float* hs, hipStream_t st) {
  const int64_t items = M_cap * (I / 8);
  swiglu_quant_kernel<<<(unsigned)((items + kThreads - 1) / kThreads), kThreads, 0, st>>>(a, offsets, E, M_cap, I, hq,
                                                                                        hs);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd_quant(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E,
                                   int64_t M_cap, int64_t I, uint8_t* daq, float* das, hipStream_t st) {
  const int64_t items = M_cap * (I / 8);
  swiglu_bwd_quant_kernel<<<(unsigned)((items + kThreads - 1) / kThreads), kThreads, 0, st>>>(a, dh, offsets, E, M_cap,
                                                                                             I, daq, das);
  return hipGetLastError();
}

hipError_t launch_swiglu_bf16(const uint16_t* a, const int32_t* offsets, int E, int64_t rows, int64_t I,
                              uint16_t* h, hipStream_t st) {
  swiglu_bf16_kernel<<<grid_for(rows * (I / 8)), kThreads, 0, st>>>(a, offsets, E, rows, I, h);
  return hipGetLastError();
}

}  // namespace ff8
