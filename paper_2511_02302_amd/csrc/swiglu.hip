// Fused SwiGLU + quantization (paper section 3.3.2) and its backward twin, for gfx950.
//
// The fc1 output A [rows, 2I] is [gate | up].  Work item (m, c) covers 8 or 16 output
// columns of row m; the items of one 1x128 output tile are consecutive lanes, so the tile
// amax is a DPP reduction and the activation goes from float32 registers straight to
// e4m3 without a bf16 round trip.  Rows at and beyond offsets[E] are skipped.
//
// FP8 checkpoint (the paper's experiments keep the activations saved for the backward in
// FP8 instead of BF16): the forward kernel can also emit A itself quantized 1x128
// (gate and up tiles, from the same registers), and the backward kernel can read that
// FP8 copy in place of the BF16 A, dequantizing it exactly in float32.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kThreads = 256;

// sigma(g) = 1 / (1 + e^-g) with the hardware reciprocal (v_rcp_f32, within 1 ulp).  A
// correctly rounded reciprocal compiles to the IEEE division sequence, about ten VALU
// instructions per element, which left the forward kernel VALU-bound.
__device__ __forceinline__ float sigmoid(float g) { return __builtin_amdgcn_rcpf(1.0f + __expf(-g)); }

// Decode 16 e4m3 bytes times a power-of-two scale (exact in float32).
__device__ __forceinline__ void dequant16(const u32x4& w, float s, float* v) {
#pragma unroll
  for (int h = 0; h < 4; ++h) {
    const f32x2 lo = dec_e4m3x2<false>(w[h]), hi = dec_e4m3x2<true>(w[h]);
    v[4 * h + 0] = lo[0] * s;
    v[4 * h + 1] = lo[1] * s;
    v[4 * h + 2] = hi[0] * s;
    v[4 * h + 3] = hi[1] * s;
  }
}

// Forward: lane c covers 16 output columns (two 16-byte loads each of gate and up), 8
// lanes one 1x128 tile, one 16-byte store per lane; one item per thread, no grid-stride
// loop.  (16 columns per lane measured faster than 8 here, and slower in the backward.)
// kKeepA: also write A as 1x128 FP8 (aq [rows, 2I], as_ [rows, 2I/128]).
template <bool kKeepA, typename S>
__global__ __launch_bounds__(kThreads) void swiglu_quant_kernel(const uint16_t* __restrict__ a,
                                                                const int32_t* __restrict__ offsets, int E,
                                                                int64_t M_cap, int64_t I, uint8_t* __restrict__ hq,
                                                                S* __restrict__ hs, uint8_t* __restrict__ aq,
                                                                S* __restrict__ as_) {
  const int64_t rows = active_rows(offsets, E, M_cap);
  const int64_t cpr = I / 16, n_items = rows * cpr, sh = I / kTile;
  const int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (it >= n_items) return;  // whole 8-lane tiles (cpr is a multiple of 8)
  const int64_t m = it / cpr, c = it - m * cpr;
  const uint16_t* row = a + m * 2 * I + c * 16;
  const u32x4 g0 = ldnt16(row), g1 = ldnt16(row + 8), u0 = ldnt16(row + I), u1 = ldnt16(row + I + 8);
  float g[16], u[16], h[16];
  unpack_bf16x8(g0, g);
  unpack_bf16x8(g1, g + 8);
  unpack_bf16x8(u0, u);
  unpack_bf16x8(u1, u + 8);
#pragma unroll
  for (int i = 0; i < 16; ++i) h[i] = g[i] * sigmoid(g[i]) * u[i];
  int t;
  const u32x4 r = quant16_tile8(h, t);
  stnt16(hq + m * I + c * 16, r);
  if ((threadIdx.x & 7) == 0) put_scale(&hs[m * sh + (c >> 3)], t);
  if (kKeepA) {
    int tg, tu;
    const u32x4 rg = quant16_tile8(g, tg);
    const u32x4 ru = quant16_tile8(u, tu);
    stnt16(aq + m * 2 * I + c * 16, rg);
    stnt16(aq + m * 2 * I + I + c * 16, ru);
    if ((threadIdx.x & 7) == 0) {
      put_scale(&as_[m * 2 * sh + (c >> 3)], tg);
      put_scale(&as_[m * 2 * sh + sh + (c >> 3)], tu);
    }
  }
}

// Backward: the same layout, three 16-byte loads per lane.
template <typename S>
__global__ __launch_bounds__(kThreads) void swiglu_bwd_quant_kernel(const uint16_t* __restrict__ a,
                                                                    const uint16_t* __restrict__ dh,
                                                                    const int32_t* __restrict__ offsets, int E,
                                                                    int64_t M_cap, int64_t I,
                                                                    uint8_t* __restrict__ daq,
                                                                    S* __restrict__ das) {
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
    put_scale(&das[m * sh + (c >> 4)], tg);
    put_scale(&das[m * sh + I / kTile + (c >> 4)], tu);
  }
}

// Backward from the FP8 checkpoint of A: lane c covers 16 columns (16-byte loads of the
// gate and up codes, two of dH), 8 lanes one 1x128 tile of each half of the output.
template <typename S>
__global__ __launch_bounds__(kThreads) void swiglu_bwd_quant_fp8a_kernel(const uint8_t* __restrict__ aq,
                                                                         const S* __restrict__ as_,
                                                                         const uint16_t* __restrict__ dh,
                                                                         const int32_t* __restrict__ offsets, int E,
                                                                         int64_t M_cap, int64_t I,
                                                                         uint8_t* __restrict__ daq,
                                                                         S* __restrict__ das) {
  const int64_t rows = active_rows(offsets, E, M_cap);
  const int64_t cpr = I / 16, n_items = rows * cpr, sh = 2 * I / kTile;
  const int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (it >= n_items) return;  // whole 8-lane tiles (cpr is a multiple of 8)
  const int64_t m = it / cpr, c = it - m * cpr;
  const uint8_t* row = aq + m * 2 * I + c * 16;
  const S* srow = as_ + m * sh;  // gate tiles, then up tiles
  const u32x4 qg = ldnt16(row), qu = ldnt16(row + I);
  const u32x4 d0 = ldnt16(dh + m * I + c * 16), d1 = ldnt16(dh + m * I + c * 16 + 8);
  float g[16], u[16], d[16], dg[16], du[16];
  dequant16(qg, scale_value(srow[c >> 3]), g);
  dequant16(qu, scale_value(srow[I / kTile + (c >> 3)]), u);
  unpack_bf16x8(d0, d);
  unpack_bf16x8(d1, d + 8);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float sg = sigmoid(g[i]);
    const float gs = g[i] * sg;  // silu(g)
    du[i] = d[i] * gs;
    dg[i] = d[i] * u[i] * sg * (1.0f + g[i] * (1.0f - sg));
  }
  int tg, tu;
  const u32x4 rg = quant16_tile8(dg, tg);
  const u32x4 ru = quant16_tile8(du, tu);
  uint8_t* out = daq + m * 2 * I + c * 16;
  stnt16(out, rg);
  stnt16(out + I, ru);
  if ((threadIdx.x & 7) == 0) {
    put_scale(&das[m * sh + (c >> 3)], tg);
    put_scale(&das[m * sh + I / kTile + (c >> 3)], tu);
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

namespace {

unsigned blocks_of(int64_t items) { return (unsigned)((items + kThreads - 1) / kThreads); }

template <typename S>
hipError_t swiglu_quant_impl(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I, uint8_t* hq,
                             S* hs, uint8_t* aq, S* as_, hipStream_t st) {
  const unsigned grid = blocks_of(M_cap * (I / 16));
  if (aq)
    swiglu_quant_kernel<true, S><<<grid, kThreads, 0, st>>>(a, offsets, E, M_cap, I, hq, hs, aq, as_);
  else
    swiglu_quant_kernel<false, S><<<grid, kThreads, 0, st>>>(a, offsets, E, M_cap, I, hq, hs, nullptr, nullptr);
  return hipGetLastError();
}

template <typename S>
hipError_t swiglu_bwd_quant_impl(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E, int64_t M_cap,
                                 int64_t I, uint8_t* daq, S* das, hipStream_t st) {
  swiglu_bwd_quant_kernel<S><<<blocks_of(M_cap * (I / 8)), kThreads, 0, st>>>(a, dh, offsets, E, M_cap, I, daq, das);
  return hipGetLastError();
}

template <typename S>
hipError_t swiglu_bwd_quant_fp8a_impl(const uint8_t* aq, const S* as_, const uint16_t* dh, const int32_t* offsets,
                                      int E, int64_t M_cap, int64_t I, uint8_t* daq, S* das, hipStream_t st) {
  swiglu_bwd_quant_fp8a_kernel<S><<<blocks_of(M_cap * (I / 16)), kThreads, 0, st>>>(aq, as_, dh, offsets, E, M_cap, I,
                                                                                    daq, das);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_swiglu_quant(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                               uint8_t* hq, float* hs, hipStream_t st) {
  return swiglu_quant_impl<float>(a, offsets, E, M_cap, I, hq, hs, nullptr, nullptr, st);
}
hipError_t launch_swiglu_quant(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                               uint8_t* hq, e8m0_t* hs, hipStream_t st) {
  return swiglu_quant_impl<e8m0_t>(a, offsets, E, M_cap, I, hq, hs, nullptr, nullptr, st);
}
hipError_t launch_swiglu_quant_keep_fp8(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                        uint8_t* hq, float* hs, uint8_t* aq, float* as_, hipStream_t st) {
  return swiglu_quant_impl(a, offsets, E, M_cap, I, hq, hs, aq, as_, st);
}
hipError_t launch_swiglu_quant_keep_fp8(const uint16_t* a, const int32_t* offsets, int E, int64_t M_cap, int64_t I,
                                        uint8_t* hq, e8m0_t* hs, uint8_t* aq, e8m0_t* as_, hipStream_t st) {
  return swiglu_quant_impl(a, offsets, E, M_cap, I, hq, hs, aq, as_, st);
}
hipError_t launch_swiglu_bwd_quant(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E,
                                   int64_t M_cap, int64_t I, uint8_t* daq, float* das, hipStream_t st) {
  return swiglu_bwd_quant_impl(a, dh, offsets, E, M_cap, I, daq, das, st);
}
hipError_t launch_swiglu_bwd_quant(const uint16_t* a, const uint16_t* dh, const int32_t* offsets, int E,
                                   int64_t M_cap, int64_t I, uint8_t* daq, e8m0_t* das, hipStream_t st) {
  return swiglu_bwd_quant_impl(a, dh, offsets, E, M_cap, I, daq, das, st);
}
hipError_t launch_swiglu_bwd_quant_fp8a(const uint8_t* aq, const float* as_, const uint16_t* dh, const int32_t* offsets,
                                        int E, int64_t M_cap, int64_t I, uint8_t* daq, float* das, hipStream_t st) {
  return swiglu_bwd_quant_fp8a_impl(aq, as_, dh, offsets, E, M_cap, I, daq, das, st);
}
hipError_t launch_swiglu_bwd_quant_fp8a(const uint8_t* aq, const e8m0_t* as_, const uint16_t* dh,
                                        const int32_t* offsets, int E, int64_t M_cap, int64_t I, uint8_t* daq,
                                        e8m0_t* das, hipStream_t st) {
  return swiglu_bwd_quant_fp8a_impl(aq, as_, dh, offsets, E, M_cap, I, daq, das, st);
}

hipError_t launch_swiglu_bf16(const uint16_t* a, const int32_t* offsets, int E, int64_t rows, int64_t I,
                              uint16_t* h, hipStream_t st) {
  swiglu_bf16_kernel<<<grid_for(rows * (I / 8)), kThreads, 0, st>>>(a, offsets, E, rows, I, h);
  return hipGetLastError();
}

}  // namespace ff8
