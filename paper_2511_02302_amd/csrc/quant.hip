// Quantization kernels for gfx950: 1x128 row-wise and 128x128 block quantization with
// power-of-two scales (paper section 3.1), element casts, and the unfused baseline
// pieces (dequantize, bf16 transpose, copy) used to reproduce the naive conversion.
//
// Row-wise layout makes the tensor a flat stream of 128-element tiles: tile i covers
// elements [128 i, 128 i + 128) and owns scale s[i].  Each lane takes 8 consecutive
// elements (one 16-byte load), 16 lanes cover one tile, and the tile maximum is a
// 16-lane DPP reduction, so loads, byte stores and scale stores are all contiguous.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kThreads = 256;
constexpr int kStreamBlocksPerCU = 1 << 20;  // streaming kernels: one tile per workgroup, no grid-stride cap

int grid_for(int64_t work_items, int per_block, int max_per_cu) {
  int64_t need = (work_items + per_block - 1) / per_block;
  int64_t cap = (int64_t)device_cu_count() * max_per_cu;
  if (need < 1) need = 1;
  return (int)(need < cap ? need : cap);
}

template <int U, typename S>
__global__ __launch_bounds__(kThreads) void quant_rowwise_kernel(const uint16_t* __restrict__ x, int64_t n_chunks,
                                                                 uint8_t* __restrict__ q, S* __restrict__ s) {
  const int64_t stride = (int64_t)gridDim.x * kThreads * U;
  for (int64_t c0 = (int64_t)blockIdx.x * kThreads * U + threadIdx.x; c0 < n_chunks; c0 += stride) {
    u32x4 w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t c = c0 + (int64_t)u * kThreads;
      if (c < n_chunks) w[u] = ldnt16(x + c * 8);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t c = c0 + (int64_t)u * kThreads;
      if (c < n_chunks) {  // uniform across each 16-lane tile group
        float v[8];
        unpack_bf16x8(w[u], v);
        int t;
        const u32x2 r = quant8_tile16(v, t);
        stnt8(q + c * 8, r);
        if ((threadIdx.x & 15) == 0) put_scale(&s[c >> 4], t);
      }
    }
  }
}

// One workgroup per 128x128 block: 16 lanes span a 128-column row segment, 16 rows per
// pass, 8 passes.  Block maximum = wave DPP reduction + a 4-entry LDS reduction.
template <typename S>
__global__ __launch_bounds__(kThreads) void quant_block128_kernel(const uint16_t* __restrict__ w, int64_t cols,
                                                                  int64_t n_col_blocks, uint8_t* __restrict__ q,
                                                                  S* __restrict__ s) {
  __shared__ uint32_t wave_max[kThreads / 64];
  const int64_t blk = blockIdx.x;
  const int64_t rb = blk / n_col_blocks, cb = blk - rb * n_col_blocks;
  const int cc = threadIdx.x & 15, r0 = threadIdx.x >> 4;
  const int64_t base = (rb * kTile + r0) * cols + cb * kTile + cc * 8;
  u32x4 v[8];
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v[i] = ldnt16(w + base + (int64_t)i * 16 * cols);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      m = max(m, abs_bits(bf16_lo(v[i][j])));
      m = max(m, abs_bits(bf16_hi(v[i][j])));
    }
  }
  m = max64_u32(m);
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = m;
  __syncthreads();
  m = max(max(wave_max[0], wave_max[1]), max(wave_max[2], wave_max[3]));
  const int t = scale_exponent(__uint_as_float(m));
  const float inv = exp2i(-t);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float f[8];
    unpack_bf16x8(v[i], f);
    u32x2 r;
    r[0] = cvt_e4m3x4(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
    r[1] = cvt_e4m3x4(f[4] * inv, f[5] * inv, f[6] * inv, f[7] * inv);
    stnt8(q + base + (int64_t)i * 16 * cols, r);
  }
  if (threadIdx.x == 0) put_scale(&s[blk], t);
}

// Two horizontally adjacent 128x128 blocks per workgroup: 32 lanes span a 256-column row
// segment (512 bytes per load instruction pair of rows), 8 rows per pass, 16 passes.
template <typename S>
__global__ __launch_bounds__(kThreads) void quant_block128x2_kernel(const uint16_t* __restrict__ w, int64_t cols,
                                                                    int64_t n_pairs, uint8_t* __restrict__ q,
                                                                    S* __restrict__ s) {
  __shared__ uint32_t wave_max[kThreads / 64][2];
  const int64_t pr = blockIdx.x;
  const int64_t rb = pr / n_pairs, cp = pr - rb * n_pairs;
  const int cc = threadIdx.x & 31, r0 = threadIdx.x >> 5;
  const int64_t base = (rb * kTile + r0) * cols + cp * 2 * kTile + cc * 8;
  u32x4 v[16];
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    v[i] = ldnt16(w + base + (int64_t)i * 8 * cols);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      m = max(m, abs_bits(bf16_lo(v[i][j])));
      m = max(m, abs_bits(bf16_hi(v[i][j])));
    }
  }
  m = max16_u32(m);                                   // per 16-lane group: one block, one row group
  m = max(m, (uint32_t)__shfl_xor((int)m, 32));       // both row groups of the wave
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (lane == 0) wave_max[wv][0] = m;
  if (lane == 16) wave_max[wv][1] = m;
  __syncthreads();
  const int h = cc >> 4;  // this lane's block
  m = max(max(wave_max[0][h], wave_max[1][h]), max(wave_max[2][h], wave_max[3][h]));
  const int t = scale_exponent(__uint_as_float(m));
  const float inv = exp2i(-t);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    float f[8];
    unpack_bf16x8(v[i], f);
    u32x2 r;
    r[0] = cvt_e4m3x4(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
    r[1] = cvt_e4m3x4(f[4] * inv, f[5] * inv, f[6] * inv, f[7] * inv);
    stnt8(q + base + (int64_t)i * 8 * cols, r);
  }
  if (threadIdx.x == 0 || threadIdx.x == 16) put_scale(&s[rb * 2 * n_pairs + cp * 2 + h], t);
}

__device__ __forceinline__ float sat448(float f) { return fminf(fmaxf(f, -448.0f), 448.0f); }

__global__ __launch_bounds__(kThreads) void cast_f32_e4m3_kernel(const float* __restrict__ x, int64_t n,
                                                                 uint8_t* __restrict__ q) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i * 4 < n; i += stride) {
    if (i * 4 + 4 <= n) {
      const u32x4 w = ldnt16(x + i * 4);
      float f[4];
      uint32_t nanmask = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f[j] = __uint_as_float(w[j]);
        if (f[j] != f[j]) nanmask |= 0x7Fu << (8 * j);
        f[j] = sat448(f[j]);
      }
      uint32_t r = cvt_e4m3x4(f[0], f[1], f[2], f[3]);
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (nanmask & (0xFFu << (8 * j))) r = (r & ~(0xFFu << (8 * j))) | (0x7Fu << (8 * j));
      *reinterpret_cast<uint32_t*>(q + i * 4) = r;
    } else {
      for (int64_t j = i * 4; j < n; ++j) {
        const float f = x[j];
        q[j] = (f != f) ? 0x7F : (uint8_t)(cvt_e4m3x2<false>(sat448(f), 0.0f, 0u) & 0xFF);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void cast_e4m3_f32_kernel(const uint8_t* __restrict__ q, int64_t n,
                                                                 float* __restrict__ x) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i * 4 < n; i += stride) {
    if (i * 4 + 4 <= n) {
      const uint32_t w = *reinterpret_cast<const uint32_t*>(q + i * 4);
      const f32x2 a = dec_e4m3x2<false>(w), b = dec_e4m3x2<true>(w);
      u32x4 o;
      o[0] = __float_as_uint(a[0]);
      o[1] = __float_as_uint(a[1]);
      o[2] = __float_as_uint(b[0]);
      o[3] = __float_as_uint(b[1]);
      stnt16(x + i * 4, o);
    } else {
      for (int64_t j = i * 4; j < n; ++j) x[j] = dec_e4m3x2<false>((uint32_t)q[j])[0];
    }
  }
}

template <typename S>
__global__ __launch_bounds__(kThreads) void dequant_rowwise_kernel(const uint8_t* __restrict__ q,
                                                                   const S* __restrict__ s, int64_t n_chunks,
                                                                   uint16_t* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t c = (int64_t)blockIdx.x * kThreads + threadIdx.x; c < n_chunks; c += stride) {
    const u32x2 b = ldnt8(q + c * 8);
    const float sc = scale_value(s[c >> 4]);
    u32x4 o;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const f32x2 lo = dec_e4m3x2<false>(b[j]), hi = dec_e4m3x2<true>(b[j]);
      o[2 * j] = pack_bf16x2(lo[0] * sc, lo[1] * sc);
      o[2 * j + 1] = pack_bf16x2(hi[0] * sc, hi[1] * sc);
    }
    stnt16(out + c * 8, o);
  }
}

// 64x64 bf16 tile transpose through LDS.
__global__ __launch_bounds__(kThreads) void transpose_bf16_kernel(const uint16_t* __restrict__ in, int64_t rows,
                                                                  int64_t cols, uint16_t* __restrict__ out) {
  __shared__ uint16_t tile[64][64 + 2];
  const int64_t n_cb = cols / 64;
  const int64_t rb = blockIdx.x / n_cb, cb = blockIdx.x - rb * n_cb;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = ty + 16 * i;
    const u32x2 v = ldnt8(in + (rb * 64 + r) * cols + cb * 64 + tx * 4);
    tile[r][tx * 4 + 0] = v[0] & 0xFFFF;
    tile[r][tx * 4 + 1] = v[0] >> 16;
    tile[r][tx * 4 + 2] = v[1] & 0xFFFF;
    tile[r][tx * 4 + 3] = v[1] >> 16;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = ty + 16 * i;
    u32x2 v;
    v[0] = (uint32_t)tile[tx * 4 + 0][c] | ((uint32_t)tile[tx * 4 + 1][c] << 16);
    v[1] = (uint32_t)tile[tx * 4 + 2][c] | ((uint32_t)tile[tx * 4 + 3][c] << 16);
    stnt8(out + (cb * 64 + c) * rows + rb * 64 + tx * 4, v);
  }
}

template <int U>
__global__ __launch_bounds__(kThreads) void copy_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                        u32x4* __restrict__ dst) {
  const int64_t stride = (int64_t)gridDim.x * kThreads * U;
  for (int64_t c0 = (int64_t)blockIdx.x * kThreads * U + threadIdx.x; c0 < n16; c0 += stride) {
    u32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c0 + u * kThreads < n16) v[u] = ldnt16(src + c0 + u * kThreads);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (c0 + u * kThreads < n16) stnt16(dst + c0 + u * kThreads, v[u]);
  }
}

}  // namespace

namespace {

template <typename S>
hipError_t quant_rowwise_impl(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, S* s, hipStream_t st) {
  const int64_t n_chunks = rows * cols / 8;
  constexpr int U = 4;
  const int grid = grid_for(n_chunks, kThreads * U, kStreamBlocksPerCU);
  quant_rowwise_kernel<U, S><<<grid, kThreads, 0, st>>>(x, n_chunks, q, s);
  return hipGetLastError();
}

template <typename S>
hipError_t quant_block128_impl(const uint16_t* w, int64_t rows, int64_t cols, uint8_t* q, S* s, hipStream_t st) {
  const int64_t nbc = cols / kTile, blocks = rows / kTile * nbc;
  if (nbc % 2 == 0) {
    quant_block128x2_kernel<S><<<(unsigned)(blocks / 2), kThreads, 0, st>>>(w, cols, nbc / 2, q, s);
    return hipGetLastError();
  }
  quant_block128_kernel<S><<<(unsigned)blocks, kThreads, 0, st>>>(w, cols, nbc, q, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_quant_rowwise(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, float* s,
                                hipStream_t st) {
  return quant_rowwise_impl(x, rows, cols, q, s, st);
}
hipError_t launch_quant_rowwise(const uint16_t* x, int64_t rows, int64_t cols, uint8_t* q, e8m0_t* s,
                                hipStream_t st) {
  return quant_rowwise_impl(x, rows, cols, q, s, st);
}
hipError_t launch_quant_block128(const uint16_t* w, int64_t rows, int64_t cols, uint8_t* q, float* s,
                                 hipStream_t st) {
  return quant_block128_impl(w, rows, cols, q, s, st);
}
hipError_t launch_quant_block128(const uint16_t* w, int64_t rows, int64_t cols, uint8_t* q, e8m0_t* s,
                                 hipStream_t st) {
  return quant_block128_impl(w, rows, cols, q, s, st);
}

hipError_t launch_cast_f32_e4m3(const float* x, int64_t n, uint8_t* q, hipStream_t st) {
  cast_f32_e4m3_kernel<<<grid_for((n + 3) / 4, kThreads, 16), kThreads, 0, st>>>(x, n, q);
  return hipGetLastError();
}

hipError_t launch_cast_e4m3_f32(const uint8_t* q, int64_t n, float* x, hipStream_t st) {
  cast_e4m3_f32_kernel<<<grid_for((n + 3) / 4, kThreads, 16), kThreads, 0, st>>>(q, n, x);
  return hipGetLastError();
}

template <typename S>
static hipError_t dequant_rowwise_impl(const uint8_t* q, const S* s, int64_t rows, int64_t cols, uint16_t* out,
                                       hipStream_t st) {
  const int64_t n_chunks = rows * cols / 8;
  dequant_rowwise_kernel<S><<<grid_for(n_chunks, kThreads, 16), kThreads, 0, st>>>(q, s, n_chunks, out);
  return hipGetLastError();
}
hipError_t launch_dequant_rowwise(const uint8_t* q, const float* s, int64_t rows, int64_t cols, uint16_t* out,
                                  hipStream_t st) {
  return dequant_rowwise_impl(q, s, rows, cols, out, st);
}
hipError_t launch_dequant_rowwise(const uint8_t* q, const e8m0_t* s, int64_t rows, int64_t cols, uint16_t* out,
                                  hipStream_t st) {
  return dequant_rowwise_impl(q, s, rows, cols, out, st);
}

hipError_t launch_transpose_bf16(const uint16_t* in, int64_t rows, int64_t cols, uint16_t* out, hipStream_t st) {
  const int64_t blocks = (rows / 64) * (cols / 64);
  transpose_bf16_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(in, rows, cols, out);
  return hipGetLastError();
}

hipError_t launch_copy(const void* src, void* dst, int64_t nbytes, hipStream_t st) {
  const int64_t n16 = nbytes / 16;
  constexpr int U = 4;
  copy_kernel<U><<<grid_for(n16, kThreads * U, kStreamBlocksPerCU), kThreads, 0, st>>>(
      reinterpret_cast<const u32x4*>(src), n16, reinterpret_cast<u32x4*>(dst));
  return hipGetLastError();
}

}  // namespace ff8
