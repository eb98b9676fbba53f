// Fused permute + padding + quantization and fused unpermute for gfx950 (paper
// section 3.3.1; the quantization is the entry cast of the FP8 dataflow, section 3.2).
//
// Routing maps are built without host synchronization and without atomics-order
// dependence, so the grouped layout is deterministic (ascending token order inside
// each expert group):
//   route_count  : one workgroup per chunk of 256 tokens counts its (token, slot)
//                  pairs per expert in LDS -> counts[chunk][e];
//   route_scan   : one workgroup turns the counts into per-chunk bases, pads every
//                  expert to a multiple of 128 rows, writes offsets[E+1] and marks the
//                  padding rows' src_row = -1;
//   route_assign : one wave per chunk walks its tokens 64 at a time; a 64-bit LDS
//                  ballot mask per expert gives each pair its rank among earlier lanes.
// Then permute_quant reads each token row ONCE, quantizes it 1x128 (16 lanes per tile,
// DPP amax), and writes it to each of its k rows; with routing weights each copy is
// scaled (float32 product) and quantized separately.  pad_fill writes the padding rows.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kChunk = 256;  // tokens per routing chunk
constexpr int kThreads = 256;

int64_t n_chunks_of(int64_t T) { return (T + kChunk - 1) / kChunk; }

__global__ __launch_bounds__(kThreads) void route_count_kernel(const int32_t* __restrict__ idx, int64_t T, int k,
                                                               int E, int32_t* __restrict__ counts) {
  __shared__ int cnt[1024];
  for (int e = threadIdx.x; e < E; e += kThreads) cnt[e] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kChunk + threadIdx.x;
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      const int e = idx[t * k + j];
      if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += kThreads) counts[(int64_t)blockIdx.x * E + e] = cnt[e];
}

__global__ __launch_bounds__(1024) void route_scan_kernel(int32_t* __restrict__ counts, int64_t n_chunks, int E,
                                                          int32_t* __restrict__ offsets, int32_t* __restrict__ src_row) {
  __shared__ int padded[1024];
  __shared__ int offs[1025];
  const int e = threadIdx.x;
  int total = 0;
  if (e < E) {
    for (int64_t c = 0; c < n_chunks; ++c) {  // counts -> exclusive per-chunk prefix (in place)
      const int v = counts[c * E + e];
      counts[c * E + e] = total;
      total += v;
    }
    padded[e] = (total + kTile - 1) / kTile * kTile;
  }
  __syncthreads();
  if (e == 0) {
    int acc = 0;
    for (int i = 0; i < E; ++i) {
      offs[i] = acc;
      acc += padded[i];
    }
    offs[E] = acc;
  }
  __syncthreads();
  if (e < E) {
    const int base = offs[e];
    for (int64_t c = 0; c < n_chunks; ++c) counts[c * E + e] += base;
    offsets[e] = base;
    for (int r = base + total; r < offs[e + 1]; ++r) src_row[r] = -1;
  }
  if (e == 0) offsets[E] = offs[E];
}

__global__ __launch_bounds__(64) void route_assign_kernel(const int32_t* __restrict__ idx, int64_t T, int k, int E,
                                                          const int32_t* __restrict__ bases,
                                                          int32_t* __restrict__ row_map, int32_t* __restrict__ src_row) {
  __shared__ int run[1024];
  __shared__ unsigned long long mask[1024];
  const int lane = threadIdx.x;
  const int64_t chunk = blockIdx.x;
  for (int e = lane; e < E; e += 64) run[e] = bases[chunk * E + e];
  const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int b = 0; b < kChunk / 64; ++b) {
    const int64_t t = chunk * kChunk + b * 64 + lane;
    if (chunk * kChunk + b * 64 >= T) break;  // uniform
    for (int e = lane; e < E; e += 64) mask[e] = 0ull;
    __syncthreads();
    const bool valid = t < T;
    for (int j = 0; j < k; ++j) {
      const int e = valid ? idx[t * k + j] : -1;
      if (e >= 0 && e < E) atomicOr(&mask[e], 1ull << lane);
    }
    __syncthreads();
    for (int j = 0; j < k && valid; ++j) {
      const int e = idx[t * k + j];
      int row = -1;
      if (e >= 0 && e < E) {
        row = run[e] + __popcll(mask[e] & below);
        src_row[row] = (int32_t)(t * k + j);
      }
      row_map[t * k + j] = row;
    }
    __syncthreads();
    for (int e = lane; e < E; e += 64) run[e] += __popcll(mask[e]);
    __syncthreads();
  }
}

// Work item (t, c): token t, 8-element chunk c of its row.  16 consecutive items share a
// 128-element tile (H / 8 is a multiple of 16), so the tile amax stays a 16-lane reduction.
template <bool kWeighted>
__global__ __launch_bounds__(kThreads) void permute_quant_kernel(const uint16_t* __restrict__ x,
                                                                 const float* __restrict__ row_w, int64_t T,
                                                                 int64_t H, int k, const int32_t* __restrict__ row_map,
                                                                 int64_t M_cap, uint8_t* __restrict__ q,
                                                                 float* __restrict__ s) {
  const int64_t cpr = H / 8;  // chunks per row
  const int64_t n_items = T * cpr;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  const int64_t sh = H / kTile;
  const bool leader = (threadIdx.x & 15) == 0;
  for (int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x; it < n_items; it += stride) {
    const int64_t t = it / cpr, c = it - t * cpr;
    float v[8];
    unpack_bf16x8(ldnt16(x + t * H + c * 8), v);
    if (!kWeighted) {
      int tq;
      const u32x2 r = quant8_tile16(v, tq);
      for (int j = 0; j < k; ++j) {
        const int row = row_map[t * k + j];
        if (row >= 0 && row < M_cap) {  // uniform across the 16 lanes of a tile
          stnt8(q + (int64_t)row * H + c * 8, r);
          if (leader) s[(int64_t)row * sh + (c >> 4)] = exp2i(tq);
        }
      }
    } else {
      for (int j = 0; j < k; ++j) {
        const int row = row_map[t * k + j];
        if (row >= 0 && row < M_cap) {
          const float w = row_w[t * k + j];
          float vw[8];
#pragma unroll
          for (int i = 0; i < 8; ++i) vw[i] = w * v[i];
          int tq;
          const u32x2 r = quant8_tile16(vw, tq);
          stnt8(q + (int64_t)row * H + c * 8, r);
          if (leader) s[(int64_t)row * sh + (c >> 4)] = exp2i(tq);
        }
      }
    }
  }
}

// Padding rows (src_row == -1 below offsets[E]): bytes 0x00, scales 2^-126.  Padding
// only occurs in the last 128-row block of a group; other blocks exit after one read.
__global__ __launch_bounds__(kThreads) void pad_fill_kernel(const int32_t* __restrict__ offsets, int E,
                                                            const int32_t* __restrict__ src_row, int64_t H,
                                                            uint8_t* __restrict__ q, float* __restrict__ s) {
  __shared__ int pad_rows[kTile];
  __shared__ int n_pad;
  const int64_t r0 = (int64_t)blockIdx.x * kTile;
  if (r0 >= offsets[E]) return;
  if (threadIdx.x == 0) n_pad = 0;
  __syncthreads();
  if (threadIdx.x < kTile && src_row[r0 + threadIdx.x] < 0) pad_rows[atomicAdd(&n_pad, 1)] = threadIdx.x;
  __syncthreads();
  const int np = n_pad;
  const int64_t c16 = H / 16, sh = H / kTile;
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t i = threadIdx.x; i < (int64_t)np * c16; i += kThreads) {
    const int64_t r = r0 + pad_rows[i / c16];
    stnt16(q + r * H + (i % c16) * 16, z);
  }
  for (int64_t i = threadIdx.x; i < (int64_t)np * sh; i += kThreads) {
    const int64_t r = r0 + pad_rows[i / sh];
    s[r * sh + i % sh] = exp2i(kTMin);
  }
}

template <bool kWeighted>
__global__ __launch_bounds__(kThreads) void unpermute_kernel(const uint16_t* __restrict__ y_perm,
                                                             const int32_t* __restrict__ row_map,
                                                             const float* __restrict__ row_w, int64_t T, int k,
                                                             int64_t H, int64_t M_cap, uint16_t* __restrict__ y) {
  const int64_t cpr = H / 8;
  const int64_t n_items = T * cpr;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t it = (int64_t)blockIdx.x * kThreads + threadIdx.x; it < n_items; it += stride) {
    const int64_t t = it / cpr, c = it - t * cpr;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const int row = row_map[t * k + j];
      if (row < 0 || row >= M_cap) continue;
      float v[8];
      unpack_bf16x8(ldnt16(y_perm + (int64_t)row * H + c * 8), v);
      if (kWeighted) {
        const float w = row_w[t * k + j];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] = fmaf(w, v[i], acc[i]);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += v[i];
      }
    }
    u32x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = pack_bf16x2(acc[2 * i], acc[2 * i + 1]);
    stnt16(y + t * H + c * 8, o);
  }
}

constexpr int kStreamBlocksPerCU = 1 << 20;  // grid cap of the permute / unpermute kernels (none: one pass)

int grid_for(int64_t items, int max_per_cu) {
  int64_t need = (items + kThreads - 1) / kThreads;
  const int64_t cap = (int64_t)device_cu_count() * max_per_cu;
  if (need < 1) need = 1;
  return (int)(need < cap ? need : cap);
}

}  // namespace

size_t permute_workspace_bytes(int64_t T, int k, int E) {
  (void)k;
  return (size_t)n_chunks_of(T) * (size_t)E * sizeof(int32_t);
}

hipError_t launch_route(const int32_t* topk_idx, int64_t T, int k, int E, int32_t* row_map, int32_t* offsets,
                        int32_t* src_row, int64_t M_cap, void* workspace, hipStream_t st) {
  (void)M_cap;
  const int64_t nc = n_chunks_of(T);
  int32_t* counts = static_cast<int32_t*>(workspace);
  if (nc > 0) route_count_kernel<<<(unsigned)nc, kThreads, 0, st>>>(topk_idx, T, k, E, counts);
  route_scan_kernel<<<1, 1024, 0, st>>>(counts, nc, E, offsets, src_row);
  if (nc > 0) route_assign_kernel<<<(unsigned)nc, 64, 0, st>>>(topk_idx, T, k, E, counts, row_map, src_row);
  return hipGetLastError();
}

hipError_t launch_permute_quant(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                int64_t M_cap, uint8_t* q, float* s, hipStream_t st) {
  const int64_t items = T * (H / 8);
  if (items > 0) {
    const int grid = grid_for(items, kStreamBlocksPerCU);
    if (row_w)
      permute_quant_kernel<true><<<grid, kThreads, 0, st>>>(x, row_w, T, H, k, row_map, M_cap, q, s);
    else
      permute_quant_kernel<false><<<grid, kThreads, 0, st>>>(x, row_w, T, H, k, row_map, M_cap, q, s);
  }
  pad_fill_kernel<<<(unsigned)(M_cap / kTile), kThreads, 0, st>>>(offsets, E, src_row, H, q, s);
  return hipGetLastError();
}

hipError_t launch_unpermute(const uint16_t* y_perm, const int32_t* row_map, const float* row_w, int64_t T, int k,
                            int64_t H, int64_t M_cap, uint16_t* y, hipStream_t st) {
  const int64_t items = T * (H / 8);
  if (items == 0) return hipSuccess;
  const int grid = grid_for(items, kStreamBlocksPerCU);
  if (row_w)
    unpermute_kernel<true><<<grid, kThreads, 0, st>>>(y_perm, row_map, row_w, T, k, H, M_cap, y);
  else
    unpermute_kernel<false><<<grid, kThreads, 0, st>>>(y_perm, row_map, row_w, T, k, H, M_cap, y);
  return hipGetLastError();
}

}  // namespace ff8
