// Fused permute + padding + quantization and fused unpermute for gfx950 (paper
// section 3.3.1; the quantization is the entry cast of the FP8 dataflow, section 3.2).
//
// Routing maps are built without host synchronization and without atomics-order
// dependence, so the grouped layout is deterministic (ascending token order inside
// each expert group):
//   route_count  : one workgroup per chunk of 256 tokens counts its (token, slot)
//                  pairs per expert in LDS -> counts[chunk][e];
//   route_scan   : one workgroup (E x parts threads) turns the counts into per-chunk
//                  bases, pads every expert to a multiple of 128 rows, writes
//                  offsets[E+1] and marks the padding rows' src_row = -1;
//   route_assign : one workgroup per chunk, one wave per 64 tokens; a 64-bit LDS mask per
//                  wave and expert gives each pair its rank among earlier lanes and waves.
// (64-token chunks, four times the workgroups, measured the same; four waves per chunk in
// route_assign instead of one wave walking it 64 tokens at a time saved 6 us of the routing
// launches' ~26 us at the DeepSeek-V3 share.)
// Then permute_quant reads each token row ONCE (one workgroup per token, 16 elements per
// lane, 8 lanes per 1x128 tile, DPP amax), quantizes it and writes it to each of its k
// rows; with routing weights each copy is scaled (float32 product) and quantized
// separately.  E more workgroups of the same launch write the padding rows, one expert
// group each.  unpermute gathers a token's k rows the same way and sums them in slot order.

#include <mutex>

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kChunk = kRouteChunk;  // tokens per routing chunk
constexpr int kThreads = 256;
constexpr int kRowThreadsMax = 512;  // one-token workgroups (permute, unpermute)

int64_t n_chunks_of(int64_t T) { return (T + kChunk - 1) / kChunk; }

__global__ __launch_bounds__(kChunk) void route_count_kernel(const int32_t* __restrict__ idx, int64_t T, int k,
                                                             int E, int32_t* __restrict__ counts) {
  __shared__ int cnt[1024];
  for (int e = threadIdx.x; e < E; e += kChunk) cnt[e] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kChunk + threadIdx.x;
  if (t < T) {
    for (int j = 0; j < k; ++j) {
      const int e = idx[t * k + j];
      if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += kChunk) counts[(int64_t)blockIdx.x * E + e] = cnt[e];
}

// Inclusive sum over the 1024 threads of the workgroup, in thread order: a 64-lane shuffle
// scan per wave, then the 16 wave totals scanned by one wave (wsum: 16 ints of LDS).
__device__ __forceinline__ int block_inclusive_sum(int v, int* wsum) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int u = __shfl_up(v, d);
    if (lane >= d) v += u;
  }
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  if (w == 0) {
    int x = lane < 16 ? wsum[lane] : 0;
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) {
      const int u = __shfl_up(x, d);
      if (lane >= d) x += u;
    }
    if (lane < 16) wsum[lane] = x;
  }
  __syncthreads();
  const int r = w > 0 ? v + wsum[w - 1] : v;
  __syncthreads();  // wsum is reused by the next call
  return r;
}

// Thread (e, part) of P = 1024 / E parts owns a contiguous range of chunks of expert e: it
// sums them; one block-wide scan of the part sums (expert-major) gives each part's base
// within its expert and each expert's total; a second scan of the padded totals gives the
// group offsets; each thread then rewrites its range as exclusive bases.  All chunk loads
// of a pass are independent.
__global__ __launch_bounds__(1024) void route_scan_kernel(int32_t* __restrict__ counts, int64_t n_chunks, int E,
                                                          int align, int32_t* __restrict__ offsets,
                                                          int32_t* __restrict__ src_row) {
  __shared__ int incl[1024];  // inclusive scan of the part sums, expert-major
  __shared__ int offs[1025];
  __shared__ int wsum[16];
  const int P = 1024 / E;  // parts per expert (E <= 1024)
  const int e = threadIdx.x / P, part = threadIdx.x - e * P;
  const int64_t per = (n_chunks + P - 1) / P;
  const int64_t c0 = (int64_t)part * per;
  const int64_t c1 = c0 + per < n_chunks ? c0 + per : n_chunks;
  int sum = 0;
  if (e < E)
    for (int64_t c = c0; c < c1; ++c) sum += counts[c * E + e];
  incl[threadIdx.x] = block_inclusive_sum(sum, wsum);
  __syncthreads();
  // expert x's rows: incl[x P + P - 1] - incl[x P - 1]; padded to the alignment, scanned
  const int x = threadIdx.x;
  int total = 0;
  if (x < E) total = incl[x * P + P - 1] - (x > 0 ? incl[x * P - 1] : 0);
  const int padded = (total + align - 1) / align * align;
  const int end = block_inclusive_sum(padded, wsum);
  if (x < E) offs[x + 1] = end;
  if (x == 0) offs[0] = 0;
  __syncthreads();
  if (e < E) {
    const int seg0 = e > 0 ? incl[e * P - 1] : 0;
    const int tot = incl[e * P + P - 1] - seg0;
    int run = offs[e] + (incl[threadIdx.x] - sum - seg0);  // the part's exclusive base in the group
    for (int64_t c = c0; c < c1; ++c) {
      const int v = counts[c * E + e];
      counts[c * E + e] = run;
      run += v;
    }
    if (part == 0) offsets[e] = offs[e];
    // padding rows of the group: src_row = -1, spread over the expert's parts
    for (int r = offs[e] + tot + part; r < offs[e + 1]; r += P) src_row[r] = -1;
  }
  if (threadIdx.x == 0) offsets[E] = offs[E];
}

// One workgroup (4 waves) per chunk: wave w takes tokens 64 w .. 64 w + 63 of the chunk and
// sets, per expert, a 64-bit LDS mask of its lanes routed there; a pair's rank is the
// chunk's base for its expert, plus the popcounts of that expert's masks in earlier waves,
// plus its position among earlier lanes of its own mask.  All four waves work at once (one
// round of routing loads per chunk instead of four).
__global__ __launch_bounds__(kChunk) void route_assign_kernel(const int32_t* __restrict__ idx, int64_t T, int k, int E,
                                                             const int32_t* __restrict__ bases,
                                                             int32_t* __restrict__ row_map, int32_t* __restrict__ src_row) {
  static_assert(kChunk == 256, "four waves of 64 tokens per chunk");
  __shared__ int run[1024];
  __shared__ unsigned long long mask[4][1024];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int64_t chunk = blockIdx.x;
  for (int e = tid; e < E; e += kChunk) {
    run[e] = bases[chunk * E + e];
#pragma unroll
    for (int w = 0; w < 4; ++w) mask[w][e] = 0ull;
  }
  __syncthreads();
  const int64_t t = chunk * kChunk + tid;
  const bool valid = t < T;
  for (int j = 0; j < k && valid; ++j) {
    const int e = idx[t * k + j];
    if (e >= 0 && e < E) atomicOr(&mask[wave][e], 1ull << lane);
  }
  __syncthreads();
  const unsigned long long below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int j = 0; j < k && valid; ++j) {
    const int e = idx[t * k + j];
    int row = -1;
    if (e >= 0 && e < E) {
      row = run[e] + __popcll(mask[wave][e] & below);
      for (int w = 0; w < wave; ++w) row += __popcll(mask[w][e]);
      src_row[row] = (int32_t)(t * k + j);
    }
    row_map[t * k + j] = row;
  }
}

// Padding rows of expert e's group (src_row == -1, below offsets[e + 1]): bytes 0x00, scales
// 2^-126.  A group is padded by fewer than 128 rows, all among its last 128; the workgroup's
// waves take those rows in turn (wave-uniform tests, one 16-byte store per lane and chunk).
template <typename S>
__device__ __forceinline__ void pad_group(int e, const int32_t* __restrict__ offsets,
                                          const int32_t* __restrict__ src_row, int64_t H, uint8_t* __restrict__ q,
                                          S* __restrict__ s) {
  const int64_t g0 = offsets[e], g1 = offsets[e + 1];
  const int64_t r0 = g1 - g0 > kTile ? g1 - kTile : g0;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int n_waves = blockDim.x >> 6;
  const int64_t c16 = H / 16, sh = H / kTile;
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (int64_t r = r0 + wave; r < g1; r += n_waves) {
    if (src_row[r] >= 0) continue;
    uint8_t* row = q + r * H;
    for (int64_t c = lane; c < c16; c += 64) stnt16(row + c * 16, z);
    for (int64_t c = lane; c < sh; c += 64) put_scale(&s[r * sh + c], kTMin);
  }
}

// One workgroup per token: lane c covers 16 elements (two 16-byte loads) of the row, 8
// lanes one 128-element tile (8-lane DPP amax).  Workgroups T.. T + E - 1 fill the padding
// rows of expert groups 0..E-1 instead.  The token's k destination rows and
// weights are workgroup-uniform (scalar loads); every copy is one 16-byte store per lane,
// so a wave writes 1 KB contiguous of one destination row.
template <bool kWeighted, typename S>
__global__ __launch_bounds__(kRowThreadsMax) void permute_quant_kernel(const uint16_t* __restrict__ x,
                                                                       const float* __restrict__ row_w, int64_t H,
                                                                       int k, const int32_t* __restrict__ row_map,
                                                                       int64_t M_cap, uint8_t* __restrict__ q,
                                                                       S* __restrict__ s, int64_t T,
                                                                       const int32_t* __restrict__ offsets,
                                                                       const int32_t* __restrict__ src_row) {
  const int64_t t = blockIdx.x;
  if (t >= T) {
    pad_group<S>((int)(t - T), offsets, src_row, H, q, s);
    return;
  }
  const int64_t n16 = H / 16, sh = H / kTile;
  for (int64_t c = threadIdx.x; c < n16; c += blockDim.x) {  // uniform per 8-lane tile
    const bool leader = (c & 7) == 0;
    float v[16];
    unpack_bf16x8(ldnt16(x + t * H + c * 16), v);
    unpack_bf16x8(ldnt16(x + t * H + c * 16 + 8), v + 8);
    if (!kWeighted) {
      int tq;
      const u32x4 r = quant16_tile8(v, tq);
      for (int j = 0; j < k; ++j) {
        const int row = row_map[t * k + j];
        if (row >= 0 && row < M_cap) {
          stnt16(q + (int64_t)row * H + c * 16, r);
          if (leader) put_scale(&s[(int64_t)row * sh + (c >> 3)], tq);
        }
      }
    } else {
      for (int j = 0; j < k; ++j) {
        const int row = row_map[t * k + j];
        if (row >= 0 && row < M_cap) {
          const float w = row_w[t * k + j];
          float vw[16];
#pragma unroll
          for (int i = 0; i < 16; ++i) vw[i] = w * v[i];
          int tq;
          const u32x4 r = quant16_tile8(vw, tq);
          stnt16(q + (int64_t)row * H + c * 16, r);
          if (leader) put_scale(&s[(int64_t)row * sh + (c >> 3)], tq);
        }
      }
    }
  }
}

// B1 with the router gradient (the backward of the routing-weighted combine): besides the
// weighted, quantized copies of dY[t], dprobs[t, j] = sum_h dY[t, h] * Y_perm[row_map[t, j], h]
// in float32 (bf16 x bf16 products are exact).  One chunk of 16 columns per lane (H <= 16 *
// kRowThreadsMax), so dY[t] stays in registers for all k dot products.  Sum order, fixed: the
// lane's 16 products in column order, a butterfly over the wave, then the waves in order.
// (Loading 2, 4 or 8 slots' Y_perm rows ahead of their dot products measured no faster: the
// registers it takes cost occupancy.)
constexpr int kMaxKDprobs = 64;
template <typename S>
__global__ __launch_bounds__(kRowThreadsMax) void permute_quant_dprobs_kernel(
    const uint16_t* __restrict__ dy, const float* __restrict__ row_w, int64_t H, int k,
    const int32_t* __restrict__ row_map, int64_t M_cap, uint8_t* __restrict__ q, S* __restrict__ s,
    const uint16_t* __restrict__ y_perm, float* __restrict__ dprobs, int64_t T, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ src_row) {
  __shared__ float part[kMaxKDprobs * (kRowThreadsMax / 64)];
  const int64_t t = blockIdx.x;
  if (t >= T) {  // padding rows of group t - T (the whole workgroup leaves before any barrier)
    pad_group<S>((int)(t - T), offsets, src_row, H, q, s);
    return;
  }
  const int64_t n16 = H / 16, sh = H / kTile;
  const int c = threadIdx.x, wave = c >> 6, n_waves = blockDim.x >> 6;
  const bool act = c < n16;  // uniform per 8-lane tile
  const bool leader = (c & 7) == 0;
  float v[16];
  if (act) {
    unpack_bf16x8(ldnt16(dy + t * H + c * 16), v);
    unpack_bf16x8(ldnt16(dy + t * H + c * 16 + 8), v + 8);
  } else {
#pragma unroll
    for (int i = 0; i < 16; ++i) v[i] = 0.0f;
  }
  for (int j = 0; j < k; ++j) {
    const int row = row_map[t * k + j];
    const bool ok = row >= 0 && row < M_cap;  // uniform
    float acc = 0.0f;
    if (ok && act) {
      const uint16_t* yp = y_perm + (int64_t)row * H + c * 16;
      float y[16];
      unpack_bf16x8(ldnt16(yp), y);
      unpack_bf16x8(ldnt16(yp + 8), y + 8);
#pragma unroll
      for (int i = 0; i < 16; ++i) acc = fmaf(v[i], y[i], acc);
      const float w = row_w[t * k + j];
      float vw[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) vw[i] = w * v[i];
      int tq;
      const u32x4 r = quant16_tile8(vw, tq);
      stnt16(q + (int64_t)row * H + c * 16, r);
      if (leader) put_scale(&s[(int64_t)row * sh + (c >> 3)], tq);
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) acc += __shfl_xor(acc, d);
    if ((c & 63) == 0) part[j * (kRowThreadsMax / 64) + wave] = acc;
  }
  __syncthreads();
  for (int j = c; j < k; j += blockDim.x) {
    const int row = row_map[t * k + j];
    float sum = 0.0f;
    for (int w = 0; w < n_waves; ++w) sum += part[j * (kRowThreadsMax / 64) + w];
    dprobs[t * k + j] = (row >= 0 && row < M_cap) ? sum : 0.0f;
  }
}

// One workgroup per token: each lane sums two 8-element chunks (c and c + blockDim, so
// that every 16-byte load instruction of a wave covers 1 KB contiguous) of the token's k
// rows in slot order (float32, routing weight applied per slot when given), one bf16
// rounding.  Up to kUnrollK slots are loaded before the sum so that their reads are in
// flight together.
constexpr int kUnrollK = 8;
template <bool kWeighted>
__global__ __launch_bounds__(kRowThreadsMax) void unpermute_kernel(const uint16_t* __restrict__ y_perm,
                                                                   const int32_t* __restrict__ row_map,
                                                                   const float* __restrict__ row_w, int k, int64_t H,
                                                                   int64_t M_cap, uint16_t* __restrict__ y) {
  const int64_t t = blockIdx.x;
  const int64_t n8 = H / 8, stride = blockDim.x;
  for (int64_t c = threadIdx.x; c < n8; c += 2 * stride) {
    const bool two = c + stride < n8;
    const int64_t c1 = two ? c + stride : c;
    float acc[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
    for (int j0 = 0; j0 < k; j0 += kUnrollK) {
      u32x4 a[kUnrollK], b[kUnrollK];
      int rows[kUnrollK];
#pragma unroll
      for (int jj = 0; jj < kUnrollK; ++jj) {
        const int j = j0 + jj;
        rows[jj] = (j < k) ? row_map[t * k + j] : -1;
        if (rows[jj] >= 0 && rows[jj] < M_cap) {
          a[jj] = ldnt16(y_perm + (int64_t)rows[jj] * H + c * 8);
          b[jj] = ldnt16(y_perm + (int64_t)rows[jj] * H + c1 * 8);
        }
      }
#pragma unroll
      for (int jj = 0; jj < kUnrollK; ++jj) {
        if (rows[jj] < 0 || rows[jj] >= M_cap) continue;
        float v[16];
        unpack_bf16x8(a[jj], v);
        unpack_bf16x8(b[jj], v + 8);
        if (kWeighted) {
          const float w = row_w[t * k + j0 + jj];
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[i] = fmaf(w, v[i], acc[i]);
        } else {
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[i] += v[i];
        }
      }
    }
    u32x4 o0, o1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o0[i] = pack_bf16x2(acc[2 * i], acc[2 * i + 1]);
      o1[i] = pack_bf16x2(acc[8 + 2 * i], acc[8 + 2 * i + 1]);
    }
    stnt16(y + t * H + c * 8, o0);
    if (two) stnt16(y + t * H + c1 * 8, o1);
  }
}

// Threads of a one-token workgroup: one lane per 16 elements, whole waves, at most 512.
unsigned row_threads(int64_t H) {
  int64_t n = (H / 16 + 63) / 64 * 64;
  return (unsigned)(n < kRowThreadsMax ? n : kRowThreadsMax);
}

}  // namespace

size_t permute_workspace_bytes(int64_t T, int k, int E) {
  (void)k;
  return (size_t)n_chunks_of(T) * (size_t)E * sizeof(int32_t);
}

hipError_t launch_route(const int32_t* topk_idx, int64_t T, int k, int E, int align, int32_t* row_map, int32_t* offsets,
                        int32_t* src_row, int64_t M_cap, void* workspace, hipStream_t st) {
  (void)M_cap;
  const int64_t nc = n_chunks_of(T);
  int32_t* counts = static_cast<int32_t*>(workspace);
  if (nc > 0) route_count_kernel<<<(unsigned)nc, kChunk, 0, st>>>(topk_idx, T, k, E, counts);
  route_scan_kernel<<<1, 1024, 0, st>>>(counts, nc, E, align, offsets, src_row);
  if (nc > 0) route_assign_kernel<<<(unsigned)nc, kChunk, 0, st>>>(topk_idx, T, k, E, counts, row_map, src_row);
  return hipGetLastError();
}

// Routing workspace of the no-allocation entry point: one array per device, resident until the
// process ends.  Host code never passes its name to a kernel (in host code the name is only a
// stand-in for the symbol): it takes the device address from hipGetSymbolAddress, once per
// device with that device current, and passes that.
static __device__ __align__(256) int32_t scratch[kRouteScratchInts];

hipError_t route_scratch(int32_t** out) {
  static std::mutex mu;
  static int32_t* addr[64] = {nullptr};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = static_cast<int32_t*>(p);
  }
  *out = addr[dev];
  return hipSuccess;
}

template <typename S>
static hipError_t permute_quant_impl(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                     const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                     int64_t M_cap, uint8_t* q, S* s, hipStream_t st) {
  const unsigned grid = (unsigned)(T + E);  // tokens, then one padding workgroup per expert group
  if (row_w)
    permute_quant_kernel<true, S><<<grid, row_threads(H), 0, st>>>(x, row_w, H, k, row_map, M_cap, q, s, T, offsets,
                                                                   src_row);
  else
    permute_quant_kernel<false, S><<<grid, row_threads(H), 0, st>>>(x, row_w, H, k, row_map, M_cap, q, s, T, offsets,
                                                                    src_row);
  return hipGetLastError();
}

hipError_t launch_permute_quant(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                int64_t M_cap, uint8_t* q, float* s, hipStream_t st) {
  return permute_quant_impl(x, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, st);
}
hipError_t launch_permute_quant(const uint16_t* x, const float* row_w, int64_t T, int64_t H, int k, int E,
                                const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                int64_t M_cap, uint8_t* q, e8m0_t* s, hipStream_t st) {
  return permute_quant_impl(x, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, st);
}

template <typename S>
static hipError_t permute_quant_dprobs_impl(const uint16_t* dy, const float* row_w, int64_t T, int64_t H, int k,
                                            int E, const int32_t* row_map, const int32_t* offsets,
                                            const int32_t* src_row, int64_t M_cap, uint8_t* q, S* s,
                                            const uint16_t* y_perm, float* dprobs, hipStream_t st) {
  permute_quant_dprobs_kernel<S><<<(unsigned)(T + E), row_threads(H), 0, st>>>(dy, row_w, H, k, row_map, M_cap, q, s,
                                                                                y_perm, dprobs, T, offsets, src_row);
  return hipGetLastError();
}
hipError_t launch_permute_quant_dprobs(const uint16_t* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                       const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                       int64_t M_cap, uint8_t* q, float* s, const uint16_t* y_perm, float* dprobs,
                                       hipStream_t st) {
  return permute_quant_dprobs_impl(dy, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, y_perm, dprobs, st);
}
hipError_t launch_permute_quant_dprobs(const uint16_t* dy, const float* row_w, int64_t T, int64_t H, int k, int E,
                                       const int32_t* row_map, const int32_t* offsets, const int32_t* src_row,
                                       int64_t M_cap, uint8_t* q, e8m0_t* s, const uint16_t* y_perm, float* dprobs,
                                       hipStream_t st) {
  return permute_quant_dprobs_impl(dy, row_w, T, H, k, E, row_map, offsets, src_row, M_cap, q, s, y_perm, dprobs, st);
}

int max_k_dprobs() { return kMaxKDprobs; }
int64_t max_h_dprobs() { return 16LL * kRowThreadsMax; }

hipError_t launch_unpermute(const uint16_t* y_perm, const int32_t* row_map, const float* row_w, int64_t T, int k,
                            int64_t H, int64_t M_cap, uint16_t* y, hipStream_t st) {
  if (T == 0) return hipSuccess;
  if (row_w)
    unpermute_kernel<true><<<(unsigned)T, row_threads(H), 0, st>>>(y_perm, row_map, row_w, k, H, M_cap, y);
  else
    unpermute_kernel<false><<<(unsigned)T, row_threads(H), 0, st>>>(y_perm, row_map, row_w, k, H, M_cap, y);
  return hipGetLastError();
}

}  // namespace ff8
