// Scaling-aware FP8 transpose for gfx950 (paper section 3.1, Algorithm 1 and the
// exponent-shift identity).
//
// Output layout: the transpose is K-blocked.  Element (c, r) of the transpose of a [rows, cols]
// tensor -- row r, column c of the input -- is byte (r / 128) * cols * 128 + c * 128 + r % 128 of
// qT: block b of 128 input rows is one contiguous [cols][128] slab, next to its column scales
// sT[b][cols] (block-major).  A 128 x 128 block of the output is then 16 KB of consecutive
// bytes, and the weight-gradient GEMM reads each K stage of an operand panel as one run.
//
// One workgroup owns one 128-row block of the input and two neighbouring 128-column tiles,
// whose output is one 32 KB run of the block's slab (measured 1-3% faster than two vertically
// stacked blocks); column-tile pairs are the fastest-varying index of the grid, so the
// workgroups an XCD runs together read the same rows (their scale lines and DRAM pages once)
// and write consecutive stretches of one slab.
//   1. up front, the row scales of both blocks give every row's exponent (to LDS) and each
//      block's S_max (wave DPP max + LDS);
//   2. both blocks' data are loaded before the first barrier: lane (db, sr, sc) holds 8 rows x
//      16 bytes of block db (16-byte non-temporal loads); the 16 lanes of both blocks' 128-byte
//      pieces of a row are consecutive, so a load instruction reads 4 rows x 256 bytes (1-2%
//      faster than 8 rows x 128 bytes of one block);
//   3. rows with k_i = log2(S_max) - log2(s_i) > 0 are re-expressed at S_max: decode (exact),
//      multiply by 2^-k (exact), hardware RNE encode -- equal to lowering the exponent field
//      by k_i while it stays >= 1, and the nearest-even subnormal below;
//   4. each 8x8 byte sub-block is transposed in registers (v_perm_b32) and written to LDS in
//      output order (8-byte units XOR-swizzled within their 128-byte block);
//   5. after one more barrier, the pair's 32 KB leave as consecutive 16-byte stores (plain
//      stores: measured faster than non-temporal ones here).
// Against the former row-major transpose [cols][rows], whose 256-byte runs per output row had
// to be spread by a diagonal grid order when the row stride was a multiple of 16 KB, the
// K-blocked output is 3-7% faster at the layer's 135168 rows and 37% faster on 32768 x 7168.
// Groups padded to 16 rows can end inside a block: the last block's S_max covers only the
// rows below m_rows (offsets[E]), and only those rows of its slab are written.
// One launch can transpose up to four tensors with the same rows (the backward pass's four
// weight-gradient operands): tensor t owns the logical workgroups [first[t], first[t + 1]), so
// the tail of one tensor's grid overlaps the head of the next instead of draining the chip
// between launches.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// 4x4 byte transpose: rows a, b, c, d (byte j of each = column j) -> columns.
__device__ __forceinline__ void transpose4x4(uint32_t a, uint32_t b, uint32_t c, uint32_t d, uint32_t& w0,
                                             uint32_t& w1, uint32_t& w2, uint32_t& w3) {
  const uint32_t p = perm(b, a, 0x06020400u);  // a0 b0 a2 b2
  const uint32_t q = perm(b, a, 0x07030501u);  // a1 b1 a3 b3
  const uint32_t r = perm(d, c, 0x06020400u);  // c0 d0 c2 d2
  const uint32_t s = perm(d, c, 0x07030501u);  // c1 d1 c3 d3
  w0 = perm(r, p, 0x05040100u);                // a0 b0 c0 d0
  w2 = perm(r, p, 0x07060302u);                // a2 b2 c2 d2
  w1 = perm(s, q, 0x05040100u);                // a1 b1 c1 d1
  w3 = perm(s, q, 0x07060302u);                // a3 b3 c3 d3
}

// Re-express 4 e4m3 bytes at a scale 2^k times larger.
__device__ __forceinline__ uint32_t shift4(uint32_t w, float f) {
  const f32x2 lo = dec_e4m3x2<false>(w), hi = dec_e4m3x2<true>(w);
  return cvt_e4m3x4(lo[0] * f, lo[1] * f, hi[0] * f, hi[1] * f);
}

__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int xcd = bid & 7, slot = bid >> 3, q = n >> 3, r = n & 7;
  return xcd * q + (xcd < r ? xcd : r) + slot;
}

// Re-express the rows of an 8 x 8 byte sub-block at the block scale (k_i octaves lower; every
// e4m3 value is below 2^9, so k >= 19 gives a signed zero and the clamp keeps 2^-k a normal
// float), transpose it and write it to the output tile at output rows o0..o0+7, 8-byte unit
// `unit` of block bi.  w0[i], w1[i]: the sub-block's row i, bytes 0-3 and 4-7.
template <int RB>
__device__ __forceinline__ void shift_transpose_store(uint32_t (&w0)[8], uint32_t (&w1)[8], const int* t_row, int t_max,
                                                      u32x2* tile, int o0, int bi, int unit) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = t_max - t_row[i];
    if (k != 0) {
      const float f = exp2i(-min(k, 64));
      w0[i] = shift4(w0[i], f);
      w1[i] = shift4(w1[i], f);
    }
  }
  uint32_t o_lo[8], o_hi[8];
  transpose4x4(w0[0], w0[1], w0[2], w0[3], o_lo[0], o_lo[1], o_lo[2], o_lo[3]);
  transpose4x4(w0[4], w0[5], w0[6], w0[7], o_hi[0], o_hi[1], o_hi[2], o_hi[3]);
  transpose4x4(w1[0], w1[1], w1[2], w1[3], o_lo[4], o_lo[5], o_lo[6], o_lo[7]);
  transpose4x4(w1[4], w1[5], w1[6], w1[7], o_hi[4], o_hi[5], o_hi[6], o_hi[7]);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int orow = o0 + c;
    u32x2 w;
    w[0] = o_lo[c];
    w[1] = o_hi[c];
    tile[orow * RB * 16 + bi * 16 + (unit ^ ((orow >> 3) & 15))] = w;
  }
}

// Output tile of the workgroup's two blocks: 128 rows (input columns of a block) x 2 x 128
// bytes (input rows), in 8-byte units: unit k of block b of output row o sits at
// b*16 + (k ^ ((o >> 3) & 15)).  Rows of the input are 8-byte units of the output; the swizzle
// keeps the sub-block writes and the row reads conflict-free.
constexpr int RB = 2;  // 128x128 blocks per workgroup

// The tensors of one launch; all have `rows` rows and the same active rows.
template <typename S>
struct SatJobs {
  const uint8_t* q[kSatMaxJobs];
  const S* s[kSatMaxJobs];
  uint8_t* qT[kSatMaxJobs];
  S* sT[kSatMaxJobs];
  int64_t cols[kSatMaxJobs];
  int first[kSatMaxJobs + 1];  // first logical workgroup of each tensor; first[n] = the grid
  int n;
};

template <typename S>
__global__ __launch_bounds__(kThreads) void sat_kernel(const SatJobs<S> jobs, int64_t rows,
                                                       const int32_t* __restrict__ offsets, int E) {
  __shared__ u32x2 tile[128 * RB * 16];
  __shared__ int t_rows[RB][128];
  __shared__ uint32_t wmax[RB][2];

  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  int t = 0;  // the tensor of this workgroup (uniform)
#pragma unroll
  for (int i = 1; i < kSatMaxJobs; ++i)
    if (i < jobs.n && logical >= jobs.first[i]) t = i;
  const uint8_t* __restrict__ q = jobs.q[t];
  const S* __restrict__ s = jobs.s[t];
  uint8_t* __restrict__ qT = jobs.qT[t];
  S* __restrict__ sT = jobs.sT[t];
  const int64_t cols = jobs.cols[t];
  const int local = logical - jobs.first[t];
  const int n_cb = (int)(cols / kTile), n_cp = (n_cb + 1) / 2;
  const int64_t rb = local / n_cp;                     // the 128-row block
  const int cb0 = 2 * (local - (int)rb * n_cp);        // its first column tile
  const int64_t m_rows = active_rows(offsets, E, rows);
  if (rb * kTile >= m_rows) return;                    // uniform: a block past the active rows
  const int n_valid = cb0 + 1 < n_cb ? 2 : 1;          // column tiles of this pair (uniform)
  const int tid = threadIdx.x;
  const int64_t r0 = rb * kTile;

  // 1. row exponents to LDS, S_max per block (wave DPP max, two waves per block); rows at and
  //    beyond m_rows (a last block cut by 16-row padding) never win S_max
  const int bl = tid >> 7;                             // block (column tile cb0 + bl) of this half
  {
    const int r = tid & 127;
    int t_row = -256;
    if (bl < n_valid && r0 + r < m_rows) t_row = scale_exp(s[(r0 + r) * n_cb + cb0 + bl]);
    t_rows[bl][r] = t_row;
    const uint32_t m = max64_u32((uint32_t)(t_row + 256));
    if ((tid & 63) == 0) wmax[bl][(tid >> 6) & 1] = m;
  }

  // 2.-4. both blocks loaded before the barrier, then shifted, transposed and staged
  // lane (db, sr, sc) = (bit 3, bits 4-7, bits 0-2 of tid): rows 8 sr.. of block db, 16 bytes
  // from 16 sc
  const int db = (tid >> 3) & 1, sr = tid >> 4, sc = tid & 7;
  u32x4 v[8];
  if (db < n_valid) {
    const uint8_t* src = q + (r0 + sr * 8) * cols + (int64_t)(cb0 + db) * kTile + sc * 16;
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = ldnt16(src + (int64_t)i * cols);
  }
  __syncthreads();
  if (db < n_valid) {
    const int t_max = (int)max(wmax[db][0], wmax[db][1]) - 256;
#pragma unroll
    for (int h = 0; h < 2; ++h) {  // the two 8-byte column halves
      uint32_t w0[8], w1[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        w0[i] = v[i][2 * h];
        w1[i] = v[i][2 * h + 1];
      }
      shift_transpose_store<RB>(w0, w1, &t_rows[db][sr * 8], t_max, tile, sc * 16 + 8 * h, db, sr);
    }
  }
  __syncthreads();

  // 5. the pair's [256 columns][128 rows] of slab rb, 32 KB of consecutive bytes from
  //    (rb * cols + cb0 * 128) * 128: lane j of 8 carries bytes 16 j.. of an output row of block
  //    blk (m_rows is a multiple of 16: whole pieces)
  constexpr int CPR = RB * 8;          // 16-byte pieces per output row (both blocks)
  constexpr int RPP = kThreads / CPR;  // output rows per pass
  const int j = tid % CPR, blk = j >> 3, u = 2 * (j & 7);
  const bool ok = blk < n_valid && r0 + (j & 7) * 16 < m_rows;
  uint8_t* const slab = qT + (rb * cols + (int64_t)(cb0 + blk) * kTile) * kTile + (j & 7) * 16;
#pragma unroll
  for (int p = 0; p < 128 / RPP; ++p) {
    const int orow = tid / CPR + p * RPP;
    const int sw = (orow >> 3) & 15;
    const u32x2 a = tile[orow * RB * 16 + blk * 16 + (u ^ sw)];
    const u32x2 b = tile[orow * RB * 16 + blk * 16 + ((u + 1) ^ sw)];
    u32x4 o;
    o[0] = a[0];
    o[1] = a[1];
    o[2] = b[0];
    o[3] = b[1];
    if (ok) st16(slab + (int64_t)orow * kTile, o);
  }

  // column-wise scales: each block's S_max for its 128 columns
  if (bl < n_valid)
    put_scale(&sT[rb * cols + (int64_t)(cb0 + bl) * kTile + (tid & 127)], (int)max(wmax[bl][0], wmax[bl][1]) - 256);
}

}  // namespace

template <typename S>
static hipError_t sat_impl(int n, const uint8_t* const* q, const S* const* s, const int64_t* cols, int64_t rows,
                           const int32_t* offsets, int E, uint8_t* const* qT, S* const* sT, hipStream_t st) {
  SatJobs<S> jobs{};
  const int64_t n_rb = rows / kTile;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    jobs.q[i] = q[i];
    jobs.s[i] = s[i];
    jobs.qT[i] = qT[i];
    jobs.sT[i] = sT[i];
    jobs.cols[i] = cols[i];
    jobs.first[i] = (int)total;
    total += n_rb * ((cols[i] / kTile + 1) / 2);
    if (total >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  }
  jobs.first[n] = (int)total;
  jobs.n = n;
  sat_kernel<S><<<(unsigned)total, kThreads, 0, st>>>(jobs, rows, offsets, E);
  return hipGetLastError();
}

hipError_t launch_sat(const uint8_t* q, const float* s, int64_t rows, int64_t cols, const int32_t* offsets, int E,
                      uint8_t* qT, float* sT, hipStream_t st) {
  return sat_impl(1, &q, &s, &cols, rows, offsets, E, &qT, &sT, st);
}
hipError_t launch_sat(const uint8_t* q, const e8m0_t* s, int64_t rows, int64_t cols, const int32_t* offsets, int E,
                      uint8_t* qT, e8m0_t* sT, hipStream_t st) {
  return sat_impl(1, &q, &s, &cols, rows, offsets, E, &qT, &sT, st);
}
hipError_t launch_sat_batch(int n, const uint8_t* const* q, const float* const* s, const int64_t* cols, int64_t rows,
                            const int32_t* offsets, int E, uint8_t* const* qT, float* const* sT, hipStream_t st) {
  return sat_impl(n, q, s, cols, rows, offsets, E, qT, sT, st);
}
hipError_t launch_sat_batch(int n, const uint8_t* const* q, const e8m0_t* const* s, const int64_t* cols, int64_t rows,
                            const int32_t* offsets, int E, uint8_t* const* qT, e8m0_t* const* sT, hipStream_t st) {
  return sat_impl(n, q, s, cols, rows, offsets, E, qT, sT, st);
}

}  // namespace ff8
