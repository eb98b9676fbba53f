// Scaling-aware FP8 transpose for gfx950 (paper section 3.1, Algorithm 1 and the
// exponent-shift identity).
//
// One workgroup owns one 128-column tile of the input and kRB consecutive 128-row
// blocks; column tiles are the fastest-varying index of the grid, so the workgroups an
// XCD runs together read the same rows (their scale lines and DRAM pages once).  When the
// output row stride (rows bytes) is a multiple of 16 KB, those workgroups would all write
// the same byte offset of output rows 16 KB apart, which crowds a few memory channels; the
// row group then advances with the column tile (a diagonal order), so that workgroups
// running together write different offsets (measured +19% at 32768 rows, -2..4% at the
// layer's 135168 rows, which keep the plain order).
//   1. up front, the row scales of all kRB blocks give every row's exponent (to LDS)
//      and each block's S_max (wave DPP max + LDS), behind a single barrier;
//   2. per block, lane (sr, sc) holds an 8x8 byte sub-block (rows 8 sr.., bytes 8 sc..;
//      16 lanes read a full 128-byte row segment); all kRB blocks are loaded up front;
//   3. rows with k_i = log2(S_max) - log2(s_i) > 0 are re-expressed at S_max: decode
//      (exact), multiply by 2^-k (exact), hardware RNE encode -- equal to lowering the
//      exponent field by k_i while it stays >= 1, and the nearest-even subnormal below;
//   4. the 8x8 sub-block is transposed in registers (v_perm_b32) and written to LDS in
//      output order (XOR-swizzled 8-byte chunks, conflict-free);
//   5. the 128x128 output block is streamed out with 16-byte non-temporal stores, 8
//      lanes per 128-byte output row segment.
// Groups padded to 16 rows can end inside a block: the last block's S_max covers only the
// rows below m_rows (offsets[E]), and only those columns of qT are written.
// The column-wise scales are block-major, sT [rows/128][cols]: block rb's S_max goes to the
// 128 consecutive floats of its column tile (one coalesced 512-byte store per block), and
// a consumer reads one contiguous run per 128-row block for any range of columns.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

constexpr int kThreads = 256;
constexpr int kRB = 2;  // 128-row blocks per workgroup (all loaded before the first is written)

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

__global__ __launch_bounds__(kThreads) void sat_kernel(const uint8_t* __restrict__ q, const float* __restrict__ s,
                                                       int64_t rows, int64_t cols, const int32_t* __restrict__ offsets,
                                                       int E, int n_rb_groups, int diagonal, uint8_t* __restrict__ qT,
                                                       float* __restrict__ sT) {
  __shared__ uint32_t tile[128 * 128 / 4];  // output block, 128 rows x 128 bytes (swizzled 8-byte chunks)
  __shared__ int t_rows[kRB][128];          // scale exponent of every input row of every block
  __shared__ uint32_t wmax[kRB][2];

  const int n_cb = (int)(cols / kTile);
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  // column tiles fastest: the workgroups an XCD runs together share the same input rows,
  // so each row's scale line and DRAM pages are fetched once for all its column tiles
  const int g = logical / n_cb;
  const int cb = logical - g * n_cb;
  const int rg = diagonal ? (g + 2 * cb) % n_rb_groups : g;  // a permutation of the groups per column tile
  const int64_t m_rows = active_rows(offsets, E, rows);
  const int64_t n_rb = rows / kTile;
  const int64_t rb0 = (int64_t)rg * kRB;
  int n_valid = 0;  // blocks of this group that hold data (uniform)
#pragma unroll
  for (int bi = 0; bi < kRB; ++bi)
    if (rb0 + bi < n_rb && (rb0 + bi) * kTile < m_rows) n_valid = bi + 1;

  const int tid = threadIdx.x;
  const int sr = tid >> 4, sc = tid & 15;

  // 1. All blocks' row scales up front: per-row exponents to LDS, S_max per block by a
  //    wave DPP max and a 2-entry LDS max; one barrier for the whole group.
  if (tid < 128) {
#pragma unroll
    for (int bi = 0; bi < kRB; ++bi) {
      int t_row = -256;  // rows at and beyond m_rows (a last block cut by 16-row padding) never win S_max
      if (bi < n_valid && (rb0 + bi) * kTile + tid < m_rows)
        t_row = (int)(__float_as_uint(s[((rb0 + bi) * kTile + tid) * n_cb + cb]) >> 23) - 127;
      t_rows[bi][tid] = t_row;
      const uint32_t m = max64_u32((uint32_t)(t_row + 256));
      if ((tid & 63) == 0) wmax[bi][tid >> 6] = m;
    }
  }
  // every block's data in flight across the barrier
  u32x2 vb[kRB][8];
#pragma unroll
  for (int bi = 0; bi < kRB; ++bi) {
    if (bi < n_valid) {
      const uint8_t* src = q + ((rb0 + bi) * kTile + sr * 8) * cols + (int64_t)cb * kTile + sc * 8;
#pragma unroll
      for (int i = 0; i < 8; ++i) vb[bi][i] = ld8(src + (int64_t)i * cols);
    }
  }
  __syncthreads();

#pragma unroll
  for (int bi = 0; bi < kRB; ++bi) {
    if (bi >= n_valid) break;
    const int64_t rb = rb0 + bi;
    u32x2* v = vb[bi];
    const int t_max = (int)max(wmax[bi][0], wmax[bi][1]) - 256;
    // 2. rows below S_max are re-expressed at S_max: decode (exact), times 2^-k (exact),
    //    RNE encode -- the exponent-field decrement, and nearest-even below the normals.
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = t_max - t_rows[bi][sr * 8 + i];
      if (k != 0) {
        // every e4m3 value is below 2^9, so any k >= 19 sends it to a signed zero; the
        // clamp keeps 2^-k a normal float for the block's full 253-octave range
        const float f = exp2i(-min(k, 64));
        v[i][0] = shift4(v[i][0], f);
        v[i][1] = shift4(v[i][1], f);
      }
    }
    // 3. transpose the 8x8 sub-block: column c of the input becomes output row 8 sc + c.
    uint32_t o_lo[8], o_hi[8];
    transpose4x4(v[0][0], v[1][0], v[2][0], v[3][0], o_lo[0], o_lo[1], o_lo[2], o_lo[3]);
    transpose4x4(v[4][0], v[5][0], v[6][0], v[7][0], o_hi[0], o_hi[1], o_hi[2], o_hi[3]);
    transpose4x4(v[0][1], v[1][1], v[2][1], v[3][1], o_lo[4], o_lo[5], o_lo[6], o_lo[7]);
    transpose4x4(v[4][1], v[5][1], v[6][1], v[7][1], o_hi[4], o_hi[5], o_hi[6], o_hi[7]);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int orow = sc * 8 + c;
      const int chunk = sr ^ (orow >> 3);  // orow >> 3 == sc
      u32x2 w;
      w[0] = o_lo[c];
      w[1] = o_hi[c];
      *reinterpret_cast<u32x2*>(&tile[orow * 32 + chunk * 2]) = w;
    }
    __syncthreads();

    // 4. stream the output block: 8 lanes per 128-byte output row, 4 passes of 32 rows;
    //    streaming stores (the transposed tensor is consumed much later, by wgrad).
    const int c16 = tid & 7;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const int orow = (tid >> 3) + 32 * p;
      const int sw = (orow >> 3) & 15;
      const u32x2 a = *reinterpret_cast<const u32x2*>(&tile[orow * 32 + ((2 * c16) ^ sw) * 2]);
      const u32x2 b = *reinterpret_cast<const u32x2*>(&tile[orow * 32 + ((2 * c16 + 1) ^ sw) * 2]);
      u32x4 o;
      o[0] = a[0];
      o[1] = a[1];
      o[2] = b[0];
      o[3] = b[1];
      if (rb * kTile + c16 * 16 < m_rows)  // m_rows is a multiple of 16: whole 16-byte pieces
        stnt16(qT + ((int64_t)cb * kTile + orow) * rows + rb * kTile + c16 * 16, o);
    }
    __syncthreads();  // the tile is rewritten by the next block
  }

  // 5. column-wise scales: S_max of each block for the tile's 128 columns.
  if (tid < 128) {
    for (int bi = 0; bi < n_valid; ++bi)
      sT[(rb0 + bi) * cols + (int64_t)cb * kTile + tid] = exp2i((int)max(wmax[bi][0], wmax[bi][1]) - 256);
  }
}

}  // namespace

hipError_t launch_sat(const uint8_t* q, const float* s, int64_t rows, int64_t cols, const int32_t* offsets, int E,
                      uint8_t* qT, float* sT, hipStream_t st) {
  const int64_t n_rb = rows / kTile;
  const int n_groups = (int)((n_rb + kRB - 1) / kRB);
  const int64_t blocks = (cols / kTile) * n_groups;
  const int diagonal = rows % 16384 == 0;
  sat_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(q, s, rows, cols, offsets, E, n_groups, diagonal, qT, sT);
  return hipGetLastError();
}

}  // namespace ff8
