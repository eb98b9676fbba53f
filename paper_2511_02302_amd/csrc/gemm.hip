// FP8 grouped GEMMs for gfx950: fprop, dgrad and wgrad of the expert layer (paper
// sections 3.1-3.2: row-wise FP8 operands for Fprop/Dgrad, column-wise operands from
// the scaling-aware transpose for Wgrad).
//
// Every mode is C[p, q] = sum_k P[p, k] * Q[q, k] * sP(p, k/128) * sQ(q, k/128) over
// one expert's data, where p indexes the output's contiguous dimension:
//   fprop: p = n (W_e rows),        q = token row m, k over K  -> out[m, n] bf16
//   dgrad: p = k (W_e columns),     q = token row m, k = n     -> out[m, k] bf16
//   wgrad: p = k (xT rows),         q = n (gT rows), k = token -> dw[e, n, k] fp32
// The wgrad operands come K-blocked from the transpose: row r's bytes of token block b at
// (b * rows + r) * 128.
//
// Matrix core: v_mfma_scale_f32_32x32x64_f8f6f4 (e4m3 x e4m3, fp32 accumulate).  The
// library's scales are powers of two, i.e. exactly E8M0 values (the fp32 exponent
// field), so the per-128 block scales of both operands are applied by the MFMA itself,
// per P row and per Q column, inside the fp32 accumulation -- no VALU promotion pass.
//
// Tiling: 256 (p) x 256 (q) per workgroup, 4 waves in 2 x 2, each wave 128 x 128 =
// 4 x 4 MFMA tiles (256 accumulators in AGPRs).  K advances 128 per stage (one scale
// block), in two half-steps of 64 (16 MFMAs each).
// Data movement is sized for the L2, whose request rate is the binding limit: every
// operand row segment of a stage is one whole 128-byte line, loaded by
// buffer_load_dwordx4 ... lds straight into LDS (8 lanes per line, no register staging);
// the scales of four K blocks arrive in one batch (four lanes per row line).  Two
// stage buffers: the DMA of stage s+2 is issued, spread over the MFMAs, during the
// second half of stage s, once a barrier has shown every wave done with stage s's
// buffer and stage s+1 landed.  Fragments are double buffered in VGPRs (one set per
// half-step), and LDS reads are threaded one or two per MFMA.
// K-major tiles (128-byte rows) use the 16-byte XOR swizzle chunk ^ ((r >> 1) & 7),
// conflict-free for the fragment reads.  dgrad reads W_e in its stored [n][k]
// orientation (256-byte rows) with ds_read_b64_tr_b8, which transposes 8x8 byte
// blocks across lanes; its rows use the swizzle chunk ^ ((2j ^ j>>2) & 15), j = n%8.
//
// Grouped scheduling is on the device: tiles are counted per expert from offsets (no
// host sync).  The kernel is persistent, one workgroup per CU walking its XCD's tiles, so
// that a tile's epilogue (output staged through one stage buffer, streaming stores)
// overlaps the next tile's first-stage DMA into the other.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) uint8_t lds_u8;

constexpr int kThreads = 256;
constexpr int kTP = 256;   // p tile
constexpr int kTQ = 256;   // q tile
constexpr int kBK = 128;   // k per stage (one scale block)
constexpr int kBQ = 8;     // q tiles per XCD block
constexpr int kBP = 4;     // p tiles per XCD block
static_assert(kBQ * kBP == 32, "an XCD block is the 32 workgroups one XCD runs at once");
constexpr int kTileBytes = kTP * kBK;  // 32 KB per operand per stage
constexpr int kScaleBatch = 4;         // K blocks per scale batch
#define FF8_STR2(x) #x
#define FF8_STR(x) FF8_STR2(x)
constexpr int kReadSlots = 6;          // MFMA slots of a half-step that carry fragment reads
// The stage buffer a stage reads is free once every wave has read its second-half fragments
// (issued over the first kReadSlots slots of the first half-step): a barrier at slot kEarly
// publishes that, and the 16 tile DMAs of stage ks+2 into it are spread evenly over the
// remaining kDmaSlots MFMA slots of the stage.  (Issued within the second half-step only, the
// 64 DMA instructions of a workgroup outran the vector-memory path, whose backpressure stalled
// the in-order waves in front of their next MFMA.)
constexpr int kEarly = 6;
constexpr int kDmaSlots = 32 - kEarly;
static_assert(kEarly >= kReadSlots && kEarly < 16, "the early barrier follows the last fragment read of half 0");
// tile DMAs issued before DMA slot j (slot j = MFMA slot kEarly + j of half 0, then of half 1)
__host__ __device__ constexpr int dma_before(int j) { return (16 * j) / kDmaSlots; }
// DMAs issued in half 0, still in flight at the mid-stage wait (the literal in that wait)
#define FF8_HALF0_DMAS 6
static_assert(dma_before(16 - kEarly) == FF8_HALF0_DMAS, "mid-stage vmcnt literal");
// Rotate each XCD block's K order (memory-channel spread).  Measured: +5.6% for fprop,
// whose two operands are row-major over K; -1% / -3% for dgrad / wgrad, which keep it off.
template <int MODE> constexpr bool kStaggerK = (MODE == kFprop);

__shared__ __attribute__((aligned(1024))) uint8_t g_st0[2 * kTileBytes], g_st1[2 * kTileBytes];  // [P | Q]
__shared__ __attribute__((aligned(1024))) float g_sc[2][2 * kTP * kScaleBatch];  // [P rows x 4 | Q rows x 4]
__shared__ int g_cum[1025];  // fprop/dgrad: cumulative 256-row tile counts per expert
__shared__ int g_off[1025];  // fprop/dgrad: expert row offsets

template <int B> __device__ __forceinline__ uint8_t* stage_buf() {
  if constexpr (B == 0) return g_st0; else return g_st1;
}
template <int B> __device__ __forceinline__ uint32_t stage_lds() {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)stage_buf<B>();
}
__device__ __forceinline__ uint32_t scale_lds(int b) {
  return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) float*)&g_sc[b][0];
}

struct GemmArgs {
  const uint8_t* P;   // fprop: w; dgrad: w; wgrad: xT
  const void* sP;     // scales: float, or UE8M0 bytes
  const uint8_t* Q;   // fprop: a; dgrad: g; wgrad: gT
  const void* sQ;
  const int32_t* offsets;
  void* out;
  int E;
  int M_cap;          // dimensions are below 2^31 (byte offsets below 2^32 are checked on the host)
  int Np;             // extent of p (output columns)
  int Nq;             // wgrad: extent of q (N); fprop/dgrad: unused
  int Kdim;           // fprop/dgrad: contraction length; wgrad: unused (per group)
  int n_pt, n_qt;     // p tiles; q tiles (wgrad only)
  int accumulate;
  int n_slots;        // workgroups per XCD in one group of the grid
  // wgrad expert shares (share = 0: none fit): each XCD takes one rect_q x rect_p-tile
  // rectangle of every expert's n_qt x n_pt tiles, the 8 rectangles tiling it (rect_b along p)
  int share, rect_q, rect_p, rect_b;
};

// K-major stage tile: 256 rows x 128 bytes, 16-byte chunk c of row r at c ^ kswz(r).  Any
// 16 consecutive rows take the 16 distinct (r % 2, chunk) slots of a 256-byte bank window,
// and the swizzle repeats every 16 rows, so fragment rows 32 apart share one address
// register (plus an immediate offset).
__device__ __forceinline__ int kswz(int r) { return (r >> 1) & 7; }
// dgrad weight stage tile: 128 rows (n) x 256 bytes, chunk c of row n at c ^ wswz(n % 8).
__device__ __forceinline__ int wswz(int j) { return ((2 * j) ^ (j >> 2)) & 15; }

// LDS DMA (buffer_load ... lds): each lane loads 16 (or 4) bytes at resource base +
// soff + voff into LDS at M0 + 16 * lane (or 4 * lane).  The resources cover exactly
// their tensor, and every operand offset is in voffset, which the hardware range-checks:
// rows past a tensor's end read zeros, so tiles at the edges need no clamping (K-blocked
// wgrad operands: rows past the end read the next block's rows, or zeros after the last
// block; those rows' accumulators are never stored).  Issued
// through inline asm so that the compiler does not serialize the pipeline with
// conservative waits; the kernel waits for its own DMA (vmcnt) before the barrier that
// publishes a stage.  The compiler's hazard checks do not look inside asm.  A buffer
// instruction needs 5 wait states after a VALU write of an SGPR it reads (the resource or M0
// may come straight from v_readfirstlane, or from v_readlane when the compiler reloads a
// spilled SGPR), and an LDS DMA 1 after an SALU write of M0; with fewer, the load can use the
// register's old value.  The DMAs issued right after a tile's setup (kLoop false) carry all 5.
// Inside the K loop the resources are loop-invariant and M0 is set by s_mov, so the DMAs there
// carry 1 (4 issue cycles fewer per DMA, 1-2% on every GEMM); the hazard scan of the compiled
// kernels checks that no VALU write of an SGPR they read comes closer.
typedef int i32x4 __attribute__((ext_vector_type(4)));
// Raw (stride 0) buffer resource: loads at offsets >= `bytes` return zeros.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, uint32_t bytes = 0xFFFFFFFFu) {
  const uint64_t a = (uint64_t)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));  // stride 0
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;   // raw 32-bit data format
  return r;
}
template <bool kLoop = false>
__device__ __forceinline__ void dma16(const i32x4& rsrc, uint32_t voff, uint32_t lds_off) {
  if constexpr (kLoop)
    asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "{m0}"(lds_off), "v"(voff), "s"(rsrc)
                 : "memory");
  else
    asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" : : "{m0}"(lds_off), "v"(voff), "s"(rsrc)
                 : "memory");
}
// 4-byte form (scales).  The scale DMAs, like the operand DMAs, keep their whole offset in
// the range-checked voffset, so a lane past a scale tensor's end reads zeros.
template <bool kLoop = false>
__device__ __forceinline__ void dma4(const i32x4& rsrc, uint32_t voff, uint32_t lds_off) {
  if constexpr (kLoop)
    asm volatile("s_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds" : : "{m0}"(lds_off), "v"(voff), "s"(rsrc)
                 : "memory");
  else
    asm volatile("s_nop 4\n\tbuffer_load_dword %1, %2, 0 offen lds" : : "{m0}"(lds_off), "v"(voff), "s"(rsrc)
                 : "memory");
}

__device__ __forceinline__ i32x8 with_half(i32x8 f, const u32x4& x, int half) {
  f[4 * half + 0] = (int)x[0];
  f[4 * half + 1] = (int)x[1];
  f[4 * half + 2] = (int)x[2];
  f[4 * half + 3] = (int)x[3];
  return f;
}

// Lane index as an opaque value: lane-dependent tile setup and epilogue arithmetic built
// on it is recomputed per tile instead of being hoisted out of the tile loop, where it
// would stay live (in registers) through the main loop.
__device__ __forceinline__ int opaque_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Per-thread state of one workgroup tile.  SC: scale storage, float (fp32 powers of two)
// or e8m0_t (UE8M0 bytes); either way the MFMA receives the E8M0 byte.
template <int MODE, typename SC>
struct Tile {
  static constexpr bool kE8 = sizeof(SC) == 1;
  static constexpr uint32_t kSB = sizeof(SC);  // bytes per stored scale
  f32x16 acc[4][4];
  i32x8 fpA[4], fqA[4], fpB[4], fqB[4];  // set A: first half-step, set B: second
  // Packed E8M0 scales of the current batch of four K blocks, per K block: byte R of
  // cp[j] is the scale of this lane's P row 128 wp + 32 R + l (cq: Q rows); np/nq are
  // the next batch, assembled during the last stage of the current one.
  uint32_t cp[4], cq[4], np[4], nq[4];
  u32x4 rsp[4], rsq[4];  // raw scale rows of the next batch, between read and pack
  uint32_t p_shift;      // dgrad with UE8M0 scales: bit offset of the wave's weight-block byte in its dword
  // DMA sources: one resource per tensor; per-lane byte offsets of this tile's stage 0
  // for the two row-group patterns of the tile DMA (instruction i uses pattern i / 4,
  // dgrad P: i % 2), and wave-uniform steps between instructions and stages.
  i32x4 p_rsrc, q_rsrc, sp_rsrc, sq_rsrc;
  uint32_t p_voff[2], q_voff[2];
  uint32_t sp_off, sq_off;       // scale DMA: this lane's source offset at K block 0
  int p_kstep, q_kstep;          // bytes per stage of the P / Q source
  int p_istep, q_istep;          // bytes between instructions of one pattern
  int sp_kb, sq_kb;              // scales per K block of the P / Q scale sources
  // fprop / dgrad: a wave's 128 P rows are one 128x128 weight block, so its P scale is one
  // value per K block (stored compactly as [tile half][4 K blocks]); wgrad: one per row.
  static constexpr bool kBlockP = (MODE != kWgrad);
  // wgrad reads and packs the next batch's per-row scales of P in the second stage of a batch
  // and those of Q in the fourth (its scale DMA lands by the middle of the second), instead of
  // both in the fourth: fewer VALU packs crowd one stage's MFMA slots (+0.6%).  fprop and dgrad
  // keep them in the fourth stage, where the packed words are not live across stages.
  static constexpr bool kSpreadScales = (MODE == kWgrad);
  int wave, lane, wp, wq;
  int nk;
  int k_rot;  // K stages this tile's loop is rotated by (fprop: a multiple of the scale batch)
  int k_lo, k_hi;  // wgrad: valid K bytes [k_lo, 128) of the first stage and [0, k_hi) of the last
  // Stage ks of the loop reads K block (ks + k_rot) mod nk.
  __device__ __forceinline__ int kphys(int ks) const {
    const int k = ks + k_rot;
    return k < nk ? k : k - nk;
  }

  // Tile DMA instruction I (0..15) of stage ks into stage buffer B: 0-7 P, 8-15 Q.
  // K-major tiles (fprop / wgrad operands, dgrad Q): instruction i of wave w carries row
  // group w + 8i (i < 4) or w + 4 + 8(i - 4) (i >= 4) -- 8 rows x 128 bytes, LDS 1 KB at
  // group * 1 KB -- so that within each pattern the swizzle (row group % 8) is constant
  // and consecutive instructions are one uniform step apart.  dgrad P (W_e rows n, 256
  // bytes): instruction i carries rows 32w + 4i .., patterns by i % 2.
  // wgrad with groups padded to 16 rows: an expert's first and last K blocks may hold tokens
  // of its neighbours (or rows past offsets[E]).  Such a tile's loop is rotated so that these
  // two blocks are its stages 0 and 1 (the last block first), whose DMAs are issued before
  // the loop with kMask: lanes whose 16 tokens lie outside the expert load from the
  // resource's end instead, which reads zeros, so those tokens add nothing and the loop
  // itself is unchanged.  A K-major lane's 16-byte chunk is (l % 8) ^ kswz(row), the same
  // for both patterns and both operands: (l % 8) ^ ((4 (w % 2) + l / 16) % 8).
  __device__ __forceinline__ uint32_t masked_off(uint32_t off, uint32_t kp, uint32_t end) const {
    const int l = lane;
    const int c16 = 16 * ((l & 7) ^ ((4 * (wave & 1) + (l >> 4)) & 7));
    const bool drop = (kp == 0 && c16 < k_lo) || ((int)kp == nk - 1 && c16 >= k_hi);
    return drop ? end : off;
  }
  template <int B, int I, bool kMask = false, bool kLoop = false>
  __device__ __forceinline__ void dma_tile(int ks) {
    const uint32_t stage = stage_lds<B>();
    const uint32_t kp = (uint32_t)__builtin_amdgcn_readfirstlane(kphys(ks));  // uniform
    if constexpr (I < 8) {
      if constexpr (MODE == kDgrad) {
        const uint32_t step = kp * (uint32_t)p_kstep + (uint32_t)(I >> 1) * (uint32_t)p_istep;
        dma16<kLoop>(p_rsrc, p_voff[I & 1] + step, stage + (uint32_t)wave * 8192u + I * 1024);
      } else {
        const uint32_t step = kp * (uint32_t)p_kstep + (uint32_t)(I & 3) * (uint32_t)p_istep;
        const uint32_t grp = (uint32_t)wave + (I < 4 ? 8 * I : 4 + 8 * (I - 4));
        uint32_t off = p_voff[I >> 2] + step;
        if constexpr (kMask) off = masked_off(off, kp, (uint32_t)p_rsrc[2]);
        dma16<kLoop>(p_rsrc, off, stage + grp * 1024u);
      }
    } else {
      constexpr int J = I - 8;
      const uint32_t step = kp * (uint32_t)q_kstep + (uint32_t)(J & 3) * (uint32_t)q_istep;
      const uint32_t grp = (uint32_t)wave + (J < 4 ? 8 * J : 4 + 8 * (J - 4));
      uint32_t off = q_voff[J >> 2] + step;
      if constexpr (kMask) off = masked_off(off, kp, (uint32_t)q_rsrc[2]);
      dma16<kLoop>(q_rsrc, off, stage + kTileBytes + grp * 1024u);
    }
  }
  // Scale DMA of batch b (K blocks kb0..kb0+3 in loop order) into batch buffer b % 2:
  //   fprop / dgrad P (kBlockP): 8 lanes carry the tile's two weight blocks' 4 floats (the
  //     rest duplicate them) -> LDS P rows 0 and 1, four floats each; with UE8M0 bytes each
  //     lane carries the dword holding its byte (fprop: the 4 K blocks' bytes of its row;
  //     dgrad: the K block's byte at bit offset p_shift);
  //   fprop / dgrad Q (row-major scales [rows][K/128]): lane l carries the four scales of
  //     tile row 64 wave + l (16 or 4 bytes) -> LDS [row][4];
  //   wgrad P and Q (block-major scales [M_cap/128][rows]): wave w carries K block kb0 + w,
  //     lane l the tile rows 4l..4l+3, one contiguous 1 KB (256-byte) run -> LDS [K block][256 rows].
  // Batches are rotated with the K order (k_rot is a multiple of the batch); blocks past
  // the last K block read neighbouring scales or zeros and are never multiplied.
  template <bool kLoop = false>
  __device__ __forceinline__ void dma_scale_p(int b) {
    const uint32_t lbase = scale_lds((int)(b & 1));
    if constexpr (kBlockP) {
      const uint32_t kb0 = (uint32_t)__builtin_amdgcn_readfirstlane(kphys(b * kScaleBatch));
      dma4<kLoop>(sp_rsrc, sp_off + kb0 * (uint32_t)sp_kb * kSB, lbase);
    } else {  // wgrad: wave w takes the block of stage 4 b + w (the rotation may wrap inside a batch)
      const uint32_t kbw = (uint32_t)__builtin_amdgcn_readfirstlane(kphys(b * kScaleBatch + wave));
      if constexpr (kE8)
        dma4<kLoop>(sp_rsrc, sp_off + kbw * (uint32_t)sp_kb, lbase + (uint32_t)wave * 256u);
      else
        dma16<kLoop>(sp_rsrc, sp_off + kbw * (uint32_t)sp_kb * 4u, lbase + (uint32_t)wave * 1024u);
    }
  }
  template <bool kLoop = false>
  __device__ __forceinline__ void dma_scale_q(int b) {
    const uint32_t lbase = scale_lds((int)(b & 1)) + kTP * kScaleBatch * 4;
    if constexpr (MODE == kWgrad) {
      const uint32_t kbw = (uint32_t)__builtin_amdgcn_readfirstlane(kphys(b * kScaleBatch + wave));
      if constexpr (kE8)
        dma4<kLoop>(sq_rsrc, sq_off + kbw * (uint32_t)sq_kb, lbase + (uint32_t)wave * 256u);
      else
        dma16<kLoop>(sq_rsrc, sq_off + kbw * (uint32_t)sq_kb * 4u, lbase + (uint32_t)wave * 1024u);
    } else {
      const uint32_t kb0 = (uint32_t)__builtin_amdgcn_readfirstlane(kphys(b * kScaleBatch));
      if constexpr (kE8)
        dma4<kLoop>(sq_rsrc, sq_off + kb0, lbase + (uint32_t)wave * 256u);
      else
        dma16<kLoop>(sq_rsrc, sq_off + kb0 * 4u, lbase + (uint32_t)wave * 1024u);
    }
  }

  // Fragment read J of half h of stage buffer B into register set kSetA.
  //   fprop / wgrad: J 0..15, 16-byte reads: J < 8 -> fq[J/2] half J%2, else fp[(J-8)/2].
  //   dgrad: J 0..7 as above for fq; J 8..23 -> fp[(J-8)/4], transposing read (J-8)%4.
  template <int B, int H, bool kSetA, int J>
  __device__ __forceinline__ void read_op() {
    i32x8 (&fp)[4] = kSetA ? fpA : fpB;
    i32x8 (&fq)[4] = kSetA ? fqA : fqB;
    const int l31 = lane & 31, g = lane >> 5;
    const uint8_t* P = stage_buf<B>();
    const uint8_t* Q = stage_buf<B>() + kTileBytes;
    if constexpr (J < 8) {
      const int r = 128 * wq + 32 * (J / 2) + l31;
      const u32x4 x = *reinterpret_cast<const u32x4*>(Q + r * kBK + (((4 * H + 2 * g + (J % 2)) ^ kswz(r)) << 4));
      fq[J / 2] = with_half(fq[J / 2], x, J % 2);
    } else if constexpr (MODE != kDgrad) {
      const int a = (J - 8) / 2, half = (J - 8) % 2;
      const int r = 128 * wp + 32 * a + l31;
      const u32x4 x = *reinterpret_cast<const u32x4*>(P + r * kBK + (((4 * H + 2 * g + half) ^ kswz(r)) << 4));
      fp[a] = with_half(fp[a], x, half);
    } else {
      const int a = (J - 8) / 4, rr = (J - 8) % 4;
      const int gg = lane >> 4, hh = lane & 1, ii = (lane & 15) >> 1;
      const int kl = 128 * wp + 32 * a + 16 * (gg & 1) + 8 * hh;
      const int n = 64 * H + 32 * (gg >> 1) + 8 * rr + ii;
      const uint8_t* addr = P + n * kTP + (((kl >> 4) ^ wswz(ii)) << 4) + (kl & 15);
      const i32x2 t =
          __builtin_amdgcn_ds_read_tr8_b64_v2i32((i32x2 __attribute__((address_space(3)))*)((lds_u8*)addr));
      fp[a][2 * rr] = t[0];
      fp[a][2 * rr + 1] = t[1];
    }
  }
  static constexpr int kFragReads = (MODE == kDgrad) ? 24 : 16;
  template <int B, int H, bool kSetA, int J>
  __device__ __forceinline__ void read_all_from() {
    if constexpr (J < kFragReads) {
      read_op<B, H, kSetA, J>();
      read_all_from<B, H, kSetA, J + 1>();
    }
  }
  // Scales of batch b (LDS buffer b % 2): read the four K-block scales of each row of one
  // operand this lane multiplies into raw[R] (kQ, or wgrad P: rows 128 w + 32 R + l for
  // R = 0..3; fprop / dgrad P: the wave's one weight-block row, raw[0] only) ...
  // Rows R0..R1-1 only (read and packed a few at a time, to keep few raw rows live).
  template <bool kQ, int R0, int R1>
  __device__ __forceinline__ void read_scale_rows(int b, u32x4 (&raw)[4]) {
    const u32x4* S = reinterpret_cast<const u32x4*>(&g_sc[b & 1][0]);
    const int l31 = opaque_lane() & 31;  // recomputed here rather than held through the tile
    if constexpr (!kQ && kBlockP) {
      if constexpr (R0 == 0) raw[0] = S[wp];
    } else if constexpr (kE8) {
      const uint8_t* B8 = reinterpret_cast<const uint8_t*>(&g_sc[b & 1][kQ ? kTP * kScaleBatch : 0]);
      if constexpr (MODE == kWgrad) {  // [K block][256 row bytes]
        const int row = (kQ ? 128 * wq : 128 * wp) + l31;
#pragma unroll
        for (int R = R0; R < R1; ++R)
#pragma unroll
          for (int j = 0; j < kScaleBatch; ++j) raw[R][j] = B8[j * kTP + row + 32 * R];
      } else {  // Q rows: one dword of four K-block bytes each
#pragma unroll
        for (int R = R0; R < R1; ++R) raw[R][0] = reinterpret_cast<const uint32_t*>(B8)[128 * wq + 32 * R + l31];
      }
    } else if constexpr (MODE == kWgrad) {  // [K block][256 rows]
      const float* F = &g_sc[b & 1][kQ ? kTP * kScaleBatch : 0];
      const int row = (kQ ? 128 * wq : 128 * wp) + l31;
#pragma unroll
      for (int R = R0; R < R1; ++R)
#pragma unroll
        for (int j = 0; j < kScaleBatch; ++j) raw[R][j] = __float_as_uint(F[j * kTP + row + 32 * R]);
    } else {  // Q rows of four K-block floats
#pragma unroll
      for (int R = R0; R < R1; ++R) raw[R] = S[kTP + 128 * wq + 32 * R + l31];
    }
  }
  // ... and pack them: word j holds the E8M0 byte (the fp32 exponent field of a
  // positive power of two, or the stored UE8M0 byte) of row R in byte R (rows R0..R1-1
  // added to the word).
  template <bool kQ, int R0, int R1>
  __device__ __forceinline__ void pack_scales(const u32x4 (&raw)[4], uint32_t (&dst)[4]) const {
    if constexpr (kE8) {
      if constexpr (!kQ && kBlockP) {
        if constexpr (R0 == 0) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            dst[j] = (((MODE == kFprop) ? raw[0][0] >> (8 * j) : raw[0][j] >> p_shift) & 0xffu) * 0x01010101u;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          uint32_t v = (R0 == 0) ? 0u : dst[j];
#pragma unroll
          for (int R = R0; R < R1; ++R)
            v |= (((MODE == kWgrad) ? raw[R][j] : raw[R][0] >> (8 * j)) & 0xffu) << (8 * R);
          dst[j] = v;
        }
      }
    } else if constexpr (!kQ && kBlockP) {
      if constexpr (R0 == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) dst[j] = (raw[0][j] >> 23) * 0x01010101u;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint32_t v = (R0 == 0) ? 0u : dst[j];
#pragma unroll
        for (int R = R0; R < R1; ++R) v |= ((raw[R][j] >> 23) & 0xffu) << (8 * R);
        dst[j] = v;
      }
    }
  }

  template <bool kSetA, int S4, int I>
  __device__ __forceinline__ void mfma_op() {
    i32x8 (&fp)[4] = kSetA ? fpA : fpB;
    i32x8 (&fq)[4] = kSetA ? fqA : fqB;
    constexpr int A = I / 4, Bq = I % 4;
    acc[A][Bq] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fp[A], fq[Bq], acc[A][Bq], 0, 0, A, (int)cp[S4], Bq,
                                                                   (int)cq[S4]);
  }
  // Tile DMA instructions D0..D1-1 of stage ks_dma into buffer B.
  template <int B, int D0, int D1>
  __device__ __forceinline__ void dma_range(int ks_dma) {
    if constexpr (D0 < D1) {
      dma_tile<B, D0, false, true>(ks_dma);
      dma_range<B, D0 + 1, D1>(ks_dma);
    }
  }
  // DMA slot J (0..kDmaSlots-1) of a stage: its share of the tile DMAs of stage ks_dma, and, in
  // the second half-step of the first stage of a scale batch, the next batch's scale DMAs
  // (slot indices of half 1 are 16 - kEarly + I).
  template <int B, int S4, int J>
  __device__ __forceinline__ void dma_slot(int ks_dma, int ks_next) {
    dma_range<B, dma_before(J), dma_before(J + 1)>(ks_dma);
    if constexpr (S4 == 0 && J == 16 - kEarly + 1) dma_scale_p<true>((ks_next >> 2) + 1);
    if constexpr (S4 == 0 && J == 16 - kEarly + 3) dma_scale_q<true>((ks_next >> 2) + 1);
  }
  // Fragment reads of MFMA slot I: the half-step's kFragReads reads spread evenly over
  // its first kReadSlots slots.
  template <int B, int H, bool kSetA, int J, int JEnd>
  __device__ __forceinline__ void reads_range() {
    if constexpr (J < JEnd) {
      read_op<B, H, kSetA, J>();
      reads_range<B, H, kSetA, J + 1, JEnd>();
    }
  }
  template <int B, int H, bool kSetA, int I>
  __device__ __forceinline__ void reads_of_slot() {
    if constexpr (I < kReadSlots)
      reads_range<B, H, kSetA, I * kFragReads / kReadSlots, (I + 1) * kFragReads / kReadSlots>();
  }

  // First half-step of stage ks (buffer B): MFMAs on set A; the reads of the second half (same
  // buffer) into set B go out over the first kReadSlots MFMAs; at slot kEarly every wave has
  // them (lgkmcnt) and a barrier frees buffer B, into which the DMA of stage ks+2 starts.
  template <int B, int S4, int I>
  __device__ __forceinline__ void half0_from(int ks_dma, int ks_next) {
    if constexpr (I < 16) {
      mfma_op<true, S4, I>();
      reads_of_slot<B, 1, false, I>();
      if constexpr (I == kEarly) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
      }
      if constexpr (I >= kEarly) dma_slot<B, S4, I - kEarly>(ks_dma, ks_next);
      __builtin_amdgcn_sched_barrier(0);
      half0_from<B, S4, I + 1>(ks_dma, ks_next);
    }
  }
  // Second half-step: MFMAs on set B.  The rest of stage ks+2's DMA (with the next scale
  // batch among it when ks % 4 == 0, landing by the middle of the next stage); the reads of
  // stage ks+1's first half (other buffer) into set A over the first kReadSlots MFMAs; in
  // the last stage of a batch the next batch's scales are read and packed (wgrad: those of P
  // in the second stage, kSpreadScales).
  template <int B, int S4, int I>
  __device__ __forceinline__ void half1_from(int ks_dma, int ks_next) {
    if constexpr (I < 16) {
      mfma_op<false, S4, I>();
      dma_slot<B, S4, 16 - kEarly + I>(ks_dma, ks_next);
      reads_of_slot<1 - B, 0, true, I>();
      if constexpr (kSpreadScales) {
        if constexpr (S4 == 1 && I == 8) read_scale_rows<false, 0, 2>((ks_next >> 2) + 1, rsp);
        if constexpr (S4 == 1 && I == 10) pack_scales<false, 0, 2>(rsp, np);
        if constexpr (S4 == 1 && I == 12) read_scale_rows<false, 2, 4>((ks_next >> 2) + 1, rsp);
        if constexpr (S4 == 1 && I == 14) pack_scales<false, 2, 4>(rsp, np);
        if constexpr (S4 == 3 && I == 8) read_scale_rows<true, 0, 2>(ks_next >> 2, rsq);
        if constexpr (S4 == 3 && I == 10) pack_scales<true, 0, 2>(rsq, nq);
        if constexpr (S4 == 3 && I == 12) read_scale_rows<true, 2, 4>(ks_next >> 2, rsq);
        if constexpr (S4 == 3 && I == 14) pack_scales<true, 2, 4>(rsq, nq);
      } else {
        if constexpr (S4 == 3 && I == 8) read_scale_rows<false, 0, 2>(ks_next >> 2, rsp);
        if constexpr (S4 == 3 && I == 9) read_scale_rows<true, 0, 2>(ks_next >> 2, rsq);
        if constexpr (S4 == 3 && I == 10) pack_scales<false, 0, 2>(rsp, np);
        if constexpr (S4 == 3 && I == 11) read_scale_rows<false, 2, 4>(ks_next >> 2, rsp);
        if constexpr (S4 == 3 && I == 11) pack_scales<true, 0, 2>(rsq, nq);
        if constexpr (S4 == 3 && I == 12) read_scale_rows<true, 2, 4>(ks_next >> 2, rsq);
        if constexpr (S4 == 3 && I == 13) pack_scales<false, 2, 4>(rsp, np);
        if constexpr (S4 == 3 && I == 14) pack_scales<true, 2, 4>(rsq, nq);
      }
      __builtin_amdgcn_sched_barrier(0);
      half1_from<B, S4, I + 1>(ks_dma, ks_next);
    }
  }

  // Stage ks, S4 = ks % 4 (buffer S4 % 2).  Between the halves, wait for this wave's DMA of
  // stage ks+1 (and older: the scale batch) -- loads complete in order, so all but the
  // FF8_HALF0_DMAS just issued for stage ks+2 -- then barrier: stage ks+1 is visible to all.
  // Stages past the end are reloads of the last one (in bounds, never multiplied).
  template <int S4>
  __device__ __forceinline__ void stage(int ks) {
    constexpr int B = S4 % 2;
    const int ks_dma = ks + 2 < nk ? ks + 2 : nk - 1;
    half0_from<B, S4, 0>(ks_dma, ks + 1);
    asm volatile("s_waitcnt vmcnt(" FF8_STR(FF8_HALF0_DMAS) ") lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    half1_from<B, S4, 0>(ks_dma, ks + 1);
    if constexpr (S4 == 3) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        cp[j] = np[j];
        cq[j] = nq[j];
      }
    }
  }
};

// One tile of the grouped product: expert e, q rows [q0, q_end) of a 256-row tile, p
// columns from p0, contraction from k0 over nk stages.
struct TileInfo {
  int e, blk;
  int q0, q_end, k0, p0, nk;  // rows, columns and stages all stay below 2^31
  int k_lo, k_hi;             // wgrad: valid K bytes of the first / last stage
};

// wgrad: the K range of expert e's tiles.  K runs over whole 128-token blocks from the one
// holding offsets[e]; with groups padded to 16 the first and last may be shared with
// neighbouring experts (masked in their DMAs).
__device__ __forceinline__ void wgrad_k_range(const GemmArgs& g, int e, TileInfo& t) {
  const int o0 = __builtin_amdgcn_readfirstlane(g.offsets[e]);
  const int o1 = __builtin_amdgcn_readfirstlane(g.offsets[e + 1]);
  const int kb0 = o0 & ~(kBK - 1);
  t.k0 = kb0;
  t.nk = o1 > o0 ? (o1 - kb0 + kBK - 1) / kBK : 0;
  t.k_lo = o0 - kb0;
  t.k_hi = o1 > o0 ? o1 - (kb0 + (t.nk - 1) * kBK) : kBK;
}

// Tile w_in of XCD block blk (kBQ x kBP tiles, p fastest).  False for tiles past the
// edges.  fprop/dgrad: q tiles are 256-row tiles of the expert groups (g_cum / g_off:
// cumulative tile counts and row offsets per expert, in LDS).
template <int MODE>
__device__ __forceinline__ bool decode_tile(const GemmArgs& g, int blk, int w_in, TileInfo& t) {
  const int n_pb = (g.n_pt + kBP - 1) / kBP;
  const int qb = blk / n_pb, pb = blk - qb * n_pb;
  const int qg = qb * kBQ + w_in / kBP;  // global q-tile index
  const int pt = pb * kBP + w_in % kBP;
  if (pt >= g.n_pt) return false;
  t.blk = blk;
  t.p0 = (int64_t)pt * kTP;
  if (MODE != kWgrad) {
    if (qg >= g_cum[g.E]) return false;
    int lo = 0, hi = g.E - 1;  // largest e with cum[e] <= qg
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (g_cum[mid] <= qg) lo = mid; else hi = mid - 1;
    }
    const int e = __builtin_amdgcn_readfirstlane(lo);
    t.e = e;
    t.q0 = __builtin_amdgcn_readfirstlane(g_off[e] + (qg - g_cum[e]) * kTQ);  // uniform (LDS values)
    t.q_end = __builtin_amdgcn_readfirstlane(g_off[e + 1]);
    t.k0 = 0;
    t.nk = g.Kdim / kBK;
    t.k_lo = 0;
    t.k_hi = kBK;
  } else {
    if (qg >= g.E * g.n_qt) return false;
    const int e = qg / g.n_qt;
    t.e = e;
    t.q0 = (int64_t)(qg - e * g.n_qt) * kTQ;
    t.q_end = g.Nq;
    wgrad_k_range(g, e, t);
  }
  return true;
}

// DMA sources of tile t: wave-uniform bases and resources, per-lane offsets (lane l of
// tile DMA instruction i writes LDS bytes 16 l .. of that instruction's 1 KB).  Offsets are
// 32-bit (the host keeps every operand under 4 GiB); past an operand's end they may wrap,
// which only feeds rows or columns that are never stored.
template <int MODE, typename SC>
__device__ __forceinline__ void setup_tile(Tile<MODE, SC>& T, const GemmArgs& g, const TileInfo& t) {
  constexpr uint32_t kSB = sizeof(SC);
  const uint32_t lane = (uint32_t)opaque_lane(), wave = (uint32_t)T.wave, e = (uint32_t)t.e;
  const uint32_t q0 = (uint32_t)t.q0, k0 = (uint32_t)t.k0, p0 = (uint32_t)t.p0;
  const uint32_t Np = (uint32_t)g.Np, Kdim = (uint32_t)g.Kdim, M_cap = (uint32_t)g.M_cap;
  T.nk = t.nk;
  T.k_lo = t.k_lo;
  T.k_hi = t.k_hi;
  const uint32_t q_ld = (MODE == kWgrad) ? M_cap : Kdim;
  const uint32_t q_rows = (MODE == kWgrad) ? (uint32_t)g.Nq : M_cap;
  // K-major row of pattern h (h = 0, 1) for this lane: group w + 4h, row 8 group + l / 8,
  // 16-byte chunk (l % 8) ^ kswz(row) (kswz depends on the group's parity and l / 16 only).
  // wgrad operands are K-blocked ([M_cap/128][rows][128]): row r's 128 bytes of K block b sit
  // at (b * rows + r) * 128, so one stage of a panel is 32 KB of consecutive bytes.
  T.q_rsrc = make_rsrc(g.Q, q_rows * q_ld);
  T.q_kstep = (MODE == kWgrad) ? (int)(q_rows * kBK) : kBK;
  T.q_istep = (MODE == kWgrad) ? 64 * kBK : (int)(64 * q_ld);
#pragma unroll
  for (uint32_t hh = 0; hh < 2; ++hh) {
    const uint32_t r = 8 * (wave + 4 * hh) + (lane >> 3);
    const uint32_t c = (lane & 7) ^ (uint32_t)kswz((int)r);
    T.q_voff[hh] = (MODE == kWgrad) ? ((k0 / kBK) * q_rows + q0 + r) * kBK + c * 16 : (q0 + r) * q_ld + k0 + c * 16;
  }
  if (MODE == kDgrad) {  // W_e [N = Kdim][K = Np], rows n = 32w + 4i + l / 16
    T.p_rsrc = make_rsrc(g.P, (uint32_t)g.E * Kdim * Np);
    T.p_kstep = kBK * Np;
    T.p_istep = 8 * Np;
#pragma unroll
    for (uint32_t hh = 0; hh < 2; ++hh) {
      const uint32_t n = 32 * wave + 4 * hh + (lane >> 4);
      const uint32_t c = (lane & 15) ^ (uint32_t)wswz((int)(n & 7));
      T.p_voff[hh] = (e * Kdim + n) * Np + p0 + c * 16;
    }
  } else {
    const uint32_t p_ld = (MODE == kWgrad) ? M_cap : Kdim;
    const uint32_t p_rows = (MODE == kWgrad) ? Np : (uint32_t)g.E * Np;  // fprop: all experts' rows
    const uint32_t p_row0 = (MODE == kFprop) ? e * Np + p0 : p0;
    T.p_rsrc = make_rsrc(g.P, p_rows * p_ld);
    T.p_kstep = (MODE == kWgrad) ? (int)(p_rows * kBK) : kBK;
    T.p_istep = (MODE == kWgrad) ? 64 * kBK : (int)(64 * p_ld);
#pragma unroll
    for (uint32_t hh = 0; hh < 2; ++hh) {
      const uint32_t r = 8 * (wave + 4 * hh) + (lane >> 3);
      const uint32_t c = (lane & 7) ^ (uint32_t)kswz((int)r);
      T.p_voff[hh] = (MODE == kWgrad) ? ((k0 / kBK) * p_rows + p_row0 + r) * kBK + c * 16
                                      : (p_row0 + r) * p_ld + k0 + c * 16;
    }
  }
  // scale DMA sources (resources range-checked to the end of each scale tensor; offsets
  // are at K block 0 of the tile, the batch adds its K-block offset)
  const SC* sp_base;
  uint32_t sp_total, sq_total;
  if (MODE == kWgrad) {  // block-major: xT_s [M_cap/128][Np], gT_s [M_cap/128][Nq]
    const uint32_t Nq = (uint32_t)g.Nq, kb_first = k0 / kTile;
    sp_base = static_cast<const SC*>(g.sP);
    T.sp_kb = (int)Np;
    T.sq_kb = (int)Nq;
    sp_total = (M_cap / kTile) * Np;
    sq_total = (M_cap / kTile) * Nq;
    T.sp_off = (kb_first * Np + p0 + 4 * lane) * kSB;
    T.sq_off = (kb_first * Nq + q0 + 4 * lane) * kSB;
  } else {
    // Q: row-major a_s / g_s [M_cap][Kdim/128], lane l of wave w carries tile row 64 w + l
    const uint32_t q_sld = Kdim / kTile;
    const uint32_t q = min(q0 + 64 * wave + lane, q_rows - 1);
    T.sq_kb = 1;
    sq_total = q_rows * q_sld;
    T.sq_off = q * q_sld * kSB;
    // P: the tile's two weight block rows, four K blocks per lane group of four
    const uint32_t pb = min(p0 / kTile + ((lane >> 2) & 1), Np / kTile - 1);
    const uint32_t j = lane & 3;
    if (MODE == kFprop) {  // w_s [E][Np/128][Kdim/128]
      sp_base = static_cast<const SC*>(g.sP) + (size_t)e * (Np / kTile) * (Kdim / kTile);
      T.sp_kb = 1;
      sp_total = ((uint32_t)g.E - e) * (Np / kTile) * (Kdim / kTile);
      // UE8M0: every lane of a row loads the dword of its four K-block bytes (K/128 and the
      // batch start are multiples of 4)
      T.sp_off = (kSB == 1) ? pb * (Kdim / kTile) : (pb * (Kdim / kTile) + j) * 4;
    } else {  // w_s [E][Kdim/128][Np/128]
      sp_base = static_cast<const SC*>(g.sP) + (size_t)e * (Kdim / kTile) * (Np / kTile);
      T.sp_kb = (int)(Np / kTile);
      sp_total = ((uint32_t)g.E - e) * (Kdim / kTile) * (Np / kTile);
      // UE8M0: the dword holding the byte (Np/128 is a multiple of 4, so the byte's offset in
      // it is pb % 4 for every K block); the wave's own block row gives the shift
      T.sp_off = (kSB == 1) ? j * (Np / kTile) + (pb & ~3u) : (j * (Np / kTile) + pb) * 4;
      T.p_shift = (uint32_t)__builtin_amdgcn_readfirstlane((int)(8 * (min(p0 / kTile + (uint32_t)T.wp, Np / kTile - 1) & 3u)));
    }
  }
  const SC* sq_base = static_cast<const SC*>(g.sQ);
  T.sp_rsrc = make_rsrc(sp_base, sp_total * kSB);
  T.sq_rsrc = make_rsrc(sq_base, sq_total * kSB);
  // Blocks start their K loops at different scale-batch-aligned stages, so that the XCDs
  // running together stream different K bands of the operand rows (spread over memory
  // channels) while the 32 tiles of one block still share every stage through their L2.
  T.k_rot = (kStaggerK<MODE> && (T.nk & (kScaleBatch - 1)) == 0 && T.nk >= 2 * kScaleBatch)
                ? ((t.blk * 5) % (T.nk / kScaleBatch)) * kScaleBatch
                : 0;
  // wgrad, an expert's K range cut by 16-row padding: the last block, then the first, as
  // stages 0 and 1, so that the only masked DMAs are the two issued before the loop
  if (MODE == kWgrad && (T.k_lo > 0 || T.k_hi < kBK) && T.nk > 1) T.k_rot = T.nk - 1;
}

// Output of one tile through stage buffer 1 only (16 KB per wave), so that the next
// tile's first stage can stream into buffer 0 meanwhile.  Every global store instruction
// writes whole 128-byte lines (16 lanes per 256-byte bf16 row, 32 lanes per 512-byte fp32
// row) instead of 16-byte pieces of 32 rows: each wave stages 64 (bf16) or 32 (fp32) rows
// of its 128 x 128 sub-tile at a time ([q][p], p contiguous), 16-byte chunks of row q
// XOR-swizzled by q, conflict-free for the fragment-order writes and the row-order reads.
// The stores are non-temporal: the output is not re-read here, and streaming it keeps the
// operand panels that the XCD's other workgroups are still reading in L2.  A wave only
// rewrites its own region, after its own reads (LDS order), so passes need no barrier.
template <int MODE, typename SC>
__device__ __forceinline__ void epilogue(Tile<MODE, SC>& T, const GemmArgs& g, const TileInfo& t) {
  const int lane = opaque_lane(), wave = T.wave, wp = T.wp, wq = T.wq;
  lds_u8* const region = (lds_u8*)g_st1 + wave * 16384;
  const int l31 = lane & 31, h = lane >> 5;
  const bool p_ok = t.p0 + 128 * wp < g.Np;  // Np is a multiple of 128: whole-wave predicate
  if (MODE == kWgrad) {
    // uniform base of this wave's 128 x 128 sub-tile, 32-bit lane offsets from it
    uint8_t* const dw = reinterpret_cast<uint8_t*>(
        static_cast<float*>(g.out) + ((size_t)t.e * g.Nq + t.q0 + 128 * wq) * g.Np + t.p0 + 128 * wp);
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      // rows ql = l31 of 512 bytes (q = 32 b + ql); chunk c = p / 4 = 8a + 2gr + h
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
          const int c = 8 * a + 2 * gr + h;
          u32x4 o;
#pragma unroll
          for (int j = 0; j < 4; ++j) o[j] = __float_as_uint(T.acc[a][b][4 * gr + j]);
          *(__attribute__((address_space(3))) u32x4*)(region + l31 * 512 + ((c ^ l31) << 4)) = o;
          __builtin_amdgcn_sched_barrier(0);  // few accumulators in VGPRs at a time
        }
      // all of the pass's row reads first, then the stores (one LDS wait, not one per store)
      u32x4 v[16];
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int ql = 2 * it + h;
        v[it] = *(__attribute__((address_space(3))) u32x4*)(region + ql * 512 + ((l31 ^ ql) << 4));
      }
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int qr = 32 * b + 2 * it + h;  // row within the wave's sub-tile
        if (!p_ok || t.q0 + 128 * wq + qr >= t.q_end) continue;
        uint8_t* dst = dw + (uint32_t)(qr * g.Np + 4 * l31) * 4u;
        if (g.accumulate) {
          const u32x4 old = ld16(dst);
          u32x4 o;
#pragma unroll
          for (int j = 0; j < 4; ++j) o[j] = __float_as_uint(__uint_as_float(old[j]) + __uint_as_float(v[it][j]));
          stnt16(dst, o);
        } else {
          stnt16(dst, v[it]);
        }
      }
    }
  } else {
    // uniform base of this wave's 128 x 128 sub-tile, 32-bit lane offsets from it
    uint8_t* const out = reinterpret_cast<uint8_t*>(static_cast<uint16_t*>(g.out) + (size_t)(t.q0 + 128 * wq) * g.Np +
                                                    t.p0 + 128 * wp);
#pragma unroll
    for (int ph = 0; ph < 2; ++ph) {
      // rows ql = 32bb + l31 of 256 bytes (q = 64 ph + ql); 8-byte piece (p = 32a + 8gr + 4h)
      // in chunk 4a + gr, half h
#pragma unroll
      for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
          for (int gr = 0; gr < 4; ++gr) {
            const int ql = 32 * bb + l31, m = 4 * a + gr;
            u32x2 o;
            o[0] = pack_bf16x2(T.acc[a][2 * ph + bb][4 * gr + 0], T.acc[a][2 * ph + bb][4 * gr + 1]);
            o[1] = pack_bf16x2(T.acc[a][2 * ph + bb][4 * gr + 2], T.acc[a][2 * ph + bb][4 * gr + 3]);
            *(__attribute__((address_space(3))) u32x2*)(region + ql * 256 + ((m ^ (ql & 15)) << 4) + 8 * h) = o;
            __builtin_amdgcn_sched_barrier(0);  // few accumulators in VGPRs at a time
          }
      // all of the pass's row reads first, then the stores (one LDS wait, not one per store)
      const int c = lane & 15;
      u32x4 v[16];
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int ql = 4 * it + (lane >> 4);
        v[it] = *(__attribute__((address_space(3))) u32x4*)(region + ql * 256 + ((c ^ (ql & 15)) << 4));
      }
#pragma unroll
      for (int it = 0; it < 16; ++it) {
        const int qr = 64 * ph + 4 * it + (lane >> 4);  // row within the wave's sub-tile
        if (!p_ok || t.q0 + 128 * wq + qr >= t.q_end) continue;
        stnt16(out + (uint32_t)(qr * g.Np + 8 * c) * 2u, v[it]);
      }
    }
  }
}

// First-stage DMA of a tile: stage 0 into buffer 0, then the scale batch 0 (buffer 0).
template <int MODE, typename SC>
__device__ __forceinline__ void dma_first_stage(Tile<MODE, SC>& T) {
  T.template dma_tile<0, 0, MODE == kWgrad>(0); T.template dma_tile<0, 1, MODE == kWgrad>(0); T.template dma_tile<0, 2, MODE == kWgrad>(0);
  T.template dma_tile<0, 3, MODE == kWgrad>(0); T.template dma_tile<0, 4, MODE == kWgrad>(0); T.template dma_tile<0, 5, MODE == kWgrad>(0);
  T.template dma_tile<0, 6, MODE == kWgrad>(0); T.template dma_tile<0, 7, MODE == kWgrad>(0); T.template dma_tile<0, 8, MODE == kWgrad>(0);
  T.template dma_tile<0, 9, MODE == kWgrad>(0); T.template dma_tile<0, 10, MODE == kWgrad>(0); T.template dma_tile<0, 11, MODE == kWgrad>(0);
  T.template dma_tile<0, 12, MODE == kWgrad>(0); T.template dma_tile<0, 13, MODE == kWgrad>(0); T.template dma_tile<0, 14, MODE == kWgrad>(0);
  T.template dma_tile<0, 15, MODE == kWgrad>(0);
  T.template dma_scale_p<false>(0);
  T.template dma_scale_q<false>(0);
}
// Second-stage DMA (stage 1, or a reload of stage 0 when nk == 1) into buffer 1: exactly
// kStage1Dma instructions per wave, the newest in flight when stage 0 is awaited.
constexpr int kStage1Dma = 16;
template <int MODE, typename SC>
__device__ __forceinline__ void dma_second_stage(Tile<MODE, SC>& T) {
  const int s1 = T.nk > 1 ? 1 : 0;
  T.template dma_tile<1, 0, MODE == kWgrad>(s1); T.template dma_tile<1, 1, MODE == kWgrad>(s1); T.template dma_tile<1, 2, MODE == kWgrad>(s1);
  T.template dma_tile<1, 3, MODE == kWgrad>(s1); T.template dma_tile<1, 4, MODE == kWgrad>(s1); T.template dma_tile<1, 5, MODE == kWgrad>(s1);
  T.template dma_tile<1, 6, MODE == kWgrad>(s1); T.template dma_tile<1, 7, MODE == kWgrad>(s1); T.template dma_tile<1, 8, MODE == kWgrad>(s1);
  T.template dma_tile<1, 9, MODE == kWgrad>(s1); T.template dma_tile<1, 10, MODE == kWgrad>(s1); T.template dma_tile<1, 11, MODE == kWgrad>(s1);
  T.template dma_tile<1, 12, MODE == kWgrad>(s1); T.template dma_tile<1, 13, MODE == kWgrad>(s1); T.template dma_tile<1, 14, MODE == kWgrad>(s1);
  T.template dma_tile<1, 15, MODE == kWgrad>(s1);
}

// Semi-persistent: the grid is a sequence of groups of S workgroups per XCD (S = 32 on
// 256 CUs, one workgroup per CU), and each workgroup runs kRoundsPerWg tiles.  Workgroups
// are dispatched round-robin over the 8 XCDs, and in order within an XCD.  XCD x owns XCD
// blocks x, x + 8, x + 16, ... (kBQ x kBP tiles each, p fastest); its work list is their
// tiles in that order, item i = k S + s going to slot s of the group that owns round k.
// With S = 32, slot s takes tile s of every block, so the 32 workgroups of an XCD work on
// one block at a time and share its 8 q panels and 4 p panels per K step in their L2, while
// the 8 XCDs together sweep one 16 x 16-tile window (about one expert).  Bounding a
// workgroup to a few rounds keeps an XCD's workgroups from drifting apart (which costs L2
// sharing) and lets faster CUs take more groups.
// wgrad under skewed routing: every expert has the same tile count, so an expert's blocks
// rarely divide evenly over the 8 XCDs, and the largest experts' extra blocks pile up on a
// few of them.  When the largest expert has more than twice the mean rows (decided in every
// workgroup from the offsets, identically), each XCD instead takes one of 8 equal rectangles
// of every expert's tile grid (at least one round of 32 tiles each), which balances the XCDs
// exactly; with near-uniform routing the blocks, which share more operand panels per round,
// are kept.
// Between tiles, the next tile's first stage (and scale batch) streams into stage buffer 0
// while the finished tile's output is staged through buffer 1 and stored; its second
// stage follows once the epilogue has left buffer 1.  All control flow is
// workgroup-uniform (tile decode from uniform values), so every barrier is reached by all
// four waves, and every wave leaves the tile loop with the same tile count.
constexpr int kPersistSlots = kBQ * kBP;  // workgroups per XCD and group
constexpr int kRoundsPerWg = 4;           // work rounds (tiles) per workgroup

// Workgroup barrier that waits for this wave's LDS accesses only: global stores may stay in
// flight across it (a __syncthreads fence would drain them).  One asm statement, so that
// no memory access moves across the barrier.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// wgrad, expert-share schedule: item i of XCD x is tile l = i % share of expert e = i / share
// in XCD x's rectangle (p fastest).  Every expert's tiles are split evenly over the 8 XCDs,
// so the XCDs' loads stay equal however skewed the routing is (with XCD blocks, an expert's
// block count is rarely a multiple of 8, and the largest experts' extra blocks pile up on a
// few XCDs).
__device__ __forceinline__ void decode_share_tile(const GemmArgs& g, int xcd, int i, TileInfo& t) {
  const int e = i / g.share, l = i - e * g.share;
  const int lq = l / g.rect_p, lp = l - lq * g.rect_p;
  const int rq = xcd / g.rect_b, rp = xcd - rq * g.rect_b;
  t.blk = 0;
  t.e = e;
  t.p0 = (rp * g.rect_p + lp) * kTP;
  t.q0 = (rq * g.rect_q + lq) * kTQ;
  t.q_end = g.Nq;
  wgrad_k_range(g, e, t);
}

// Next tile of this workgroup from round k on, below round k_end (k advances past empty
// edge tiles).
template <int MODE>
__device__ __forceinline__ bool next_tile(const GemmArgs& g, int xcd, int slot, int n_slots, int n_blocks, int k_end,
                                          bool use_share, int& k, TileInfo& t) {
  for (; k < k_end; ++k) {
    const int i = k * n_slots + slot;
    if (MODE == kWgrad && use_share) {
      if (i >= g.E * g.share) return false;
      decode_share_tile(g, xcd, i, t);
      return true;
    }
    const int blk = (i / kPersistSlots) * 8 + xcd;
    if (blk >= n_blocks) return false;
    if (decode_tile<MODE>(g, blk, i % kPersistSlots, t)) return true;
  }
  return false;
}

template <int MODE, typename SC>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_kernel(GemmArgs g) {
  const int tid = threadIdx.x;
  Tile<MODE, SC> T;
  T.lane = tid & 63;
  T.wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  T.wp = T.wave & 1;
  T.wq = T.wave >> 1;
  const int n_slots = g.n_slots, group_size = 8 * n_slots;
  const int group = blockIdx.x / group_size, in_group = blockIdx.x - group * group_size;
  const int xcd = in_group & 7, slot = in_group >> 3;
  const int k_end = (group + 1) * kRoundsPerWg;

  int n_qg;  // q tiles
  if (MODE != kWgrad) {
    // cumulative 256-row tile counts and row offsets per expert: one wave, 64 per pass
    if (tid < 64) {
      int carry = 0;
      for (int base = 0; base < g.E; base += 64) {
        const int i = base + tid;
        const int o0 = i < g.E ? g.offsets[i] : 0, o1 = i < g.E ? g.offsets[i + 1] : 0;
        int v = i < g.E ? (o1 - o0 + kTQ - 1) / kTQ : 0;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const int u = __shfl_up(v, d);
          if (tid >= d) v += u;
        }
        if (i < g.E) {
          g_cum[i + 1] = carry + v;
          g_off[i + 1] = o1;
        }
        carry += __shfl(v, 63);
      }
      if (tid == 0) {
        g_cum[0] = 0;
        g_off[0] = g.offsets[0];
      }
    }
    __syncthreads();
    n_qg = __builtin_amdgcn_readfirstlane(g_cum[g.E]);
  } else {
    n_qg = g.E * g.n_qt;
  }
  // wgrad: expert shares when the largest expert has more than twice the mean rows (one
  // wave reduces the offsets; the flag is the same in every workgroup of the launch)
  bool use_share = false;
  if (MODE == kWgrad && g.share > 0) {
    if (tid < 64) {
      int mx = 0;
      for (int base = 0; base < g.E; base += 64) {
        const int i = base + tid;
        const int r = i < g.E ? g.offsets[i + 1] - g.offsets[i] : 0;
        mx = max(mx, r);
      }
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) mx = max(mx, __shfl_xor(mx, d));
      if (tid == 0) g_cum[0] = (int64_t)mx * g.E > 2 * (int64_t)(g.offsets[g.E] - g.offsets[0]);
    }
    __syncthreads();
    use_share = __builtin_amdgcn_readfirstlane(g_cum[0]) != 0;
  }
  const int n_blocks = ((g.n_pt + kBP - 1) / kBP) * ((n_qg + kBQ - 1) / kBQ);
  int k = group * kRoundsPerWg;
  TileInfo t;
  if (!next_tile<MODE>(g, xcd, slot, n_slots, n_blocks, k_end, use_share, k, t)) return;
  setup_tile<MODE, SC>(T, g, t);
  if (T.nk > 0) dma_first_stage<MODE, SC>(T);
  // Loop invariant: tile t is set up, its stage 0 and scale batch 0 are in flight (if it
  // has any K), and stage buffer 1 is free.
  for (;;) {
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int v = 0; v < 16; ++v) T.acc[a][b][v] = 0.0f;
    const int nk = T.nk;
    if (nk > 0) {
      dma_second_stage<MODE, SC>(T);
      // stage 0 and scale batch 0 have landed when at most the stage-1 DMAs are in flight
      // (loads retire in order; older epilogue stores still in flight only make this wait longer)
      asm volatile("s_waitcnt vmcnt(16)\n\ts_barrier" ::: "memory");
      static_assert(kStage1Dma == 16, "the wait count above is the stage-1 DMA count");
      T.template read_all_from<0, 0, true, 0>();
      {
        u32x4 raw[4];
        T.template read_scale_rows<false, 0, 4>(0, raw);
        T.template pack_scales<false, 0, 4>(raw, T.cp);
        T.template read_scale_rows<true, 0, 4>(0, raw);
        T.template pack_scales<true, 0, 4>(raw, T.cq);
      }
      for (int ks = 0; ks < nk; ks += 4) {
        T.template stage<0>(ks);
        if (ks + 1 < nk) T.template stage<1>(ks + 1);
        if (ks + 2 < nk) T.template stage<2>(ks + 2);
        if (ks + 3 < nk) T.template stage<3>(ks + 3);
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the tail's reload DMAs have landed
    }
    lds_barrier();  // every wave is done with the stage buffers and the scale batches
    TileInfo tn;
    ++k;
    const bool more = next_tile<MODE>(g, xcd, slot, n_slots, n_blocks, k_end, use_share, k, tn);
    if (more) {
      setup_tile<MODE, SC>(T, g, tn);
      if (T.nk > 0) dma_first_stage<MODE, SC>(T);  // buffer 0 and scale batch 0, under the epilogue
    }
    if (!(MODE == kWgrad && t.nk == 0 && g.accumulate)) epilogue<MODE, SC>(T, g, t);
    if (!more) break;
    t = tn;
    lds_barrier();  // buffer 1 is free for the next tile's second stage
  }
}

// Grid: groups of n_slots workgroups per XCD (one per CU, the same number on each of the
// 8 XCDs, at most kPersistSlots), enough groups of kRoundsPerWg rounds for `items` tiles per
// XCD, or for n_blocks_max XCD blocks (workgroups past the work actually present exit at once).
unsigned grid_items(int64_t items, int& n_slots) {  // items: work items (tiles) per XCD
  int cus = (device_cu_count() / 8) * 8;
  if (cus > 8 * kPersistSlots) cus = 8 * kPersistSlots;
  if (cus < 8) cus = 8;
  n_slots = cus / 8;
  const int64_t rounds = (items + n_slots - 1) / n_slots;
  const int64_t groups = (rounds + kRoundsPerWg - 1) / kRoundsPerWg;
  return (unsigned)((groups > 0 ? groups : 1) * 8 * n_slots);
}
unsigned grid_blocks(int64_t n_blocks_max, int& n_slots) {
  return grid_items((n_blocks_max + 7) / 8 * kPersistSlots, n_slots);
}
int64_t blocks_of(int n_pt, int64_t n_qg) { return (int64_t)((n_pt + kBP - 1) / kBP) * ((n_qg + kBQ - 1) / kBQ); }

}  // namespace

template <typename SC>
static hipError_t grouped_gemm_impl(GemmMode mode, const uint8_t* a, const SC* a_s, const uint8_t* b, const SC* b_s,
                                    const int32_t* offsets, int E, int64_t M_cap, int64_t N, int64_t K, void* out,
                                    int accumulate, hipStream_t st) {
  GemmArgs g{};
  g.offsets = offsets;
  g.out = out;
  g.E = E;
  g.M_cap = M_cap;
  g.accumulate = accumulate;
  g.P = b; g.sP = b_s; g.Q = a; g.sQ = a_s;
  unsigned grid;
  // fprop / dgrad q tiles: expert e has ceil(rows_e / 256) <= rows_e / 256 + 1 of them, so
  // at most M_cap / 256 + E in all, whatever the groups' padding (with 16-row padding and
  // many small experts nearly every expert adds a partial tile)
  const int64_t qt_bound = (M_cap + kTQ - 1) / kTQ + E;
  if (mode == kFprop) {  // out[m, n] = a[m, :] . w[e, n, :]
    g.Np = N; g.Kdim = K;
    g.n_pt = (int)((N + kTP - 1) / kTP);
    grid = grid_blocks(blocks_of(g.n_pt, qt_bound), g.n_slots);
    grouped_gemm_kernel<kFprop, SC><<<grid, kThreads, 0, st>>>(g);
  } else if (mode == kDgrad) {  // out[m, k] = g[m, :] . w[e, :, k]
    g.Np = K; g.Kdim = N;
    g.n_pt = (int)((K + kTP - 1) / kTP);
    grid = grid_blocks(blocks_of(g.n_pt, qt_bound), g.n_slots);
    grouped_gemm_kernel<kDgrad, SC><<<grid, kThreads, 0, st>>>(g);
  } else {  // dw[e, n, k] = sum_m gT[n, m] xT[k, m]
    g.Np = K; g.Nq = N;
    g.n_pt = (int)((K + kTP - 1) / kTP);
    g.n_qt = (int)((N + kTQ - 1) / kTQ);
    // expert shares: the a x b split (a b = 8) of an expert's tiles into equal rectangles
    // whose 32-tile rounds touch the fewest operand panels (ceil(32 / rect_p) + rect_p);
    // XCD blocks when no split divides the tile grid
    int best = 1 << 30;
    for (int a = 1; a <= 8; a *= 2) {
      const int b = 8 / a;
      if (g.n_qt % a != 0 || g.n_pt % b != 0 || (g.n_qt / a) * (g.n_pt / b) < kPersistSlots) continue;
      const int rq = g.n_qt / a, rp = g.n_pt / b;
      const int panels = (kPersistSlots + rp - 1) / rp + rp;
      if (panels < best) {
        best = panels;
        g.rect_q = rq; g.rect_p = rp; g.rect_b = b; g.share = rq * rp;
      }
    }
    // either schedule may be chosen on the device: the grid covers both
    const int64_t blocks_items = (blocks_of(g.n_pt, (int64_t)E * g.n_qt) + 7) / 8 * kPersistSlots;
    const int64_t share_items = (int64_t)E * g.share;
    grid = grid_items(share_items > blocks_items ? share_items : blocks_items, g.n_slots);
    grouped_gemm_kernel<kWgrad, SC><<<grid, kThreads, 0, st>>>(g);
  }
  return hipGetLastError();
}

hipError_t launch_grouped_gemm(GemmMode mode, const uint8_t* a, const float* a_s, const uint8_t* b,
                               const float* b_s, const int32_t* offsets, int E, int64_t M_cap, int64_t N,
                               int64_t K, void* out, int accumulate, hipStream_t st) {
  return grouped_gemm_impl(mode, a, a_s, b, b_s, offsets, E, M_cap, N, K, out, accumulate, st);
}
hipError_t launch_grouped_gemm(GemmMode mode, const uint8_t* a, const e8m0_t* a_s, const uint8_t* b,
                               const e8m0_t* b_s, const int32_t* offsets, int E, int64_t M_cap, int64_t N,
                               int64_t K, void* out, int accumulate, hipStream_t st) {
  return grouped_gemm_impl(mode, a, a_s, b, b_s, offsets, E, M_cap, N, K, out, accumulate, st);
}

}  // namespace ff8
