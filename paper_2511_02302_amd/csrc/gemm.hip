// FP8 grouped GEMMs for gfx950: fprop, dgrad and wgrad of the expert layer (paper
// sections 3.1-3.2: row-wise FP8 operands for Fprop/Dgrad, column-wise operands from
// the scaling-aware transpose for Wgrad).
//
// Every mode is C[p, q] = sum_k P[p, k] * Q[q, k] * sP(p, k/128) * sQ(q, k/128) over
// one expert's data, where p indexes the output's contiguous dimension:
//   fprop: p = n (W_e rows),        q = token row m, k over K  -> out[m, n] bf16
//   dgrad: p = k (W_e columns),     q = token row m, k = n     -> out[m, k] bf16
//   wgrad: p = k (xT rows),         q = n (gT rows), k = token -> dw[e, n, k] fp32
//
// MFMA: v_mfma_scale_f32_32x32x64_f8f6f4 (e4m3 x e4m3).  The library's scales are
// powers of two, i.e. exactly E8M0 values (the fp32 exponent field), so each 128-wide
// K block's scales are applied by the matrix core itself, per P row and per Q column,
// inside the float32 accumulation -- no VALU scale-promotion pass.
//
// Tiling: 256 (p) x 256 (q) x 128 (k) per workgroup, 4 waves in 2 x 2, each wave
// 128 x 128 = 4 x 4 MFMA tiles (256 accumulator registers).  LDS holds two stages of
// both operand tiles (2 x 64 KB) plus their E8M0 scale bytes; global loads for step
// k+1 are in flight while step k runs on the matrix cores.  K-major tiles use a 16-byte
// XOR swizzle (chunk ^ row%8), so the 16-byte fragment reads are bank-conflict-free.
// dgrad reads W_e in its stored [n][k] orientation with ds_read_b64_tr_b8, which
// transposes 8x8 byte blocks across lanes on the way out of LDS.
//
// Grouped scheduling is on the device: tiles are counted per expert from offsets
// (no host sync); surplus workgroups of the host-sized grid exit at once.

#include "ff8_device.hpp"
#include "ff8_launch.hpp"

namespace ff8 {

namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kTP = 256;  // p tile
constexpr int kTQ = 256;  // q tile
constexpr int kTK = 128;  // k step (one scale block)
constexpr int kStageBytes = kTP * kTK + kTQ * kTK;  // 64 KB

struct GemmArgs {
  const uint8_t* P;   // fprop: w; dgrad: w; wgrad: xT
  const float* sP;
  const uint8_t* Q;   // fprop: a; dgrad: g; wgrad: gT
  const float* sQ;
  const int32_t* offsets;
  void* out;
  int E;
  int64_t M_cap;
  int64_t Np;         // extent of p (output columns)
  int64_t Nq;         // wgrad: extent of q (N); fprop/dgrad: unused
  int64_t Kdim;       // fprop/dgrad: contraction length; wgrad: unused (per group)
  int n_pt, n_qt;     // p tiles; q tiles (wgrad only)
  int accumulate;
};

__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int xcd = bid & 7, slot = bid >> 3, q = n >> 3, r = n & 7;
  return xcd * q + (xcd < r ? xcd : r) + slot;
}

__device__ __forceinline__ uint32_t e8m0(float s) { return (__float_as_uint(s) >> 23) & 0xFFu; }

// One scaled MFMA on sub-tile (A, B); the opsel byte selectors must be constants.
template <int A, int B>
__device__ __forceinline__ void mma(f32x16 (&acc)[4][4], const i32x8 (&fp)[4], const i32x8 (&fq)[4], int sp, int sq) {
  acc[A][B] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fp[A], fq[B], acc[A][B], 0, 0, A, sp, B, sq);
}
template <int A>
__device__ __forceinline__ void mma_row(f32x16 (&acc)[4][4], const i32x8 (&fp)[4], const i32x8 (&fq)[4], int sp,
                                        int sq) {
  mma<A, 0>(acc, fp, fq, sp, sq);
  mma<A, 1>(acc, fp, fq, sp, sq);
  mma<A, 2>(acc, fp, fq, sp, sq);
  mma<A, 3>(acc, fp, fq, sp, sq);
}

__device__ __forceinline__ int kmaj_off(int r, int c) { return r * kTK + ((c ^ (r & 7)) << 4); }
__device__ __forceinline__ int wt_off(int n, int c) { return n * kTP + ((c ^ (n & 7)) << 4); }

template <int MODE>
__global__ __launch_bounds__(kThreads, 1) void grouped_gemm_kernel(GemmArgs g) {
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint8_t* sc_base = smem + 2 * kStageBytes;  // [2][512] scale bytes: sP then sQ
  __shared__ int cum[1025];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wp = wave & 1, wq = wave >> 1;
  const int logical = xcd_remap(blockIdx.x, gridDim.x);

  // ---- tile decode ----
  int e, pt;
  int64_t q0, q_end, k0, nk;
  if (MODE != kWgrad) {
    for (int i = tid; i < g.E; i += kThreads) cum[i + 1] = (g.offsets[i + 1] - g.offsets[i] + kTQ - 1) / kTQ;
    __syncthreads();
    if (tid == 0) {
      int acc = 0;
      cum[0] = 0;
      for (int i = 1; i <= g.E; ++i) {
        acc += cum[i];
        cum[i] = acc;
      }
    }
    __syncthreads();
    pt = logical % g.n_pt;
    const int qg = logical / g.n_pt;
    if (qg >= cum[g.E]) return;
    int lo = 0, hi = g.E - 1;  // largest e with cum[e] <= qg
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cum[mid] <= qg) lo = mid; else hi = mid - 1;
    }
    e = lo;
    q0 = g.offsets[e] + (int64_t)(qg - cum[e]) * kTQ;
    q_end = g.offsets[e + 1];
    k0 = 0;
    nk = g.Kdim / kTK;
  } else {
    const int per_e = g.n_pt * g.n_qt;
    e = logical / per_e;
    const int rem = logical - e * per_e;
    const int qt = rem / g.n_pt;
    pt = rem - qt * g.n_pt;
    q0 = (int64_t)qt * kTQ;
    q_end = g.Nq;
    k0 = g.offsets[e];
    nk = (g.offsets[e + 1] - k0) / kTK;
  }
  const int64_t p0 = (int64_t)pt * kTP;

  // ---- global load assignment ----
  // Q tile (always K-major): rows q0 + (tid>>3) + 32 i, 16-byte chunk tid & 7.
  const int64_t q_ld = (MODE == kWgrad) ? g.M_cap : g.Kdim;
  const int64_t q_rows_max = (MODE == kWgrad) ? g.Nq : g.M_cap;
  const uint8_t* qptr[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int64_t r = q0 + (tid >> 3) + 32 * i;
    r = r < q_rows_max ? r : q_rows_max - 1;
    qptr[i] = g.Q + r * q_ld + k0 + (tid & 7) * 16;
  }
  // P tile: fprop / wgrad K-major rows p0 + (tid>>3) + 32 i; dgrad W rows n (16 per pass).
  const uint8_t* pptr[8];
  int64_t p_step;  // bytes to advance per k step
  if (MODE == kDgrad) {
    const uint8_t* w = g.P + (int64_t)e * g.Kdim * g.Np;  // W_e [N = Kdim][K = Np]
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int n = (tid >> 4) + 16 * i;
      int64_t col = p0 + (tid & 15) * 16;
      col = col < g.Np ? col : g.Np - 16;
      pptr[i] = w + (int64_t)n * g.Np + col;
    }
    p_step = (int64_t)kTK * g.Np;
  } else {
    const int64_t p_ld = (MODE == kWgrad) ? g.M_cap : g.Kdim;
    const uint8_t* base = (MODE == kFprop) ? g.P + (int64_t)e * g.Np * g.Kdim : g.P;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      int64_t r = p0 + (tid >> 3) + 32 * i;
      r = r < g.Np ? r : g.Np - 1;
      pptr[i] = base + r * p_ld + k0 + (tid & 7) * 16;
    }
    p_step = kTK;
  }
  // Scales: thread tid loads the P scale of p0 + tid and the Q scale of q0 + tid.
  const float* sp_ptr;
  int64_t sp_step;
  {
    int64_t p = p0 + tid;
    p = p < g.Np ? p : g.Np - 1;
    if (MODE == kFprop) {  // w_s [E][Np/128][Kdim/128]
      sp_ptr = g.sP + ((int64_t)e * (g.Np / kTile) + p / kTile) * (g.Kdim / kTile);
      sp_step = 1;
    } else if (MODE == kDgrad) {  // w_s [E][Kdim/128][Np/128]: block (n/128, p/128)
      sp_ptr = g.sP + (int64_t)e * (g.Kdim / kTile) * (g.Np / kTile) + p / kTile;
      sp_step = g.Np / kTile;
    } else {  // xT_s [Np][M_cap/128]
      sp_ptr = g.sP + p * (g.M_cap / kTile) + k0 / kTile;
      sp_step = 1;
    }
  }
  const float* sq_ptr;
  {
    int64_t q = q0 + tid;
    q = q < q_rows_max ? q : q_rows_max - 1;
    const int64_t ld = (MODE == kWgrad) ? g.M_cap / kTile : g.Kdim / kTile;
    sq_ptr = g.sQ + q * ld + k0 / kTile;
  }
  const int sc_idx = (tid & 31) * 8 + (tid >> 5);  // LDS byte of p (or q) = tid

  // ---- accumulators ----
  f32x16 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.0f;

  u32x4 rp[8], rq[8];
  float rsp = 0.f, rsq = 0.f;

  auto gload = [&](int64_t ks) {
#pragma unroll
    for (int i = 0; i < 8; ++i) rq[i] = ld16(qptr[i] + ks * kTK);
#pragma unroll
    for (int i = 0; i < 8; ++i) rp[i] = ld16(pptr[i] + ks * p_step);
    rsp = sp_ptr[ks * sp_step];
    rsq = sq_ptr[ks];
  };
  auto lstore = [&](int s) {
    uint8_t* P_l = (smem + s * kStageBytes);
    uint8_t* Q_l = (smem + s * kStageBytes) + kTP * kTK;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4*>(Q_l + kmaj_off((tid >> 3) + 32 * i, tid & 7)) = rq[i];
    if (MODE == kDgrad) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<u32x4*>(P_l + wt_off((tid >> 4) + 16 * i, tid & 15)) = rp[i];
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *reinterpret_cast<u32x4*>(P_l + kmaj_off((tid >> 3) + 32 * i, tid & 7)) = rp[i];
    }
    uint8_t* sc = sc_base + s * 512;
    sc[sc_idx] = (uint8_t)e8m0(rsp);
    sc[256 + sc_idx] = (uint8_t)e8m0(rsq);
  };

  if (nk > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();

  for (int64_t ks = 0; ks < nk; ++ks) {
    const int cur = (int)(ks & 1);
    if (ks + 1 < nk) gload(ks + 1);
    const uint8_t* P_l = (smem + cur * kStageBytes);
    const uint8_t* Q_l = (smem + cur * kStageBytes) + kTP * kTK;
    const uint8_t* sc = sc_base + cur * 512;
    const int scale_p = *reinterpret_cast<const int*>(sc + (lane & 31) * 8 + 4 * wp);
    const int scale_q = *reinterpret_cast<const int*>(sc + 256 + (lane & 31) * 8 + 4 * wq);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      i32x8 fp[4], fq[4];
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int r = 128 * wq + 32 * a + (lane & 31);
        const int c0 = 4 * h + 2 * (lane >> 5);
        const u32x4 x0 = *reinterpret_cast<const u32x4*>(Q_l + kmaj_off(r, c0));
        const u32x4 x1 = *reinterpret_cast<const u32x4*>(Q_l + kmaj_off(r, c0 + 1));
        fq[a] = i32x8{(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3], (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
      }
      if (MODE == kDgrad) {
        const int gg = lane >> 4, hh = lane & 1, ii = (lane & 15) >> 1;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int kl = 128 * wp + 32 * a + 16 * (gg & 1) + 8 * hh;
          i32x8 f;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int n = 64 * h + 32 * (gg >> 1) + 8 * r + ii;
            const uint8_t* addr = P_l + n * kTP + (((kl >> 4) ^ (n & 7)) << 4) + (kl & 15);
            const i32x2 t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
                (i32x2 __attribute__((address_space(3)))*)((__attribute__((address_space(3))) uint8_t*)(addr)));
            f[2 * r] = t[0];
            f[2 * r + 1] = t[1];
          }
          fp[a] = f;
        }
      } else {
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int r = 128 * wp + 32 * a + (lane & 31);
          const int c0 = 4 * h + 2 * (lane >> 5);
          const u32x4 x0 = *reinterpret_cast<const u32x4*>(P_l + kmaj_off(r, c0));
          const u32x4 x1 = *reinterpret_cast<const u32x4*>(P_l + kmaj_off(r, c0 + 1));
          fp[a] = i32x8{(int)x0[0], (int)x0[1], (int)x0[2], (int)x0[3], (int)x1[0], (int)x1[1], (int)x1[2], (int)x1[3]};
        }
      }
      mma_row<0>(acc, fp, fq, scale_p, scale_q);
      mma_row<1>(acc, fp, fq, scale_p, scale_q);
      mma_row<2>(acc, fp, fq, scale_p, scale_q);
      mma_row<3>(acc, fp, fq, scale_p, scale_q);
    }
    if (ks + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue ----
  if (MODE == kWgrad) {
    if (nk == 0 && g.accumulate) return;
    float* dw = static_cast<float*>(g.out) + (int64_t)e * g.Nq * g.Np;
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int64_t q = q0 + 128 * wq + 32 * b + (lane & 31);
        if (q >= q_end) continue;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
          const int64_t p = p0 + 128 * wp + 32 * a + 8 * gr + 4 * (lane >> 5);
          if (p >= g.Np) continue;
          float* dst = dw + q * g.Np + p;
          u32x4 o;
          if (g.accumulate) {
            const u32x4 old = ld16(dst);
#pragma unroll
            for (int j = 0; j < 4; ++j) o[j] = __float_as_uint(__uint_as_float(old[j]) + acc[a][b][4 * gr + j]);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) o[j] = __float_as_uint(acc[a][b][4 * gr + j]);
          }
          st16(dst, o);
        }
      }
  } else {
    uint16_t* out = static_cast<uint16_t*>(g.out);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int64_t q = q0 + 128 * wq + 32 * b + (lane & 31);
        if (q >= q_end) continue;
#pragma unroll
        for (int gr = 0; gr < 4; ++gr) {
          const int64_t p = p0 + 128 * wp + 32 * a + 8 * gr + 4 * (lane >> 5);
          if (p >= g.Np) continue;
          u32x2 o;
          o[0] = pack_bf16x2(acc[a][b][4 * gr + 0], acc[a][b][4 * gr + 1]);
          o[1] = pack_bf16x2(acc[a][b][4 * gr + 2], acc[a][b][4 * gr + 3]);
          st8(out + q * g.Np + p, o);
        }
      }
  }
}

}  // namespace

hipError_t launch_grouped_gemm(GemmMode mode, const uint8_t* a, const float* a_s, const uint8_t* b,
                               const float* b_s, const int32_t* offsets, int E, int64_t M_cap, int64_t N,
                               int64_t K, void* out, int accumulate, hipStream_t st) {
  GemmArgs g{};
  g.offsets = offsets;
  g.out = out;
  g.E = E;
  g.M_cap = M_cap;
  g.accumulate = accumulate;
  const size_t smem = 2 * kStageBytes + 2 * 512;
  unsigned grid;
  if (mode == kFprop) {  // out[m, n] = a[m, :] . w[e, n, :]
    g.P = b; g.sP = b_s; g.Q = a; g.sQ = a_s;
    g.Np = N; g.Kdim = K;
    g.n_pt = (int)((N + kTP - 1) / kTP);
    grid = (unsigned)(g.n_pt * ((M_cap + kTQ - 1) / kTQ + (E + 1) / 2));
    (void)hipFuncSetAttribute((const void*)grouped_gemm_kernel<kFprop>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    grouped_gemm_kernel<kFprop><<<grid, kThreads, smem, st>>>(g);
  } else if (mode == kDgrad) {  // out[m, k] = g[m, :] . w[e, :, k]
    g.P = b; g.sP = b_s; g.Q = a; g.sQ = a_s;
    g.Np = K; g.Kdim = N;
    g.n_pt = (int)((K + kTP - 1) / kTP);
    grid = (unsigned)(g.n_pt * ((M_cap + kTQ - 1) / kTQ + (E + 1) / 2));
    (void)hipFuncSetAttribute((const void*)grouped_gemm_kernel<kDgrad>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    grouped_gemm_kernel<kDgrad><<<grid, kThreads, smem, st>>>(g);
  } else {  // dw[e, n, k] = sum_m gT[n, m] xT[k, m]
    g.P = b; g.sP = b_s; g.Q = a; g.sQ = a_s;
    g.Np = K; g.Nq = N;
    g.n_pt = (int)((K + kTP - 1) / kTP);
    g.n_qt = (int)((N + kTQ - 1) / kTQ);
    grid = (unsigned)(E * g.n_pt * g.n_qt);
    (void)hipFuncSetAttribute((const void*)grouped_gemm_kernel<kWgrad>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
    grouped_gemm_kernel<kWgrad><<<grid, kThreads, smem, st>>>(g);
  }
  return hipGetLastError();
}

}  // namespace ff8
