// Device-side numerics shared by the gfx950 kernels: bf16 <-> f32, the OCP e4m3
// conversions (hardware v_cvt_pk_fp8_f32 / v_cvt_pk_f32_fp8, round-to-nearest-even),
// the power-of-two tile scale rule, and 16/64-lane max reductions on DPP.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ff8 {

constexpr int kTile = 128;       // quantization tile / block edge
constexpr int kTMin = -126;      // smallest scale exponent (all-zero tiles)

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Round-to-nearest-even float -> bf16: the hardware packed convert (v_cvt_pk_bf16_f32),
// bit-identical to the integer rule u + 0x7FFF + ((u >> 16) & 1) on every finite input,
// denormals included, and quiet-NaN preserving.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16x2(f, 0.0f) & 0xFFFFu; }

// Unpack 8 bf16 (one 16-byte load) into floats.
__device__ __forceinline__ void unpack_bf16x8(const u32x4& w, float* v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_lo(w[i]);
    v[2 * i + 1] = bf16_hi(w[i]);
  }
}

// Scale exponent T of a tile: the smallest integer with amax <= 448 * 2^T, clamped
// to >= -126 (an all-zero or subnormal amax gives -126).  amax = m * 2^e with
// m in [1, 2): T = e - 8 if m <= 1.75 (448 = 1.75 * 2^8), else e - 7.
__device__ __forceinline__ int scale_exponent(float amax) {
  uint32_t u = __float_as_uint(amax);
  uint32_t eb = u >> 23;
  if (eb == 0) return kTMin;
  int t = (int)eb - 127 - 8 + ((u & 0x7FFFFFu) > 0x600000u ? 1 : 0);
  return t < kTMin ? kTMin : t;
}
__device__ __forceinline__ float exp2i(int t) { return __uint_as_float((uint32_t)(t + 127) << 23); }

// Scale storage.  A power-of-two scale 2^T is stored either as float32 (its exponent field
// holds T + 127, mantissa zero) or as one UE8M0 byte holding the same T + 127.
typedef uint8_t e8m0_t;
__device__ __forceinline__ void put_scale(float* p, int t) { *p = exp2i(t); }
__device__ __forceinline__ void put_scale(e8m0_t* p, int t) { *p = (e8m0_t)(t + 127); }
__device__ __forceinline__ int scale_exp(float s) { return (int)(__float_as_uint(s) >> 23) - 127; }
__device__ __forceinline__ int scale_exp(e8m0_t b) { return (int)b - 127; }
__device__ __forceinline__ float scale_value(float s) { return s; }
__device__ __forceinline__ float scale_value(e8m0_t b) { return exp2i((int)b - 127); }

// Encode two floats already in [-448, 448] into the low (kHi = false) or high
// (kHi = true) 16 bits of `old` with the hardware RNE conversion.
template <bool kHi>
__device__ __forceinline__ uint32_t cvt_e4m3x2(float a, float b, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(a, b, (int)old, kHi);
}
// Four floats in [-448, 448] -> one dword of e4m3 bytes (element 0 in the low byte).
__device__ __forceinline__ uint32_t cvt_e4m3x4(float a, float b, float c, float d) {
  uint32_t w = cvt_e4m3x2<false>(a, b, 0u);
  return cvt_e4m3x2<true>(c, d, w);
}
// Decode two e4m3 bytes (kHi = false: bytes 0,1; true: bytes 2,3) to floats.
template <bool kHi>
__device__ __forceinline__ f32x2 dec_e4m3x2(uint32_t w) {
  return __builtin_amdgcn_cvt_pk_f32_fp8((int)w, kHi);
}

// Max of non-negative float bit patterns across aligned groups of 16 lanes (DPP:
// xor 1, xor 2 inside quads, then half-row and row mirrors).
__device__ __forceinline__ uint32_t max16_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false));
  return v;
}
// Max across the 64 lanes of a wave (every lane gets the result).
__device__ __forceinline__ uint32_t max64_u32(uint32_t v) {
  v = max16_u32(v);
  v = max(v, (uint32_t)__shfl_xor((int)v, 16));
  v = max(v, (uint32_t)__shfl_xor((int)v, 32));
  return v;
}
__device__ __forceinline__ uint32_t abs_bits(float f) { return __float_as_uint(f) & 0x7FFFFFFFu; }

// Plain vector loads/stores.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ u32x2 ld8(const void* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ void st8(void* p, const u32x2& v) { *reinterpret_cast<u32x2*>(p) = v; }
// Streaming (non-temporal) vector loads/stores for data touched once: the lines are
// marked for early eviction instead of displacing reusable data in L2 / MALL.
__device__ __forceinline__ u32x4 ldnt16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void stnt16(void* p, const u32x4& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(p));
}
__device__ __forceinline__ u32x2 ldnt8(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
}
__device__ __forceinline__ void stnt8(void* p, const u32x2& v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x2*>(p));
}

// Quantize 8 values that belong to one 1x128 tile shared by 16 consecutive lanes:
// tile amax across the 16 lanes, power-of-two scale, RNE e4m3.  Returns the 8 bytes
// and the tile's scale exponent.
__device__ __forceinline__ u32x2 quant8_tile16(const float* v, int& t_out) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) m = max(m, abs_bits(v[i]));
  m = max16_u32(m);
  int t = scale_exponent(__uint_as_float(m));
  float inv = exp2i(-t);
  u32x2 r;
  r[0] = cvt_e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
  r[1] = cvt_e4m3x4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
  t_out = t;
  return r;
}

// Max of non-negative float bit patterns across aligned groups of 8 lanes (DPP).
__device__ __forceinline__ uint32_t max8_u32(uint32_t v) {
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false));
  v = max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false));
  return v;
}
// 16 values of one 1x128 tile shared by 8 consecutive lanes -> 16 e4m3 bytes and the
// tile's scale exponent.
__device__ __forceinline__ u32x4 quant16_tile8(const float* v, int& t_out) {
  uint32_t m = 0;
#pragma unroll
  for (int i = 0; i < 16; ++i) m = max(m, abs_bits(v[i]));
  m = max8_u32(m);
  const int t = scale_exponent(__uint_as_float(m));
  const float inv = exp2i(-t);
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = cvt_e4m3x4(v[4 * i] * inv, v[4 * i + 1] * inv, v[4 * i + 2] * inv, v[4 * i + 3] * inv);
  t_out = t;
  return r;
}

// Rows of the grouped tensor that hold data: offsets[E] when offsets are given.
__device__ __forceinline__ int64_t active_rows(const int32_t* offsets, int E, int64_t rows) {
  if (offsets == nullptr) return rows;
  int64_t m = offsets[E];
  return m < rows ? m : rows;
}

}  // namespace ff8
