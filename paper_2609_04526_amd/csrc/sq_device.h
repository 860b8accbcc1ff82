// Device-side helpers for the frozen-code FP4 layer on gfx950: element codecs,
// bf16 packing and the on-chip dequantisation of packed E2M1 codes.
//
// Storage (paper Section 2, "Native FP4 microscaling storage"):
//   W[o,i] = code[o,i] * eff[o, i / B]
//   code  E2M1 nibble (sign | 2 exponent bits, bias 1 | 1 mantissa bit), the
//         low nibble of a byte holds the even column;
//   MXFP4 eff = 2^(byte-127) (E8M0, B = 32);
//   NVFP4 eff = e4m3(byte) * ws2 (E4M3 "fn", B = 16), ws2 one fp32 per tensor.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

enum Fmt { kMX = 0, kNV = 1 };

__device__ __forceinline__ uint32_t bits_of(bf16x2 v) {
  uint32_t u;
  __builtin_memcpy(&u, &v, 4);
  return u;
}

// ---------------------------------------------------------------- scalars
// E8M0 byte as the fp32 whose exponent field is that byte: 2^(b-127) for
// 1 <= b <= 254.  The scaled FP4 converts read only the exponent field of
// their fp32 scale operand, which is exactly an E8M0 scale.
__device__ __forceinline__ float e8m0_as_scale_operand(uint32_t b) {
  return __uint_as_float(b << 23);
}

// E8M0 byte -> fp32 value (0 -> 2^-127, an fp32 subnormal; 0xFF -> NaN).
__device__ __forceinline__ float e8m0_to_f32(uint32_t b) {
  uint32_t bits = (b == 0u) ? 0x00400000u : ((b == 0xFFu) ? 0x7FC00000u : (b << 23));
  return __uint_as_float(bits);
}

// E4M3 "fn" byte -> fp32 (bias 7, subnormals, 0x7F/0xFF NaN, no infinities).
__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {
  // gfx950's fp8 convert reads the OCP E4M3 ("fn") format: exact for every
  // byte, 0x7F / 0xFF decode to NaN.
  return __builtin_amdgcn_cvt_f32_fp8((int)(b & 0xFFu), 0);
}

// E2M1 nibble -> fp32.  Magnitudes in half units: 0,1,2,3,4,6,8,12.
__device__ __forceinline__ float e2m1_to_f32(uint32_t n) {
  const uint32_t half_units = __builtin_amdgcn_perm(0x0C080604u, 0x03020100u, 0x0C0C0C00u | (n & 7u)) & 0xFFu;
  const float mag = (float)half_units * 0.5f;
  return (n & 8u) ? -mag : mag;
}

// fp32 -> bf16 bits, round to nearest even; NaN -> quiet NaN.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return ((u >> 16) | 0x40u) & 0xFFFFu;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

// ---------------------------------------------------------------- dequant
// 8 packed codes (one dword, code 2p in the low nibble of byte p) times one
// block scale -> 8 bf16 in 4 dwords (element 2p in the low half of dword p).
// Every product code * scale is exact in bf16: an E2M1 value has 2 significant
// bits and an E8M0 scale none, an E4M3 scale 4, so no rounding happens here.
//
// MX: one hardware convert per byte; the instruction multiplies by 2 to the
// exponent of its scale operand, which is the E8M0 byte itself.
__device__ __forceinline__ uint4 dequant8_mx(uint32_t w, float e8m0_operand) {
  uint4 r;
  r.x = bits_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, e8m0_operand, 0));
  r.y = bits_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, e8m0_operand, 1));
  r.z = bits_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, e8m0_operand, 2));
  r.w = bits_of(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, e8m0_operand, 3));
  return r;
}

// NV: the scaled converts ignore a scale's mantissa, so decode to fp32 at unit
// scale, multiply by the full E4M3 value (exact) and keep the top 16 bits
// (exact, so truncation is the correct rounding).
__device__ __forceinline__ uint32_t pack_hi16(float lo, float hi) {
  return __builtin_amdgcn_perm(__float_as_uint(hi), __float_as_uint(lo), 0x07060302u);
}
template <int SEL>
__device__ __forceinline__ uint32_t dequant2_nv_sel(uint32_t w, float s) {
  f32x2 v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w, 1.0f, SEL);
  return pack_hi16(v.x * s, v.y * s);
}
__device__ __forceinline__ uint4 dequant8_nv(uint32_t w, float e4m3_value) {
  uint4 r;
  r.x = dequant2_nv_sel<0>(w, e4m3_value);
  r.y = dequant2_nv_sel<1>(w, e4m3_value);
  r.z = dequant2_nv_sel<2>(w, e4m3_value);
  r.w = dequant2_nv_sel<3>(w, e4m3_value);
  return r;
}

template <int FMT>
struct ScaleOperand;
template <>
struct ScaleOperand<kMX> {
  static __device__ __forceinline__ float of(uint32_t byte) { return e8m0_as_scale_operand(byte); }
  static __device__ __forceinline__ uint4 dequant8(uint32_t w, float s) { return dequant8_mx(w, s); }
  static constexpr int kBlock = 32;
};
template <>
struct ScaleOperand<kNV> {
  static __device__ __forceinline__ float of(uint32_t byte) { return e4m3_to_f32(byte); }
  static __device__ __forceinline__ uint4 dequant8(uint32_t w, float s) { return dequant8_nv(w, s); }
  static constexpr int kBlock = 16;
};

// ---------------------------------------------------------------- transposes
// 8x8 transpose of 16-bit elements held as 8 rows of 4 dwords: in[r][c/2]
// holds element (r, c) in its low (c even) or high (c odd) half; out[c][r/2]
// receives element (r, c).  One byte permute per output dword.
__device__ __forceinline__ void transpose8x8_b16(const uint32_t (&in)[8][4], uint32_t (&out)[8][4]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = in[2 * q][c >> 1];
      const uint32_t hi = in[2 * q + 1][c >> 1];
      out[c][q] = __builtin_amdgcn_perm(hi, lo, (c & 1) ? 0x07060302u : 0x05040100u);
    }
  }
}

}  // namespace sq
