// The grid-and-clamp path of the block scales, shared by the scale-plane
// merge (sq_elem.hip) and the QAST forward (sq_qast.hip): paper Section 3,
// stability recipe item (iii), requires the merge to round and clamp exactly
// as the training forward did, so both call grid_update below.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"

namespace sq {

// ------------------------------------------------------------------ encoders
// fp32 -> E8M0 byte of 2^round(log2 x), nearest in the log domain: with
// x = m * 2^k, m in [1, 2), round up iff m > sqrt(2), i.e. iff the 23-bit
// fraction field is >= 0x3504F4 (fp32(sqrt 2) = 0x3FB504F3 lies below sqrt 2).
// Exponent clamped to [-127, 127]; x <= 0 -> 0x00, +inf -> 0xFE, NaN -> 0xFF.
__device__ __forceinline__ uint32_t e8m0_encode_log(float x) {
  if (x != x) return 0xFFu;
  if (!(x > 0.0f)) return 0x00u;
  uint32_t u = __float_as_uint(x);
  if (u >= 0x7F800000u) return 0xFEu;
  int e = (int)(u >> 23);
  uint32_t frac = u & 0x7FFFFFu;
  int k;
  if (e == 0) {                             // subnormal: x = frac * 2^-149
    const int p = 31 - __clz(frac);         // top set bit
    k = p - 149;
    frac = (frac << (23 - p)) & 0x7FFFFFu;
  } else {
    k = e - 127;
  }
  if (frac >= 0x3504F4u) k += 1;
  k = k < -127 ? -127 : (k > 127 ? 127 : k);
  return (uint32_t)(k + 127);
}

// fp32 -> E4M3 "fn" byte, round to nearest, ties to even mantissa, saturating
// at +-448; NaN -> 0x7F.
__device__ __forceinline__ uint32_t e4m3_encode_rne_sat(float x) {
  // gfx950's fp8 convert rounds to the nearest OCP E4M3 value, ties to even;
  // clamping to +-448 first makes it saturate (448 is the largest finite
  // value, so the clamp changes no in-range rounding).  NaN -> 0x7F.
  if (x != x) return 0x7Fu;
  const float c = __builtin_fminf(__builtin_fmaxf(x, -448.0f), 448.0f);
  return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, c, 0, false) & 0xFFu;
}

// ------------------------------------------------------------------ division
// A divisor with its correctly rounded reciprocal r = fp32(1 / d).
struct RcpDivisor {
  float d, r;
  bool fast;      // d in [2^-64, 2^64]: divide through r (div_exact)
};
__device__ __forceinline__ RcpDivisor make_rcp_divisor(float d) {
  RcpDivisor v;
  v.d = d;
  v.r = __fdiv_rn(1.0f, d);
  v.fast = d >= 0x1p-64f && d <= 0x1p64f;
  return v;
}

// fp32(x / d), correctly rounded (nearest even).  q0 = fp32(x r) is within
// two ulps of the quotient; a Newton step with the remainder x - d q0 taken by
// a fused multiply-add makes it faithful, and a second one rounds it correctly
// (Markstein's theorem: a faithful quotient corrected through the correctly
// rounded reciprocal).  That needs the remainders to stay clear of underflow;
// with d in [2^-64, 2^64] they do for every quotient at or above 2^-26, and
// the callers round smaller quotients to a signed zero (E4M3 or E2M1)
// whichever way their last bit goes.  Zeros keep their sign and a quotient
// past the fp32 range stays infinite (q0); NaN stays NaN.  Other divisors
// divide directly.  FAST = 1 or 0 takes that path without looking at
// v.fast (callers that branch once per plane); -1 looks.
template <int FAST = -1>
__device__ __forceinline__ float div_exact(float x, const RcpDivisor& v) {
  if (FAST == 0 || (FAST < 0 && !v.fast)) return __fdiv_rn(x, v.d);
  const float q0 = __fmul_rn(x, v.r);
  const float q1 = __builtin_fmaf(__builtin_fmaf(-q0, v.d, x), v.r, q0);
  const float q2 = __builtin_fmaf(__builtin_fmaf(-q1, v.d, x), v.r, q1);
  return (x == 0.0f || __builtin_isinf(q0)) ? q0 : q2;
}

// ------------------------------------------------------------------ NVFP4 step
// A tensor's ws2 with what the NVFP4 grid step needs of it: the divisor and
// the ceiling fp32(448 ws2).
struct Ws2Div {
  RcpDivisor div;
  float ws2, cap;
};
__device__ __forceinline__ Ws2Div make_ws2_div(float ws2) {
  Ws2Div w;
  w.div = make_rcp_divisor(ws2);
  w.ws2 = ws2;
  w.cap = __fmul_rn(448.0f, ws2);
  return w;
}

// q = fp32(e2 / ws2) of the NVFP4 step for stored byte b (given as the low
// byte of `word` shifted to byte SEL) and delta d; `clamped` reports whether
// the ceiling bound.  The result is at most fp32(cap / ws2) < 449.
template <int SEL, int FAST = -1>
__device__ __forceinline__ float nv_step_q(uint32_t word, float d, const Ws2Div& w, bool& clamped) {
  const float e = __fmul_rn(__builtin_amdgcn_cvt_f32_fp8((int)word, SEL), w.ws2);
  float e2 = __fadd_rn(e, d);
  clamped = e2 > w.cap;                       // NaN compares false and is kept
  e2 = clamped ? w.cap : e2;
  return div_exact<FAST>(e2, w.div);
}

// Step results go to E4M3 through gfx950's fp8 convert (nearest even).  They
// lie below 449, whose nearest E4M3 value is 448, so only the lower side needs
// the clamp at -448 that makes the convert saturate; NaN compares false and
// passes.  The convert writes NaN as 0xFF: e4m3_nan_canon turns every NaN
// byte (0x7F or 0xFF; finite values stop at 0x7E / 0xFE) into 0x7F.
__device__ __forceinline__ float e4m3_prep(float q) { return q < -448.0f ? -448.0f : q; }
__device__ __forceinline__ uint32_t e4m3_nan_canon(uint32_t w) {
  const uint32_t nan_bytes = ((w & 0x7F7F7F7Fu) + 0x01010101u) & 0x80808080u;   // bit 7 of each NaN byte
  return w & ~nan_bytes;
}

// ------------------------------------------------------------------ update
// New scale byte for eff' = eff + d rounded onto the grid (round_grid of
// Section 3); `clamped` reports whether the NVFP4 ceiling min(eff', 448 ws2)
// bound (the gradient does not pass it there).
//   NVFP4: e = fp32(e4m3(b) ws2), e2 = fp32(e + d), e2 = min(e2, fp32(448 ws2)),
//          q = fp32(e2 / ws2), b' = E4M3 nearest-even, saturating.
//   MXFP4: e2 = fp32(2^(b-127) + d), b' = E8M0 of 2^round(log2 e2).
template <int FMT>
__device__ __forceinline__ uint32_t grid_update(uint32_t b, float d, const Ws2Div& w, bool& clamped) {
  if (FMT == kNV) {
    const float q = e4m3_prep(nv_step_q<0>(b, d, w, clamped));
    return e4m3_nan_canon((uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(q, q, 0, false) & 0xFFu);
  }
  clamped = false;
  return e8m0_encode_log(__fadd_rn(e8m0_to_f32(b), d));
}

template <int FMT>
__device__ __forceinline__ uint32_t merge_one_t(uint32_t b, float d, const Ws2Div& w) {
  bool clamped;
  return grid_update<FMT>(b, d, w, clamped);
}

// NVFP4 step of the four bytes of `word` (byte k with delta d[k]).  The same
// arithmetic as grid_update<kNV>, byte for byte; two converts pack the word.
typedef float sq_f32x4 __attribute__((ext_vector_type(4)));
template <int FAST>
__device__ __forceinline__ uint32_t nv_merge_word(uint32_t word, sq_f32x4 d, const Ws2Div& w) {
  bool c;
  const float q0 = e4m3_prep(nv_step_q<0, FAST>(word, d[0], w, c));
  const float q1 = e4m3_prep(nv_step_q<1, FAST>(word, d[1], w, c));
  const float q2 = e4m3_prep(nv_step_q<2, FAST>(word, d[2], w, c));
  const float q3 = e4m3_prep(nv_step_q<3, FAST>(word, d[3], w, c));
  const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(q0, q1, 0, false);
  return e4m3_nan_canon((uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(q2, q3, lo, true));
}

}  // namespace sq
