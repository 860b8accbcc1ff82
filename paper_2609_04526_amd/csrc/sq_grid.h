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

// ------------------------------------------------------------------ update
// New scale byte for eff' = eff + d rounded onto the grid (round_grid of
// Section 3); `clamped` reports whether the NVFP4 ceiling min(eff', 448 ws2)
// bound (the gradient does not pass it there).
//   NVFP4: e = fp32(e4m3(b) ws2), e2 = fp32(e + d), e2 = min(e2, fp32(448 ws2)),
//          q = fp32(e2 / ws2), b' = E4M3 nearest-even, saturating.
//   MXFP4: e2 = fp32(2^(b-127) + d), b' = E8M0 of 2^round(log2 e2).
template <int FMT>
__device__ __forceinline__ uint32_t grid_update(uint32_t b, float d, float ws2, bool& clamped) {
  if (FMT == kNV) {
    const float e = __fmul_rn(e4m3_to_f32(b), ws2);
    float e2 = __fadd_rn(e, d);
    const float cap = __fmul_rn(448.0f, ws2);
    clamped = e2 > cap;                         // NaN compares false and is kept
    e2 = clamped ? cap : e2;
    return e4m3_encode_rne_sat(__fdiv_rn(e2, ws2));
  }
  clamped = false;
  return e8m0_encode_log(__fadd_rn(e8m0_to_f32(b), d));
}

template <int FMT>
__device__ __forceinline__ uint32_t merge_one_t(uint32_t b, float d, float ws2) {
  bool clamped;
  return grid_update<FMT>(b, d, ws2, clamped);
}

}  // namespace sq
