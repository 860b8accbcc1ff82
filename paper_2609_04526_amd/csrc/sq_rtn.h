// Round-to-nearest (and deploy-rule) re-quantisation of one chunk of 8 bf16
// weights into E2M1 codes and the block scale: the device side shared by the
// RTN kernels and the fused QAT-LoRA re-quantiser.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"

namespace sq {

// ceil(log2 x) for positive finite fp32 x (subnormals included).
__device__ __forceinline__ int ceil_log2_pos(float x) {
  const uint32_t u = __float_as_uint(x);
  const uint32_t e = u >> 23, frac = u & 0x7FFFFFu;
  if (e == 0u) {
    const int p = 31 - __clz(frac);
    return p - 149 + ((frac & (frac - 1u)) != 0u);
  }
  return (int)e - 127 + (frac != 0u);
}

// The 128-bit product a * m as (hi, lo) from four 32 x 32 -> 64-bit
// multiply-adds; no partial sum overflows 64 bits.
__device__ __forceinline__ void mulhilo64(uint64_t a, uint64_t m, uint64_t& hi, uint64_t& lo) {
  const uint32_t a0 = (uint32_t)a, a1 = (uint32_t)(a >> 32), m0 = (uint32_t)m, m1 = (uint32_t)(m >> 32);
  const uint64_t p00 = (uint64_t)a0 * m0;
  const uint64_t t = (uint64_t)a1 * m0 + (p00 >> 32);
  const uint64_t u = (uint64_t)a0 * m1 + (uint32_t)t;
  hi = (uint64_t)a1 * m1 + (t >> 32) + (u >> 32);
  lo = (u << 32) | (uint32_t)p00;
}

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC 2011) with counter
// (c, 0, 0, 0) and key (key, 0): ten rounds of two 64 x 64 -> 128-bit
// products recombined with the other counter words and the key, the key
// bumped by two Weyl constants between rounds.  Written from the published
// definition; it feeds the stochastic deploy rule.
__device__ __forceinline__ void philox4x64_10(uint64_t c, uint64_t key, uint64_t out[4]) {
  uint64_t x0 = c, x1 = 0, x2 = 0, x3 = 0, k0 = key, k1 = 0;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B97F4A7C15ull;
      k1 += 0xBB67AE8584CAA73Bull;
    }
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(x0, 0xD2E7470EE14C6C93ull, hi0, lo0);
    mulhilo64(x2, 0xCA5A826395121157ull, hi1, lo1);
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

// E2M1 magnitude of index m (0..7): twice the values 0, .5, 1, 1.5, 2, 3, 4, 6
// sit in the nibbles of 0xC8643210.
__device__ __forceinline__ float e2m1_mag(uint32_t m) {
  return (float)((0xC8643210u >> (4u * m)) & 0xFu) * 0.5f;
}

// E2M1 code of q rounded toward zero (magnitude index of the largest grid
// value at or below min(|q|, 6), and the sign bit of q), from q's bits: bits
// 22..30 hold the exponent and the first fraction bit, b = 254 + 2e + f1 for
// |q| = (1.f1...) 2^e, so |q| in [1, 8) has index b - 252 (1 -> 2, 1.5 -> 3,
// 2 -> 4, 3 -> 5, 4 -> 6, 6 -> 7); larger magnitudes, infinity included, stop
// at 7, [0.5, 1) (b = 252 or 253) has index 1 and smaller magnitudes 0.  A
// NaN q gives 7 and is fixed up by the caller.
__device__ __forceinline__ uint32_t e2m1_rtz_code(float q) {
  const uint32_t u = __float_as_uint(q);
  const int b = (int)((u >> 22) & 0x1FFu);
  const int m = min(max(b - 252, 0), 7) | (b == 252 ? 1 : 0);
  return (uint32_t)m | ((u >> 28) & 8u);
}

// Rounding rules of the re-quantiser.  The nearest rules and round-toward-zero
// and stochastic rounding keep the per-block scale; the whole-tensor rule
// takes one scale from the tensor amax (the deploy-side quantisers of the
// out-of-family sweep, Appendix B threat model (a) and the deployment-quantizer
// sweep).
enum : int { kRuleEven = 0, kRuleAway = 1, kRuleRtz = 2, kRuleStochastic = 3, kRuleWholeTensor = 4 };

// One chunk of 8 consecutive weights of a row (16 bytes of bf16, already
// loaded); the B/8 lanes of a block are adjacent and share the block amax.
// amax_t: the tensor amax (whole-tensor rule); seed: the Philox key
// (stochastic rule; element e = 8c + k draws word e % 4 of block e / 4).
// pack_below > 0: the lanes hold consecutive chunks from a multiple of 64 on,
// the scale plane is 4-byte aligned, and chunks below pack_below are whole
// groups of four blocks, written as one 4-byte store by the group's first
// lane (the wave's lanes must all take part: the bytes cross lanes).
// ws2d: the NVFP4 ws2 with its reciprocal, taken once per thread by the
// caller (null: derived here from ws2_ptr / ws2_val).  NVFAST = 1: the caller
// has checked that ws2 lies in [2^-55, 2^55], so ws2 and every block scale
// e4m3 * ws2 (E4M3 values lie in [2^-9, 448]) are divisors div_exact takes
// through their reciprocal: the quotients skip the per-element range check
// (same results).
template <int FMT, int RULE, int NVFAST = -1>
__device__ __forceinline__ void rtn_chunk(const uint4 v, int64_t c, bool valid, const float* ws2_ptr, float ws2_val,
                                          const float* amax_t, uint64_t seed,
                                          uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                          int64_t pack_below = 0, const RcpDivisor* ws2d = nullptr) {
  constexpr int B = ScaleOperand<FMT>::kBlock;
  constexpr int LPB = B / 8;
  const uint32_t h[4] = {v.x, v.y, v.z, v.w};
  // amax as a bit pattern: for |x| the integer order of the bits is the
  // numeric order, with NaN above +inf, so NaN propagates like a max.
  uint32_t am = 0;
  if (RULE == kRuleWholeTensor) {
    am = __float_as_uint(*amax_t) >> 16;                    // bf16 bits, written by rtn_amax
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      am = max(am, h[k] & 0x7FFFu);
      am = max(am, (h[k] >> 16) & 0x7FFFu);
    }
    am = max(am, (uint32_t)__shfl_xor((int)am, 1));
    if (LPB == 4) am = max(am, (uint32_t)__shfl_xor((int)am, 2));
  }
  const float amax = __uint_as_float(am << 16);
  // fp32(amax / 6) through the reciprocal of 6: correctly rounded for every
  // bf16 amax at or above 2^-120 (all 31,744 of them were checked against
  // true division with an exact emulation); smaller, zero and NaN divide
  const float sixth = amax >= 0x1p-120f ? div_exact<1>(amax, RcpDivisor{6.0f, 0x1.555556p-3f, true})
                                        : __fdiv_rn(amax, 6.0f);

  uint32_t sbyte;
  float eff;            // effective block scale (what q divides by)
  if (FMT == kMX) {
    int k;
    if (sixth != sixth) {
      sbyte = 0xFFu;
      k = 0;
    } else {
      if (sixth == 0.0f) k = -127;
      else if (sixth > 3.4028234e38f) k = 127;
      else k = ceil_log2_pos(sixth);
      k = k < -127 ? -127 : (k > 127 ? 127 : k);
      sbyte = (uint32_t)(k + 127);
    }
    // 2^-k as fp32 (2^-127 is subnormal, 2^127 normal): exact
    const float inv = (k == 127) ? __uint_as_float(0x00400000u) : __uint_as_float((uint32_t)(127 - k) << 23);
    eff = (sbyte == 0xFFu) ? __uint_as_float(0x7FC00000u) : inv;   // used as a multiplier below
  } else {
    float ws2;
    RcpDivisor wd;
    if (RULE == kRuleWholeTensor && !(ws2_val > 0.0f)) {    // recomputed from the same amax
      ws2 = __fdiv_rn(sixth, 448.0f);
      if (ws2 == 0.0f) ws2 = 1.0f;
      wd = make_rcp_divisor(ws2);
    } else if (ws2d) {
      wd = *ws2d;
      ws2 = wd.d;
    } else {
      ws2 = ws2_ptr ? *ws2_ptr : ws2_val;
      wd = make_rcp_divisor(ws2);
    }
    // fp32(sixth / ws2): div_exact is correctly rounded for quotients at or
    // above 2^-26, and the E4M3 encoder turns every smaller one into 0
    sbyte = e4m3_encode_rne_sat(div_exact<NVFAST>(sixth, wd));
    eff = __fmul_rn(e4m3_to_f32(sbyte), ws2);
  }

  // Codes: gfx950's fp32 -> E2M1 convert rounds |q| to the nearest E2M1
  // magnitude with ties to even and saturates at 6 (it equals the threshold
  // rounding on every non-NaN fp32 input); ties away differ from it exactly at
  // |q| = 0.25, 1.25, 2.5 and 5, where they take the next magnitude.  A NaN q
  // codes as magnitude 0, and the sign bit is always the sign of w.
  float q[8];
  RcpDivisor ed;                                            // NVFP4: q = w / eff, exactly (div_exact)
  if (FMT == kNV) ed = make_rcp_divisor(eff);
  auto weight = [&](int k) { return __uint_as_float(((h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu) << 16); };
  // NVFAST: a block whose scale is nonzero and whose quotients stay below
  // 2^100 (|w| <= amax <= 2^100 eff) takes div_exact's refinement without
  // its zero and overflow cases: the refined quotient is exact, and of the
  // signs only that of a zero w can be lost, which copysign restores.  Zero
  // scales, NaN blocks and overflowing quotients take the general path.
  if (FMT == kNV && NVFAST == 1 && eff != 0.0f && amax <= __fmul_rn(eff, 0x1p100f)) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float w = weight(k);
      const float q0 = __fmul_rn(w, ed.r);
      const float q1 = __builtin_fmaf(__builtin_fmaf(-q0, ed.d, w), ed.r, q0);
      const float q2 = __builtin_fmaf(__builtin_fmaf(-q1, ed.d, w), ed.r, q1);
      q[k] = __builtin_copysignf(q2, w);
    }
  } else {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float w = weight(k);
      if (FMT == kMX) q[k] = __fmul_rn(w, eff);             // w / 2^k, one rounding
      else q[k] = (eff == 0.0f) ? 0.0f : div_exact<NVFAST>(w, ed);
    }
  }
  // the convert writes its two codes into byte p of its first operand and
  // keeps the other bytes, so four of them build the word
  uint32_t packed = 0;
  if (RULE == kRuleRtz) {
#pragma unroll
    for (int k = 0; k < 8; ++k) packed |= e2m1_rtz_code(q[k]) << (4 * k);
  } else {
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, q[0], q[1], 1.0f, 0);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, q[2], q[3], 1.0f, 1);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, q[4], q[5], 1.0f, 2);
    packed = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(packed, q[6], q[7], 1.0f, 3);
  }
  if (RULE == kRuleAway) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {                           // a tie magnitude is below 6: no carry
      const float a = fabsf(q[k]);
      packed += (a == 0.25f || a == 1.25f || a == 2.5f || a == 5.0f) ? (1u << (4 * k)) : 0u;
    }
  }
  if (RULE == kRuleStochastic) {
    // The nearest magnitude is the truncated one or the one above it: step
    // down where it lies above min(|q|, 6).  Stochastic rounding then goes up
    // from the truncated magnitude lo iff u * gap < a - m(lo), which is
    // u < (a - m(lo)) / gap with both sides exact in fp32 (u has 24 bits and
    // gap is 0 or a power of two; a - m(lo) is a multiple of ulp(a)).
    uint64_t rw[8];
    if (RULE == kRuleStochastic) {
      philox4x64_10((uint64_t)(2 * c), seed, rw);
      philox4x64_10((uint64_t)(2 * c + 1), seed, rw + 4);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float a = fminf(fabsf(q[k]), 6.0f);
      uint32_t m = (packed >> (4 * k)) & 7u;
      const uint32_t dn = (e2m1_mag(m) > a) ? 1u : 0u;
      m -= dn;
      uint32_t up = 0;
      if (RULE == kRuleStochastic) {
        const float u = (float)(uint32_t)(rw[k] >> 40) * 5.9604644775390625e-08f;   // 2^-24
        const uint32_t hi = m < 7u ? m + 1u : 7u;
        up = (__fmul_rn(u, e2m1_mag(hi) - e2m1_mag(m)) < a - e2m1_mag(m)) ? 1u : 0u;
      }
      packed = packed - (dn << (4 * k)) + (up << (4 * k));   // stays within the magnitude bits
    }
  }
  // The convert carries the sign of q, which is the sign of w unless q is NaN
  // (possible only when the block amax is NaN) or forced to +0 by a zero
  // NVFP4 scale; only those blocks need the general fix-up.
  if (am > 0x7F80u || (FMT == kNV && eff == 0.0f)) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const uint32_t hb = (h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
      const uint32_t mag = (q[k] != q[k]) ? 0u : ((packed >> (4 * k)) & 7u);
      packed = (packed & ~(15u << (4 * k))) | ((mag | ((hb >> 12) & 8u)) << (4 * k));
    }
  }
  if (pack_below > 0) {
    constexpr int kGroup = 4 * LPB;                         // lanes of 4 blocks
    const uint32_t b1 = (uint32_t)__shfl_down((int)sbyte, LPB);
    const uint32_t b2 = (uint32_t)__shfl_down((int)sbyte, 2 * LPB);
    const uint32_t b3 = (uint32_t)__shfl_down((int)sbyte, 3 * LPB);
    if (valid) {
      __builtin_nontemporal_store(packed, reinterpret_cast<uint32_t*>(codes) + c);   // streaming store
      if (c < pack_below) {
        if ((c % kGroup) == 0)
          reinterpret_cast<uint32_t*>(scales)[c / kGroup] = sbyte | (b1 << 8) | (b2 << 16) | (b3 << 24);
      } else if ((c % LPB) == 0) {
        scales[c / LPB] = (uint8_t)sbyte;
      }
    }
    return;
  }
  if (valid) {
    reinterpret_cast<uint32_t*>(codes)[c] = packed;
    if ((c % LPB) == 0) scales[c / LPB] = (uint8_t)sbyte;
  }
}

// NVFP4 nearest (RULE even or away) and round-toward-zero re-quantisation
// of one whole 16-weight block per lane (its two chunks of 8, already
// loaded), the same arithmetic as rtn_chunk: the block's amax, scale byte,
// block scale and its reciprocal are taken once per block instead of once in
// each of the block's two lanes, and the amax needs no shuffle.  NVFAST as in
// rtn_chunk.  blk is the block index within the weight (codes at byte 8 blk,
// the scale at byte blk).  pack_below > 0: the lanes hold consecutive blocks
// from a multiple of 64 on and the scale plane is 4-byte aligned; blocks
// below pack_below are whole groups of four, whose scale bytes leave as one
// 4-byte store from the group's first lane (every lane of the wave must take
// part: the bytes cross lanes).
// tab[2 b], tab[2 b + 1] hold fp32(e4m3(b) * ws2) and its correctly rounded
// reciprocal for every non-negative scale byte b (the caller's per-workgroup
// table).
template <int RULE, int NVFAST>
__device__ __forceinline__ void rtn_block16_nv(const uint4 lo, const uint4 hi, int64_t blk, bool valid,
                                               const RcpDivisor& wd, const __attribute__((address_space(3))) float* tab,
                                               uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                               int64_t pack_below) {
  static_assert(RULE == kRuleEven || RULE == kRuleAway || RULE == kRuleRtz, "nearest and toward-zero rules");
  const uint32_t h[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
  // the amax on bit patterns, two bf16 magnitudes per packed 16-bit max
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 m2 = {0, 0};
#pragma unroll
  for (int k = 0; k < 8; ++k) m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(u16x2, h[k] & 0x7FFF7FFFu));
  const uint32_t am = max((uint32_t)m2[0], (uint32_t)m2[1]);
  const float amax = __uint_as_float(am << 16);
  const float sixth = amax >= 0x1p-120f ? div_exact<1>(amax, RcpDivisor{6.0f, 0x1.555556p-3f, true})
                                        : __fdiv_rn(amax, 6.0f);
  const uint32_t sbyte = e4m3_encode_rne_sat(div_exact<NVFAST>(sixth, wd));
  const uint32_t ti = 2u * (sbyte & 127u);          // sbyte <= 0x7F: sixth / ws2 is never negative
  const float eff = tab[ti];
  RcpDivisor ed;
  ed.d = eff;
  ed.r = tab[ti + 1];
  ed.fast = eff >= 0x1p-64f && eff <= 0x1p64f;
  auto weight = [&](int k) { return __uint_as_float(((h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu) << 16); };
  float q[16];
  // fast: codes from the products (below); tie: ties away from zero found
  // there, one per code nibble
  bool fast = false;
  uint32_t tie[2] = {0u, 0u};
  if (NVFAST == 1 && eff != 0.0f && amax <= __fmul_rn(eff, 0x1p100f)) {
    // q0 = RN(w r) with r = RN(1 / eff) is w / eff (1 + e1)(1 + e2), |e1|, |e2|
    // <= 2^-24, so q0 and RN(w / eff) lie within 3 float steps of each other
    // (2^-23 |w / eff| is at most 2 steps of the binade, 4 just below a power
    // of two, where the steps halve, and the exact quotient adds half a
    // step).  Every value at which an E2M1 code changes under the three rules
    // (rounding boundaries 0.25, 0.75, ..., 5 and grid points 0.5, 1, ..., 6)
    // has a significand with at most two fraction bits: its bit pattern is a
    // multiple of 2^21.  When q0 lies more than 3 steps from every such
    // pattern, no such value lies between q0 and the exact quotient, and the
    // code taken from q0 is the exact quotient's under each rule (the sign
    // too: r > 0).  A block scale that is a power of two has an exact
    // reciprocal, and q0 is then the exact quotient.  Otherwise each weight
    // whose q0 falls in the window is corrected, in a branch the wave takes
    // only when one of its lanes needs it (with ws2 = fp32(1 / 448), weights
    // and scales that share an odd factor put about 1 quotient in 150 on a
    // tie).  Ties away from zero keep the window there too: an exact quotient
    // can sit on a midpoint, and a midpoint lies in the window, so the
    // midpoint test runs in the window's branch only.
    const bool pow2 = (__float_as_uint(eff) & 0x7FFFFFu) == 0u;
    uint32_t lim = RULE != kRuleAway && pow2 ? 0u : (7u << 11);
    asm("" : "+v"(lim));   // one register compare per weight, not a scale test and a constant compare
    fast = true;
#pragma unroll
    for (int k = 0; k < 16; ++k) q[k] = __fmul_rn(weight(k), ed.r);
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      // ((bits + 3) mod 2^21) << 11 in one instruction with inline operands
      uint32_t dk;
      asm("v_add_lshl_u32 %0, %1, 3, 11" : "=v"(dk) : "v"(__float_as_uint(q[k])));
      if (__builtin_amdgcn_ballot_w64(dk < lim) != 0) {
        asm volatile("" ::: "memory");   // keeps the branch (no speculation of its body)
        // Markstein's correction, twice: q1 is faithful, q2 = RN(w / eff)
        const float w = weight(k);
        const float q0 = q[k];
        const float q1 = __builtin_fmaf(__builtin_fmaf(-q0, ed.d, w), ed.r, q0);
        const float q2 = __builtin_fmaf(__builtin_fmaf(-q1, ed.d, w), ed.r, q1);
        q[k] = dk < lim ? __builtin_copysignf(q2, w) : q0;
        if (RULE == kRuleAway) {
          const float a = fabsf(q[k]);
          tie[k >> 3] |= (a == 0.25f || a == 1.25f || a == 2.5f || a == 5.0f) ? (1u << (4 * (k & 7))) : 0u;
        }
      }
    }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k) q[k] = (eff == 0.0f) ? 0.0f : div_exact<NVFAST>(weight(k), ed);
  }
  uint32_t packed[2];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {                // byte-selected converts, as in rtn_chunk
    uint32_t w = 0;
    if (RULE == kRuleRtz) {
#pragma unroll
      for (int k = 0; k < 8; ++k) w |= e2m1_rtz_code(q[8 * hf + k]) << (4 * k);
    } else {
      w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, q[8 * hf + 0], q[8 * hf + 1], 1.0f, 0);
      w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, q[8 * hf + 2], q[8 * hf + 3], 1.0f, 1);
      w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, q[8 * hf + 4], q[8 * hf + 5], 1.0f, 2);
      w = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(w, q[8 * hf + 6], q[8 * hf + 7], 1.0f, 3);
    }
    packed[hf] = w;
  }
  // ties away from zero take the next magnitude (a tie magnitude is below 6:
  // no carry out of the nibble)
  if (RULE == kRuleAway) {
    if (fast) {
      packed[0] += tie[0];
      packed[1] += tie[1];
    } else {
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float a = fabsf(q[k]);
        packed[k >> 3] += (a == 0.25f || a == 1.25f || a == 2.5f || a == 5.0f) ? (1u << (4 * (k & 7))) : 0u;
      }
    }
  }
  if (am > 0x7F80u || eff == 0.0f) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const uint32_t hb = (h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
      const uint32_t mag = (q[k] != q[k]) ? 0u : ((packed[k >> 3] >> (4 * (k & 7))) & 7u);
      packed[k >> 3] = (packed[k >> 3] & ~(15u << (4 * (k & 7)))) | ((mag | ((hb >> 12) & 8u)) << (4 * (k & 7)));
    }
  }
  uint32_t* c32 = reinterpret_cast<uint32_t*>(codes);
  if (pack_below > 0) {
    // lanes 1, 2, 3 of each quad to its lane 0 (DPP quad permutations)
    const uint32_t b1 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)sbyte, 0x55, 0xF, 0xF, false);
    const uint32_t b2 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)sbyte, 0xAA, 0xF, 0xF, false);
    const uint32_t b3 = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)sbyte, 0xFF, 0xF, 0xF, false);
    if (valid) {
      __builtin_nontemporal_store(packed[0], c32 + 2 * blk);
      __builtin_nontemporal_store(packed[1], c32 + 2 * blk + 1);
      if (blk < pack_below) {
        if ((blk & 3) == 0) reinterpret_cast<uint32_t*>(scales)[blk >> 2] = sbyte | (b1 << 8) | (b2 << 16) | (b3 << 24);
      } else {
        scales[blk] = (uint8_t)sbyte;
      }
    }
    return;
  }
  if (valid) {
    c32[2 * blk] = packed[0];
    c32[2 * blk + 1] = packed[1];
    scales[blk] = (uint8_t)sbyte;
  }
}

}  // namespace sq
