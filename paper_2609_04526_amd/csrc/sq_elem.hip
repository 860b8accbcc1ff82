// Bandwidth-bound kernels of the frozen-code FP4 layer on gfx950:
//   * the scale-plane merge / swap (paper Section 3, "QAST makes merge exact
//     by construction" and stability recipe items (ii)-(iii); Appendix B
//     "Payoff 2" hot swap), which reads and writes scale bytes only;
//   * round-to-nearest re-quantisation of a bf16 weight (Section 2, "The naive
//     re-quantized merge is the failure mode"), the baseline that rewrites
//     every code.
// Every fp32 step is an explicitly correctly rounded operation (__fmul_rn,
// __fadd_rn, __fdiv_rn); fp32 subnormals are kept (E8M0 2^-127 is one).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"
#include "sq_launch.h"

namespace sq {

// ------------------------------------------------------------------ merge
// The planes of a launch are cut into spans: kDeltaSpan scale bytes (delta
// mode: kDeltaSteps steps of 4 scales and a 16-byte fp32 delta per lane) or
// kCopySpan bytes (copy mode: kCopySteps steps of 16 bytes per lane).  Workgroup w takes spans w, w + grid,
// w + 2 grid, ...: at any moment the whole grid streams through one window of
// the planes, which keeps the DRAM accesses of all workgroups together (a
// workgroup walking a private region of its own streams markedly slower).
// Consecutive lanes touch consecutive 4-byte scale words and 16-byte delta
// words; delta and copy sources are read once, with streaming loads.  The
// plane pointers are restrict: a scale store cannot alias a later load.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// One delta span: kDeltaSteps steps of 4 scales per lane, all loads issued
// before any compute.
template <int FMT>
__device__ __forceinline__ void merge_delta_span(uint8_t* __restrict__ sc, const float* __restrict__ dl, int64_t n,
                                                 int64_t off, float ws2, int tid) {
  if (off + kDeltaSpan <= n) {
    uint32_t sv[kDeltaSteps];
    f32x4_t dv[kDeltaSteps];
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g) {
      const int64_t i = off + g * 1024 + tid * 4;
      sv[g] = *reinterpret_cast<const uint32_t*>(sc + i);
      dv[g] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(dl + i));
    }
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g) {
      const uint32_t v = sv[g];
      sv[g] = merge_one_t<FMT>(v & 0xFFu, dv[g][0], ws2) | (merge_one_t<FMT>((v >> 8) & 0xFFu, dv[g][1], ws2) << 8) |
              (merge_one_t<FMT>((v >> 16) & 0xFFu, dv[g][2], ws2) << 16) |
              (merge_one_t<FMT>(v >> 24, dv[g][3], ws2) << 24);
    }
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g) *reinterpret_cast<uint32_t*>(sc + off + g * 1024 + tid * 4) = sv[g];
  } else {
    for (int64_t k = off + tid; k < n && k < off + kDeltaSpan; k += 256)
      sc[k] = (uint8_t)merge_one_t<FMT>(sc[k], dl[k], ws2);
  }
}

// One copy span: kCopySteps steps of 16 bytes per lane, loads first.
__device__ __forceinline__ void merge_copy_span(uint8_t* __restrict__ sc, const uint8_t* __restrict__ sr, int64_t n,
                                                int64_t off, int tid) {
  if (off + kCopySpan <= n) {
    u32x4_t v[kCopySteps];
#pragma unroll
    for (int g = 0; g < kCopySteps; ++g)
      v[g] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(sr + off + g * 4096 + tid * 16));
#pragma unroll
    for (int g = 0; g < kCopySteps; ++g) *reinterpret_cast<u32x4_t*>(sc + off + g * 4096 + tid * 16) = v[g];
  } else {
    for (int64_t k = off + tid; k < n && k < off + kCopySpan; k += 256) sc[k] = sr[k];
  }
}

__global__ __launch_bounds__(256) void merge_kernel(MergeBatch batch_arg) {
  (void)batch_arg;
  // The batch is the kernel's only explicit argument, so it sits at offset 0
  // of the kernarg segment; reading it there (constant address space) keeps
  // the workgroup-uniform plane data in scalar registers.
  const __attribute__((address_space(4))) MergeBatch& batch =
      *(const __attribute__((address_space(4))) MergeBatch*)__builtin_amdgcn_kernarg_segment_ptr();
  const int tid = threadIdx.x;
  int pi = 0;
  for (int span = blockIdx.x; span < batch.spans; span += gridDim.x) {
    // spans only grow, so the plane index only moves forward
    while (pi + 1 < batch.count && batch.span_begin[pi + 1] <= span) ++pi;
    uint8_t* __restrict__ sc = batch.scales[pi];
    const int64_t n = batch.n[pi];
    const int64_t rel = span - batch.span_begin[pi];
    if (batch.mode[pi] == 1) {                                // copy
      merge_copy_span(sc, static_cast<const uint8_t*>(batch.aux[pi]), n, rel * kCopySpan, tid);
    } else {
      const float* __restrict__ dl = static_cast<const float*>(batch.aux[pi]);
      if (batch.fmt[pi] == kNV)
        merge_delta_span<kNV>(sc, dl, n, rel * kDeltaSpan, batch.ws2[pi], tid);
      else
        merge_delta_span<kMX>(sc, dl, n, rel * kDeltaSpan, batch.ws2[pi], tid);
    }
  }
}

int merge_launch(const MergeBatch& b, hipStream_t s) {
  if (b.spans <= 0) return 0;
  // Measured on the 8B model's planes (medians of interleaved runs): copies
  // stream best from 2048 workgroups, MXFP4 deltas from 4096, and NVFP4
  // deltas, whose division keeps more lanes busy, from 8192.
  const int64_t cap = b.copy_only ? 2048 : (b.nv_delta ? 8192 : 4096);
  const int64_t grid = b.spans < cap ? b.spans : cap;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)grid), dim3(256), 0, s, b);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ------------------------------------------------------------------ RTN
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
template <int FMT, int RULE>
__device__ __forceinline__ void rtn_chunk(const uint4 v, int64_t c, bool valid, const float* ws2_ptr, float ws2_val,
                                          const float* amax_t, uint64_t seed,
                                          uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
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
  const float sixth = __fdiv_rn(amax, 6.0f);

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
    float ws2 = ws2_ptr ? *ws2_ptr : ws2_val;
    if (RULE == kRuleWholeTensor && !(ws2_val > 0.0f)) {    // recomputed from the same amax
      ws2 = __fdiv_rn(sixth, 448.0f);
      if (ws2 == 0.0f) ws2 = 1.0f;
    }
    sbyte = e4m3_encode_rne_sat(__fdiv_rn(sixth, ws2));
    eff = __fmul_rn(e4m3_to_f32(sbyte), ws2);
  }

  // Codes: gfx950's fp32 -> E2M1 convert rounds |q| to the nearest E2M1
  // magnitude with ties to even and saturates at 6 (it equals the threshold
  // rounding on every non-NaN fp32 input); ties away differ from it exactly at
  // |q| = 0.25, 1.25, 2.5 and 5, where they take the next magnitude.  A NaN q
  // codes as magnitude 0, and the sign bit is always the sign of w.
  float q[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const float w = __uint_as_float(((h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu) << 16);
    if (FMT == kMX) q[k] = __fmul_rn(w, eff);               // w / 2^k, one rounding
    else q[k] = (eff == 0.0f) ? 0.0f : __fdiv_rn(w, eff);
  }
  uint32_t packed = 0;
#pragma unroll
  for (int p = 0; p < 4; ++p)
    packed |= (__builtin_amdgcn_cvt_scalef32_pk_fp4_f32(0u, q[2 * p], q[2 * p + 1], 1.0f, 0) & 0xFFu) << (8 * p);
  if (RULE == kRuleAway) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {                           // a tie magnitude is below 6: no carry
      const float a = fabsf(q[k]);
      packed += (a == 0.25f || a == 1.25f || a == 2.5f || a == 5.0f) ? (1u << (4 * k)) : 0u;
    }
  }
  if (RULE == kRuleRtz || RULE == kRuleStochastic) {
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
  if (valid) {
    reinterpret_cast<uint32_t*>(codes)[c] = packed;
    if ((c % LPB) == 0) scales[c / LPB] = (uint8_t)sbyte;
  }
}

// Each workgroup takes 512 chunks: a lane loads its two chunks (c and c + 256)
// before working on either, so two 16-byte loads are in flight per lane.
template <int FMT, int RULE>
__global__ __launch_bounds__(256) void rtn_kernel(const uint16_t* __restrict__ W, int64_t n_chunks,
                                                  const float* ws2_ptr, float ws2_val, const float* amax_t,
                                                  uint64_t seed, uint8_t* __restrict__ codes,
                                                  uint8_t* __restrict__ scales) {
  const int64_t c0 = (int64_t)blockIdx.x * 512 + threadIdx.x, c1 = c0 + 256;
  const bool ok0 = c0 < n_chunks, ok1 = c1 < n_chunks;
  const uint4 v0 = ok0 ? *reinterpret_cast<const uint4*>(W + 8 * c0) : make_uint4(0, 0, 0, 0);
  const uint4 v1 = ok1 ? *reinterpret_cast<const uint4*>(W + 8 * c1) : make_uint4(0, 0, 0, 0);
  rtn_chunk<FMT, RULE>(v0, c0, ok0, ws2_ptr, ws2_val, amax_t, seed, codes, scales);
  rtn_chunk<FMT, RULE>(v1, c1, ok1, ws2_ptr, ws2_val, amax_t, seed, codes, scales);
}

__global__ void rtn_amax_init(float* slot) { *reinterpret_cast<uint32_t*>(slot) = 0u; }

// Tensor amax (as bf16 bits) for the recomputed ws2: 4 loads in flight per
// lane, one integer atomicMax per workgroup (a max of bit patterns is
// order-independent, so the result is deterministic).
__global__ __launch_bounds__(256) void rtn_amax(const uint16_t* __restrict__ W, int64_t n_chunks, float* slot) {
  __shared__ uint32_t red[4];
  uint32_t am = 0;
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; c + 3 * stride < n_chunks; c += 4 * stride) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const uint4*>(W + 8 * (c + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const uint32_t h[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) am = max(am, max(h[k] & 0x7FFFu, (h[k] >> 16) & 0x7FFFu));
    }
  }
  for (; c < n_chunks; c += stride) {
    const uint4 v = *reinterpret_cast<const uint4*>(W + 8 * c);
    const uint32_t h[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) am = max(am, max(h[k] & 0x7FFFu, (h[k] >> 16) & 0x7FFFu));
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) am = max(am, (uint32_t)__shfl_xor((int)am, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = am;
  __syncthreads();
  if (threadIdx.x == 0)
    atomicMax(reinterpret_cast<unsigned int*>(slot), max(max(red[0], red[1]), max(red[2], red[3])) << 16);
}

__global__ void rtn_ws2_store(float* slot, float v) { *slot = v; }

__global__ void rtn_ws2_finalize(float* slot) {
  const float amax = *slot;
  float ws2 = __fdiv_rn(__fdiv_rn(amax, 6.0f), 448.0f);
  if (ws2 == 0.0f) ws2 = 1.0f;
  *slot = ws2;
}

namespace {
template <int FMT, int RULE>
void rtn_grid(int64_t n_chunks, const uint16_t* w, const float* ws2_ptr, float ws2_val, const float* amax_t,
              uint64_t seed, uint8_t* codes, uint8_t* scales, hipStream_t s) {
  if (n_chunks <= 0) return;
  const unsigned grid = (unsigned)((n_chunks + 511) / 512);
  hipLaunchKernelGGL((rtn_kernel<FMT, RULE>), dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_ptr, ws2_val, amax_t,
                     seed, codes, scales);
}

template <int RULE>
void rtn_fmt(int fmt, int64_t n_chunks, const uint16_t* w, const float* ws2_ptr, float ws2_val, const float* amax_t,
             uint64_t seed, uint8_t* codes, uint8_t* scales, hipStream_t s) {
  if (fmt == kMX) rtn_grid<kMX, RULE>(n_chunks, w, ws2_ptr, 1.0f, amax_t, seed, codes, scales, s);
  else rtn_grid<kNV, RULE>(n_chunks, w, ws2_ptr, ws2_val, amax_t, seed, codes, scales, s);
}

// The tensor amax (as the bits of an fp32 holding a bf16 value) into *slot.
void tensor_amax(const uint16_t* w, int64_t n_chunks, float* slot, hipStream_t s) {
  hipLaunchKernelGGL(rtn_amax_init, dim3(1), dim3(1), 0, s, slot);
  const int64_t want = (n_chunks + 1023) / 1024;
  const unsigned grid = (unsigned)(want < 1024 ? (want > 0 ? want : 1) : 1024);
  hipLaunchKernelGGL(rtn_amax, dim3(grid), dim3(256), 0, s, w, n_chunks, slot);
}
}  // namespace

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s) {
  return rtn_rule_launch(fmt, O, I, W, ws2_in, tie == 1 ? kRuleAway : kRuleEven, 0, codes, scales, ws2_out, s);
}

int rtn_rule_launch(int fmt, int O, int I, const void* W, float ws2_in, int rule, uint64_t seed,
                    uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s) {
  const int64_t n_chunks = (int64_t)O * I / 8;
  const uint16_t* w = static_cast<const uint16_t*>(W);
  if (rule == kRuleWholeTensor) {
    // ws2_out holds the tensor amax while the codes are written, then the
    // ws2 used (1 for MXFP4); the launches are stream-ordered.
    tensor_amax(w, n_chunks, ws2_out, s);
    rtn_fmt<kRuleWholeTensor>(fmt, n_chunks, w, nullptr, fmt == kNV && ws2_in > 0.0f ? ws2_in : 0.0f, ws2_out,
                              seed, codes, scales, s);
    if (fmt == kNV && !(ws2_in > 0.0f)) hipLaunchKernelGGL(rtn_ws2_finalize, dim3(1), dim3(1), 0, s, ws2_out);
    else hipLaunchKernelGGL(rtn_ws2_store, dim3(1), dim3(1), 0, s, ws2_out, fmt == kNV ? ws2_in : 1.0f);
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }
  const float* ws2_ptr = nullptr;
  if (fmt == kNV) {
    if (ws2_in > 0.0f) {
      if (ws2_out) hipLaunchKernelGGL(rtn_ws2_store, dim3(1), dim3(1), 0, s, ws2_out, ws2_in);
    } else {
      tensor_amax(w, n_chunks, ws2_out, s);
      hipLaunchKernelGGL(rtn_ws2_finalize, dim3(1), dim3(1), 0, s, ws2_out);
      ws2_ptr = ws2_out;
    }
  }
  switch (rule) {
    case kRuleEven: rtn_fmt<kRuleEven>(fmt, n_chunks, w, ws2_ptr, ws2_in, nullptr, seed, codes, scales, s); break;
    case kRuleAway: rtn_fmt<kRuleAway>(fmt, n_chunks, w, ws2_ptr, ws2_in, nullptr, seed, codes, scales, s); break;
    case kRuleRtz: rtn_fmt<kRuleRtz>(fmt, n_chunks, w, ws2_ptr, ws2_in, nullptr, seed, codes, scales, s); break;
    case kRuleStochastic:
      rtn_fmt<kRuleStochastic>(fmt, n_chunks, w, ws2_ptr, ws2_in, nullptr, seed, codes, scales, s);
      break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
