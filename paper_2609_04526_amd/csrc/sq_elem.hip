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

// E2M1 magnitude index (0..7 for 0,.5,1,1.5,2,3,4,6) of |q| with ties to the
// even mantissa or away from zero; >= 6 saturates, NaN gives 0.
template <bool AWAY>
__device__ __forceinline__ uint32_t e2m1_round_index(float a) {
  uint32_t i = 0;
  if (AWAY) {
    i += (a >= 0.25f); i += (a >= 0.75f); i += (a >= 1.25f); i += (a >= 1.75f);
    i += (a >= 2.5f);  i += (a >= 3.5f);  i += (a >= 5.0f);
  } else {
    // a tie goes to whichever neighbour has an even index: 0.25->0, 0.75->1.0,
    // 1.25->1.0, 1.75->2.0, 2.5->2.0, 3.5->4.0, 5->4.0
    i += (a > 0.25f); i += (a >= 0.75f); i += (a > 1.25f); i += (a >= 1.75f);
    i += (a > 2.5f);  i += (a >= 3.5f);  i += (a > 5.0f);
  }
  return i;
}

// ------------------------------------------------------------------ merge
// One workgroup per batch.chunk scale bytes of one plane (a multiple of
// kMergeUnit, chosen per launch so the grid fills the chip).  In each pass a
// lane issues all of its loads before computing (the plane pointers are
// restrict: a scale store cannot alias a later load); consecutive lanes touch
// consecutive 4-byte scale words and 16-byte delta words; delta and copy
// sources are read once, with streaming (non-temporal) loads.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#ifndef SQ_MERGE_PASS
#define SQ_MERGE_PASS 8
#endif
// Delta merge of the scale bytes [base, end) of one plane, in
// passes of SQ_MERGE_PASS steps of 4 scales per lane: all loads of a pass are issued before
// any compute.
template <int FMT>
__device__ __forceinline__ void merge_delta_chunk(uint8_t* __restrict__ sc, const float* __restrict__ dl,
                                                  int64_t n, int64_t base, int64_t end, float ws2, int tid) {
  constexpr int kPass = SQ_MERGE_PASS;
  constexpr int kPassBytes = kPass * 1024;
  for (int64_t b = base; b < end && b < n; b += kPassBytes) {
    if (b + kPassBytes <= n) {
      uint32_t sv[kPass];
      f32x4_t dv[kPass];
#pragma unroll
      for (int g = 0; g < kPass; ++g) {
        const int64_t i = b + g * 1024 + tid * 4;
        sv[g] = *reinterpret_cast<const uint32_t*>(sc + i);
        dv[g] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(dl + i));
      }
#pragma unroll
      for (int g = 0; g < kPass; ++g) {
        const uint32_t s = sv[g];
        sv[g] = merge_one_t<FMT>(s & 0xFFu, dv[g][0], ws2) |
                (merge_one_t<FMT>((s >> 8) & 0xFFu, dv[g][1], ws2) << 8) |
                (merge_one_t<FMT>((s >> 16) & 0xFFu, dv[g][2], ws2) << 16) |
                (merge_one_t<FMT>(s >> 24, dv[g][3], ws2) << 24);
      }
#pragma unroll
      for (int g = 0; g < kPass; ++g)
        *reinterpret_cast<uint32_t*>(sc + b + g * 1024 + tid * 4) = sv[g];
    } else {
      for (int64_t k = b + tid; k < n && k < b + kPassBytes; k += 256)
        sc[k] = (uint8_t)merge_one_t<FMT>(sc[k], dl[k], ws2);
    }
  }
}

__global__ __launch_bounds__(256) void merge_kernel(MergeBatch batch_arg) {
  (void)batch_arg;
  // The batch is the kernel's only explicit argument, so it sits at offset 0
  // of the kernarg segment; reading it there (constant address space) turns a
  // workgroup-uniform plane index into scalar loads instead of a private copy.
  const __attribute__((address_space(4))) MergeBatch& batch =
      *(const __attribute__((address_space(4))) MergeBatch*)__builtin_amdgcn_kernarg_segment_ptr();
  const int chunk = blockIdx.x;
  // plane of this workgroup: the last plane whose first chunk is <= chunk
  // (binary search over the workgroup-uniform chunk_begin array)
  int lo = 0, hi = batch.count - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (batch.chunk_begin[mid] <= chunk) lo = mid;
    else hi = mid - 1;
  }
  const int pi = lo;
  uint8_t* __restrict__ sc = batch.scales[pi];
  const int64_t n = batch.n[pi];
  const int fmt = batch.fmt[pi];
  const float ws2 = batch.ws2[pi];
  const int64_t base = (int64_t)(chunk - batch.chunk_begin[pi]) * batch.chunk;
  const int64_t end = base + batch.chunk;
  const int tid = threadIdx.x;
  if (batch.mode[pi] == 1) {                                  // copy: 16 bytes per lane per step
    constexpr int kCopyPass = kMergeUnit / 4096;
    const uint8_t* __restrict__ sr = static_cast<const uint8_t*>(batch.aux[pi]);
    for (int64_t b = base; b < end && b < n; b += kMergeUnit) {
      if (b + kMergeUnit <= n) {
        u32x4_t v[kCopyPass];
#pragma unroll
        for (int g = 0; g < kCopyPass; ++g)
          v[g] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(sr + b + g * 4096 + tid * 16));
#pragma unroll
        for (int g = 0; g < kCopyPass; ++g) *reinterpret_cast<u32x4_t*>(sc + b + g * 4096 + tid * 16) = v[g];
      } else {
        for (int64_t k = b + tid; k < n && k < b + kMergeUnit; k += 256) sc[k] = sr[k];
      }
    }
    return;
  }
  const float* __restrict__ dl = static_cast<const float*>(batch.aux[pi]);
  if (fmt == kNV)
    merge_delta_chunk<kNV>(sc, dl, n, base, end, ws2, tid);
  else
    merge_delta_chunk<kMX>(sc, dl, n, base, end, ws2, tid);
}

int64_t merge_chunk_for(int64_t total) {
  // about 8 workgroups per CU on 256 CUs, between 1 and 8 units each
  int64_t units = (total + 2048 * (int64_t)kMergeUnit - 1) / (2048 * (int64_t)kMergeUnit);
  units = units < 1 ? 1 : (units > 8 ? 8 : units);
  return units * kMergeUnit;
}

int merge_launch(const MergeBatch& b, int64_t total_chunks, hipStream_t s) {
  if (total_chunks <= 0) return 0;
  hipLaunchKernelGGL(merge_kernel, dim3((unsigned)total_chunks), dim3(256), 0, s, b);
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

// One thread per 8 consecutive weights of a row (16 bytes of bf16); the
// B/8 threads of a block are adjacent lanes and share the block amax.
template <int FMT, bool AWAY>
__global__ __launch_bounds__(256) void rtn_kernel(const uint16_t* __restrict__ W, int64_t n_chunks,
                                                  const float* ws2_ptr, float ws2_val,
                                                  uint8_t* __restrict__ codes, uint8_t* __restrict__ scales) {
  constexpr int B = ScaleOperand<FMT>::kBlock;
  constexpr int LPB = B / 8;
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool valid = c < n_chunks;
  uint4 v = valid ? *reinterpret_cast<const uint4*>(W + 8 * c) : make_uint4(0, 0, 0, 0);
  const uint32_t h[4] = {v.x, v.y, v.z, v.w};
  // amax as a bit pattern: for |x| the integer order of the bits is the
  // numeric order, with NaN above +inf, so NaN propagates like a max.
  uint32_t am = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    am = max(am, h[k] & 0x7FFFu);
    am = max(am, (h[k] >> 16) & 0x7FFFu);
  }
  am = max(am, (uint32_t)__shfl_xor((int)am, 1));
  if (LPB == 4) am = max(am, (uint32_t)__shfl_xor((int)am, 2));
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
    const float ws2 = ws2_ptr ? *ws2_ptr : ws2_val;
    sbyte = e4m3_encode_rne_sat(__fdiv_rn(sixth, ws2));
    eff = __fmul_rn(e4m3_to_f32(sbyte), ws2);
  }

  uint32_t packed = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t hb = (h[k >> 1] >> (16 * (k & 1))) & 0xFFFFu;
    const float w = __uint_as_float(hb << 16);
    float q;
    if (FMT == kMX) q = __fmul_rn(w, eff);                  // w / 2^k, one rounding
    else q = (eff == 0.0f) ? 0.0f : __fdiv_rn(w, eff);
    const uint32_t mag = e2m1_round_index<AWAY>(fabsf(q));
    packed |= (mag | ((hb >> 12) & 8u)) << (4 * k);
  }
  if (valid) {
    reinterpret_cast<uint32_t*>(codes)[c] = packed;
    if ((c % LPB) == 0) scales[c / LPB] = (uint8_t)sbyte;
  }
}

__global__ void rtn_amax_init(float* slot) { *reinterpret_cast<uint32_t*>(slot) = 0u; }

__global__ __launch_bounds__(256) void rtn_amax(const uint16_t* __restrict__ W, int64_t n_chunks, float* slot) {
  uint32_t am = 0;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < n_chunks; c += (int64_t)gridDim.x * 256) {
    const uint4 v = *reinterpret_cast<const uint4*>(W + 8 * c);
    const uint32_t h[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      am = max(am, h[k] & 0x7FFFu);
      am = max(am, (h[k] >> 16) & 0x7FFFu);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) am = max(am, (uint32_t)__shfl_xor((int)am, off));
  if ((threadIdx.x & 63) == 0) atomicMax(reinterpret_cast<unsigned int*>(slot), am << 16);
}

__global__ void rtn_ws2_store(float* slot, float v) { *slot = v; }

__global__ void rtn_ws2_finalize(float* slot) {
  const float amax = *slot;
  float ws2 = __fdiv_rn(__fdiv_rn(amax, 6.0f), 448.0f);
  if (ws2 == 0.0f) ws2 = 1.0f;
  *slot = ws2;
}

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s) {
  const int64_t n_chunks = (int64_t)O * I / 8;
  const uint16_t* w = static_cast<const uint16_t*>(W);
  const float* ws2_ptr = nullptr;
  if (fmt == kNV) {
    if (ws2_in > 0.0f) {
      if (ws2_out) hipLaunchKernelGGL(rtn_ws2_store, dim3(1), dim3(1), 0, s, ws2_out, ws2_in);
    } else {
      hipLaunchKernelGGL(rtn_amax_init, dim3(1), dim3(1), 0, s, ws2_out);
      const int64_t want = (n_chunks + 255) / 256;
      const unsigned grid = (unsigned)(want < 4096 ? (want > 0 ? want : 1) : 4096);
      hipLaunchKernelGGL(rtn_amax, dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_out);
      hipLaunchKernelGGL(rtn_ws2_finalize, dim3(1), dim3(1), 0, s, ws2_out);
      ws2_ptr = ws2_out;
    }
  }
  if (n_chunks > 0) {
    const unsigned grid = (unsigned)((n_chunks + 255) / 256);
    if (fmt == kMX) {
      if (tie == 1) hipLaunchKernelGGL((rtn_kernel<kMX, true>), dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_ptr, 1.0f, codes, scales);
      else hipLaunchKernelGGL((rtn_kernel<kMX, false>), dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_ptr, 1.0f, codes, scales);
    } else {
      if (tie == 1) hipLaunchKernelGGL((rtn_kernel<kNV, true>), dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_ptr, ws2_in, codes, scales);
      else hipLaunchKernelGGL((rtn_kernel<kNV, false>), dim3(grid), dim3(256), 0, s, w, n_chunks, ws2_ptr, ws2_in, codes, scales);
    }
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
