// Merge rollback and the byte audit on gfx950 (paper Appendix B, "Payoff 3:
// invertible merges and rollback" and "Payoff 5: verifiability").
//
//   applied[i]  = value(after[i]) - value(before[i])      one fp32 subtraction
//   rollback:     b[i] = grid(value(b[i]) - applied[i])    one fp32 subtraction
//   diff:         counts += (differing bytes, differing 4-bit nibbles)
//
// value() is the stored field's own value: the E4M3 value for NVFP4 (the
// per-tensor ws2 is common to both sides and stays out), 2^(b-127) for
// MXFP4.  Two such values within 24 binades differ by an fp32-representable
// amount, so the subtraction is exact and rollback re-encodes the exact base.
// All three stream with the merge's grid-stride order, the whole grid inside
// one window of the planes.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"
#include "sq_launch.h"

namespace sq {

typedef float f32x4a_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4a_t __attribute__((ext_vector_type(4)));

template <int FMT>
__device__ __forceinline__ float field_value(uint32_t b) {
  return FMT == kNV ? e4m3_to_f32(b) : e8m0_to_f32(b);
}
template <int FMT>
__device__ __forceinline__ uint32_t field_encode(float v) {
  return FMT == kNV ? e4m3_encode_rne_sat(v) : e8m0_encode_log(v);
}

// Both kernels take spans of kAuditSteps x 1024 scales: a lane issues all
// kAuditSteps of its 4-scale loads before computing, and workgroup w takes
// spans w, w + grid, ...  Outputs are written with streaming stores, and the
// scale planes of NVFP4 (the larger ones) are read with streaming loads, as
// in the merge.
constexpr int kAuditSteps = 8;
constexpr int64_t kAuditSpan = 1024 * kAuditSteps;

template <int FMT>
__device__ __forceinline__ uint32_t load_scales4(const uint8_t* p) {
  if constexpr (FMT == kNV) return __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(p));
  else return *reinterpret_cast<const uint32_t*>(p);
}

template <int FMT>
__global__ __launch_bounds__(256) void applied_kernel(const uint8_t* __restrict__ before,
                                                      const uint8_t* __restrict__ after, float* __restrict__ applied,
                                                      int64_t n) {
  const int tid = threadIdx.x;
  for (int64_t off = (int64_t)blockIdx.x * kAuditSpan; off < n; off += (int64_t)gridDim.x * kAuditSpan) {
    if (off + kAuditSpan <= n) {
      uint32_t b0[kAuditSteps], b1[kAuditSteps];
#pragma unroll
      for (int g = 0; g < kAuditSteps; ++g) {
        const int64_t i = off + g * 1024 + tid * 4;
        b0[g] = load_scales4<FMT>(before + i);
        b1[g] = load_scales4<FMT>(after + i);
      }
#pragma unroll
      for (int g = 0; g < kAuditSteps; ++g) {
        f32x4a_t d;
#pragma unroll
        for (int k = 0; k < 4; ++k)
          d[k] = __fsub_rn(field_value<FMT>((b1[g] >> (8 * k)) & 0xFFu), field_value<FMT>((b0[g] >> (8 * k)) & 0xFFu));
        __builtin_nontemporal_store(d, reinterpret_cast<f32x4a_t*>(applied + off + g * 1024 + tid * 4));
      }
    } else {
      for (int64_t k = off + tid; k < n && k < off + kAuditSpan; k += 256)
        applied[k] = __fsub_rn(field_value<FMT>(after[k]), field_value<FMT>(before[k]));
    }
  }
}

template <int FMT>
__global__ __launch_bounds__(256) void rollback_kernel(uint8_t* __restrict__ sc, const float* __restrict__ applied,
                                                       int64_t n) {
  const int tid = threadIdx.x;
  for (int64_t off = (int64_t)blockIdx.x * kAuditSpan; off < n; off += (int64_t)gridDim.x * kAuditSpan) {
    if (off + kAuditSpan <= n) {
      uint32_t b[kAuditSteps];
      f32x4a_t d[kAuditSteps];
#pragma unroll
      for (int g = 0; g < kAuditSteps; ++g) {
        const int64_t i = off + g * 1024 + tid * 4;
        b[g] = load_scales4<FMT>(sc + i);
        d[g] = __builtin_nontemporal_load(reinterpret_cast<const f32x4a_t*>(applied + i));
      }
#pragma unroll
      for (int g = 0; g < kAuditSteps; ++g) {
        uint32_t out = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k)
          out |= field_encode<FMT>(__fsub_rn(field_value<FMT>((b[g] >> (8 * k)) & 0xFFu), d[g][k])) << (8 * k);
        __builtin_nontemporal_store(out, reinterpret_cast<uint32_t*>(sc + off + g * 1024 + tid * 4));
      }
    } else {
      for (int64_t k = off + tid; k < n && k < off + kAuditSpan; k += 256)
        sc[k] = (uint8_t)field_encode<FMT>(__fsub_rn(field_value<FMT>(sc[k]), applied[k]));
    }
  }
}

// differing nibbles and bytes of one 32-bit word of a ^ b
__device__ __forceinline__ void diff_word(uint32_t x, uint32_t& bytes, uint32_t& nibbles) {
  const uint32_t y = (x | (x >> 1) | (x >> 2) | (x >> 3)) & 0x11111111u;    // a bit per nonzero nibble
  nibbles += __popc(y);
  bytes += __popc((y | (y >> 4)) & 0x01010101u);
}

__global__ __launch_bounds__(256) void byte_diff_kernel(const uint8_t* __restrict__ a, const uint8_t* __restrict__ b,
                                                        int64_t n, unsigned long long* counts) {
  __shared__ uint32_t red[2][4];
  uint32_t nb = 0, nn = 0;
  const int64_t stride = (int64_t)gridDim.x * 4096;
  int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 16;
  for (; i + 3 * stride + 16 <= n; i += 4 * stride) {      // four 16-byte pairs in flight
    u32x4a_t x[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      x[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4a_t*>(a + i + u * stride)) ^
             __builtin_nontemporal_load(reinterpret_cast<const u32x4a_t*>(b + i + u * stride));
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k) diff_word(x[u][k], nb, nn);
  }
  for (; i < n; i += stride) {
    if (i + 16 <= n) {
      const u32x4a_t x = __builtin_nontemporal_load(reinterpret_cast<const u32x4a_t*>(a + i)) ^
                         __builtin_nontemporal_load(reinterpret_cast<const u32x4a_t*>(b + i));
#pragma unroll
      for (int k = 0; k < 4; ++k) diff_word(x[k], nb, nn);
    } else {
      for (int64_t k = i; k < n; ++k) diff_word((uint32_t)(a[k] ^ b[k]), nb, nn);
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    nb += (uint32_t)__shfl_xor((int)nb, off);
    nn += (uint32_t)__shfl_xor((int)nn, off);
  }
  if ((threadIdx.x & 63) == 0) { red[0][threadIdx.x >> 6] = nb; red[1][threadIdx.x >> 6] = nn; }
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicAdd(&counts[0], (unsigned long long)red[0][0] + red[0][1] + red[0][2] + red[0][3]);
    atomicAdd(&counts[1], (unsigned long long)red[1][0] + red[1][1] + red[1][2] + red[1][3]);
  }
}

static unsigned stream_grid(int64_t n, int64_t per_wg) {
  const int64_t want = (n + per_wg - 1) / per_wg;
  return (unsigned)(want < 4096 ? (want > 0 ? want : 1) : 4096);
}

constexpr int64_t kAuditGrid = 16384;
static unsigned span_grid(int64_t n) {
  const int64_t want = (n + kAuditSpan - 1) / kAuditSpan;
  return (unsigned)(want < kAuditGrid ? want : kAuditGrid);
}

int applied_launch(int fmt, int64_t n, const uint8_t* before, const uint8_t* after, float* applied, hipStream_t s) {
  if (n <= 0) return 0;
  const unsigned g = span_grid(n);
  if (fmt == kMX) hipLaunchKernelGGL(applied_kernel<kMX>, dim3(g), dim3(256), 0, s, before, after, applied, n);
  else hipLaunchKernelGGL(applied_kernel<kNV>, dim3(g), dim3(256), 0, s, before, after, applied, n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int rollback_launch(int fmt, int64_t n, uint8_t* scales, const float* applied, hipStream_t s) {
  if (n <= 0) return 0;
  const unsigned g = span_grid(n);
  if (fmt == kMX) hipLaunchKernelGGL(rollback_kernel<kMX>, dim3(g), dim3(256), 0, s, scales, applied, n);
  else hipLaunchKernelGGL(rollback_kernel<kNV>, dim3(g), dim3(256), 0, s, scales, applied, n);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int byte_diff_launch(int64_t n, const uint8_t* a, const uint8_t* b, uint64_t* counts, hipStream_t s) {
  if (n <= 0) return 0;
  // One workgroup per CU streams best: on the 8B model's planes the audit ran
  // at 3.5 / 4.7 TB/s (MXFP4 / NVFP4) from 4096 workgroups and 5.8-6.0 /
  // 6.7 TB/s from 256, each lane keeping its four 16-byte pairs in flight.
  constexpr int64_t kDiffGrid = 256;
  const int64_t want = (n + 16383) / 16384;
  const unsigned grid = (unsigned)(want < kDiffGrid ? (want > 0 ? want : 1) : kDiffGrid);
  hipLaunchKernelGGL(byte_diff_kernel, dim3(grid), dim3(256), 0, s, a, b, n,
                     reinterpret_cast<unsigned long long*>(counts));
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
