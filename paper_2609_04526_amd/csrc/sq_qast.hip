// One QAST low-rank scale step on gfx950 (paper Section 3, "Scale-QLoRA
// forward" and "QAST makes merge exact by construction"; stability recipe
// items (ii)-(iii)).
//
//   Delta_S = (alpha/r) B A            B bf16 [O, r], A bf16 [r, G]
//   eff'    = eff + Delta_S            rounded onto the grid by grid_update,
//                                      the same function the merge uses
//   dB = (alpha/r) (dS * m) A^T        m = 0 where the NVFP4 ceiling clamp bound
//   dA = (alpha/r) B^T (dS * m)
//
// Delta_S adds the r rank-one terms in increasing k in fp32; each product of
// two bf16 values is exact in fp32, so the fused multiply-add below rounds
// exactly like a separate multiply and add, and the scale bytes are fixed bit
// for bit.  The factor gradients accumulate in fp32 in a fixed order (lanes,
// then a butterfly; row chunks, then chunk index order): deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"
#include "sq_launch.h"

namespace sq {

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// ------------------------------------------------------------------ scales
// A wave per row o, 4 consecutive blocks per lane (256 per wave).
template <int FMT>
__global__ __launch_bounds__(256) void qast_scales_kernel(const uint8_t* __restrict__ base,
                                                          const uint16_t* __restrict__ B,
                                                          const uint16_t* __restrict__ A, int O, int G, int r,
                                                          float c, float ws2, uint8_t* out, uint8_t* mask) {
  // 1-D grid: block = (row group of 4) * gchunks + chunk of 256 blocks
  const int gchunks = (G + 255) / 256;
  const int o = (int)(blockIdx.x / gchunks) * 4 + (threadIdx.x >> 6);
  if (o >= O) return;
  const int g0 = (int)(blockIdx.x % gchunks) * 256 + (threadIdx.x & 63) * 4;
  if (g0 >= G) return;
  float acc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int k = 0; k < r; ++k) {
    const float bk = bf16_bits_to_f32(B[(size_t)o * r + k]);
    const uint16_t* ak = A + (size_t)k * G;
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (g0 + j < G) acc[j] = __builtin_fmaf(bk, bf16_bits_to_f32(ak[g0 + j]), acc[j]);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int g = g0 + j;
    if (g >= G) continue;
    const size_t at = (size_t)o * G + g;
    bool clamped;
    const uint32_t nb = grid_update<FMT>(base[at], __fmul_rn(acc[j], c), ws2, clamped);
    out[at] = (uint8_t)nb;
    if (mask) mask[at] = clamped ? 0 : 1;
  }
}

// ------------------------------------------------------------------ dB
// A wave per row o: lanes stride over the blocks, then a butterfly sum.
template <int RMAX>
__global__ __launch_bounds__(256) void qast_db_kernel(const float* __restrict__ dS, const uint8_t* __restrict__ mask,
                                                      const uint16_t* __restrict__ A, int O, int G, int r, float c,
                                                      float* __restrict__ dB) {
  const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (o >= O) return;
  const int lane = threadIdx.x & 63;
  float acc[RMAX];
#pragma unroll
  for (int k = 0; k < RMAX; ++k) acc[k] = 0.0f;
  for (int g = lane; g < G; g += 64) {
    const size_t at = (size_t)o * G + g;
    const float v = mask ? dS[at] * (float)mask[at] : dS[at];
#pragma unroll
    for (int k = 0; k < RMAX; ++k)
      if (k < r) acc[k] = __builtin_fmaf(v, bf16_bits_to_f32(A[(size_t)k * G + g]), acc[k]);
  }
  float mine = 0.0f;
#pragma unroll
  for (int k = 0; k < RMAX; ++k) {
    if (k >= r) continue;
    float s = acc[k];
#pragma unroll
    for (int w = 32; w >= 1; w >>= 1) s += __shfl_xor(s, w);
    if (lane == k) mine = s;
  }
  if (lane < r) dB[(size_t)o * r + lane] = __fmul_rn(mine, c);
}

// ------------------------------------------------------------------ dA
// Partial dA over a chunk of kDaRows rows: lanes over blocks, each of the 4
// waves over a quarter of the rows in order, the waves added in order.
constexpr int kDaRows = 64;
template <int RMAX>
__global__ __launch_bounds__(256) void qast_da_partial_kernel(const float* __restrict__ dS,
                                                              const uint8_t* __restrict__ mask,
                                                              const uint16_t* __restrict__ B, int O, int G, int r,
                                                              float* __restrict__ part) {
  __shared__ float red[4][RMAX][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int gchunks = (G + 63) / 64;
  const int g = (int)(blockIdx.x % gchunks) * 64 + lane;
  const int chunk = (int)(blockIdx.x / gchunks);
  float acc[RMAX];
#pragma unroll
  for (int k = 0; k < RMAX; ++k) acc[k] = 0.0f;
  const int o_begin = chunk * kDaRows + wave * (kDaRows / 4);
  const int o_end = min(o_begin + kDaRows / 4, O);
  if (g < G) {
    for (int o = o_begin; o < o_end; ++o) {
      const size_t at = (size_t)o * G + g;
      const float v = mask ? dS[at] * (float)mask[at] : dS[at];
#pragma unroll
      for (int k = 0; k < RMAX; ++k)
        if (k < r) acc[k] = __builtin_fmaf(bf16_bits_to_f32(B[(size_t)o * r + k]), v, acc[k]);
    }
  }
#pragma unroll
  for (int k = 0; k < RMAX; ++k) red[wave][k][lane] = acc[k];
  __syncthreads();
  if (g >= G) return;
  // thread (wave, lane) adds the four waves' partials for k = wave, wave+4, ...
  for (int k = wave; k < r; k += 4) {
    const float s = ((red[0][k][lane] + red[1][k][lane]) + red[2][k][lane]) + red[3][k][lane];
    part[((size_t)chunk * r + k) * G + g] = s;
  }
}

__global__ __launch_bounds__(256) void qast_da_reduce_kernel(const float* __restrict__ part, int chunks, int r,
                                                             int G, float c, float* __restrict__ dA) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = (int64_t)r * G;
  if (i >= n) return;
  float s = part[i];
  for (int ch = 1; ch < chunks; ++ch) s += part[(size_t)ch * n + i];
  dA[i] = __fmul_rn(s, c);
}

// ------------------------------------------------------------------ launch
int qast_scales_launch(int fmt, int O, int G, int r, const uint8_t* base, const void* B, const void* A,
                       float c, float ws2, uint8_t* out, uint8_t* mask, hipStream_t s) {
  const dim3 grid((unsigned)(((G + 255) / 256) * (int64_t)((O + 3) / 4)));
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  if (fmt == kMX)
    hipLaunchKernelGGL(qast_scales_kernel<kMX>, grid, dim3(256), 0, s, base, b, a, O, G, r, c, ws2, out, mask);
  else
    hipLaunchKernelGGL(qast_scales_kernel<kNV>, grid, dim3(256), 0, s, base, b, a, O, G, r, c, ws2, out, mask);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

size_t qast_grads_workspace(int O, int G, int r) {
  return (size_t)((O + kDaRows - 1) / kDaRows) * r * G * sizeof(float);
}

template <int RMAX>
static void qast_grads_r(int O, int G, int r, const float* dS, const uint8_t* mask, const uint16_t* B,
                         const uint16_t* A, float c, float* dB, float* dA, float* part, hipStream_t s) {
  hipLaunchKernelGGL(qast_db_kernel<RMAX>, dim3((unsigned)((O + 3) / 4)), dim3(256), 0, s, dS, mask, A, O, G, r, c, dB);
  const int chunks = (O + kDaRows - 1) / kDaRows;
  hipLaunchKernelGGL(qast_da_partial_kernel<RMAX>, dim3((unsigned)(((G + 63) / 64) * (int64_t)chunks)), dim3(256), 0, s,
                     dS, mask, B, O, G, r, part);
  const int64_t n = (int64_t)r * G;
  hipLaunchKernelGGL(qast_da_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, part, chunks, r, G, c,
                     dA);
}

int qast_grads_launch(int O, int G, int r, const float* dS, const uint8_t* mask, const void* B, const void* A,
                      float c, float* dB, float* dA, void* workspace, hipStream_t s) {
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  float* part = static_cast<float*>(workspace);
  if (r <= 16) qast_grads_r<16>(O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  else if (r <= 32) qast_grads_r<32>(O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  else qast_grads_r<64>(O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
