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
// The MoE path stacks E experts (rows e*O .. e*O + O - 1 of every [rows, G]
// or [rows, r] plane; A as [E, r, G]) and runs every expert's step in the
// same launches.
//
// Delta_S adds the r rank-one terms in increasing k in fp32; each product of
// two bf16 values is exact in fp32, so the fused multiply-add below rounds
// exactly like a separate multiply and add, and the scale bytes are fixed bit
// for bit.  The factor gradients accumulate in fp32 in a fixed order (dB: over
// the blocks in order; dA: rows in order within 32-row chunks, then the chunk
// partials through a fixed per-lane order and butterfly): deterministic.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"
#include "sq_launch.h"

namespace sq {

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// ------------------------------------------------------------------ scales
// One thread per scale (o, g), consecutive threads along g: the A reads are
// coalesced and a row's B entries are shared by its threads.
// Experts are stacked: rows e*O .. e*O + O - 1 of base, B, out and mask
// belong to expert e, whose A is A + e*r*G and whose ws2 is ws2[e].
template <int FMT>
__global__ __launch_bounds__(256) void qast_scales_kernel(const uint8_t* __restrict__ base,
                                                          const uint16_t* __restrict__ B,
                                                          const uint16_t* __restrict__ A, int E, int O, int G, int r,
                                                          float c, Ws2Table ws2, uint8_t* out, uint8_t* mask) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)E * O * G) return;
  const int64_t row = idx / G;
  const int g = (int)(idx - row * G);
  const int e = (int)(row / O);
  const uint16_t* brow = B + (size_t)row * r;
  const uint16_t* ae = A + (size_t)e * r * G;
  float acc = 0.0f;
  for (int k = 0; k < r; ++k)
    acc = __builtin_fmaf(bf16_bits_to_f32(brow[k]), bf16_bits_to_f32(ae[(size_t)k * G + g]), acc);
  bool clamped;
  const uint32_t nb = grid_update<FMT>(base[idx], __fmul_rn(acc, c), ws2.v[e], clamped);
  out[idx] = (uint8_t)nb;
  if (mask) mask[idx] = clamped ? 0 : 1;
}

// ------------------------------------------------------------------ dB
// A thread per (o, k): dB[o,k] = c sum_g v[o,g] A[k,g] over g in order, with
// A staged transposed in LDS ([g][k], consecutive k in consecutive lanes) in
// tiles of kDbTile blocks.  RP lanes per row (RP >= r, a power of two),
// 256 / RP rows per workgroup.
constexpr int kDbTile = 256;
template <int RP>
__global__ __launch_bounds__(256) void qast_db_kernel(const float* __restrict__ dS, const uint8_t* __restrict__ mask,
                                                      const uint16_t* __restrict__ A, int O, int G, int r, float c,
                                                      float* __restrict__ dB) {
  __shared__ float at[kDbTile * RP];                     // [g - g0][k]
  const int e = blockIdx.y;                              // expert: its rows, its A
  dS += (size_t)e * O * G;
  if (mask) mask += (size_t)e * O * G;
  A += (size_t)e * r * G;
  dB += (size_t)e * O * r;
  const int k = threadIdx.x % RP;
  const int o = blockIdx.x * (256 / RP) + threadIdx.x / RP;
  const bool active = o < O && k < r;
  const float* vrow = dS + (size_t)(active ? o : 0) * G;
  const uint8_t* mrow = mask ? mask + (size_t)(active ? o : 0) * G : nullptr;
  float acc = 0.0f;
  for (int g0 = 0; g0 < G; g0 += kDbTile) {
    const int gn = min(kDbTile, G - g0);
    __syncthreads();                                     // the previous tile is consumed
    for (int i = threadIdx.x; i < gn * RP; i += 256) {
      const int gi = i / RP, kk = i - gi * RP;
      at[i] = kk < r ? bf16_bits_to_f32(A[(size_t)kk * G + g0 + gi]) : 0.0f;
    }
    __syncthreads();
    if (active) {
      int gi = 0;
      for (; gi + 8 <= gn; gi += 8) {                    // 8 loads in flight, then 8 FMAs in order
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = vrow[g0 + gi + j];
        if (mrow) {
#pragma unroll
          for (int j = 0; j < 8; ++j) v[j] *= (float)mrow[g0 + gi + j];
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) acc = __builtin_fmaf(v[j], at[(gi + j) * RP + k], acc);
      }
      for (; gi < gn; ++gi) {
        const int g = g0 + gi;
        const float v = mrow ? vrow[g] * (float)mrow[g] : vrow[g];
        acc = __builtin_fmaf(v, at[gi * RP + k], acc);
      }
    }
  }
  if (active) dB[(size_t)o * r + k] = __fmul_rn(acc, c);
}

// ------------------------------------------------------------------ dA
// Partial dA over a chunk of kDaRows rows, rows in order: lanes along g, the
// four waves of a workgroup each own a quarter of the ranks (RMAX / 4).
constexpr int kDaRows = 32;
template <int RMAX>
__global__ __launch_bounds__(256) void qast_da_partial_kernel(const float* __restrict__ dS,
                                                              const uint8_t* __restrict__ mask,
                                                              const uint16_t* __restrict__ B, int O, int G, int r,
                                                              float* __restrict__ part) {
  constexpr int KW = RMAX / 4;
  const int e = blockIdx.y;                              // expert: its rows, its partial planes
  dS += (size_t)e * O * G;
  if (mask) mask += (size_t)e * O * G;
  B += (size_t)e * O * r;
  part += (size_t)e * ((O + kDaRows - 1) / kDaRows) * r * G;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int gchunks = (G + 63) / 64;
  const int g = (int)(blockIdx.x % gchunks) * 64 + lane;
  const int chunk = (int)(blockIdx.x / gchunks);
  const int k0 = wave * KW;
  if (g >= G || k0 >= r) return;
  float acc[KW];
#pragma unroll
  for (int j = 0; j < KW; ++j) acc[j] = 0.0f;
  const int o_end = min((chunk + 1) * kDaRows, O);
  int o = chunk * kDaRows;
  for (; o + 8 <= o_end; o += 8) {                       // 8 rows of loads in flight, rows added in order
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = dS[(size_t)(o + u) * G + g];
    if (mask) {
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] *= (float)mask[(size_t)(o + u) * G + g];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint16_t* brow = B + (size_t)(o + u) * r + k0;
#pragma unroll
      for (int j = 0; j < KW; ++j)
        if (k0 + j < r) acc[j] = __builtin_fmaf(bf16_bits_to_f32(brow[j]), v[u], acc[j]);
    }
  }
  for (; o < o_end; ++o) {
    const size_t at = (size_t)o * G + g;
    const float v = mask ? dS[at] * (float)mask[at] : dS[at];
    const uint16_t* brow = B + (size_t)o * r + k0;
#pragma unroll
    for (int j = 0; j < KW; ++j)
      if (k0 + j < r) acc[j] = __builtin_fmaf(bf16_bits_to_f32(brow[j]), v, acc[j]);
  }
#pragma unroll
  for (int j = 0; j < KW; ++j)
    if (k0 + j < r) part[((size_t)chunk * r + k0 + j) * G + g] = acc[j];
}

// dA[i] = c sum over the chunk partials: a wave per output, lane l adds the
// chunks l, l + 64, ... in order, then a fixed butterfly across the lanes.
__global__ __launch_bounds__(256) void qast_da_reduce_kernel(const float* __restrict__ part, int chunks, int r,
                                                             int G, int E, float c, float* __restrict__ dA) {
  const int64_t n = (int64_t)r * G;
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i >= (int64_t)E * n) return;
  const int64_t e = i / n, ie = i - e * n;
  const float* pe = part + (size_t)e * chunks * n;
  const int lane = threadIdx.x & 63;
  float s = 0.0f;
  for (int ch = lane; ch < chunks; ch += 64) s += pe[(size_t)ch * n + ie];
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) s += __shfl_xor(s, w);
  if (lane == 0) dA[i] = __fmul_rn(s, c);
}

// ------------------------------------------------------------------ launch
int qast_scales_launch(int fmt, int E, int O, int G, int r, const uint8_t* base, const void* B, const void* A,
                       float c, const float* ws2, uint8_t* out, uint8_t* mask, hipStream_t s) {
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  for (int e0 = 0; e0 < E; e0 += kWs2TableMax) {          // per-expert ws2 travels by value
    const int m = E - e0 < kWs2TableMax ? E - e0 : kWs2TableMax;
    Ws2Table t;
    for (int e = 0; e < m; ++e) t.v[e] = fmt == kNV ? ws2[e0 + e] : 1.0f;
    const size_t rows0 = (size_t)e0 * O;
    const int64_t n = (int64_t)m * O * G;
    const dim3 grid((unsigned)((n + 255) / 256));
    if (fmt == kMX)
      hipLaunchKernelGGL(qast_scales_kernel<kMX>, grid, dim3(256), 0, s, base + rows0 * G, b + rows0 * r,
                         a + (size_t)e0 * r * G, m, O, G, r, c, t, out + rows0 * G, mask ? mask + rows0 * G : nullptr);
    else
      hipLaunchKernelGGL(qast_scales_kernel<kNV>, grid, dim3(256), 0, s, base + rows0 * G, b + rows0 * r,
                         a + (size_t)e0 * r * G, m, O, G, r, c, t, out + rows0 * G, mask ? mask + rows0 * G : nullptr);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

size_t qast_grads_workspace(int E, int O, int G, int r) {
  return (size_t)E * ((O + kDaRows - 1) / kDaRows) * r * G * sizeof(float);
}

template <int RMAX>
static int qast_grads_r(int E, int O, int G, int r, const float* dS, const uint8_t* mask, const uint16_t* B,
                        const uint16_t* A, float c, float* dB, float* dA, float* part, hipStream_t s) {
  hipLaunchKernelGGL(qast_db_kernel<RMAX>, dim3((unsigned)((O + 256 / RMAX - 1) / (256 / RMAX)), (unsigned)E),
                     dim3(256), 0, s, dS, mask, A, O, G, r, c, dB);
  const int chunks = (O + kDaRows - 1) / kDaRows;
  hipLaunchKernelGGL(qast_da_partial_kernel<RMAX>, dim3((unsigned)(((G + 63) / 64) * (int64_t)chunks), (unsigned)E),
                     dim3(256), 0, s, dS, mask, B, O, G, r, part);
  const int64_t n = (int64_t)E * r * G;
  hipLaunchKernelGGL(qast_da_reduce_kernel, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, s, part, chunks, r, G, E, c,
                     dA);
  return 0;
}

int qast_grads_launch(int E, int O, int G, int r, const float* dS, const uint8_t* mask, const void* B, const void* A,
                      float c, float* dB, float* dA, void* workspace, hipStream_t s) {
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  float* part = static_cast<float*>(workspace);
  int rc;
  if (r <= 8) rc = qast_grads_r<8>(E, O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  else if (r <= 16) rc = qast_grads_r<16>(E, O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  else if (r <= 32) rc = qast_grads_r<32>(E, O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  else rc = qast_grads_r<64>(E, O, G, r, dS, mask, b, a, c, dB, dA, part, s);
  if (rc != 0) return rc;
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
