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
// partials through a fixed per-lane order and butterfly): deterministic.  The
// backward kernels stage tiles of dS * m in LDS with all of a tile's loads in
// flight together.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_grid.h"
#include "sq_launch.h"

namespace sq {

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// ------------------------------------------------------------------ scales
// A workgroup per tile of 32 TB rows x 32 blocks of one expert (blockIdx.y):
// the tile's A columns [RMAX][32] and B rows, transposed to [RMAX][32 TB], are
// staged in LDS as fp32 (every load issued together; ranks past r are 0 and
// add exact zeros), and thread (row group, block group) adds the r terms of
// its 4 rows x TB blocks in increasing k, with a 16-byte LDS read of B and a
// TB-wide one of A per 4 TB fused multiply-adds.  TB = 4 where the tiles
// still give every CU two workgroups (the stacked experts of an MoE layer),
// else TB = 1 (one linear: four times the workgroups).  With TB = 4, where
// G % 4 == 0 and the byte planes are 4-byte aligned (vec), a thread's four
// blocks of a row are one 4-byte load and store.  Experts are stacked: rows
// e*O .. e*O + O - 1 of base, B, out and mask belong to expert e, whose A is
// A + e*r*G and whose ws2 is ws2[e].
constexpr int kScCols = 32;
template <int TB>
constexpr int sc_rows() { return 32 * TB; }

template <int FMT, int RMAX, int TB>
__global__ __launch_bounds__(256) void qast_scales_kernel(const uint8_t* __restrict__ base,
                                                          const uint16_t* __restrict__ B,
                                                          const uint16_t* __restrict__ A, int O, int G, int r,
                                                          float c, Ws2Table ws2, uint8_t* out, uint8_t* mask,
                                                          int vec) {
  constexpr int ROWS = sc_rows<TB>();
  constexpr int kAPad = kScCols + 4, kBPad = ROWS + 4;      // rows stay 16-byte aligned
  __shared__ __attribute__((aligned(16))) float at[RMAX][kAPad];
  __shared__ __attribute__((aligned(16))) float bt[RMAX][kBPad];
  const int e = blockIdx.y;
  const size_t rows0 = (size_t)e * O;
  const uint16_t* ae = A + (size_t)e * r * G;
  const int gtiles = (G + kScCols - 1) / kScCols;
  const int o0 = ((int)blockIdx.x / gtiles) * ROWS, g0 = ((int)blockIdx.x % gtiles) * kScCols;
#pragma unroll
  for (int u = 0; u < RMAX * kScCols / 256; ++u) {
    const int i = threadIdx.x + 256 * u, k = i / kScCols, gi = i % kScCols;
    at[k][gi] = (k < r && g0 + gi < G) ? bf16_bits_to_f32(ae[(size_t)k * G + g0 + gi]) : 0.0f;
  }
#pragma unroll
  for (int u = 0; u < ROWS * RMAX / 256; ++u) {
    const int i = threadIdx.x + 256 * u, ro = i / RMAX, k = i % RMAX;
    bt[k][ro] = (k < r && o0 + ro < O) ? bf16_bits_to_f32(B[(rows0 + o0 + ro) * r + k]) : 0.0f;
  }
  __syncthreads();
  const int gq = (threadIdx.x % (kScCols / TB)) * TB, rq = (threadIdx.x / (kScCols / TB)) * 4;
  float acc[4][TB];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int j = 0; j < TB; ++j) acc[q][j] = 0.0f;
#pragma unroll 4
  for (int k = 0; k < RMAX; ++k) {
    float av[TB];
    if constexpr (TB == 4) {
      const float4 a = *reinterpret_cast<const float4*>(&at[k][gq]);
      av[0] = a.x; av[1] = a.y; av[2] = a.z; av[3] = a.w;
    } else {
#pragma unroll
      for (int j = 0; j < TB; ++j) av[j] = at[k][gq + j];
    }
    const float4 b = *reinterpret_cast<const float4*>(&bt[k][rq]);
    const float bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int j = 0; j < TB; ++j) acc[q][j] = __builtin_fmaf(bv[q], av[j], acc[q][j]);
  }
  const int g = g0 + gq;
  if (g >= G) return;
  const Ws2Div wd = make_ws2_div(ws2.v[e]);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int o = o0 + rq + q;
    if (o >= O) break;
    const size_t idx = (rows0 + o) * G + g;
    if (TB == 4 && vec) {                       // blocks g .. g + 3, one word each way
      const uint32_t in = *reinterpret_cast<const uint32_t*>(base + idx);
      uint32_t nw = 0, mw = 0;
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        bool clamped;
        nw |= grid_update<FMT>((in >> (8 * j)) & 0xFFu, __fmul_rn(acc[q][j], c), wd, clamped) << (8 * j);
        mw |= (clamped ? 0u : 1u) << (8 * j);
      }
      *reinterpret_cast<uint32_t*>(out + idx) = nw;
      if (mask) *reinterpret_cast<uint32_t*>(mask + idx) = mw;
    } else {
#pragma unroll
      for (int j = 0; j < TB; ++j) {
        if (g + j >= G) break;
        bool clamped;
        out[idx + j] = (uint8_t)grid_update<FMT>(base[idx + j], __fmul_rn(acc[q][j], c), wd, clamped);
        if (mask) mask[idx + j] = clamped ? 0 : 1;
      }
    }
  }
}

// ------------------------------------------------------------------ dB, dA
// Both backward products stage tiles of v = dS * m (fp32) in LDS with every
// load of the tile issued together, plus the matching factor tile, and give
// each thread a 4 x 4 (dA: 4 x TG) block of outputs.  blockIdx.y is the
// expert (its rows, its A).  dA is summed over 32-row chunks (partials in the
// workspace, then a fixed-order reduction).
constexpr int kDaRows = 32;         // rows per dA chunk

// v = dS * m at blocks g .. g + 3 of row o (G % 4 == 0, dS 16-byte and mask
// 4-byte aligned: one 16-byte and one 4-byte load); zeros past the plane.
__device__ __forceinline__ float4 load_v4(const float* __restrict__ dS, const uint8_t* __restrict__ mask, int O,
                                          int G, int o, int g) {
  float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  if (o < O && g < G) {
    const size_t at_ = (size_t)o * G + g;
    v = *reinterpret_cast<const float4*>(dS + at_);
    if (mask) {
      const uint32_t m = *reinterpret_cast<const uint32_t*>(mask + at_);
      v.x *= (float)(m & 0xFFu);
      v.y *= (float)((m >> 8) & 0xFFu);
      v.z *= (float)((m >> 16) & 0xFFu);
      v.w *= (float)(m >> 24);
    }
  }
  return v;
}

// dB[o, k] = c sum over g in increasing order of v[o, g] A[k, g]: a workgroup
// owns 1024 RT / RMAX rows and walks the blocks in tiles of 32, staging v and
// A transposed ([g][row], [g][k]) so that thread (row group, rank group)
// reads its RT rows and four ranks of a block with two LDS reads and adds
// 4 RT products.  RT = 4 where that still gives every CU two workgroups,
// else RT = 1.
constexpr int kDbCols = 32;
template <int RMAX, int RT>
constexpr int db_rows() { return RT * (256 / (RMAX / 4)); }

template <int RMAX, int RT>
constexpr int db_lds_floats() { return kDbCols * (db_rows<RMAX, RT>() + 4) + kDbCols * (RMAX + 4); }

template <int RMAX, int RT>
__device__ __forceinline__ void db_tile(int bx, int e, float* lds, const float* __restrict__ dS,
                                        const uint8_t* __restrict__ mask, const uint16_t* __restrict__ A, int O,
                                        int G, int r, float c, float* __restrict__ dB, int vec) {
  constexpr int KQ = RMAX / 4, ROWS = db_rows<RMAX, RT>();
  float (*vt)[ROWS + 4] = reinterpret_cast<float (*)[ROWS + 4]>(lds);
  float (*at)[RMAX + 4] = reinterpret_cast<float (*)[RMAX + 4]>(lds + kDbCols * (ROWS + 4));
  dS += (size_t)e * O * G;
  if (mask) mask += (size_t)e * O * G;
  A += (size_t)e * r * G;
  dB += (size_t)e * O * r;
  const int o0 = bx * ROWS;
  const int kq = (threadIdx.x % KQ) * 4, rq = (threadIdx.x / KQ) * RT;
  float acc[RT][4];
#pragma unroll
  for (int q = 0; q < RT; ++q)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[q][j] = 0.0f;
  for (int g0 = 0; g0 < G; g0 += kDbCols) {
    __syncthreads();                                     // the previous tiles are consumed
    if (vec) {
#pragma unroll
      for (int u = 0; u < (ROWS * kDbCols / 4 + 255) / 256; ++u) {
        const int i = threadIdx.x + 256 * u, ro = i / (kDbCols / 4), gq = (i % (kDbCols / 4)) * 4;
        if (ROWS * kDbCols / 4 % 256 != 0 && i >= ROWS * kDbCols / 4) break;
        const float4 v = load_v4(dS, mask, O, G, o0 + ro, g0 + gq);
        vt[gq][ro] = v.x;
        vt[gq + 1][ro] = v.y;
        vt[gq + 2][ro] = v.z;
        vt[gq + 3][ro] = v.w;
      }
    } else {
#pragma unroll 4
      for (int u = 0; u < ROWS * kDbCols / 256; ++u) {
        const int i = threadIdx.x + 256 * u, ro = i / kDbCols, gi = i % kDbCols;
        const int o = o0 + ro, g = g0 + gi;
        float v = 0.0f;
        if (o < O && g < G) {
          const size_t at_ = (size_t)o * G + g;
          v = dS[at_];
          if (mask) v *= (float)mask[at_];
        }
        vt[gi][ro] = v;
      }
    }
#pragma unroll
    for (int u = 0; u < RMAX * kDbCols / 256; ++u) {
      const int i = threadIdx.x + 256 * u, kk = i / kDbCols, gi = i % kDbCols;
      at[gi][kk] = (kk < r && g0 + gi < G) ? bf16_bits_to_f32(A[(size_t)kk * G + g0 + gi]) : 0.0f;
    }
    __syncthreads();
    const int gn = min(kDbCols, G - g0);
    for (int gi = 0; gi < gn; ++gi) {
      const float4 a = *reinterpret_cast<const float4*>(&at[gi][kq]);
      const float av[4] = {a.x, a.y, a.z, a.w};
      float vv[RT];
      if constexpr (RT == 4) {
        const float4 v = *reinterpret_cast<const float4*>(&vt[gi][rq]);
        vv[0] = v.x; vv[1] = v.y; vv[2] = v.z; vv[3] = v.w;
      } else {
#pragma unroll
        for (int q = 0; q < RT; ++q) vv[q] = vt[gi][rq + q];
      }
#pragma unroll
      for (int q = 0; q < RT; ++q)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) acc[q][jj] = __builtin_fmaf(vv[q], av[jj], acc[q][jj]);
    }
  }
#pragma unroll
  for (int q = 0; q < RT; ++q) {
    const int o = o0 + rq + q;
    if (o >= O) break;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj)
      if (kq + jj < r) dB[(size_t)o * r + kq + jj] = __fmul_rn(acc[q][jj], c);
  }
}

// Partial dA over one 32-row chunk: part[chunk][k][g] = sum over the chunk's
// rows in increasing order of B[o, k] v[o, g].  A workgroup takes the chunk's
// rows for 1024 TG / RMAX blocks; thread (rank group, block group) holds four
// ranks and TG blocks (TG = RMAX / 16, at least 1) and per row reads them
// with one 16-byte and one TG-wide LDS read.
template <int RMAX>
constexpr int da_tg() { return RMAX >= 16 ? RMAX / 16 : 1; }
template <int RMAX>
constexpr int da_cols() { return 1024 * da_tg<RMAX>() / RMAX; }

template <int RMAX>
constexpr int da_lds_floats() { return kDaRows * (da_cols<RMAX>() + 4) + kDaRows * (RMAX + 4); }

template <int RMAX>
__device__ __forceinline__ void da_tile(int bx, int e, float* lds, const float* __restrict__ dS,
                                        const uint8_t* __restrict__ mask, const uint16_t* __restrict__ B, int O,
                                        int G, int r, float* __restrict__ part, int vec) {
  constexpr int TG = da_tg<RMAX>(), GT = da_cols<RMAX>(), KQ = RMAX / 4;
  static_assert(KQ * (GT / TG) == 256, "a thread per rank group and block group");
  float (*vt)[GT + 4] = reinterpret_cast<float (*)[GT + 4]>(lds);
  float (*bt)[RMAX + 4] = reinterpret_cast<float (*)[RMAX + 4]>(lds + kDaRows * (GT + 4));
  const int chunks = (O + kDaRows - 1) / kDaRows;
  dS += (size_t)e * O * G;
  if (mask) mask += (size_t)e * O * G;
  B += (size_t)e * O * r;
  part += (size_t)e * chunks * r * G;
  const int gtiles = (G + GT - 1) / GT;
  const int chunk = bx / gtiles, g0 = (bx % gtiles) * GT;
  const int o0 = chunk * kDaRows;
  static_assert(kDaRows * GT % 1024 == 0, "whole 16-byte loads per thread");
  if (vec) {
#pragma unroll
    for (int u = 0; u < kDaRows * GT / 1024; ++u) {
      const int i = threadIdx.x + 256 * u, ro = i / (GT / 4), gq = (i % (GT / 4)) * 4;
      *reinterpret_cast<float4*>(&vt[ro][gq]) = load_v4(dS, mask, O, G, o0 + ro, g0 + gq);
    }
  } else {
#pragma unroll 4
    for (int u = 0; u < kDaRows * GT / 256; ++u) {
      const int i = threadIdx.x + 256 * u, ro = i / GT, gi = i % GT;
      const int o = o0 + ro, g = g0 + gi;
      float v = 0.0f;
      if (o < O && g < G) {
        const size_t at_ = (size_t)o * G + g;
        v = dS[at_];
        if (mask) v *= (float)mask[at_];
      }
      vt[ro][gi] = v;
    }
  }
#pragma unroll
  for (int u = 0; u < (kDaRows * RMAX + 255) / 256; ++u) {
    const int i = threadIdx.x + 256 * u;
    if (i < kDaRows * RMAX) {
      const int ro = i / RMAX, kk = i % RMAX;
      bt[ro][kk] = (kk < r && o0 + ro < O) ? bf16_bits_to_f32(B[(size_t)(o0 + ro) * r + kk]) : 0.0f;
    }
  }
  __syncthreads();
  const int kq = (threadIdx.x % KQ) * 4, gq = (threadIdx.x / KQ) * TG;
  float acc[4][TG];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int t = 0; t < TG; ++t) acc[j][t] = 0.0f;
  const int on = min(kDaRows, O - o0);
  for (int ro = 0; ro < on; ++ro) {
    const float4 b = *reinterpret_cast<const float4*>(&bt[ro][kq]);
    const float bv[4] = {b.x, b.y, b.z, b.w};
    float vv[TG];
#pragma unroll
    for (int t = 0; t < TG; ++t) vv[t] = vt[ro][gq + t];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < TG; ++t) acc[j][t] = __builtin_fmaf(bv[j], vv[t], acc[j][t]);
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (kq + j >= r) break;
#pragma unroll
    for (int t = 0; t < TG; ++t)
      if (g0 + gq + t < G) part[((size_t)chunk * r + kq + j) * G + g0 + gq + t] = acc[j][t];
  }
}

// dB and the dA partials read the same v but are independent: one launch runs
// both, workgroups below ndb taking dB rows and the rest dA chunks, so the
// two short passes overlap instead of running one after the other.
template <int RMAX, int RT>
__global__ __launch_bounds__(256) void qast_grads_kernel(const float* __restrict__ dS,
                                                         const uint8_t* __restrict__ mask,
                                                         const uint16_t* __restrict__ A,
                                                         const uint16_t* __restrict__ B, int O, int G, int r,
                                                         float c, float* __restrict__ dB, float* __restrict__ part,
                                                         int ndb, int vec) {
  constexpr int kDb = db_lds_floats<RMAX, RT>(), kDa = da_lds_floats<RMAX>();
  __shared__ __attribute__((aligned(16))) float lds[kDb > kDa ? kDb : kDa];
  const int bx = (int)blockIdx.x, e = (int)blockIdx.y;
  if (bx < ndb)
    db_tile<RMAX, RT>(bx, e, lds, dS, mask, A, O, G, r, c, dB, vec);
  else
    da_tile<RMAX>(bx - ndb, e, lds, dS, mask, B, O, G, r, part, vec);
}

// dA[i] = c sum over the chunk partials.  Up to 64 chunks: a thread per
// output adds the chunks in order (loads eight at a time); more: a wave per
// output, lane l adds the chunks l, l + 64, ... in order, then a fixed
// butterfly across the lanes.  Either order depends only on the shape.
constexpr int kDaFewChunks = 64;
__global__ __launch_bounds__(256) void qast_da_reduce_kernel(const float* __restrict__ part, int chunks, int r,
                                                             int G, int E, float c, float* __restrict__ dA) {
  const int64_t n = (int64_t)r * G;
  if (chunks <= kDaFewChunks) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)E * n) return;
    const int64_t e = i / n, ie = i - e * n;
    const float* pe = part + (size_t)e * chunks * n + ie;
    float s = 0.0f;
    int ch = 0;
    for (; ch + 8 <= chunks; ch += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = pe[(size_t)(ch + u) * n];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; ch < chunks; ++ch) s += pe[(size_t)ch * n];
    dA[i] = __fmul_rn(s, c);
    return;
  }
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
constexpr int kQastCUs = 256;        // MI355X compute units

template <int F, int R>
static void scales_tb(bool tb4, dim3 grid, hipStream_t s, const uint8_t* bp, const uint16_t* Bp, const uint16_t* Ap,
                      int O, int G, int r, float c, const Ws2Table& t, uint8_t* op, uint8_t* mp, int vec) {
  if (tb4)
    hipLaunchKernelGGL((qast_scales_kernel<F, R, 4>), grid, dim3(256), 0, s, bp, Bp, Ap, O, G, r, c, t, op, mp, vec);
  else
    hipLaunchKernelGGL((qast_scales_kernel<F, R, 1>), grid, dim3(256), 0, s, bp, Bp, Ap, O, G, r, c, t, op, mp, 0);
}
int qast_scales_launch(int fmt, int E, int O, int G, int r, const uint8_t* base, const void* B, const void* A,
                       float c, const float* ws2, uint8_t* out, uint8_t* mask, hipStream_t s) {
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  for (int e0 = 0; e0 < E; e0 += kWs2TableMax) {          // per-expert ws2 travels by value
    const int m = E - e0 < kWs2TableMax ? E - e0 : kWs2TableMax;
    Ws2Table t;
    for (int e = 0; e < m; ++e) t.v[e] = fmt == kNV ? ws2[e0 + e] : 1.0f;
    const size_t rows0 = (size_t)e0 * O;
    const int64_t gtiles = (G + kScCols - 1) / kScCols;
    const int64_t wide = ((O + sc_rows<4>() - 1) / sc_rows<4>()) * gtiles * m;   // workgroups with TB = 4
    const bool tb4 = wide >= 2 * kQastCUs;
    const int rows = tb4 ? sc_rows<4>() : sc_rows<1>();
    const dim3 grid((unsigned)(((O + rows - 1) / rows) * gtiles), (unsigned)m);
    const uint8_t* bp = base + rows0 * G;
    const uint16_t* Bp = b + rows0 * r;
    const uint16_t* Ap = a + (size_t)e0 * r * G;
    uint8_t* op = out + rows0 * G;
    uint8_t* mp = mask ? mask + rows0 * G : nullptr;
    const auto al4 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 3) == 0; };
    const int vec = G % 4 == 0 && al4(bp) && al4(op) && (mp == nullptr || al4(mp)) ? 1 : 0;
#define SQ_QAST_SCALES(F, R) scales_tb<F, R>(tb4, grid, s, bp, Bp, Ap, O, G, r, c, t, op, mp, vec)
    if (fmt == kMX) {
      if (r <= 8) SQ_QAST_SCALES(kMX, 8);
      else if (r <= 16) SQ_QAST_SCALES(kMX, 16);
      else if (r <= 32) SQ_QAST_SCALES(kMX, 32);
      else SQ_QAST_SCALES(kMX, 64);
    } else {
      if (r <= 8) SQ_QAST_SCALES(kNV, 8);
      else if (r <= 16) SQ_QAST_SCALES(kNV, 16);
      else if (r <= 32) SQ_QAST_SCALES(kNV, 32);
      else SQ_QAST_SCALES(kNV, 64);
    }
#undef SQ_QAST_SCALES
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

size_t qast_grads_workspace(int E, int O, int G, int r) {
  return (size_t)E * ((O + kDaRows - 1) / kDaRows) * r * G * sizeof(float);
}

template <int RMAX>
static int qast_grads_r(int E, int O, int G, int r, const float* dS, const uint8_t* mask, const uint16_t* B,
                        const uint16_t* A, float c, float* dB, float* dA, float* part, hipStream_t s) {
  const int chunks = (O + kDaRows - 1) / kDaRows;
  const int vec = G % 4 == 0 && (reinterpret_cast<uintptr_t>(dS) & 15) == 0 &&
                  (mask == nullptr || (reinterpret_cast<uintptr_t>(mask) & 3) == 0) ? 1 : 0;
  constexpr int kWide = db_rows<RMAX, 4>(), kNarrow = db_rows<RMAX, 1>();
  const int nda = ((G + da_cols<RMAX>() - 1) / da_cols<RMAX>()) * chunks;
  if ((int64_t)((O + kWide - 1) / kWide) * E >= 2 * kQastCUs) {
    const int ndb = (O + kWide - 1) / kWide;
    hipLaunchKernelGGL((qast_grads_kernel<RMAX, 4>), dim3((unsigned)(ndb + nda), (unsigned)E), dim3(256), 0, s, dS,
                       mask, A, B, O, G, r, c, dB, part, ndb, vec);
  } else {
    const int ndb = (O + kNarrow - 1) / kNarrow;
    hipLaunchKernelGGL((qast_grads_kernel<RMAX, 1>), dim3((unsigned)(ndb + nda), (unsigned)E), dim3(256), 0, s, dS,
                       mask, A, B, O, G, r, c, dB, part, ndb, vec);
  }
  const int64_t n = (int64_t)E * r * G;
  const int64_t rblocks = chunks <= kDaFewChunks ? (n + 255) / 256 : (n + 3) / 4;
  hipLaunchKernelGGL(qast_da_reduce_kernel, dim3((unsigned)rblocks), dim3(256), 0, s, part, chunks, r, G, E, c, dA);
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
