// bf16-MFMA GEMMs of the frozen-code FP4 linear layer on gfx950.
//
// Three products share one kernel template (paper Section 2 storage equation,
// Section 3 "Scale-QLoRA forward"; the backward follows from the chain rule
// through W = code * eff with the codes frozen):
//
//   FWD  Y[t,o]  = sum_i X[t,i] W[o,i]          M=T  N=O  K=I
//   DX   dX[t,i] = sum_o dY[t,o] W[o,i]         M=T  N=I  K=O
//   DS   dS[o,b] = sum_{j in b} code[o,j] sum_t dY[t,o] X[t,j]
//                                                M=I  N=O  K=T
//
// Every operand tile is staged in LDS as bf16 rows that are contiguous along
// K, so all three products feed v_mfma_f32_32x32x16_bf16 from the same
// fragment reads.  What differs is how a tile reaches LDS:
//   * X (FWD) and dY (DX) are already K-contiguous: 16-byte copies;
//   * W (FWD) is K-contiguous in its packed code plane: each 4-byte word of 8
//     codes is dequantised in registers (exact, see sq_device.h) and written
//     as 16 bytes of bf16;
//   * W^T (DX) and X^T, dY^T (DS) are contiguous along N/M: a thread loads an
//     8x8 block (8 rows of 16 bytes, or 8 rows of one code word that it
//     dequantises first), transposes it in registers with byte permutes and
//     writes 8 K-contiguous 16-byte rows.
// LDS rows are 64 bf16 (128 bytes) with the 16-byte chunk index XOR-swizzled
// by (row ^ row/8) & 7, which keeps the fragment reads and both write
// patterns free of bank conflicts within each group of 8 lanes.
//
// The DS epilogue multiplies each accumulator dW[o,j] by its E2M1 code and
// sums over the block in registers (the 32x32 MFMA output puts 8 of a
// 16-row block's rows in one lane and the other 8 in the lane 32 away), so
// dW never leaves the chip and dS is written once, without atomics.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_launch.h"

namespace sq {

enum Mode { kFwd = 0, kDx = 1, kDs = 2 };

constexpr int kBK = 64;           // K per LDS stage (one 128-byte row)
constexpr int kXcds = 8;          // MI355X: workgroups are dealt round-robin to 8 XCDs

struct GemmArgs {
  const uint16_t* a;      // FWD: X [T,I]   DX: dY [T,O]   DS: X [T,I]
  const uint16_t* b;      // DS: dY [T,O]
  const uint8_t* codes;   // [O, I/2]
  const uint8_t* scales;  // [O, G]  (FWD, DX)
  void* out;              // FWD: Y [T,O]  DX: dX [T,I]  DS: dS [O,G] fp32
  int M, N, K;
  int T, O, I, G;
  float ws2;              // NV epilogue factor (1 for MX)
  int out_bf16;
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * kBK + (((chunk ^ row ^ (row >> 3)) & 7) << 3);
}

__device__ __forceinline__ void st_lds16(uint16_t* s, int row, int chunk, uint4 v) {
  *reinterpret_cast<uint4*>(s + lds_off(row, chunk)) = v;
}

__device__ __forceinline__ uint4 ld_global16(const uint16_t* p) {
  return *reinterpret_cast<const uint4*>(p);
}

// ------------------------------------------------------------------ loaders
// K-contiguous bf16 tile: rows [r0, r0+R) of a [rows_total, ld] matrix,
// columns [k0, k0+64).  Out-of-range rows or 8-element chunks read as zero.
template <int R, int NT>
struct LoadKContig {
  static constexpr int kPer = R * 8 / NT;         // 16-byte chunks per thread
  static_assert(kPer * NT == R * 8, "tile rows must split evenly");
  uint4 v[kPer];
  __device__ __forceinline__ void fetch(const uint16_t* src, int ld, int rows_total, int kdim, int r0, int k0, int tid) {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int idx = tid + p * NT;
      const int row = idx >> 3, chunk = idx & 7;
      const int gr = r0 + row, gk = k0 + chunk * 8;
      if (gr < rows_total && gk < kdim)
        v[p] = ld_global16(src + (size_t)gr * ld + gk);
      else
        v[p] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void commit(uint16_t* s, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int idx = tid + p * NT;
      st_lds16(s, idx >> 3, idx & 7, v[p]);
    }
  }
};

// W tile for FWD: rows o in [n0, n0+R), K = i in [k0, k0+64), from packed codes.
template <int R, int FMT, int NT>
struct LoadWKContig {
  static constexpr int kPer = R * 8 / NT;
  static_assert(kPer * NT == R * 8, "tile rows must split evenly");
  uint32_t w[kPer];
  uint32_t sb[kPer];
  __device__ __forceinline__ void fetch(const GemmArgs& g, int n0, int k0, int tid) {
    constexpr int B = ScaleOperand<FMT>::kBlock;
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int idx = tid + p * NT;
      const int row = idx >> 3, chunk = idx & 7;
      const int o = n0 + row, i = k0 + chunk * 8;
      if (o < g.O && i < g.I) {
        w[p] = *reinterpret_cast<const uint32_t*>(g.codes + (size_t)o * (g.I >> 1) + (i >> 1));
        sb[p] = g.scales[(size_t)o * g.G + i / B];
      } else {
        w[p] = 0u;
        sb[p] = 0x38u;   // any finite scale: the codes are zero
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* s, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int idx = tid + p * NT;
      const float so = ScaleOperand<FMT>::of(sb[p]);
      st_lds16(s, idx >> 3, idx & 7, ScaleOperand<FMT>::dequant8(w[p], so));
    }
  }
};

// W^T tile for DX: LDS rows are i in [n0, n0+R), K = o in [k0, k0+64).
// The tile holds R 8x8 blocks (R/8 along i, 8 along o); block q is taken by
// thread q % NT, item q / NT.
template <int R, int FMT, int NT>
struct LoadWTrans {
  static constexpr int kBlocks = R;
  static constexpr int kPer = (kBlocks + NT - 1) / NT;
  uint32_t w[kPer][8];
  uint32_t sb[kPer][8];
  __device__ __forceinline__ void fetch(const GemmArgs& g, int n0, int k0, int tid) {
    constexpr int B = ScaleOperand<FMT>::kBlock;
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int q = tid + p * NT;
      if (q >= kBlocks) break;
      const int ib = q % (R / 8), ob = q / (R / 8);
      const int i = n0 + ib * 8;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int o = k0 + ob * 8 + r;
        if (o < g.O && i < g.I) {
          w[p][r] = *reinterpret_cast<const uint32_t*>(g.codes + (size_t)o * (g.I >> 1) + (i >> 1));
          sb[p][r] = g.scales[(size_t)o * g.G + i / B];
        } else {
          w[p][r] = 0u;
          sb[p][r] = 0x38u;
        }
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* s, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int q = tid + p * NT;
      if (q >= kBlocks) break;
      const int ib = q % (R / 8), ob = q / (R / 8);
      uint32_t rows[8][4], cols[8][4];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const uint4 d = ScaleOperand<FMT>::dequant8(w[p][r], ScaleOperand<FMT>::of(sb[p][r]));
        rows[r][0] = d.x; rows[r][1] = d.y; rows[r][2] = d.z; rows[r][3] = d.w;
      }
      transpose8x8_b16(rows, cols);
#pragma unroll
      for (int c = 0; c < 8; ++c)
        st_lds16(s, ib * 8 + c, ob, make_uint4(cols[c][0], cols[c][1], cols[c][2], cols[c][3]));
    }
  }
};

// Both DS tiles (X^T rows j in [m0, m0+BM), dY^T rows o in [n0, n0+BN), K = t
// in [k0, k0+64)) from sources [T, ld] that are contiguous along the tile
// rows.  The BM + BN 8x8 blocks (A blocks first) are dealt to the threads.
template <int BM, int BN, int NT>
struct LoadTransDS {
  static constexpr int kBlocks = BM + BN;
  static constexpr int kPer = (kBlocks + NT - 1) / NT;
  uint4 v[kPer][8];
  __device__ __forceinline__ void fetch(const GemmArgs& g, int m0, int n0, int k0, int tid) {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int q = tid + p * NT;
      if (q >= kBlocks) break;
      const bool isA = q < BM;
      const int lq = isA ? q : q - BM;
      const int rows8 = (isA ? BM : BN) / 8;
      const int mb = lq % rows8, kb = lq / rows8;
      const int m = (isA ? m0 : n0) + mb * 8;
      const int mdim = isA ? g.I : g.O;
      const uint16_t* src = isA ? g.a : g.b;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const int k = k0 + kb * 8 + r;
        if (k < g.T && m < mdim)
          v[p][r] = ld_global16(src + (size_t)k * mdim + m);
        else
          v[p][r] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void commit(uint16_t* sa, uint16_t* sb, int tid) const {
#pragma unroll
    for (int p = 0; p < kPer; ++p) {
      const int q = tid + p * NT;
      if (q >= kBlocks) break;
      const bool isA = q < BM;
      const int lq = isA ? q : q - BM;
      const int rows8 = (isA ? BM : BN) / 8;
      const int mb = lq % rows8, kb = lq / rows8;
      uint32_t rows[8][4], cols[8][4];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        rows[r][0] = v[p][r].x; rows[r][1] = v[p][r].y; rows[r][2] = v[p][r].z; rows[r][3] = v[p][r].w;
      }
      transpose8x8_b16(rows, cols);
      uint16_t* s = isA ? sa : sb;
#pragma unroll
      for (int c = 0; c < 8; ++c)
        st_lds16(s, mb * 8 + c, kb, make_uint4(cols[c][0], cols[c][1], cols[c][2], cols[c][3]));
    }
  }
};

// ------------------------------------------------------------------ tile order
// Workgroup w runs on XCD w % 8, and each XCD has its own L2.  Tiles are
// enumerated in groups of kGroupM tile-rows (column by column inside a group)
// and each XCD is given one contiguous stretch of that order, so the
// workgroups that share an L2 also share operand panels.
constexpr int kGroupM = 8;

__device__ __forceinline__ void tile_of(int bid, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int x = bid % kXcds, q = nb / kXcds, r = nb % kXcds;
  const int idx = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + bid / kXcds;
  const int per_group = kGroupM * tiles_n;
  const int group = idx / per_group;
  const int first_m = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first_m);
  const int in = idx - group * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

// ------------------------------------------------------------------ kernel
// Block tile BM x BN, WGM x WGN waves, each wave (BM/WGM) x (BN/WGN) built
// from 32x32 MFMA tiles.
template <int MODE, int FMT, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_kernel(GemmArgs g) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t* sA = smem;                       // [2][BM][64]
  uint16_t* sB = smem + 2 * BM * kBK;        // [2][BN][64]

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  int tm, tn;
  tile_of(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  LoadKContig<BM, NT> la_k;          // FWD: X, DX: dY
  LoadWKContig<BN, FMT, NT> lb_w;    // FWD
  LoadWTrans<BN, FMT, NT> lb_wt;     // DX
  LoadTransDS<BM, BN, NT> l_ds;      // DS

  auto fetch = [&](int k0) {
    if constexpr (MODE == kFwd) {
      la_k.fetch(g.a, g.I, g.T, g.I, m0, k0, tid);
      lb_w.fetch(g, n0, k0, tid);
    } else if constexpr (MODE == kDx) {
      la_k.fetch(g.a, g.O, g.T, g.O, m0, k0, tid);
      lb_wt.fetch(g, n0, k0, tid);
    } else {
      l_ds.fetch(g, m0, n0, k0, tid);
    }
  };
  auto commit = [&](int buf) {
    uint16_t* a = sA + buf * BM * kBK;
    uint16_t* b = sB + buf * BN * kBK;
    if constexpr (MODE == kFwd) {
      la_k.commit(a, tid);
      lb_w.commit(b, tid);
    } else if constexpr (MODE == kDx) {
      la_k.commit(a, tid);
      lb_wt.commit(b, tid);
    } else {
      l_ds.commit(a, b, tid);
    }
  };

  const int nk = (g.K + kBK - 1) / kBK;
  if (nk > 0) {
    fetch(0);
    commit(0);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) fetch((kt + 1) * kBK);
    const uint16_t* a = sA + buf * BM * kBK;
    const uint16_t* b = sB + buf * BN * kBK;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      const int chunk = kk * 2 + (lane >> 5);
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        fa[i] = *reinterpret_cast<const bf16x8*>(a + lds_off(wm0 + i * 32 + (lane & 31), chunk));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        fb[j] = *reinterpret_cast<const bf16x8*>(b + lds_off(wn0 + j * 32 + (lane & 31), chunk));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) commit(buf ^ 1);
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // 32x32 output tile: lane l, register r holds row 8*(r/4) + 4*(l/32) + r%4,
  // column l%32.
  const int lrow = 4 * (lane >> 5), lcol = lane & 31;
  if constexpr (MODE == kFwd || MODE == kDx) {
    const float f = g.ws2;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn0 + j * 32 + lcol;
        if (col >= g.N) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = m0 + wm0 + i * 32 + 8 * (r >> 2) + lrow + (r & 3);
          if (row >= g.M) continue;
          const float v = (FMT == kNV) ? acc[i][j][r] * f : acc[i][j][r];
          if (g.out_bf16)
            reinterpret_cast<uint16_t*>(g.out)[(size_t)row * g.N + col] = (uint16_t)f32_to_bf16_rne(v);
          else
            reinterpret_cast<float*>(g.out)[(size_t)row * g.N + col] = v;
        }
      }
  } else {
    // rows are input features j, columns output features o
    float* dS = reinterpret_cast<float*>(g.out);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int o = n0 + wn0 + j * 32 + lcol;
      const bool o_ok = o < g.O;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int jb = m0 + wm0 + i * 32;          // first feature of this 32-row tile
        float prod[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int j0 = jb + 8 * q + lrow;        // 4 consecutive features j0..j0+3
          uint32_t cw = 0;
          if (o_ok && j0 < g.I)
            cw = *reinterpret_cast<const uint16_t*>(g.codes + (size_t)o * (g.I >> 1) + (j0 >> 1));
#pragma unroll
          for (int e = 0; e < 4; ++e) prod[4 * q + e] = acc[i][j][4 * q + e] * e2m1_to_f32((cw >> (4 * e)) & 15u);
        }
        if constexpr (FMT == kMX) {
          float s = 0.0f;
#pragma unroll
          for (int r = 0; r < 16; ++r) s += prod[r];
          s += __shfl_xor(s, 32);
          if (lane < 32 && o_ok && jb < g.I) dS[(size_t)o * g.G + jb / 32] = s;
        } else {
          float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
          for (int r = 0; r < 8; ++r) { s0 += prod[r]; s1 += prod[8 + r]; }
          s0 += __shfl_xor(s0, 32);
          s1 += __shfl_xor(s1, 32);
          const int b = jb / 16 + (lane >> 5);
          const float s = (lane < 32) ? s0 : s1;
          if (o_ok && b * 16 < g.I) dS[(size_t)o * g.G + b] = s;
        }
      }
    }
  }
}

// Tile configurations (compile-time; SQ_CFG_* selects one per product for
// tuning builds).  Each entry: BM, BN, waves along M, waves along N.
#ifndef SQ_CFG_FWD
#define SQ_CFG_FWD 256, 256, 4, 2
#endif
#ifndef SQ_CFG_DX
#define SQ_CFG_DX 256, 256, 2, 2
#endif
#ifndef SQ_CFG_DS
#define SQ_CFG_DS 256, 256, 4, 2
#endif

template <int MODE, int FMT, int BM, int BN, int WGM, int WGN>
static int launch_gemm(const GemmArgs& g, hipStream_t s) {
  const size_t lds = (size_t)2 * (BM + BN) * kBK * sizeof(uint16_t);
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  if (tiles == 0) return 0;
  auto kern = gemm_kernel<MODE, FMT, BM, BN, WGM, WGN>;
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)lds) != hipSuccess)
      return -1;
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3(tiles), dim3(64 * WGM * WGN), lds, s, g);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ------------------------------------------------------------------ entry
int gemm_fwd(int fmt, int T, int O, int I, const void* X, const uint8_t* codes,
             const uint8_t* scales, float ws2, void* Y, int y_bf16, hipStream_t s) {
  GemmArgs g{};
  g.a = static_cast<const uint16_t*>(X);
  g.codes = codes; g.scales = scales; g.out = Y;
  g.T = T; g.O = O; g.I = I; g.G = I / (fmt == kMX ? 32 : 16);
  g.M = T; g.N = O; g.K = I;
  g.ws2 = (fmt == kNV) ? ws2 : 1.0f;
  g.out_bf16 = y_bf16;
  return fmt == kMX ? launch_gemm<kFwd, kMX, SQ_CFG_FWD>(g, s) : launch_gemm<kFwd, kNV, SQ_CFG_FWD>(g, s);
}

int gemm_dx(int fmt, int T, int O, int I, const void* dY, const uint8_t* codes,
            const uint8_t* scales, float ws2, void* dX, int dx_bf16, hipStream_t s) {
  GemmArgs g{};
  g.a = static_cast<const uint16_t*>(dY);
  g.codes = codes; g.scales = scales; g.out = dX;
  g.T = T; g.O = O; g.I = I; g.G = I / (fmt == kMX ? 32 : 16);
  g.M = T; g.N = I; g.K = O;
  g.ws2 = (fmt == kNV) ? ws2 : 1.0f;
  g.out_bf16 = dx_bf16;
  return fmt == kMX ? launch_gemm<kDx, kMX, SQ_CFG_DX>(g, s) : launch_gemm<kDx, kNV, SQ_CFG_DX>(g, s);
}

int gemm_dscale(int fmt, int T, int O, int I, const void* X, const void* dY,
                const uint8_t* codes, float* dS, hipStream_t s) {
  GemmArgs g{};
  g.a = static_cast<const uint16_t*>(X);
  g.b = static_cast<const uint16_t*>(dY);
  g.codes = codes; g.out = dS;
  g.T = T; g.O = O; g.I = I; g.G = I / (fmt == kMX ? 32 : 16);
  g.M = I; g.N = O; g.K = T;
  g.ws2 = 1.0f;
  g.out_bf16 = 0;
  return fmt == kMX ? launch_gemm<kDs, kMX, SQ_CFG_DS>(g, s) : launch_gemm<kDs, kNV, SQ_CFG_DS>(g, s);
}

}  // namespace sq
