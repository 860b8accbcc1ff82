// QAT-LoRA weight-space STE step on gfx950: the comparator the paper measures
// Scale-QLoRA against (Section 2 related work, "Merge-aware weight-space";
// Appendix "Training cost per step").  The adapter is ordinary LoRA on the
// weight, W = W_base + (alpha/r) B A, and the forward runs on quantize(W).
//
// * qat_requant_kernel builds W_eff = bf16(fp32(base + fp32(alpha/r * S))),
//   S[o,i] = sum over k in increasing order of B[o,k] A[k,i] (fp32, each
//   product exact), and re-quantises it with the nearest rule in the same
//   pass, so W_eff never reaches HBM.  The fake-quantised weight is exactly
//   the new (codes, scales) pair, so the forward and dX run on the FP4 GEMM.
// * The straight-through gradients factor through the rank:
//     dB = (alpha/r) dY^T (X A^T),  dA = (alpha/r) (dY B)^T X,
//   so dW = dY^T X is never formed.  P = X A^T and Q = dY B contract over the
//   contiguous dimension (thin_n: MFMA fed straight from global memory);
//   dA and dB contract over tokens (thin_m: MFMA again, with P and Q carried
//   as bf16 hi + lo pairs so the fp32 values pass at about 16 bits, and
//   partial sums over token ranges reduced in a fixed order, so the result is
//   deterministic).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sq_device.h"
#include "sq_launch.h"
#include "sq_rtn.h"

namespace sq {

// ------------------------------------------------------------ requant
constexpr int kReqRows = 32;        // rows per workgroup: 4 waves x 8 rows
constexpr int kReqRowsPerWave = 8;
constexpr int kReqCols = 512;       // columns per workgroup: 64 lanes x 8

constexpr int kReqRankTile = 32;    // ranks staged in LDS at a time

// The rank is walked in tiles of 32 (A tile [32][512] and B tile [16][32] in
// LDS), k in increasing order throughout; ranks past r read as 0, which adds
// exact zeros.  grid.z is the expert of a stack (expert e0 + z, planes
// [E, O, *] contiguous, its ws2 in the table).
template <int FMT>
__global__ __launch_bounds__(256) void qat_requant_kernel(const uint8_t* __restrict__ codes,
                                                          const uint8_t* __restrict__ scales, Ws2Table ws2t,
                                                          const uint16_t* __restrict__ B,
                                                          const uint16_t* __restrict__ A, int O, int I, int r,
                                                          float c, uint8_t* __restrict__ codes_out,
                                                          uint8_t* __restrict__ scales_out, int e0) {
  constexpr int BLK = ScaleOperand<FMT>::kBlock;
  {
    const int64_t e = (int64_t)e0 + blockIdx.z;
    const int64_t code_plane = (int64_t)O * (I / 2), scale_plane = (int64_t)O * (I / BLK);
    codes += e * code_plane;
    codes_out += e * code_plane;
    scales += e * scale_plane;
    scales_out += e * scale_plane;
    B += e * O * r;
    A += e * r * I;
  }
  const float ws2 = FMT == kMX ? 1.0f : ws2t.v[blockIdx.z];
  __shared__ __align__(16) uint16_t a_lds[kReqRankTile][kReqCols];
  __shared__ __align__(16) uint16_t b_lds[kReqRows][kReqRankTile];
  const int tid = threadIdx.x;
  const int col0 = blockIdx.x * kReqCols, row0 = blockIdx.y * kReqRows;
  const int wave = tid >> 6, lane = tid & 63;
  const int cc = (col0 >> 3) + lane;                       // chunk column in the row
  const bool col_ok = 8 * cc < I;
  float acc[kReqRowsPerWave][8];
#pragma unroll
  for (int j = 0; j < kReqRowsPerWave; ++j)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[j][e] = 0.0f;

  const int rp = (r + 7) & ~7;
  for (int kb = 0; kb < rp; kb += kReqRankTile) {
    if (kb > 0) __syncthreads();                           // the previous tile is consumed
    // A tile: 64 threads per rank row of 512 columns, 16 bytes each.
    for (int e = tid; e < kReqRankTile * (kReqCols / 8); e += 256) {
      const int k = e / (kReqCols / 8), q = e % (kReqCols / 8);
      const int col = col0 + 8 * q;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (kb + k < r && col < I) v = *reinterpret_cast<const uint4*>(A + (int64_t)(kb + k) * I + col);
      *reinterpret_cast<uint4*>(&a_lds[k][8 * q]) = v;
    }
    for (int e = tid; e < kReqRows * kReqRankTile; e += 256) {
      const int j = e / kReqRankTile, k = e % kReqRankTile;
      const int o = row0 + j;
      b_lds[j][k] = (kb + k < r && o < O) ? B[(int64_t)o * r + kb + k] : (uint16_t)0;
    }
    __syncthreads();
    const int kn = min(kReqRankTile, rp - kb);
    for (int kg = 0; kg < kn; kg += 8) {
      uint4 bq[kReqRowsPerWave];
#pragma unroll
      for (int j = 0; j < kReqRowsPerWave; ++j)
        bq[j] = *reinterpret_cast<const uint4*>(&b_lds[wave * kReqRowsPerWave + j][kg]);
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        const uint4 av = *reinterpret_cast<const uint4*>(&a_lds[kg + kk][8 * lane]);
        const uint32_t aw[4] = {av.x, av.y, av.z, av.w};
        float a[8];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          a[2 * p] = __uint_as_float(aw[p] << 16);
          a[2 * p + 1] = __uint_as_float(aw[p] & 0xFFFF0000u);
        }
#pragma unroll
        for (int j = 0; j < kReqRowsPerWave; ++j) {
          const uint32_t bw[4] = {bq[j].x, bq[j].y, bq[j].z, bq[j].w};
          const uint32_t h = bw[kk >> 1];
          const float b = __uint_as_float((kk & 1) ? (h & 0xFFFF0000u) : (h << 16));
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[j][e] = __builtin_fmaf(b, a[e], acc[j][e]);   // b*a exact in fp32
        }
      }
    }
  }

  const int64_t cpr = I / 8;                               // chunks per row
#pragma unroll
  for (int j = 0; j < kReqRowsPerWave; ++j) {
    const int o = row0 + wave * kReqRowsPerWave + j;
    const bool ok = col_ok && o < O;
    uint32_t cw = 0, sb = 0;
    if (ok) {
      cw = *reinterpret_cast<const uint32_t*>(codes + (int64_t)o * (I / 2) + 4 * cc);
      sb = scales[(int64_t)o * (I / BLK) + (8 * cc) / BLK];
    }
    float eff;
    if (FMT == kMX) eff = e8m0_to_f32(sb);
    else eff = __fmul_rn(e4m3_to_f32(sb), ws2);
    uint32_t wb[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      uint32_t h2[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int e = 2 * p + q;
        const float base = __fmul_rn(e2m1_to_f32((cw >> (4 * e)) & 15u), eff);
        const float w = __fadd_rn(base, __fmul_rn(c, acc[j][e]));
        h2[q] = (w != w) ? 0x7FC0u : f32_to_bf16_rne(w);
      }
      wb[p] = h2[0] | (h2[1] << 16);
    }
    rtn_chunk<FMT, kRuleEven>(make_uint4(wb[0], wb[1], wb[2], wb[3]), (int64_t)o * cpr + cc, ok, nullptr, ws2,
                              nullptr, 0, codes_out, scales_out);
  }
}

int qat_requant_launch(int fmt, int E, int O, int I, int r, const uint8_t* codes, const uint8_t* scales,
                       const float* ws2, const void* B, const void* A, float c, uint8_t* codes_out,
                       uint8_t* scales_out, hipStream_t s) {
  const uint16_t* b = static_cast<const uint16_t*>(B);
  const uint16_t* a = static_cast<const uint16_t*>(A);
  for (int e0 = 0; e0 < E; e0 += kWs2TableMax) {
    const int n = E - e0 < kWs2TableMax ? E - e0 : kWs2TableMax;
    Ws2Table t{};
    for (int k = 0; k < n; ++k) t.v[k] = fmt == kMX ? 1.0f : ws2[e0 + k];
    const dim3 grid((unsigned)((I + kReqCols - 1) / kReqCols), (unsigned)((O + kReqRows - 1) / kReqRows),
                    (unsigned)n);
    if (fmt == kMX)
      hipLaunchKernelGGL(qat_requant_kernel<kMX>, grid, dim3(256), 0, s, codes, scales, t, b, a, O, I, r, c,
                         codes_out, scales_out, e0);
    else
      hipLaunchKernelGGL(qat_requant_kernel<kNV>, grid, dim3(256), 0, s, codes, scales, t, b, a, O, I, r, c,
                         codes_out, scales_out, e0);
    if (hipGetLastError() != hipSuccess) return -1;
  }
  return 0;
}

// ------------------------------------------------------------ thin_n
// Partial products part[kc][t][j] = sum over K-chunk kc of L[t, k] Rt[j, k]
// for a list of independent products per launch (each expert has two,
// P = X A^T and Q = dY B, which share its tokens M, the rank and its padded
// token count).  bf16 operands, both contiguous along K (a multiple of 8);
// rows of Rt at or past r and rows of L at or past M read as 0.  A workgroup
// owns 32 rows and one K-chunk of one product; its 8 waves take the chunk's
// 16-wide steps round-robin and reduce through LDS in a fixed order.
// thin_n_finish then sums the chunks in order and writes the transposed bf16
// hi/lo pair Lt[hl][j][t].
constexpr int kThinWaves = 8;
constexpr int kThinKChunk = 1024;
constexpr int kLoraExperts = 32;    // experts per launch set (two products each)

struct ThinNProb {
  const uint16_t* L;                // [M, K]
  const uint16_t* Rt;               // [RW, K]
  float* part;                      // [chunks][Tp][RW]
  uint16_t* Lt;                     // [2][RW][Tp]
  int K, chunks, M, Tp;
  int blk0;                         // first thin_n workgroup of the product
  int fblk0;                        // first thin_n_finish workgroup
};
struct ThinNList {
  ThinNProb p[2 * kLoraExperts];
  int n;
};
static_assert(sizeof(ThinNList) <= 4096, "kernel argument budget");

// The last product whose first workgroup is at or before b (first[] ascending).
template <typename F>
__device__ __forceinline__ int find_product(int b, int n, F first) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first(mid) <= b) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

template <int NT>
__global__ __launch_bounds__(512) void thin_n_kernel(ThinNList pl, int r) {
  constexpr int RW = 32 * NT;
  __shared__ float red[kThinWaves / 2][32][RW + 1];
  const int b = (int)blockIdx.x;
  const int pi = find_product(b, pl.n, [&](int q) { return pl.p[q].blk0; });
  const ThinNProb& pr = pl.p[pi];
  const int rows = pr.Tp / 32;
  const int local = b - pr.blk0;
  const int kc = local / rows;
  const int K = pr.K, M = pr.M, Tp = pr.Tp;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int row0 = (local % rows) * 32;
  const int lr = lane & 31, kh = lane >> 5;
  const bool row_ok = row0 + lr < M;
  const uint16_t* lp = pr.L + (int64_t)(row0 + lr) * K + 8 * kh;
  const uint16_t* rp[NT];
  bool r_ok[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    r_ok[t] = 32 * t + lr < r;
    rp[t] = pr.Rt + (int64_t)(32 * t + lr) * K + 8 * kh;
  }
  f32x16 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[t][e] = 0.0f;

  auto frag = [&](const uint16_t* p, bool ok, int st) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (ok && 16 * st + 8 * kh < K) v = *reinterpret_cast<const uint4*>(p + 16 * st);
    bf16x8 f;
    __builtin_memcpy(&f, &v, 16);
    return f;
  };
  // The chunk's steps st = s0 + wave, s0 + wave + 8, ... (8 per wave): all
  // loads in flight before the MFMAs.
  constexpr int kSteps = kThinKChunk / (16 * kThinWaves);
  static_assert(kThinKChunk == 16 * kSteps * kThinWaves, "whole steps per wave");
  const int s0 = kc * (kThinKChunk / 16);
  bf16x8 fa[kSteps], fb[kSteps][NT];
#pragma unroll
  for (int u = 0; u < kSteps; ++u) {
    const int st = s0 + wave + u * kThinWaves;
    fa[u] = frag(lp, row_ok, st);
#pragma unroll
    for (int t = 0; t < NT; ++t) fb[u][t] = frag(rp[t], r_ok[t], st);
  }
#pragma unroll
  for (int u = 0; u < kSteps; ++u)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[u], fb[u][t], acc[t], 0, 0, 0);

  // lane l, register e: row 8(e/4) + 4(l/32) + e%4, column l%32.  Waves 4..7
  // store, waves 0..3 add theirs, then the four are summed in order.
  const int half = kThinWaves / 2;
  if (wave >= half) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) red[wave - half][8 * (e >> 2) + 4 * kh + (e & 3)][32 * t + lr] = acc[t][e];
  }
  __syncthreads();
  if (wave < half) {
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        float& d = red[wave][8 * (e >> 2) + 4 * kh + (e & 3)][32 * t + lr];
        d = acc[t][e] + d;
      }
  }
  __syncthreads();
  float* out = pr.part + ((int64_t)kc * Tp + row0) * RW;
  for (int e = tid; e < 32 * RW; e += 512) {
    const int row = e / RW, j = e % RW;
    out[e] = ((red[0][row][j] + red[1][row][j]) + red[2][row][j]) + red[3][row][j];
  }
}

// Lt[p][0][j][t] = hi, Lt[p][1][j][t] = lo of the fp32 sum over K-chunks (in
// order) of part[p][kc][t][j]: hi = bf16(s), lo = bf16(s - hi).  A workgroup
// takes 32 tokens of one product (RW / 8 sums per thread, their loads issued
// together) and transposes them through LDS.
template <int RW>
__global__ __launch_bounds__(256) void thin_n_finish_kernel(ThinNList pl) {
  constexpr int kPer = 32 * RW / 256;
  __shared__ float t_s[32][RW + 1];
  const int b = (int)blockIdx.x;
  const int pi = find_product(b, pl.n, [&](int q) { return pl.p[q].fblk0; });
  const ThinNProb& pr = pl.p[pi];
  const int Tp = pr.Tp;
  const int t0 = (b - pr.fblk0) * 32;
  const float* part = pr.part + (int64_t)t0 * RW;
  const int chunks = pr.chunks;
  float sum[kPer];
#pragma unroll
  for (int u = 0; u < kPer; ++u) sum[u] = 0.0f;
  for (int kc = 0; kc < chunks; ++kc) {
    float v[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) v[u] = part[(int64_t)kc * Tp * RW + threadIdx.x + 256 * u];
#pragma unroll
    for (int u = 0; u < kPer; ++u) sum[u] += v[u];
  }
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = threadIdx.x + 256 * u;
    t_s[e / RW][e % RW] = sum[u];
  }
  __syncthreads();
  uint16_t* Lt = pr.Lt;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    const int e = threadIdx.x + 256 * u;
    const int j = e >> 5, tt = e & 31;
    const float v = t_s[tt][j];
    const uint32_t hi = f32_to_bf16_rne(v);
    const uint32_t lo = f32_to_bf16_rne(v - __uint_as_float(hi << 16));
    Lt[(int64_t)j * Tp + t0 + tt] = (uint16_t)hi;
    Lt[((int64_t)RW + j) * Tp + t0 + tt] = (uint16_t)lo;
  }
}

// ------------------------------------------------------------ thin_m
// part[split][j][n] = sum over the split's tokens t of (hi + lo)[j][t] R[t, n]
// on the matrix cores: out^T = Lt R with K = tokens.  A workgroup owns 256
// columns (64 per wave, two 32-column MFMA tiles) and one token range, walked
// in stages of 64 tokens: R [64][256] is staged in LDS in its natural layout
// and read with the transpose read; the hi/lo rows of Lt for the stage sit in
// LDS as [2*RW][64].  The next stage's global loads are in flight while the
// current one computes.
typedef short v4i16 __attribute__((ext_vector_type(4)));
#define SQ_LDS __attribute__((address_space(3)))
constexpr int kTmCols = 256;
constexpr int kTmTok = 64;

// [64][256] bf16, 16-byte chunk c of token row k at chunk c ^ (4 (k % 8)):
// the four rows one transpose read spans fall in different banks.
__device__ __forceinline__ int tm_r_off(int k, int col) {
  return k * kTmCols + ((((col >> 3) ^ (4 * (k & 7))) & 31) << 3) + (col & 7);
}
// [2*RW][64] bf16, chunk c of row q at chunk c ^ (q % 8).
__device__ __forceinline__ int tm_a_off(int q, int c) { return q * kTmTok + ((c ^ (q & 7)) << 3); }

// Tokens k0 .. k0+3 and k0+4 .. k0+7 of the four columns at col, through two
// transpose reads: the MFMA operand of one lane.
__device__ __forceinline__ bf16x8 tm_frag(const uint16_t* rt, int k0, int col) {
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SQ_LDS v4i16*)(rt + tm_r_off(k0, col)));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SQ_LDS v4i16*)(rt + tm_r_off(k0 + 4, col)));
  bf16x8 r;
  __builtin_memcpy(&r, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&r) + 8, &hi, 8);
  return r;
}

// One stage's global loads into registers: R [64][256] (zeros past T and N)
// and the 2*RW rows of Lt over the stage's 64 tokens; all zeros when !live.
template <int AC>
__device__ __forceinline__ void tm_load(const uint16_t* __restrict__ R, const uint16_t* __restrict__ Lt, int T, int Tp,
                                        int N, int n0, int t0, bool live, int tid, uint4 (&rreg)[8],
                                        uint4 (&areg)[AC]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int q = tid + 256 * i, k = q >> 5, c = q & 31;
    const int col = n0 + 8 * c;
    rreg[i] = (live && t0 + k < T && col < N) ? *reinterpret_cast<const uint4*>(R + (int64_t)(t0 + k) * N + col)
                                              : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < AC; ++i) {
    const int q = tid + 256 * i, row = q >> 3, c = q & 7;
    areg[i] = live ? *reinterpret_cast<const uint4*>(Lt + (int64_t)row * Tp + t0 + 8 * c) : make_uint4(0, 0, 0, 0);
  }
}

// One product of the token contraction: Lt hi/lo [2][RW][Tp], R [T, N];
// tiles * splits workgroups from blk0 on, local workgroup b takes column tile
// b % tiles and token range b / tiles.  trans: partials as [split][N][RW]
// (the output is [N, r]), else [split][RW][N].
struct TmProblem {
  const uint16_t* Lt;
  const uint16_t* R;
  float* part;
  int N, tiles, tps, splits, trans, T, Tp, blk0;
};
struct TmList {
  TmProblem p[2 * kLoraExperts];
  int n;
};
static_assert(sizeof(TmList) <= 4096, "kernel argument budget");

template <int JT>
__global__ __launch_bounds__(256) void thin_m_kernel(TmList pl) {
  constexpr int RW = 32 * JT;
  constexpr int kAChunks = 2 * RW * (kTmTok / 8) / 256;   // 16-byte A chunks per thread per stage
  __shared__ __align__(16) uint16_t rt[kTmTok * kTmCols];
  __shared__ __align__(16) uint16_t at[2 * RW * kTmTok];
  const int pi = find_product((int)blockIdx.x, pl.n, [&](int q) { return pl.p[q].blk0; });
  const TmProblem& P = pl.p[pi];
  const uint16_t* __restrict__ Lt = P.Lt;
  const uint16_t* __restrict__ R = P.R;
  const int N = P.N, T = P.T, Tp = P.Tp;
  const int local = (int)blockIdx.x - P.blk0;
  const int tile = local % P.tiles, split = local / P.tiles;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n0 = tile * kTmCols;
  const int t_begin = split * P.tps, t_end = min(Tp, t_begin + P.tps);

  uint4 rreg[8], areg[kAChunks];
  f32x16 acc[JT][2];
#pragma unroll
  for (int jt = 0; jt < JT; ++jt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[jt][nt][e] = 0.0f;

  const int i16 = lane & 15, g = lane >> 4;
  tm_load<kAChunks>(R, Lt, T, Tp, N, n0, t_begin, t_begin < t_end, tid, rreg, areg);
  for (int t0 = t_begin; t0 < t_end; t0 += kTmTok) {
    __syncthreads();                                       // the previous stage is consumed
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + 256 * i, k = q >> 5, c = q & 31;
      *reinterpret_cast<uint4*>(rt + tm_r_off(k, 8 * c)) = rreg[i];
    }
#pragma unroll
    for (int i = 0; i < kAChunks; ++i) {
      const int q = tid + 256 * i;
      *reinterpret_cast<uint4*>(at + tm_a_off(q >> 3, q & 7)) = areg[i];
    }
    __syncthreads();
    tm_load<kAChunks>(R, Lt, T, Tp, N, n0, t0 + kTmTok, t0 + kTmTok < t_end, tid, rreg, areg);
#pragma unroll
    for (int kk = 0; kk < kTmTok / 16; ++kk) {
      // lane l receives tokens 16kk + 8(l/32) + 0..7 of column 64 wave + 32 nt + l%32
      const int col = 64 * wave + 16 * (g & 1) + 4 * (i16 & 3);
      const int k0 = 16 * kk + 8 * (g >> 1) + (i16 >> 2);
      const bf16x8 fb[2] = {tm_frag(rt, k0, col), tm_frag(rt, k0, col + 32)};
#pragma unroll
      for (int jt = 0; jt < JT; ++jt)
#pragma unroll
        for (int hl = 0; hl < 2; ++hl) {
          const int q = hl * RW + 32 * jt + (lane & 31);
          bf16x8 fa;
          const uint4 v = *reinterpret_cast<const uint4*>(at + tm_a_off(q, 2 * kk + (lane >> 5)));
          __builtin_memcpy(&fa, &v, 16);
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
            acc[jt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa, fb[nt], acc[jt][nt], 0, 0, 0);
        }
    }
  }
  // lane l, register e: row j = 32 jt + 8(e/4) + 4(l/32) + e%4, column l%32
  float* pp = P.part + (int64_t)split * RW * N;
#pragma unroll
  for (int jt = 0; jt < JT; ++jt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const int n = n0 + 64 * wave + 32 * nt + (lane & 31);
      if (n >= N) continue;
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int j = 32 * jt + 8 * e4 + 4 * (lane >> 5);
        if (P.trans) {
          float4 v;
          v.x = acc[jt][nt][4 * e4];
          v.y = acc[jt][nt][4 * e4 + 1];
          v.z = acc[jt][nt][4 * e4 + 2];
          v.w = acc[jt][nt][4 * e4 + 3];
          *reinterpret_cast<float4*>(pp + (int64_t)n * RW + j) = v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) pp[(int64_t)(j + e) * N + n] = acc[jt][nt][4 * e4 + e];
        }
      }
    }
}

// Per expert: dA[j, i] = c * sum over splits (in order) of partA[s][j][i]
// (i < I, j < r), then dB[o, j] = c * sum over splits of partB[s][o][j]: one
// thread per output.  An expert without tokens (no splits) gets zeros.
struct RedProb {
  const float* partA;
  const float* partB;
  float* dA;
  float* dB;
  int splitsA, splitsB, blk0;
};
struct RedList {
  RedProb p[kLoraExperts];
  int n;
};
static_assert(sizeof(RedList) <= 4096, "kernel argument budget");

__global__ __launch_bounds__(256) void thin_m_reduce_kernel(RedList pl, int RW, int r, int I, int O, float c) {
  const int ei = find_product((int)blockIdx.x, pl.n, [&](int q) { return pl.p[q].blk0; });
  const RedProb& P = pl.p[ei];
  const int64_t e = (int64_t)((int)blockIdx.x - P.blk0) * 256 + threadIdx.x;
  const int64_t nA = (int64_t)r * I;
  if (e < nA) {
    const int j = (int)(e / I), i = (int)(e % I);
    float s = 0.0f;
    for (int q = 0; q < P.splitsA; ++q) s += P.partA[((int64_t)q * RW + j) * I + i];
    P.dA[e] = P.splitsA ? __fmul_rn(c, s) : 0.0f;
    return;
  }
  const int64_t f = e - nA;
  if (f >= (int64_t)r * O) return;
  const int o = (int)(f / r), j = (int)(f % r);
  float s = 0.0f;
  for (int q = 0; q < P.splitsB; ++q) s += P.partB[((int64_t)q * O + o) * RW + j];
  P.dB[f] = P.splitsB ? __fmul_rn(c, s) : 0.0f;
}

// Bt[RW, O] = B[O, r]^T with rows r .. RW-1 zero, for the experts of a launch
// set (grid.y; an expert without tokens has no Bt and is skipped); a
// workgroup moves 64 rows of B (at most 64 x 64 elements, 16 per thread, all
// loads issued first) through LDS so both sides are read and written
// contiguously.
struct BtList {
  const uint16_t* B[kLoraExperts];
  uint16_t* Bt[kLoraExperts];
};
__global__ __launch_bounds__(256) void transpose_b_kernel(BtList bl, int O, int r, int RW) {
  __shared__ uint16_t t[64][65];
  const uint16_t* __restrict__ B = bl.B[blockIdx.y];
  uint16_t* __restrict__ Bt = bl.Bt[blockIdx.y];
  if (Bt == nullptr) return;
  const int o0 = blockIdx.x * 64;
  const int rows = min(64, O - o0);
  const int n = rows * r;
  uint16_t v[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int e = threadIdx.x + 256 * u;
    v[u] = e < n ? B[(int64_t)o0 * r + e] : (uint16_t)0;
  }
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const int e = threadIdx.x + 256 * u;
    if (e < n) t[e / r][e % r] = v[u];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < RW * 64; e += 256) {
    const int k = e >> 6, ol = e & 63;
    if (ol < rows) Bt[(int64_t)k * O + o0 + ol] = k < r ? t[ol][k] : (uint16_t)0;
  }
}

namespace {
int rank_width(int r) { return r <= 32 ? 32 : 64; }
size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }
int64_t padded_tokens(int64_t T) { return (T + kTmTok - 1) / kTmTok * kTmTok; }

// Token range per workgroup of the token contraction: about 256 workgroups
// per product over its column tiles, in whole 64-token stages (chosen per
// expert, as for a single call, so a batched expert computes exactly what
// its own call computes).
int tokens_per_split(int64_t T, int N) {
  const int64_t Tp = padded_tokens(T);
  const int64_t tiles = (N + kTmCols - 1) / kTmCols;
  int64_t want = 256 / tiles;
  if (want < 1) want = 1;
  int64_t tps = (Tp + want - 1) / want;
  tps = (tps + kTmTok - 1) / kTmTok * kTmTok;
  return (int)(tps < kTmTok ? kTmTok : tps);
}
int64_t splits_of(int64_t T, int N) {
  const int tps = tokens_per_split(T, N);
  return (padded_tokens(T) + tps - 1) / tps;
}

TmProblem tm_problem(const uint16_t* Lt, const uint16_t* R, int T, int N, float* part, int trans) {
  TmProblem p;
  p.Lt = Lt;
  p.R = R;
  p.part = part;
  p.N = N;
  p.tiles = (N + kTmCols - 1) / kTmCols;
  p.tps = tokens_per_split(T, N);
  p.splits = (int)splits_of(T, N);
  p.trans = trans;
  p.T = T;
  p.Tp = (int)padded_tokens(T);
  p.blk0 = 0;
  return p;
}

// One expert's scratch: P and Q transposed as bf16 hi/lo [2][RW][Tp], B^T
// [RW][O], the token-range partials of dA and dB and the K-chunk partials of
// P and Q.  Nothing for an expert without tokens.
struct ExpertScratch {
  uint16_t *Pt, *Qt, *Bt;
  float *partA, *partB, *partP, *partQ;
};
size_t expert_scratch(int64_t T, int O, int I, int r, char* base, ExpertScratch* out) {
  if (T <= 0) {
    if (out) *out = ExpertScratch{};
    return 0;
  }
  const size_t RW = rank_width(r);
  const size_t Tp = (size_t)padded_tokens(T);
  const size_t kcI = (I + kThinKChunk - 1) / kThinKChunk, kcO = (O + kThinKChunk - 1) / kThinKChunk;
  const size_t sz[7] = {align256(2 * RW * Tp * 2), align256(2 * RW * Tp * 2), align256(RW * O * 2),
                        align256((size_t)splits_of(T, I) * I * RW * 4), align256((size_t)splits_of(T, O) * O * RW * 4),
                        align256(kcI * Tp * RW * 4), align256(kcO * Tp * RW * 4)};
  size_t at = 0;
  char* ptr[7];
  for (int k = 0; k < 7; ++k) {
    ptr[k] = base ? base + at : nullptr;
    at += sz[k];
  }
  if (out) {
    out->Pt = reinterpret_cast<uint16_t*>(ptr[0]);
    out->Qt = reinterpret_cast<uint16_t*>(ptr[1]);
    out->Bt = reinterpret_cast<uint16_t*>(ptr[2]);
    out->partA = reinterpret_cast<float*>(ptr[3]);
    out->partB = reinterpret_cast<float*>(ptr[4]);
    out->partP = reinterpret_cast<float*>(ptr[5]);
    out->partQ = reinterpret_cast<float*>(ptr[6]);
  }
  return at;
}
}  // namespace

size_t lora_grads_workspace(int T, int O, int I, int r) { return expert_scratch(T, O, I, r, nullptr, nullptr); }

size_t lora_grads_batched_workspace(int E, const int64_t* T, int O, int I, int r) {
  size_t total = 0;
  for (int e = 0; e < E; ++e) total += expert_scratch(T[e], O, I, r, nullptr, nullptr);
  return total;
}

// Experts e0 .. e0 + n - 1 (n <= kLoraExperts) in one launch set: B^T, P and
// Q, their transposed hi/lo pairs, the token contractions and the reduction.
// X and dY hold the experts' token rows one after another (tok0: the first
// row of expert e0); B, A, dB, dA are stacked [E, O, r], [E, r, I].
static int lora_set(int e0, int n, const int64_t* T, int64_t tok0, int O, int I, int r, const uint16_t* X,
                    const uint16_t* dY, const uint16_t* B, const uint16_t* A, float c, float* dB, float* dA,
                    char*& ws, hipStream_t s) {
  const int RW = rank_width(r);
  const int kcI = (I + kThinKChunk - 1) / kThinKChunk, kcO = (O + kThinKChunk - 1) / kThinKChunk;
  BtList bl{};
  ThinNList nl{};
  TmList ml{};
  RedList rl{};
  int nblk = 0, fblk = 0, mblk = 0, rblk = 0;
  int64_t tok = tok0;
  const int red_per = (int)(((int64_t)r * (I + O) + 255) / 256);
  for (int k = 0; k < n; ++k) {
    const int e = e0 + k;
    const int Te = (int)T[e];
    ExpertScratch w;
    ws += expert_scratch(Te, O, I, r, ws, &w);
    const uint16_t* xe = X + tok * I;
    const uint16_t* dye = dY + tok * O;
    tok += Te;
    bl.B[k] = B + (int64_t)e * O * r;
    bl.Bt[k] = w.Bt;
    RedProb rp{};
    rp.dA = dA + (int64_t)e * r * I;
    rp.dB = dB + (int64_t)e * O * r;
    rp.blk0 = rblk;
    rblk += red_per;
    if (Te > 0) {
      const int Tp = (int)padded_tokens(Te);
      ThinNProb P{xe, A + (int64_t)e * r * I, w.partP, w.Pt, I, kcI, Te, Tp, nblk, fblk};
      nblk += Tp / 32 * kcI;
      fblk += Tp / 32;
      ThinNProb Q{dye, w.Bt, w.partQ, w.Qt, O, kcO, Te, Tp, nblk, fblk};
      nblk += Tp / 32 * kcO;
      fblk += Tp / 32;
      nl.p[nl.n++] = P;
      nl.p[nl.n++] = Q;
      TmProblem ma = tm_problem(w.Qt, xe, Te, I, w.partA, 0);   // dA = c Q^T X
      ma.blk0 = mblk;
      mblk += ma.tiles * ma.splits;
      TmProblem mb = tm_problem(w.Pt, dye, Te, O, w.partB, 1);  // dB = c (P^T dY)^T
      mb.blk0 = mblk;
      mblk += mb.tiles * mb.splits;
      ml.p[ml.n++] = ma;
      ml.p[ml.n++] = mb;
      rp.partA = w.partA;
      rp.partB = w.partB;
      rp.splitsA = ma.splits;
      rp.splitsB = mb.splits;
    }
    rl.p[rl.n++] = rp;
  }
  if (nl.n > 0) {
    hipLaunchKernelGGL(transpose_b_kernel, dim3((unsigned)((O + 63) / 64), (unsigned)n), dim3(256), 0, s, bl, O,
                       r, RW);
    if (RW == 32) {
      hipLaunchKernelGGL(thin_n_kernel<1>, dim3((unsigned)nblk), dim3(512), 0, s, nl, r);
      hipLaunchKernelGGL(thin_n_finish_kernel<32>, dim3((unsigned)fblk), dim3(256), 0, s, nl);
      hipLaunchKernelGGL(thin_m_kernel<1>, dim3((unsigned)mblk), dim3(256), 0, s, ml);
    } else {
      hipLaunchKernelGGL(thin_n_kernel<2>, dim3((unsigned)nblk), dim3(512), 0, s, nl, r);
      hipLaunchKernelGGL(thin_n_finish_kernel<64>, dim3((unsigned)fblk), dim3(256), 0, s, nl);
      hipLaunchKernelGGL(thin_m_kernel<2>, dim3((unsigned)mblk), dim3(256), 0, s, ml);
    }
  }
  hipLaunchKernelGGL(thin_m_reduce_kernel, dim3((unsigned)rblk), dim3(256), 0, s, rl, RW, r, I, O, c);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int lora_grads_batched_launch(int E, const int64_t* T, int O, int I, int r, const void* X, const void* dY,
                              const void* B, const void* A, float c, float* dB, float* dA, void* workspace,
                              hipStream_t s) {
  char* ws = static_cast<char*>(workspace);
  int64_t tok = 0;
  for (int e0 = 0; e0 < E; e0 += kLoraExperts) {
    const int n = E - e0 < kLoraExperts ? E - e0 : kLoraExperts;
    if (lora_set(e0, n, T, tok, O, I, r, static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(dY),
                 static_cast<const uint16_t*>(B), static_cast<const uint16_t*>(A), c, dB, dA, ws, s) != 0)
      return -1;
    for (int k = 0; k < n; ++k) tok += T[e0 + k];
  }
  return 0;
}

int lora_grads_launch(int T, int O, int I, int r, const void* X, const void* dY, const void* B, const void* A,
                      float c, float* dB, float* dA, void* workspace, hipStream_t s) {
  const int64_t t = T;
  return lora_grads_batched_launch(1, &t, O, I, r, X, dY, B, A, c, dB, dA, workspace, s);
}

}  // namespace sq
