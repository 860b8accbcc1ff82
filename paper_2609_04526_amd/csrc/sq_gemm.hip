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
// All three feed v_mfma_f32_32x32x16_bf16 (fp32 accumulation) from LDS, in
// K stages of 64, on 256 x 256 tiles of 8 waves (128 x 64 each in the MXFP4
// forward, dX and dS; 64 x 128 in the LDS-dequantised forward) with two LDS
// stages; grids that would leave CUs idle use 128 x 128 tiles, and a grid
// ending in a short partial wave runs that remainder as half tiles.
// How each operand reaches the matrix cores:
//   * bf16 activations are copied global -> LDS by buffer loads that write LDS
//     directly (no registers), with reads past the operand's end returning
//     zeros (ragged tiles need no branches);
//   * K-contiguous tiles (X in FWD, dY in DX) are stored as 128-byte rows and
//     read with ds_read_b128;
//   * tiles that are contiguous along M or N (X and dY in DS, W in DX) are
//     stored in their natural [k][m] layout and read with the gfx950 LDS
//     transpose read ds_read_b64_tr_b16: within each 16-lane group, lane i
//     receives column i of the 4x16 block whose rows the group's lanes supply,
//     so two reads give a lane the 8 consecutive k of its MFMA operand;
//   * W in the MXFP4 forward: the packed codes are copied to LDS as they are
//     and each wave dequantises its own operand in registers (kFwdC);
//   * W elsewhere (dX, the NVFP4 forward): packed codes and scale bytes are
//     loaded into registers two stages ahead, dequantised exactly to bf16
//     (sq_device.h) and written to a double-buffered LDS tile once per
//     workgroup.
// Two schedules: the late-barrier one (MXFP4 forward, dX, dS; see `step2`)
// reads each slice's operands one slice ahead and publishes the next stage
// before the last slice's MFMAs; the LDS-dequantised forward waits for its
// stage, passes one s_barrier, issues the W loads, then runs four 16-deep
// MFMA slices with the next stage's DMA issued in quarters between them.
// Waits are explicit vmcnt counts and the barrier is the raw s_barrier, so
// later loads stay in flight across it.
//
// The DS epilogue multiplies each accumulator dW[o,j] by its E2M1 code and
// sums over the block in registers (the 32x32 MFMA output puts 8 of a
// 16-row block's rows in one lane and the other 8 in the lane 32 away), so
// dW never leaves the chip and dS is written once, without atomics.
//
// MoE experts (grouped calls) run the same tile code over one tile order of
// all experts, dealt to XCDs in contiguous stretches; grouped dS over short
// token sums runs as resident workgroups that stream their tiles' stages
// back to back (ds_stream_kernel).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <mutex>
#include <type_traits>
#include <vector>

#include "sq_device.h"
#include "sq_launch.h"

namespace sq {

// The three products.  Two forms of the forward:
//   kFwdR  W dequantised once per workgroup into a bf16 K-contiguous LDS tile;
//   kFwdC  (MXFP4) the packed codes are copied to LDS as they are and every
//          wave dequantises its own MFMA operand in registers: one
//          v_cvt_scalef32_pk_bf16_fp4 per code byte, with the E8M0 scale byte
//          as the convert's scale operand.  LDS carries 4 bits per weight
//          instead of 16, and no bf16 W tile is written.
enum Mode { kDx = 1, kDs = 2, kFwdR = 3, kFwdC = 4 };

constexpr int kBK = 64;                 // K per LDS stage
constexpr int kXcds = 8;                // MI355X: workgroups are dealt round-robin to 8 XCDs
constexpr uint32_t kOOB = 0x80000000u;  // a buffer offset past every operand: reads zero

#define SQ_LDS __attribute__((address_space(3)))
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

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
  int ksplit;             // DS: K (token) ranges per tile; >1 writes partial planes to `out`
  int ksteps_per;         // DS: K stages per range
  // the launch covers output rows [m_off, m_off + m_cnt) and columns
  // [n_off, n_off + n_cnt) (a count of 0: up to M or N)
  int m_off, m_cnt, n_off, n_cnt;
};

// Up to kGroupMax experts per grouped launch, passed by value (kernel
// arguments stay under 4 KiB): each kind of pointer is a base and a 32-bit
// byte offset per expert, so the run of experts a launch takes is cut short
// where the pointers of one kind would span 4 GiB or more.  The second
// operand is dS's dY, or the forward's and dX's scale plane.  An operand an
// expert does not have (null, read with a size of zero) gets offset 0.
struct GemmGroup {
  GemmArgs base;                  // shared: O, I, G, N (fwd/dx) or M, N (ds), out_bf16
  const uint8_t* a0;
  const uint8_t* p0;
  const uint8_t* codes0;
  uint8_t* out0;
  uint32_t a[kGroupMax];
  uint32_t p[kGroupMax];
  uint32_t codes[kGroupMax];
  uint32_t out[kGroupMax];
  int T[kGroupMax];
  float ws2[kGroupMax];
  int tile_begin[kGroupMax];
  int count;
  __device__ const uint16_t* act(int e) const { return reinterpret_cast<const uint16_t*>(a0 + a[e]); }
  __device__ const uint8_t* second(int e) const { return p0 + p[e]; }
  __device__ const uint8_t* code_plane(int e) const { return codes0 + codes[e]; }
  __device__ void* output(int e) const { return out0 + out[e]; }
};
static_assert(sizeof(GemmGroup) <= 4096, "kernel argument budget");

// Bases and offsets of experts p[0, n) (dS: the second operand is b, else
// the scale plane); false when one kind's pointers span 4 GiB or more.
static bool set_experts(GemmGroup& gg, const ExpertProblem* p, int n, bool ds) {
  auto pack = [&](auto get, const uint8_t*& base, uint32_t* off) {
    uintptr_t lo = UINTPTR_MAX, hi = 0;
    for (int e = 0; e < n; ++e) {
      const uintptr_t v = reinterpret_cast<uintptr_t>(get(p[e]));
      if (v == 0) continue;
      lo = v < lo ? v : lo;
      hi = v > hi ? v : hi;
    }
    if (lo == UINTPTR_MAX) lo = hi = 0;
    if (hi - lo > 0xFFFFFFFFu) return false;
    base = reinterpret_cast<const uint8_t*>(lo);
    for (int e = 0; e < n; ++e) {
      const uintptr_t v = reinterpret_cast<uintptr_t>(get(p[e]));
      off[e] = v == 0 ? 0u : (uint32_t)(v - lo);
    }
    return true;
  };
  const uint8_t* out0 = nullptr;
  const bool ok = pack([](const ExpertProblem& x) { return x.a; }, gg.a0, gg.a) &&
                  pack([ds](const ExpertProblem& x) { return ds ? x.b : static_cast<const void*>(x.scales); },
                       gg.p0, gg.p) &&
                  pack([](const ExpertProblem& x) { return x.codes; }, gg.codes0, gg.codes) &&
                  pack([](const ExpertProblem& x) { return x.out; }, out0, gg.out);
  gg.out0 = const_cast<uint8_t*>(out0);
  return ok;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

// Buffer descriptor of the global -> LDS copies: base, num_records = bytes
// (offsets at or past it read zeros), raw buffer flags.
typedef int i32x4 __attribute__((ext_vector_type(4)));
struct DmaRsrc {
  i32x4 v;
};
__device__ __forceinline__ DmaRsrc make_dma_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  DmaRsrc r;
  r.v = i32x4{__builtin_amdgcn_readfirstlane((int)(uint32_t)a), __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32) & 0xFFFF),
              __builtin_amdgcn_readfirstlane((int)bytes), 0x00020000};
  return r;
}

// 16 bytes per lane, global -> LDS; lane l writes dst + 16 l.  Written as
// the instruction itself: the compiler's wait insertion cannot tell the LDS
// tile a copy fills from the tile being read, and would otherwise stall
// every later LDS read until the copy lands.  The loop waits for the copies
// explicitly (vmcnt) before the barrier that publishes a stage.
__device__ __forceinline__ void dma16(DmaRsrc r, SQ_LDS void* dst, uint32_t voff) {
  const int lds = __builtin_amdgcn_readfirstlane((int)(uint32_t)reinterpret_cast<uintptr_t>(dst));
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds), "v"(voff), "s"(r.v)
               : "memory", "m0");
}

// Wait until at most n vector-memory loads of this wave are outstanding and
// all of its LDS operations are done (raw s_barrier has no memory semantics).
template <int n>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(n >= 0 && n < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0070 | (n & 15) | ((n >> 4) << 14));
}

// ------------------------------------------------------------------ layouts
// KC: K-contiguous [rows][64] bf16; 16-byte chunk c of row r lives at chunk
// c ^ swz_kc(r), so 8 consecutive rows read at one logical chunk hit 8
// different bank groups.
__device__ __forceinline__ int swz_kc(int r) { return (r ^ (r >> 3)) & 7; }
__device__ __forceinline__ int kc_off(int r, int c) { return r * kBK + ((c ^ swz_kc(r)) << 3); }

// NAT: [BK][R] bf16 with R elements per k-row; 16-byte chunk c of row k lives
// at chunk c ^ swz_nat(k): each of the 4 rows a 16-lane transpose read spans
// lands in its own 64-byte slot.
template <int R>
__device__ __forceinline__ int swz_nat(int k) { return (4 * (k & 7)) & (R / 8 - 1); }
template <int R>
__device__ __forceinline__ int nat_off(int k, int col) {
  return k * R + ((((col >> 3) ^ swz_nat<R>(k))) << 3) + (col & 7);
}

// MFMA operand (8 consecutive k at one m) from a NAT tile: rows
// 16*kk + 8*(lane/32) + 0..7 of column mbase + lane%32.
template <int R>
__device__ __forceinline__ bf16x8 nat_frag(const SQ_LDS uint16_t* s, int kk, int mbase, int lane) {
  const int i = lane & 15, g = lane >> 4;
  const int col = mbase + 16 * (g & 1) + 4 * (i & 3);
  const int row0 = 16 * kk + 8 * (g >> 1) + (i >> 2);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SQ_LDS v4i16*)(s + nat_off<R>(row0, col)));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SQ_LDS v4i16*)(s + nat_off<R>(row0 + 4, col)));
  bf16x8 r;
  __builtin_memcpy(&r, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&r) + 8, &hi, 8);
  return r;
}

// ------------------------------------------------------------------ DMA issue
// Each thread issues the same set of 16-byte buffer->LDS loads every stage,
// at byte offsets that advance by a fixed step per stage.  The offsets, their
// per-stage step and the K limit of each load are computed once.
//
// KC tile: rows [r0, r0+R) of a [rows_total, ld] bf16 matrix, k in
// [k0, k0+64); one wave instruction fills 8 consecutive LDS rows (1 KiB).
// Rows past the matrix read zeros from the buffer bound; k past kdim is
// masked explicitly on a ragged last stage.
template <int R, int NT>
struct DmaKC {
  static constexpr int kInst = R / 8 / (NT / 64);
  static_assert(kInst * (NT / 64) * 8 == R, "tile rows must split over the waves");
  uint32_t off[kInst];      // byte offset at k0 = 0 (kOOB if the row is outside)
  int klim[kInst];          // the load is valid while k0 < klim
  __device__ __forceinline__ void init(int ld, int rows_total, int kdim, int r0, int tid) {
    const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      const int blk = q * (NT / 64) + wave;
      const int r = blk * 8 + (lane >> 3);
      const int c = (lane & 7) ^ swz_kc(r);
      const int gr = r0 + r;
      off[q] = gr < rows_total ? (uint32_t)((size_t)gr * ld + c * 8) * 2u : kOOB;
      klim[q] = kdim - c * 8;
    }
  }
  __device__ __forceinline__ void issue(DmaRsrc rs, SQ_LDS uint16_t* s, int k0, bool full,
                                        int wave) const {
    issue_part<0, kInst>(rs, s, k0, full, wave);
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_part(DmaRsrc rs, SQ_LDS uint16_t* s, int k0, bool full,
                                             int wave) const {
#pragma unroll
    for (int q = Q0; q < Q1; ++q) {
      const int blk = q * (NT / 64) + wave;
      uint32_t o = off[q] + (uint32_t)k0 * 2u;
      if (!full && k0 >= klim[q]) o = kOOB;
      dma16(rs, s + blk * 8 * kBK, o);
    }
  }
};

// NAT tile: k-rows [k0, k0+BK) of a [kdim, ld] bf16 matrix, columns [m0, m0+R).
// Rows past kdim fall past the buffer's end and read zeros; columns past mdim
// only feed accumulators of rows/columns that are never stored.
template <int R, int NT, int BK>
struct DmaNat {
  static constexpr int kCpr = R / 8;                       // chunks per row
  static constexpr int kInst = BK * kCpr / 64 / (NT / 64);
  static_assert(kInst * (NT / 64) * 64 == BK * kCpr, "tile must split over the waves");
  uint32_t off[kInst];
  __device__ __forceinline__ void init(int ld, int mdim, int m0, int tid) {
    const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      const int blk = q * (NT / 64) + wave;
      const int p = blk * 64 + lane;
      const int k = p / kCpr, pc = p % kCpr;
      const int c = pc ^ swz_nat<R>(k);
      const int gm = m0 + c * 8;
      off[q] = gm < mdim ? (uint32_t)((size_t)k * ld + gm) * 2u : kOOB;
    }
  }
  __device__ __forceinline__ void issue(DmaRsrc rs, SQ_LDS uint16_t* s, uint32_t kstep_bytes,
                                        int wave) const {
    issue_part<0, kInst>(rs, s, kstep_bytes, wave);
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_part(DmaRsrc rs, SQ_LDS uint16_t* s, uint32_t kstep_bytes,
                                             int wave) const {
#pragma unroll
    for (int q = Q0; q < Q1; ++q) {
      const int blk = q * (NT / 64) + wave;
      const uint32_t o = off[q] == kOOB ? kOOB : off[q] + kstep_bytes;
      dma16(rs, s + blk * 64 * 8, o);
    }
  }
};

// Code tile (kFwdC): rows [r0, r0+R) of the packed [O, I/2] code plane, the 32
// bytes (64 codes) of one K stage per row, stored row after row, 16-byte half
// h of row r at half h ^ swz_codes(r): the 16 (or 8) lanes a ds_read_b128
// serves together read 16 consecutive rows at one logical half and so land
// in 16 distinct 16-byte bank slots.  One wave instruction fills 32 rows
// (lane l: row l/2, stored half l%2).  Rows past O read zeros from the buffer
// bound; a half past I is masked on the last stage.
__device__ __forceinline__ int swz_codes(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }
template <int R, int NT>
struct DmaCodes {
  // wave instructions per stage (32 rows each), spread over the waves; when
  // there are fewer than waves, the first ones issue one each
  static constexpr int kWaveInst = R / 32;
  static constexpr int kInst = kWaveInst >= NT / 64 ? kWaveInst / (NT / 64) : 1;
  static_assert(kWaveInst >= NT / 64 ? kInst * (NT / 64) == kWaveInst : (NT / 64) % kWaveInst == 0,
                "code rows must split over the waves");
  uint32_t off[kInst];
  int klim[kInst];
  __device__ __forceinline__ void init(int I, int O, int r0, int tid) {
    const int wave = tid >> 6, lane = tid & 63;
#pragma unroll
    for (int q = 0; q < kInst; ++q) {
      const int r = (q * (NT / 64) + wave) * 32 + (lane >> 1);
      const int h = (lane & 1) ^ swz_codes(r);
      const int gr = r0 + r;
      off[q] = gr < O && r < R ? (uint32_t)gr * (uint32_t)(I >> 1) + 16u * (uint32_t)h : kOOB;
      klim[q] = I - 32 * h;
    }
  }
  template <int Q0, int Q1>
  __device__ __forceinline__ void issue_part(DmaRsrc rs, SQ_LDS uint8_t* s, int k0, int wave) const {
    if (kWaveInst < NT / 64 && wave >= kWaveInst) return;     // wave-uniform
#pragma unroll
    for (int q = Q0; q < Q1; ++q) {
      const int blk = q * (NT / 64) + wave;
      const uint32_t o = (off[q] == kOOB || k0 >= klim[q]) ? kOOB : off[q] + (uint32_t)(k0 >> 1);
      dma16(rs, s + blk * 1024, o);
    }
  }
};

// 16-byte DMA loads each thread issues per stage (only the mode's own
// operand layouts are instantiated)
template <int MODE, int BM, int BN, int NT, int BK>
__host__ __device__ constexpr int dma_count() {
  if constexpr (MODE == kDx || MODE == kFwdR) return DmaKC<BM, NT>::kInst;
  else if constexpr (MODE == kFwdC) return DmaKC<BM, NT>::kInst + DmaCodes<BN, NT>::kInst;
  else return DmaNat<BM, NT, BK>::kInst + DmaNat<BN, NT, BK>::kInst;
}

// ------------------------------------------------------------------ tile order
// Workgroup w runs on XCD w % 8, and each XCD has its own L2.  Tiles are
// enumerated in groups of kGroupM tile-rows (column by column inside a group)
// and each XCD is given one contiguous stretch of that order, so the
// workgroups that share an L2 also share operand panels.  With 32 tiles per
// XCD, a height of 4 gives each XCD 4 activation panels (2 MiB each at 4096
// tokens) and 8 code panels (0.5 MiB): 96 MiB fetched per 4096^3 forward or
// dX against 144 MiB at height 8, in the same time.  For dS both operands are
// 2 MiB panels and heights 4 and 8 fetch the same.
template <int MODE>
constexpr int group_m() {
  return MODE == kDs ? 8 : 4;
}

// Position in the tile order of workgroup bid of nb: XCD x = bid % 8 takes
// the x-th contiguous stretch of the order (stretches differ by at most one).
__device__ __forceinline__ int xcd_stretch(int bid, int nb) {
  const int x = bid % kXcds, q = nb / kXcds, r = nb % kXcds;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + bid / kXcds;
}

// Tile (tm, tn) at position idx of the grouped column-by-column order.
template <int kGroupM>
__device__ __forceinline__ void tile_at(int idx, int tiles_m, int tiles_n, int& tm, int& tn) {
  const int per_group = kGroupM * tiles_n;
  const int group = idx / per_group;
  const int first_m = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first_m);
  const int in = idx - group * per_group;
  tm = first_m + in % gm;
  tn = in / gm;
}

template <int kGroupM>
__device__ __forceinline__ void tile_of(int bid, int nb, int tiles_m, int tiles_n, int& tm, int& tn) {
  tile_at<kGroupM>(xcd_stretch(bid, nb), tiles_m, tiles_n, tm, tn);
}

template <int MODE, int BM, int BN, int STAGES, int BK, int NW>
struct SmemLayout {
  static constexpr int kA = BM * BK * 2;                                      // bytes per A stage
  static constexpr int kB = BK * BN * 2;                                      // bytes per B stage
  static constexpr bool kWReg = MODE == kDx || MODE == kFwdR;                 // W staged through registers
  static constexpr int kCodes = MODE == kFwdC ? BN * (BK / 2) : 0;            // packed codes per stage
  static constexpr int kStage = kA + (kWReg || MODE == kFwdC ? 0 : kB) + kCodes;   // DMA bytes per stage
  static constexpr int kWBytes = kWReg ? 2 * kB : 0;                          // bf16 W double buffer
  // kFwdC has no W buffer: its stage arrays are sized to also hold the bf16
  // output staging of every wave (one (BM x BN / NW) bf16 region per wave,
  // whole regions per stage array)
  static constexpr int kEpiRegion = BM * BN * 2 / NW;
  static constexpr int kEpiPer = (NW + STAGES - 1) / STAGES * kEpiRegion;
  static constexpr int kStageAlloc = MODE == kFwdC && kEpiPer > kStage ? kEpiPer : kStage;
  static constexpr int kBytes = STAGES * kStageAlloc + kWBytes;
};

// ------------------------------------------------------------------ output
// Output element offsets stay below 2^31: every output holds fewer than 2^31
// elements, since each of T, O and I times the other operand dimension does.
template <bool CHECK, int FMT, int TM, int TN>
__device__ __forceinline__ void epi_store_direct(const f32x16 (&acc)[TM][TN], const GemmArgs& g, int r0, int c0,
                                                 int lane) {
  const int lrow = 4 * (lane >> 5), lcol = lane & 31;
  const float f = g.ws2;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = c0 + j * 32 + lcol;
      if (CHECK && col >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = r0 + i * 32 + 8 * (r >> 2) + lrow + (r & 3);
        if (CHECK && row >= g.M) continue;
        const float v = (FMT == kNV) ? acc[i][j][r] * f : acc[i][j][r];
        const uint32_t at = (uint32_t)row * (uint32_t)g.N + (uint32_t)col;
        if (g.out_bf16)
          reinterpret_cast<uint16_t*>(g.out)[at] = (uint16_t)f32_to_bf16_rne(v);
        else
          reinterpret_cast<float*>(g.out)[at] = v;
      }
    }
}

// Staged bf16 store of one wave's (32*TM) x (32*TN) block, fully inside the
// output.  LDS holds the block column-major in 8-byte units of 4 rows; unit
// (col, q) sits at col * (WM/4) + (q ^ (4*(col%4) + (col/4)%4) % (WM/4)), so
// the 4-row writes of 16 consecutive columns and the transposing reads of a
// 4-column x 16-row patch each touch 16 distinct 8-byte bank slots.  A
// transposing read gives lane i of a 16-lane group row i of 4 consecutive
// columns; two of them make one 16-byte store.
template <int WM>
__device__ __forceinline__ int epi_unit(int col, int q) {
  const int f = 4 * (col & 3) + ((col >> 2) & 3);
  return col * (WM / 4) + ((q ^ f) & (WM / 4 - 1));
}
template <int FMT, int TM, int TN>
__device__ __forceinline__ void epi_store_bf16(const f32x16 (&acc)[TM][TN], SQ_LDS uint16_t* s, const GemmArgs& g,
                                               int r0, int c0, int lane) {
  constexpr int WM = 32 * TM, WN = 32 * TN;
  const float f = g.ws2;
  const int lq = lane >> 5, lcol = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        typedef float f2 __attribute__((ext_vector_type(2)));
        typedef __bf16 b2 __attribute__((ext_vector_type(2)));
        f2 lo = {acc[i][j][4 * q], acc[i][j][4 * q + 1]};
        f2 hi = {acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if constexpr (FMT == kNV) { lo = lo * f; hi = hi * f; }
        const b2 blo = __builtin_convertvector(lo, b2), bhi = __builtin_convertvector(hi, b2);
        v4i16 v;
        __builtin_memcpy(&v, &blo, 4);
        __builtin_memcpy(reinterpret_cast<char*>(&v) + 4, &bhi, 4);
        // rows i*32 + 8q + 4*lq .. +3 of column j*32 + lcol
        *(SQ_LDS v4i16*)(s + 4 * epi_unit<WM>(j * 32 + lcol, i * 8 + 2 * q + lq)) = v;
      }
  // lane i of group gq: row 16p + i, columns cb*32 + 8gq .. +7
  const int li = lane & 15, gq = lane >> 4;
  uint16_t* out = reinterpret_cast<uint16_t*>(g.out);
#pragma unroll
  for (int p = 0; p < WM / 16; ++p)
#pragma unroll
    for (int cb = 0; cb < WN / 32; ++cb) {
      v4i16 h[2];
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const int col = cb * 32 + 8 * gq + 4 * e + (li >> 2);
        const int q = 4 * p + (li & 3);
        h[e] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SQ_LDS v4i16*)(s + 4 * epi_unit<WM>(col, q)));
      }
      u32x4 w;
      __builtin_memcpy(&w, h, 16);
      const uint32_t at = (uint32_t)(r0 + 16 * p + li) * (uint32_t)g.N + (uint32_t)(c0 + cb * 32 + 8 * gq);
      *reinterpret_cast<u32x4*>(out + at) = w;
    }
}

// ------------------------------------------------------------------ dS epilogue
// A dS tile's rows are input features j, its columns output features o.  In
// 32x32 MFMA tile (i, j) lane l holds rows 8 q + 4 (l / 32) + 0..3 (q = 0..3)
// of column l % 32, and each group of 4 rows takes its 4 codes from one
// 16-bit pair of the packed plane.  The 16 bytes of codes of row o and the
// tile's 32 features hold the pairs of both lane halves; cw[j TM + i] is that
// chunk, zeros for a row outside the layer.  The chunk starts at byte
// o I / 2 + jb / 2: 16-byte aligned for MXFP4 (I is a multiple of 32), 8-byte
// aligned for NVFP4 (a multiple of 16), which loads it as two halves.
template <int FMT, int TM, int TN>
__device__ __forceinline__ void ds_codes(u32x4 (&cw)[TM * TN], const uint8_t* codes, int O, int I, int r0, int c0,
                                         int lane) {
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(codes, (uint32_t)((size_t)O * (I >> 1)));
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int o = c0 + j * 32 + (lane & 31);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int jb = r0 + i * 32;
      const uint32_t off = o < O && jb < I ? (uint32_t)o * (uint32_t)(I >> 1) + (uint32_t)(jb >> 1) : kOOB;
      if constexpr (FMT == kMX) {
        cw[j * TM + i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0));
      } else {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)off, 0, 0));
        const u32x2 hi = __builtin_bit_cast(
            u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)(off == kOOB ? kOOB : off + 8u), 0, 0));
        cw[j * TM + i] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      }
    }
  }
}

// Products with the codes, summed over each scale block (32 features for
// MXFP4, 16 for NVFP4; the 32 rows of an MFMA tile are split over the two
// lane halves) and stored to dS[o, block].
// INTERIOR: the tile lies inside the layer (every row below I, every column
// below O), so no element needs a range check.
template <int FMT, int TM, int TN, bool INTERIOR>
__device__ __forceinline__ void ds_store(const f32x16 (&acc)[TM][TN], const u32x4 (&cw)[TM * TN], float* dS, int O,
                                         int I, int G, int r0, int c0, int lane) {
  const int lrow = 4 * (lane >> 5);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int o = c0 + j * 32 + (lane & 31);
    const bool o_ok = INTERIOR || o < O;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int jb = r0 + i * 32;          // first feature of this 32-row tile
      float prod[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        // the pair of rows jb + 8 q + lrow .. + 3: bytes 4 q + lrow / 2 of the
        // chunk, decoded two codes per convert (E2M1 values are exact in fp32)
        const uint32_t c = INTERIOR || jb + 8 * q + lrow < I ? cw[j * TM + i][q] >> (4 * lrow) : 0u;
        typedef float f32x2 __attribute__((ext_vector_type(2)));
        const f32x2 v01 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 0);
        const f32x2 v23 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(c, 1.0f, 1);
        prod[4 * q + 0] = acc[i][j][4 * q + 0] * v01[0];
        prod[4 * q + 1] = acc[i][j][4 * q + 1] * v01[1];
        prod[4 * q + 2] = acc[i][j][4 * q + 2] * v23[0];
        prod[4 * q + 3] = acc[i][j][4 * q + 3] * v23[1];
      }
      if constexpr (FMT == kMX) {
        float s = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) s += prod[r];
        s += __shfl_xor(s, 32);
        if (lane < 32 && o_ok && (INTERIOR || jb < I)) dS[(size_t)o * G + jb / 32] = s;
      } else {
        float s0 = 0.0f, s1 = 0.0f;
#pragma unroll
        for (int r = 0; r < 8; ++r) { s0 += prod[r]; s1 += prod[8 + r]; }
        s0 += __shfl_xor(s0, 32);
        s1 += __shfl_xor(s1, 32);
        const int b = jb / 16 + (lane >> 5);
        const float s = (lane < 32) ? s0 : s1;
        if (o_ok && (INTERIOR || b * 16 < I)) dS[(size_t)o * G + b] = s;
      }
    }
  }
}

// ------------------------------------------------------------------ kernel
// Block tile BM x BN, WGM x WGN waves, each wave (BM/WGM) x (BN/WGN) built
// from 32x32 MFMA tiles; STAGES LDS stages for the DMA operands.
// One workgroup's tile: bid is its index among the nb workgroups of one
// product, dealt to XCDs by bid % 8; with ORDERED, bid is already the tile's
// position in the product's tile order (the grouped launch deals its XCD
// stretches over all experts at once).
template <int MODE, int FMT, int BM, int BN, int WGM, int WGN, int STAGES, int BK, bool ORDERED = false>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int bid, int nb) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int B = ScaleOperand<FMT>::kBlock;
  // every schedule reads a stage as four 16-deep MFMA slices
  static_assert(BK == kBK, "64-deep stages");
  using L = SmemLayout<MODE, BM, BN, STAGES, BK, WGM * WGN>;
  constexpr bool kWReg = L::kWReg;
  constexpr int kDma = dma_count<MODE, BM, BN, NT, BK>();   // DMA loads per thread per stage
  // One static array per DMA stage (distinct objects, so the compiler can see
  // that a stage being filled does not alias the stage being read).
  __shared__ __attribute__((aligned(16))) uint8_t lds0[L::kStageAlloc];
  __shared__ __attribute__((aligned(16))) uint8_t lds1[L::kStageAlloc];
  __shared__ __attribute__((aligned(16))) uint8_t lds2[STAGES > 2 ? L::kStageAlloc : 16];
  __shared__ __attribute__((aligned(16))) uint8_t lds3[STAGES > 3 ? L::kStageAlloc : 16];
  __shared__ __attribute__((aligned(16))) uint8_t ldsw[kWReg ? L::kWBytes : 16];
  static_assert(STAGES >= 2 && STAGES <= 4, "2 to 4 stages");
  // The bf16 output staging reuses the operand LDS: one WM x WN bf16 region
  // per wave, taken from the stage arrays and the W buffer in turn.
  constexpr int kEpiRegion = WM * WN * 2;
  constexpr int kEpiPerStage = L::kStageAlloc / kEpiRegion, kEpiPerW = (kWReg ? L::kWBytes : 0) / kEpiRegion;
  constexpr bool kEpiStaged =
      MODE != kDs && WM >= 16 && (WM & (WM - 1)) == 0 && WN % 32 == 0 && STAGES * kEpiPerStage + kEpiPerW >= WGM * WGN;
  auto epi_region = [&](int w) -> SQ_LDS uint16_t* {
    SQ_LDS uint8_t* base;
    if (w < kEpiPerStage) base = (SQ_LDS uint8_t*)lds0 + w * kEpiRegion;
    else if (w < 2 * kEpiPerStage) base = (SQ_LDS uint8_t*)lds1 + (w - kEpiPerStage) * kEpiRegion;
    else if (STAGES > 2 && w < 3 * kEpiPerStage) base = (SQ_LDS uint8_t*)lds2 + (w - 2 * kEpiPerStage) * kEpiRegion;
    else if (STAGES > 3 && w < 4 * kEpiPerStage) base = (SQ_LDS uint8_t*)lds3 + (w - 3 * kEpiPerStage) * kEpiRegion;
    else base = (SQ_LDS uint8_t*)ldsw + (w - STAGES * kEpiPerStage) * kEpiRegion;
    return (SQ_LDS uint16_t*)base;
  };

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int tiles_m = ((g.m_cnt ? g.m_cnt : g.M) + BM - 1) / BM, tiles_n = ((g.n_cnt ? g.n_cnt : g.N) + BN - 1) / BN;
  // a DS launch with split K runs ksplit workgroups per tile, each over its
  // own range of K stages
  const int tiles = tiles_m * tiles_n;
  const int split = (MODE == kDs && g.ksplit > 1) ? bid / tiles : 0;
  int tm, tn;
  if constexpr (ORDERED) tile_at<group_m<MODE>()>(bid, tiles_m, tiles_n, tm, tn);
  else tile_of<group_m<MODE>()>((MODE == kDs && g.ksplit > 1) ? bid - split * tiles : bid, (MODE == kDs && g.ksplit > 1) ? tiles : nb,
                                tiles_m, tiles_n, tm, tn);
  const int m0 = g.m_off + tm * BM, n0 = g.n_off + tn * BN;

  auto stage = [&](auto SC) -> SQ_LDS uint8_t* {
    constexpr int S = decltype(SC)::value;
    if constexpr (S == 0) return (SQ_LDS uint8_t*)lds0;
    else if constexpr (S == 1) return (SQ_LDS uint8_t*)lds1;
    else if constexpr (S == 2) return (SQ_LDS uint8_t*)lds2;
    else return (SQ_LDS uint8_t*)lds3;
  };

  DmaRsrc ra, rb;
  if constexpr (MODE == kFwdR) {
    ra = make_dma_rsrc(g.a, (uint32_t)((size_t)g.T * g.I * 2));
  } else if constexpr (MODE == kFwdC) {
    ra = make_dma_rsrc(g.a, (uint32_t)((size_t)g.T * g.I * 2));
    rb = make_dma_rsrc(g.codes, (uint32_t)((size_t)g.O * g.I / 2));
  } else if constexpr (MODE == kDx) {
    ra = make_dma_rsrc(g.a, (uint32_t)((size_t)g.T * g.O * 2));
  } else {
    ra = make_dma_rsrc(g.a, (uint32_t)((size_t)g.T * g.I * 2));
    rb = make_dma_rsrc(g.b, (uint32_t)((size_t)g.T * g.O * 2));
  }

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk_all = (g.K + BK - 1) / BK;
  const int kofs = (MODE == kDs && g.ksplit > 1) ? split * g.ksteps_per : 0;   // first K stage of this range
  const int nk = (MODE == kDs && g.ksplit > 1) ? min(g.ksteps_per, nk_all - kofs) : nk_all;

  // ---- DMA of one K stage into stage buffer SC
  using DA_kc = std::conditional_t<MODE != kDs, DmaKC<BM, NT>, DmaKC<8 * NT / 64, NT>>;  // unused in DS
  using DA_nat = std::conditional_t<MODE == kDs, DmaNat<BM, NT, BK>, DmaNat<512, NT, 64>>;
  using DB_nat = std::conditional_t<MODE == kDs, DmaNat<BN, NT, BK>, DmaNat<512, NT, 64>>;
  using DC = std::conditional_t<MODE == kFwdC, DmaCodes<BN, NT>, DmaCodes<NT / 2, NT>>;   // used by kFwdC
  DA_kc dA_kc;
  DA_nat dA_nat;
  DB_nat dB_nat;
  DC dC;
  if constexpr (MODE == kFwdR) {
    dA_kc.init(g.I, g.T, g.I, m0, tid);
  } else if constexpr (MODE == kFwdC) {
    dA_kc.init(g.I, g.T, g.I, m0, tid);
    dC.init(g.I, g.O, n0, tid);
  } else if constexpr (MODE == kDx) {
    dA_kc.init(g.O, g.T, g.O, m0, tid);
  } else {
    dA_nat.init(g.I, g.I, m0, tid);
    dB_nat.init(g.O, g.O, n0, tid);
  }
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto issue_dma = [&](auto SC, int kt) {
    SQ_LDS uint8_t* st = stage(SC);
    const int k0 = (kofs + kt) * BK;
    const bool full = k0 + BK <= g.K;
    if constexpr (MODE == kFwdR || MODE == kDx) {
      dA_kc.issue(ra, (SQ_LDS uint16_t*)st, k0, full, wave_u);
    } else if constexpr (MODE == kFwdC) {
      dA_kc.issue(ra, (SQ_LDS uint16_t*)st, k0, full, wave_u);
      dC.template issue_part<0, DC::kInst>(rb, st + L::kA, k0, wave_u);
    } else {
      dA_nat.issue(ra, (SQ_LDS uint16_t*)st, (uint32_t)k0 * (uint32_t)g.I * 2u, wave_u);
      dB_nat.issue(rb, (SQ_LDS uint16_t*)(st + L::kA), (uint32_t)k0 * (uint32_t)g.O * 2u, wave_u);
    }
  };

  // Quarter PART of the DMA of stage kt (the spread schedule issues one
  // quarter after each 16-deep slice of MFMAs instead of all at the start).
  auto dma_part = [&](auto SC, int kt, auto PART) {
    constexpr int P = decltype(PART)::value;
    SQ_LDS uint8_t* st = stage(SC);
    const int k0 = (kofs + kt) * BK;
    const bool full = k0 + BK <= g.K;
    if constexpr (MODE == kFwdR || MODE == kDx || MODE == kFwdC) {
      constexpr int n = decltype(dA_kc)::kInst;
      dA_kc.template issue_part<P * n / 4, (P + 1) * n / 4>(ra, (SQ_LDS uint16_t*)st, k0, full, wave_u);
      if constexpr (MODE == kFwdC && P == 0) dC.template issue_part<0, DC::kInst>(rb, st + L::kA, k0, wave_u);
    } else if constexpr (MODE == kDs) {
      constexpr int na = decltype(dA_nat)::kInst, nb = decltype(dB_nat)::kInst;
      dA_nat.template issue_part<P * na / 4, (P + 1) * na / 4>(ra, (SQ_LDS uint16_t*)st,
                                                              (uint32_t)k0 * (uint32_t)g.I * 2u, wave_u);
      dB_nat.template issue_part<P * nb / 4, (P + 1) * nb / 4>(rb, (SQ_LDS uint16_t*)(st + L::kA),
                                                              (uint32_t)k0 * (uint32_t)g.O * 2u, wave_u);
    }
  };
  // The LDS-dequantised forward (kFwdR) runs the two-stage schedule of
  // `step`; the MXFP4 register forward, dX and dS run the late-barrier
  // schedule of `step2`.
  constexpr bool kLate = MODE == kFwdC || MODE == kDs || MODE == kDx;
  static_assert(kLate || STAGES == 2, "the early-barrier schedule keeps two stages");

  // ---- W through registers (DX: W^T tile [64 o][BN i]; FWDR: W tile
  // [BN o][64 i]), one dword of 8 codes along i per item, dequantised and
  // written to LDS as bf16
  constexpr int kWPer = kWReg ? kBK * (BN / 8) / NT : 1;
  static_assert(!kWReg || kWPer * NT == kBK * (BN / 8), "W tile must split over the threads");
  // The forward fetches W two stages ahead through branch-free buffer loads
  // (an item outside the layer reads at an offset past the operand: zeros),
  // so the wait before a dequantisation leaves the newer loads in flight.
  // dX tiles below 256 x 256 convert a stage's W items in the middle of the
  // step before it (see step2), which takes a second register set; the
  // 256 x 256 tile has no registers to spare and converts them right after
  // the barrier that frees their buffer
  constexpr bool kWMid = MODE == kDx && BM * BN < 256 * 256;
  constexpr int kWAhead = (MODE == kFwdR || kWMid) ? 2 : 1;   // register sets of W items
  uint32_t w_reg[kWAhead][kWPer], w_sb[kWAhead][kWPer];
  // Forward W items: row o = n0 + idx/8 is fixed, the 8 columns start at
  // kt*64 + (idx%8)*8, so each item keeps byte offsets at kt = 0 (past the
  // operand for rows outside the layer) and a column limit.
  __amdgpu_buffer_rsrc_t rw_codes, rw_scales;
  constexpr bool kFwdAhead = MODE == kFwdR && kWAhead == 2;
  uint32_t wc0[kFwdAhead ? kWPer : 1], ws0[kFwdAhead ? kWPer : 1];
  int wklim = 0;
  // dX W items: item p of thread tid is row kt*64 + tid/(BN/8) + p*NT/(BN/8)
  // of W^T's stage and the 8 columns from n0 + (tid % (BN/8))*8, the same
  // columns for every p; a column block outside the layer is marked kOOB and
  // a row past O reads at kOOB, so the loads take no branches.
  constexpr bool kDxFree = MODE == kDx;
  uint32_t dxc = 0, dxs = 0;
  if constexpr (kDxFree) {
    static_assert(NT % (BN / 8) == 0, "every item of a thread keeps its columns");
    rw_codes = make_rsrc(g.codes, (uint32_t)((size_t)g.O * g.I / 2));
    rw_scales = make_rsrc(g.scales, (uint32_t)((size_t)g.O * g.G));
    const int i = n0 + (tid % (BN / 8)) * 8;
    dxc = i < g.I ? (uint32_t)(i >> 1) : kOOB;
    dxs = i < g.I ? (uint32_t)(i / B) : kOOB;
  }
  if constexpr (kFwdAhead) {
    rw_codes = make_rsrc(g.codes, (uint32_t)((size_t)g.O * g.I / 2));
    rw_scales = make_rsrc(g.scales, (uint32_t)((size_t)g.O * g.G));
    const int c8 = (tid % 8) * 8;
    wklim = g.I - c8;                       // the item is inside while kt*64 < wklim
#pragma unroll
    for (int p = 0; p < kWPer; ++p) {
      const int o = n0 + (tid + p * NT) / 8;
      wc0[p] = o < g.O ? (uint32_t)o * (uint32_t)(g.I >> 1) + (uint32_t)(c8 >> 1) : kOOB;
      ws0[p] = o < g.O ? (uint32_t)o * (uint32_t)g.G + (uint32_t)(c8 / B) : kOOB;
    }
  }
  auto load_w = [&](int kt, auto BUF) {
    constexpr int u = decltype(BUF)::value;
    if constexpr (kWReg) {
#pragma unroll
      for (int p = 0; p < kWPer; ++p) {
        if constexpr (kFwdAhead) {
          const bool in = kt * kBK < wklim;
          const uint32_t oc = in ? wc0[p] + (uint32_t)kt * (kBK / 2) : kOOB;
          const uint32_t os = in ? ws0[p] + (uint32_t)kt * (kBK / B) : kOOB;
          w_reg[u][p] = __builtin_amdgcn_raw_buffer_load_b32(rw_codes, (int)oc, 0, 0);
          w_sb[u][p] = __builtin_amdgcn_raw_buffer_load_b8(rw_scales, (int)os, 0, 0);
          continue;
        }
        if constexpr (kDxFree) {
          const int o = kt * kBK + tid / (BN / 8) + p * (NT / (BN / 8));
          const bool in = o < g.O && dxc != kOOB;
          const uint32_t oc = in ? (uint32_t)o * (uint32_t)(g.I >> 1) + dxc : kOOB;
          const uint32_t os = in ? (uint32_t)o * (uint32_t)g.G + dxs : kOOB;
          w_reg[u][p] = __builtin_amdgcn_raw_buffer_load_b32(rw_codes, (int)oc, 0, 0);
          w_sb[u][p] = __builtin_amdgcn_raw_buffer_load_b8(rw_scales, (int)os, 0, 0);
        }
      }
    }
  };
  auto wbuf = [&](int kt) { return (SQ_LDS uint16_t*)((SQ_LDS uint8_t*)ldsw + (kt & 1) * L::kB); };
  auto commit_w = [&](int kt, auto BUF) {
    constexpr int u = decltype(BUF)::value;
    if constexpr (kWReg) {
      SQ_LDS uint16_t* s = wbuf(kt);
#pragma unroll
      for (int p = 0; p < kWPer; ++p) {
        const int idx = tid + p * NT;
        const uint4 d = ScaleOperand<FMT>::dequant8(w_reg[u][p], ScaleOperand<FMT>::of(w_sb[u][p]));
        u32x4 v;
        __builtin_memcpy(&v, &d, 16);
        if constexpr (MODE == kDx)
          *(SQ_LDS u32x4*)(s + nat_off<BN>(idx / (BN / 8), (idx % (BN / 8)) * 8)) = v;
        else
          *(SQ_LDS u32x4*)(s + kc_off(idx / 8, idx % 8)) = v;
      }
    }
  };

  // ---- kFwdC: the E8M0 scale bytes of the wave's code rows.  Lane (n, h) of
  // 32-row slice j uses row n0 + wn0 + 32 j + n, block 2 kt + h (the 32 codes
  // of that block are the lane's half of stage kt).  Two 8-byte loads per
  // slice bring the row's 16 blocks of 8 stages; the next 16 bytes are
  // loaded during the last of those stages, into the same registers, once
  // that stage's scale operands have been taken.  The launcher takes this
  // path only when G is a multiple of 8 (I % 256 == 0), so every stage is
  // whole and each 8-byte half starts 8-byte aligned; the last chunk of a row
  // may run into the next row (bytes no stage uses).  A row outside the
  // layer, and a half past the plane, read zeros.
  constexpr int kSc = MODE == kFwdC ? TN : 1;
  u32x4 scw[kSc];
  uint32_t sc0[kSc];
  __amdgpu_buffer_rsrc_t rs_sc;
  if constexpr (MODE == kFwdC) {
    static_assert(FMT == kMX && BK == 64, "register dequantisation: MXFP4, 64-deep stages");
    rs_sc = make_rsrc(g.scales, (uint32_t)((size_t)g.O * g.G));
#pragma unroll
    for (int j = 0; j < kSc; ++j) {
      const int row = n0 + wn0 + 32 * j + (lane & 31);
      sc0[j] = row < g.O ? (uint32_t)row * (uint32_t)g.G : kOOB;
    }
  }
  auto load_sc = [&](int chunk) {
    if constexpr (MODE == kFwdC) {
#pragma unroll
      for (int j = 0; j < kSc; ++j) {
        typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
        const uint32_t off = sc0[j] + 16u * (uint32_t)chunk;
        const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs_sc, (int)off, 0, 0));
        const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs_sc, (int)(off + 8u), 0, 0));
        scw[j] = u32x4{lo[0], lo[1], hi[0], hi[1]};
      }
    }
  };

  // ---- one K stage of the early-barrier schedule (kFwdR): wait for its
  // data, refill the oldest stage, multiply
  static_assert(kLate || MODE == kFwdR, "the early-barrier schedule serves the LDS-dequantised forward");
  auto step = [&](auto SC, int kt) {
    constexpr int S = decltype(SC)::value;
    constexpr int SNEXT = (S + STAGES - 1) % STAGES;          // stage that receives kt + STAGES - 1
    // stage kt is complete once every load this thread issued has landed:
    // the last DMA quarter went out at the end of the previous step, and the
    // W registers of stage kt + 2 are loaded after this wait
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (kWAhead == 2) load_w(kt + 2, std::integral_constant<int, S % 2>{});
    __builtin_amdgcn_sched_barrier(0);

    // quarters 2 s and 2 s + 1 of the next stage's DMA are issued between the
    // operand reads and the MFMAs of slice s (s = 0, 1)
    auto slot_of = [](int q) { return q / 2; };
    auto before_mfma = [&](int kk) {
      if constexpr (!kLate) {
        if (kWAhead == 2 || kt + STAGES - 1 < nk) {
          if (slot_of(0) == kk) dma_part(std::integral_constant<int, SNEXT>{}, kt + 1, std::integral_constant<int, 0>{});
          if (slot_of(1) == kk) dma_part(std::integral_constant<int, SNEXT>{}, kt + 1, std::integral_constant<int, 1>{});
          if (slot_of(2) == kk) dma_part(std::integral_constant<int, SNEXT>{}, kt + 1, std::integral_constant<int, 2>{});
          if (slot_of(3) == kk) dma_part(std::integral_constant<int, SNEXT>{}, kt + 1, std::integral_constant<int, 3>{});
        }
      }
    };
    SQ_LDS uint8_t* st = stage(SC);
    if constexpr (MODE == kFwdR) {
      const SQ_LDS uint16_t* a = (const SQ_LDS uint16_t*)st;
      const SQ_LDS uint16_t* b = wbuf(kt);
#pragma unroll
      for (int kk = 0; kk < kBK / 16; ++kk) {
        const int chunk = 2 * kk + (lane >> 5);
        bf16x8 fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i)
          fa[i] = *(const SQ_LDS bf16x8*)(a + kc_off(wm0 + i * 32 + (lane & 31), chunk));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          fb[j] = *(const SQ_LDS bf16x8*)(b + kc_off(wn0 + j * 32 + (lane & 31), chunk));
        before_mfma(kk);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      }
      if (kt + 1 < nk) commit_w(kt + 1, std::integral_constant<int, (S + 1) % 2>{});
    }
  };

  if constexpr (!kLate) {
  // ---- prologue: the first STAGES-1 stages in flight
  if constexpr (kWReg) {
    if (nk > 0) {
      load_w(0, std::integral_constant<int, 0>{});
      commit_w(0, std::integral_constant<int, 0>{});
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  if (0 < nk) issue_dma(std::integral_constant<int, 0>{}, 0);
  if constexpr (kWAhead == 2) {
    if (0 < nk) load_w(1, std::integral_constant<int, 1>{});
  }
  __builtin_amdgcn_sched_barrier(0);

  for (int kt0 = 0; kt0 < nk; kt0 += 2) {
    step(std::integral_constant<int, 0>{}, kt0);
    if (kt0 + 1 < nk) step(std::integral_constant<int, 1>{}, kt0 + 1);
  }
  } else {
  // ---- Late-barrier schedule.  The operands of slice kk + 1 are read from
  // LDS while slice kk multiplies, and the barrier that publishes stage
  // kt + 1 sits before the MFMAs of stage kt's last slice: those MFMAs cover
  // the latency of stage kt + 1's first reads, so the matrix cores do not
  // drain at every barrier.  Right after the barrier the buffer of stage kt
  // is free: half of the DMA of stage kt + STAGES goes out there, the other
  // half in the first slice of stage kt + 1, so each stage's copy has
  // STAGES - 1 stages to land.  dX's W items for stage kt + 2 are loaded at
  // the start of step kt and converted to its LDS tile right after that
  // step's barrier (see the end of step2).
  struct Frag {
    bf16x8 a[TM];
    bf16x8 b[TN];
    uint32_t cd[MODE == kFwdC ? TN : 1];     // kFwdC: this slice's 8 codes per row slice
  };
  Frag F0, F1;
  u32x4 cst[MODE == kFwdC ? TN : 1];         // kFwdC: the stage's codes, read with slice 0
  float sop[MODE == kFwdC ? TN : 1];         // kFwdC: the stage's scale operands
  const int h32 = lane >> 5;

  auto read = [&](auto SC, int kt, auto KK, Frag& f) {
    constexpr int kk = decltype(KK)::value;
    SQ_LDS uint8_t* st = stage(SC);
    if constexpr (MODE == kFwdC) {
      const SQ_LDS uint16_t* a = (const SQ_LDS uint16_t*)st;
#pragma unroll
      for (int i = 0; i < TM; ++i)
        f.a[i] = *(const SQ_LDS bf16x8*)(a + kc_off(wm0 + i * 32 + (lane & 31), 4 * h32 + kk));
      if constexpr (kk == 0) {
        const SQ_LDS uint8_t* cs = st + L::kA;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = wn0 + 32 * j + (lane & 31);
          cst[j] = *(const SQ_LDS u32x4*)(cs + r * (kBK / 2) + 16 * (h32 ^ swz_codes(r)));
        }
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) f.cd[j] = cst[j][kk];
    } else if constexpr (MODE == kDx) {
      const SQ_LDS uint16_t* a = (const SQ_LDS uint16_t*)st;
      const SQ_LDS uint16_t* b = wbuf(kt);
#pragma unroll
      for (int i = 0; i < TM; ++i)
        f.a[i] = *(const SQ_LDS bf16x8*)(a + kc_off(wm0 + i * 32 + (lane & 31), 2 * kk + h32));
#pragma unroll
      for (int j = 0; j < TN; ++j) f.b[j] = nat_frag<BN>(b, kk, wn0 + j * 32, lane);
    } else {
      const SQ_LDS uint16_t* a = (const SQ_LDS uint16_t*)st;
      const SQ_LDS uint16_t* b = (const SQ_LDS uint16_t*)(st + L::kA);
#pragma unroll
      for (int i = 0; i < TM; ++i) f.a[i] = nat_frag<BM>(a, kk, wm0 + i * 32, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j) f.b[j] = nat_frag<BN>(b, kk, wn0 + j * 32, lane);
    }
  };
  auto mma = [&](Frag& f) {
    if constexpr (MODE == kFwdC) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const uint4 d = dequant8_mx(f.cd[j], sop[j]);
        __builtin_memcpy(&f.b[j], &d, 16);
      }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  };
  // kFwdC: scale operands of stage kt, byte 2 (kt % 8) + h of the slice's
  // 16-byte chunk; the next chunk is loaded during the chunk's last stage
  auto take_scales = [&](int kt) {
    if constexpr (MODE == kFwdC) {
      const int q = (kt >> 1) & 3;
      const uint32_t sh = 8u * (2u * (uint32_t)(kt & 1) + (uint32_t)h32);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const uint32_t w = q == 0 ? scw[j][0] : q == 1 ? scw[j][1] : q == 2 ? scw[j][2] : scw[j][3];
        sop[j] = e8m0_as_scale_operand((w >> sh) & 0xFFu);
      }
      if ((kt & 7) == 7 && kt + 1 < nk) load_sc((kt + 1) >> 3);
    }
  };
  // DMA quarters [Q0, Q0 + 2) of stage kt into buffer SC
  auto dma_half = [&](auto SC, int kt, auto Q0) {
    constexpr int q = decltype(Q0)::value;
    dma_part(SC, kt, std::integral_constant<int, q>{});
    dma_part(SC, kt, std::integral_constant<int, q + 1>{});
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  // DMA loads a thread issues for the stages after kt + 1 (the wait at the
  // barrier leaves those in flight; anything issued later is younger still)
  constexpr int kAhead = (STAGES - 2) * kDma < 63 ? (STAGES - 2) * kDma : 63;
  // kFwdC tiles with fewer 32-row code slices than waves leave the code DMA to
  // the first waves; the others issue one load per stage fewer
  constexpr bool kCodesSplit = MODE == kFwdC && DC::kWaveInst < NT / 64;
  constexpr int kDmaLow = kCodesSplit ? kDma - DC::kInst : kDma;
  constexpr int kAheadLow = (STAGES - 2) * kDmaLow < 63 ? (STAGES - 2) * kDmaLow : 63;
  const bool codes_wave = !kCodesSplit || wave_u < DC::kWaveInst;

  // The register forward issues each stage's whole DMA right after the
  // barrier that frees its buffer (the 14336 x 4096 forward 394 -> 386 us,
  // the MoE gate forward -3%); dX and dS keep the second half for the next
  // step's first slice (issued whole they ran 1% and 3% slower).
  constexpr bool kWhole = MODE == kFwdC;
  auto step2 = [&](auto SC, int kt) {
    constexpr int S = decltype(SC)::value;
    using SN = std::integral_constant<int, (S + 1) % STAGES>;            // stage kt + 1
    using SP = std::integral_constant<int, (S + STAGES - 1) % STAGES>;   // stage kt + STAGES - 1
    take_scales(kt);
    // slice 0 (operands in F0): the W loads (dX), then read slice 1 and
    // (but for the forward) issue the second half of stage kt + STAGES - 1's
    // DMA
    if constexpr (kWMid) {            // dX: the W items of stage kt + 2, in the set of its parity
      if (kt + 2 < nk) load_w(kt + 2, std::integral_constant<int, S % 2>{});
    } else if constexpr (kWReg) {     // dX: the W items of stage kt + 2
      if (kt + 2 < nk) load_w(kt + 2, I0{});
    }
    read(SC, kt, I1{}, F1);
    if (!kWhole && kt + STAGES - 1 < nk) dma_half(SP{}, kt + STAGES - 1, I2{});
    mma(F0);
    // dX below 256 x 256: stage kt + 1's W tile, from the items loaded a
    // step ago (the last barrier's wait completed them), into the buffer of
    // stage kt - 1 (read before that barrier); the next barrier publishes
    // it.  Written here, in the middle of the step, the tile's LDS writes do
    // not meet the burst of stage copies and operand reads that follows each
    // barrier.
    if constexpr (kWMid) {
      if (kt + 1 < nk) commit_w(kt + 1, std::integral_constant<int, (S + 1) % 2>{});
    }
    read(SC, kt, I2{}, F0);
    mma(F1);
    read(SC, kt, I3{}, F1);
    mma(F0);
    // stage kt + 1 has landed once at most kAhead (kAheadLow) loads are
    // outstanding, if the DMA of stages kt + 2 .. kt + STAGES - 1 all went out
    // after it; in the last stages fewer did, and everything is waited for
    if (kt + STAGES - 1 < nk) {
      if (codes_wave) wait_vm_lgkm0<kAhead>();
      else wait_vm_lgkm0<kAheadLow>();
    } else {
      wait_vm_lgkm0<0>();
    }
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if (kt + 1 < nk) read(SN{}, kt + 1, I0{}, F0);
    if (kt + STAGES < nk) {
      dma_half(SC, kt + STAGES, I0{});
      if (kWhole) dma_half(SC, kt + STAGES, I2{});
    }
    mma(F1);
    // dX 256 x 256: stage kt + 2's W tile into the buffer stage kt used
    // (every read of it came before the barrier).  Its items were loaded
    // before the wait at the barrier, so converting them waits for nothing;
    // loading them a stage ahead of their conversion keeps the round trip of
    // the W items off the step's critical path (converting a stage's items
    // in the step that loaded them cost dX 12-14%).  The next barrier
    // publishes the tile.
    if constexpr (kWReg && !kWMid) {
      if (kt + 2 < nk) commit_w(kt + 2, I0{});
    }
  };

  // prologue: stage 0 in LDS and its slice 0 read, then the DMA of stages
  // 1 .. STAGES - 2 and the first half of stage STAGES - 1 (the forward: all
  // of it)
  if (nk > 0) {
    if constexpr (kWMid) {            // dX below 256 x 256: stage 0's W tile and stage 1's items
      load_w(0, I0{});
      commit_w(0, I0{});
      if (1 < nk) load_w(1, I1{});
    } else if constexpr (kWReg) {     // dX: the W tiles of stages 0 and 1
      load_w(0, I0{});
      commit_w(0, I0{});
      if (1 < nk) {
        load_w(1, I0{});
        commit_w(1, I0{});
      }
    }
    if constexpr (MODE == kFwdC) load_sc(0);
    issue_dma(I0{}, 0);
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    read(I0{}, 0, I0{}, F0);
    if constexpr (STAGES > 2) {
      if (1 < nk) issue_dma(I1{}, 1);
    }
    if constexpr (STAGES > 3) {
      if (2 < nk) issue_dma(I2{}, 2);
    }
    if (STAGES - 1 < nk) {
      dma_half(std::integral_constant<int, STAGES - 1>{}, STAGES - 1, I0{});
      if (kWhole) dma_half(std::integral_constant<int, STAGES - 1>{}, STAGES - 1, I2{});
    }
  }
  for (int kt0 = 0; kt0 < nk; kt0 += STAGES) {
    step2(I0{}, kt0);
    if (kt0 + 1 < nk) step2(I1{}, kt0 + 1);
    if constexpr (STAGES > 2) {
      if (kt0 + 2 < nk) step2(I2{}, kt0 + 2);
    }
    if constexpr (STAGES > 3) {
      if (kt0 + 3 < nk) step2(I3{}, kt0 + 3);
    }
  }
  }

  wait_vm_lgkm0<0>();   // loads issued past the last stage have landed before LDS is reused

  // ---------------------------------------------------------------- epilogue
  // 32x32 output tile: lane l, register r holds row 8*(r/4) + 4*(l/32) + r%4,
  // column l%32.
  if constexpr (MODE != kDs) {
    const bool interior = m0 + BM <= g.M && n0 + BN <= g.N;
    if constexpr (kEpiStaged) {
      if (g.out_bf16 && interior) {
        // Every wave is done with the operand tiles; each stages its own
        // WM x WN bf16 block in LDS and leaves it as 16-byte row pieces.
        __syncthreads();
        epi_store_bf16<FMT, TM, TN>(acc, epi_region(wave), g, m0 + wm0, n0 + wn0, lane);
        return;
      }
    }
    if (interior)
      epi_store_direct<false, FMT, TM, TN>(acc, g, m0 + wm0, n0 + wn0, lane);
    else
      epi_store_direct<true, FMT, TM, TN>(acc, g, m0 + wm0, n0 + wn0, lane);
  } else {
    float* dS = reinterpret_cast<float*>(g.out) + (size_t)split * g.O * g.G;   // partial plane when split
    u32x4 cw[TM * TN];
    ds_codes<FMT, TM, TN>(cw, g.codes, g.O, g.I, m0 + wm0, n0 + wn0, lane);
    if (m0 + BM <= g.I && n0 + BN <= g.O)
      ds_store<FMT, TM, TN, true>(acc, cw, dS, g.O, g.I, g.G, m0 + wm0, n0 + wn0, lane);
    else
      ds_store<FMT, TM, TN, false>(acc, cw, dS, g.O, g.I, g.G, m0 + wm0, n0 + wn0, lane);
  }
}

template <int MODE, int FMT, int BM, int BN, int WGM, int WGN, int STAGES, int BK>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_kernel(GemmArgs g) {
  gemm_tile<MODE, FMT, BM, BN, WGM, WGN, STAGES, BK>(g, (int)blockIdx.x, (int)gridDim.x);
}

// Grouped products (one per MoE expert, same O and I, own tokens and
// weights): the experts' tiles form one order, expert by expert, expert e
// holding positions [tile_begin[e], tile_begin[e + 1]).  Each XCD takes one
// contiguous stretch of that order, so the workgroups of an expert share an
// L2 and read its activation and weight panels from HBM about once; dealing
// every expert's tiles over all 8 XCDs made each L2 fetch them again (the
// 128-expert MoE layer moved 4 to 8 times its operand bytes).
template <int MODE, int FMT, int BM, int BN, int WGM, int WGN, int STAGES, int BK>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_grouped_kernel(GemmGroup gg) {
  const int b = xcd_stretch((int)blockIdx.x, (int)gridDim.x);
  int lo = 0, hi = gg.count - 1;                 // last e with tile_begin[e] <= b
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (gg.tile_begin[mid] <= b) lo = mid;
    else hi = mid - 1;
  }
  const int e = lo;
  GemmArgs g = gg.base;
  g.a = gg.act(e);
  g.b = MODE == kDs ? reinterpret_cast<const uint16_t*>(gg.second(e)) : nullptr;
  g.codes = gg.code_plane(e);
  g.scales = MODE == kDs ? nullptr : gg.second(e);
  g.out = gg.output(e);
  g.T = gg.T[e];
  g.ws2 = gg.ws2[e];
  if (MODE == kDs) g.K = g.T;
  else g.M = g.T;
  const int tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const int local = b - gg.tile_begin[e];
  if (local >= tiles) return;
  gemm_tile<MODE, FMT, BM, BN, WGM, WGN, STAGES, BK, true>(g, local, tiles);
}

// Streamed grouped dS.  With a few hundred tokens per expert a dS tile holds
// only a few 64-token stages, and a workgroup per tile spends most of its
// life filling the pipeline (the first stage's round trip) and draining it
// (the epilogue's code loads and stores): 128 experts of 768 x 2048 at 256
// tokens ran at a third of the rate of the same tiles over 2048 tokens.
// Here each workgroup stays resident and runs its share of the tiles as one
// pipeline of stages: the DMA of the stage after a tile's last one (the next
// tile's first) goes out while the last is multiplied, and the block sums are
// stored while the next tile's stages are in flight.
//
// Every expert has the same tile grid (I x O in BM x BN tiles), so position p
// of the order is tile p % tiles (column-by-column order) of expert p / tiles.
// XCD x takes the x-th contiguous stretch of positions and its workgroups
// deal it round robin, so the tiles in flight on one XCD are neighbours in
// the order and share their experts' panels in L2.  Stages run the two-stage
// late schedule of gemm_tile (every barrier waits for all loads), with a DMA
// cursor and a compute cursor walking the same sequence of (tile, stage)
// pairs; an expert without tokens runs one stage of zeros, so its dS is 0.
// Each output element is summed in the same order as in gemm_tile.
template <int FMT, int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void ds_stream_kernel(GemmGroup gg) {
  constexpr int NT = 64 * WGM * WGN;
  constexpr int WM = BM / WGM, WN = BN / WGN;
  constexpr int TM = WM / 32, TN = WN / 32;
  using L = SmemLayout<kDs, BM, BN, 2, kBK, WGM * WGN>;
  using DA = DmaNat<BM, NT, kBK>;
  using DB = DmaNat<BN, NT, kBK>;
  constexpr int na = DA::kInst, nb = DB::kInst;
  __shared__ __attribute__((aligned(16))) uint8_t lds0[L::kStageAlloc];
  __shared__ __attribute__((aligned(16))) uint8_t lds1[L::kStageAlloc];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int wm0 = (wave / WGN) * WM, wn0 = (wave % WGN) * WN;
  const int O = gg.base.O, I = gg.base.I, G = gg.base.G;
  const int tiles_m = (I + BM - 1) / BM, tiles_n = (O + BN - 1) / BN, per = tiles_m * tiles_n;
  const int total = per * gg.count;

  // positions first, first + step, ... below end
  const int w = (int)blockIdx.x, nwg = (int)gridDim.x, x = w % kXcds;
  const int step = nwg / kXcds + (x < nwg % kXcds ? 1 : 0);
  const int tq = total / kXcds, tr = total % kXcds;
  const int s0 = x < tr ? x * (tq + 1) : tr * (tq + 1) + (x - tr) * tq;
  const int first = s0 + w / kXcds, end = s0 + (x < tr ? tq + 1 : tq);
  if (first >= end) return;

  struct Tile {
    int e, m0, n0, nk;
  };
  auto locate = [&](int pos, Tile& t) {
    t.e = pos / per;
    int tm, tn;
    tile_at<group_m<kDs>()>(pos - t.e * per, tiles_m, tiles_n, tm, tn);
    t.m0 = tm * BM;
    t.n0 = tn * BN;
    const int T = gg.T[t.e];
    t.nk = T > 0 ? (T + kBK - 1) / kBK : 1;
  };

  // DMA cursor: stage dkt of the tile at position dpos
  Tile dt;
  int dpos = first, dkt = 0;
  bool dvalid = true;
  DmaRsrc ra, rb;
  DA dA;
  DB dB;
  auto dma_tile = [&]() {
    locate(dpos, dt);
    const int T = gg.T[dt.e];
    ra = make_dma_rsrc(gg.act(dt.e), (uint32_t)((size_t)T * I * 2));
    rb = make_dma_rsrc(gg.second(dt.e), (uint32_t)((size_t)T * O * 2));
    dA.init(I, I, dt.m0, tid);
    dB.init(O, O, dt.n0, tid);
  };
  dma_tile();
  // quarters Q0 and Q0 + 1 of the cursor's stage into stage buffer st
  auto dma_half = [&](SQ_LDS uint8_t* st, auto Q0) {
    constexpr int q = decltype(Q0)::value;
    const uint32_t k0 = (uint32_t)dkt * kBK;
    dA.template issue_part<q * na / 4, (q + 1) * na / 4>(ra, (SQ_LDS uint16_t*)st, k0 * (uint32_t)I * 2u, wave_u);
    dB.template issue_part<q * nb / 4, (q + 1) * nb / 4>(rb, (SQ_LDS uint16_t*)(st + L::kA), k0 * (uint32_t)O * 2u,
                                                        wave_u);
    dA.template issue_part<(q + 1) * na / 4, (q + 2) * na / 4>(ra, (SQ_LDS uint16_t*)st, k0 * (uint32_t)I * 2u,
                                                              wave_u);
    dB.template issue_part<(q + 1) * nb / 4, (q + 2) * nb / 4>(rb, (SQ_LDS uint16_t*)(st + L::kA),
                                                              k0 * (uint32_t)O * 2u, wave_u);
  };
  auto dma_advance = [&]() {
    if (++dkt == dt.nk) {
      dkt = 0;
      dpos += step;
      dvalid = dpos < end;
      if (dvalid) dma_tile();
    }
  };

  // compute cursor: stage ckt of the tile at position cpos
  Tile ct;
  int cpos = first, ckt = 0;
  locate(cpos, ct);
  u32x4 cw[TM * TN];
  auto tile_codes = [&]() {
    ds_codes<FMT, TM, TN>(cw, gg.code_plane(ct.e), O, I, ct.m0 + wm0, ct.n0 + wn0, lane);
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  struct Frag {
    bf16x8 a[TM];
    bf16x8 b[TN];
  };
  Frag F0, F1;
  auto read = [&](SQ_LDS uint8_t* st, auto KK, Frag& f) {
    constexpr int kk = decltype(KK)::value;
    const SQ_LDS uint16_t* a = (const SQ_LDS uint16_t*)st;
    const SQ_LDS uint16_t* b = (const SQ_LDS uint16_t*)(st + L::kA);
#pragma unroll
    for (int i = 0; i < TM; ++i) f.a[i] = nat_frag<BM>(a, kk, wm0 + i * 32, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) f.b[j] = nat_frag<BN>(b, kk, wn0 + j * 32, lane);
  };
  auto mma = [&](Frag& f) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  // One stage in buffer cur (its slice 0 already in F0): every load is
  // waited for at the barrier (the next stage's, issued a whole stage
  // earlier), then the next stage's slice 0 is read and the whole DMA of the
  // stage after it is issued into cur.  (Issuing the second half of each
  // stage's DMA mid-step instead, after slice 1 is read, gave it three
  // quarters of a stage: the MoE split's dS 218 -> 211 us with the whole copy
  // one stage ahead.)  Returns false after the workgroup's last stage.
  auto stage_step = [&](SQ_LDS uint8_t* cur, SQ_LDS uint8_t* nxt) -> bool {
    read(cur, I1{}, F1);
    mma(F0);
    read(cur, I2{}, F0);
    mma(F1);
    read(cur, I3{}, F1);
    mma(F0);
    wait_vm_lgkm0<0>();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    const bool last = ckt + 1 == ct.nk;
    const bool more = !last || cpos + step < end;
    if (more) read(nxt, I0{}, F0);
    if (dvalid) {
      dma_half(cur, I0{});
      dma_half(cur, I2{});
      dma_advance();
    }
    mma(F1);
    if (!last) {
      ++ckt;
      return true;
    }
    float* const dS = reinterpret_cast<float*>(gg.output(ct.e));
    if (ct.m0 + BM <= I && ct.n0 + BN <= O)
      ds_store<FMT, TM, TN, true>(acc, cw, dS, O, I, G, ct.m0 + wm0, ct.n0 + wn0, lane);
    else
      ds_store<FMT, TM, TN, false>(acc, cw, dS, O, I, G, ct.m0 + wm0, ct.n0 + wn0, lane);
    if (!more) return false;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    cpos += step;
    ckt = 0;
    locate(cpos, ct);
    tile_codes();
    return true;
  };

  // prologue: the first stage whole, the first tile's codes, then the whole
  // second stage
  dma_half((SQ_LDS uint8_t*)lds0, I0{});
  dma_half((SQ_LDS uint8_t*)lds0, I2{});
  dma_advance();
  tile_codes();
  wait_vm_lgkm0<0>();
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_sched_barrier(0);
  read((SQ_LDS uint8_t*)lds0, I0{}, F0);
  if (dvalid) {
    dma_half((SQ_LDS uint8_t*)lds1, I0{});
    dma_half((SQ_LDS uint8_t*)lds1, I2{});
    dma_advance();
  }
  SQ_LDS uint8_t* cur = (SQ_LDS uint8_t*)lds0;
  SQ_LDS uint8_t* nxt = (SQ_LDS uint8_t*)lds1;
  while (stage_step(cur, nxt)) {
    SQ_LDS uint8_t* t = cur;
    cur = nxt;
    nxt = t;
  }
}

// Tile configurations.  Each entry: BM, BN, waves along M, waves along N, stages,
// K per stage.  The large tile's 8 waves take 128 x 64 each (2 along M, 4
// along N) in the MXFP4 forward, dX and dS: every wave dequantises or reads
// only its own 64 columns of the weight operand, so the register forward
// converts each code tile in 2 waves instead of 4 (4096^3 forward 117 -> 106
// us, the 8B MLP forwards -7%, dS -2%, dX -1%; the per-element summation
// order, and so every result, is unchanged).  The NVFP4 forward timed the
// same either way and keeps 64 x 128.  The large tile is used when its grid still gives every CU a
// workgroup; smaller grids (the 1024-wide key/value projections, MoE experts
// of a few hundred rows) take the 128 x 128 tile, with four times as many
// workgroups.  That tile runs 8 waves of 64 x 32 (two workgroups fit a CU):
// against 4 waves of 64 x 64, the key/value forward gained 16% and the MoE
// stack 10%.
#define SQ_CFG_FWD 256, 256, 4, 2, 2, 64
#define SQ_CFG_DX 256, 256, 2, 4, 2, 64
#define SQ_CFG_DS 256, 256, 2, 4, 2, 64
#define SQ_CFG_FWDC 256, 256, 2, 4, 2, 64
#define SQ_CFG_SMALL 128, 128, 2, 4, 2, 64
constexpr int kCUs = 256;   // MI355X compute units

template <int MODE, int FMT, int BM, int BN, int WGM, int WGN, int STAGES, int BK>
static int launch_gemm(const GemmArgs& g, hipStream_t s) {
  using L = SmemLayout<MODE, BM, BN, STAGES, BK, WGM * WGN>;
  static_assert(L::kBytes <= 160 * 1024, "LDS budget");
  const int tiles = (((g.m_cnt ? g.m_cnt : g.M) + BM - 1) / BM) * (((g.n_cnt ? g.n_cnt : g.N) + BN - 1) / BN);
  if (tiles == 0) return 0;
  const int blocks = tiles * (MODE == kDs && g.ksplit > 1 ? g.ksplit : 1);
  hipLaunchKernelGGL((gemm_kernel<MODE, FMT, BM, BN, WGM, WGN, STAGES, BK>), dim3(blocks), dim3(64 * WGM * WGN), 0, s, g);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// The MXFP4 forward's small tile keeps four stages in flight (80 KiB of LDS:
// its code tiles are a quarter of a bf16 W tile).
#define SQ_CFG_SMALL_FWDC 128, 128, 2, 4, 4, 64
#define SQ_CFG_HALF_N 256, 128, 4, 2, 2, 64
#define SQ_CFG_HALF_M 128, 256, 2, 4, 2, 64
// Per-product knobs for the second launch: dS's half tiles run three stages
// (144 KiB of LDS; the split dS products of the 8B MLP 389.5 -> 385.7 us);
// four stages for the MXFP4 forward's half tile timed slower (383.5 ->
// 393.7 us).
#define SQ_CFG_HALF_N_FWDC SQ_CFG_HALF_N
#define SQ_CFG_HALF_N_DS 256, 128, 4, 2, 3, 64
#define SQ_CFG_HALF_M_DS 128, 256, 2, 4, 3, 64

// A grid of 256 x 256 tiles that ends in a partial wave (at most half the
// CUs busy) leaves the other CUs idle while it runs.  When that last partial
// wave is whole tile-columns (or tile-rows) of the output, those columns
// (rows) go to a second launch of 256 x 128 (128 x 256) tiles of 8 waves of
// 64 x 64, twice as many workgroups, which fill the chip.  The first launch
// keeps the whole waves.  On the 8B MLP products at 4096 tokens (896 tiles,
// three waves and a half) this took 4-5% off the forward and dX; 4 waves of
// 64 x 128 in the second launch gained about half as much.  Each output
// element is still summed in one workgroup in K order, so results do not
// depend on the split.
template <int MODE, int FMT, int BM, int BN, int... REST>
static int launch_sized(const GemmArgs& g, hipStream_t s) {
  const int tm = (g.M + BM - 1) / BM, tn = (g.N + BN - 1) / BN;
  const int64_t big = (int64_t)tm * tn;
  if (big < kCUs) {
    if constexpr (MODE == kFwdC) return launch_gemm<MODE, FMT, SQ_CFG_SMALL_FWDC>(g, s);
    else return launch_gemm<MODE, FMT, SQ_CFG_SMALL>(g, s);
  }
  const int rem = (int)(big % kCUs);
  if (BM == 256 && BN == 256 && rem > 0 && rem <= kCUs / 2 && g.ksplit <= 1) {
    if (rem % tm == 0) {                                  // the last rem / tm tile-columns
      const int cols = (tn - rem / tm) * BN;
      GemmArgs a = g, b = g;
      a.n_cnt = cols;
      b.n_off = cols;
      b.n_cnt = g.N - cols;
      const int rc = launch_gemm<MODE, FMT, BM, BN, REST...>(a, s);
      if (rc != 0) return rc;
      if constexpr (MODE == kFwdC) return launch_gemm<MODE, FMT, SQ_CFG_HALF_N_FWDC>(b, s);
      else if constexpr (MODE == kDs) return launch_gemm<MODE, FMT, SQ_CFG_HALF_N_DS>(b, s);
      else return launch_gemm<MODE, FMT, SQ_CFG_HALF_N>(b, s);
    }
    if (rem % tn == 0) {                                  // the last rem / tn tile-rows
      const int rows = (tm - rem / tn) * BM;
      GemmArgs a = g, b = g;
      a.m_cnt = rows;
      b.m_off = rows;
      b.m_cnt = g.M - rows;
      const int rc = launch_gemm<MODE, FMT, BM, BN, REST...>(a, s);
      if (rc != 0) return rc;
      if constexpr (MODE == kDs) return launch_gemm<MODE, FMT, SQ_CFG_HALF_M_DS>(b, s);
      else return launch_gemm<MODE, FMT, SQ_CFG_HALF_M>(b, s);
    }
  }
  return launch_gemm<MODE, FMT, BM, BN, REST...>(g, s);
}

// The MXFP4 forward dequantises in registers (kFwdC) when every row's scales
// split into 8-byte runs (G % 8 == 0), the code planes are 16-byte aligned
// and the scale planes 8-byte aligned;
// the grouped forward makes the same choice as the single one, so an
// expert's output equals the single product's bit for bit.
static bool regs_dequant_ok(int G, const ExpertProblem* p, int n) {
  if (G % 8 != 0) return false;
  for (int e = 0; e < n; ++e)
    if ((reinterpret_cast<uintptr_t>(p[e].codes) & 15) != 0 || (reinterpret_cast<uintptr_t>(p[e].scales) & 7) != 0)
      return false;
  return true;
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
  // registers dequantise when the code and scale planes are 16-byte aligned
  // and every row's scales split into 16-byte runs
  ExpertProblem one{};
  one.codes = codes;
  one.scales = scales;
  if (fmt == kMX && regs_dequant_ok(g.G, &one, 1)) return launch_sized<kFwdC, kMX, SQ_CFG_FWDC>(g, s);
  return fmt == kMX ? launch_sized<kFwdR, kMX, SQ_CFG_FWD>(g, s) : launch_sized<kFwdR, kNV, SQ_CFG_FWD>(g, s);
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
  return fmt == kMX ? launch_sized<kDx, kMX, SQ_CFG_DX>(g, s) : launch_sized<kDx, kNV, SQ_CFG_DX>(g, s);
}

// ------------------------------------------------------------------ grouped
// One launch per kGroupMax experts, one workgroup per tile.
template <int MODE, int FMT, int BM, int BN, int WGM, int WGN, int STAGES, int BK>
static int launch_grouped(GemmGroup& gg, const ExpertProblem* p, int n, hipStream_t s) {
  using L = SmemLayout<MODE, BM, BN, STAGES, BK, WGM * WGN>;
  static_assert(L::kBytes <= 160 * 1024, "LDS budget");
  int blocks = 0;
  gg.count = n;
  for (int e = 0; e < n; ++e) {
    const int M = MODE == kDs ? gg.base.M : p[e].T;
    const int tiles = ((M + BM - 1) / BM) * ((gg.base.N + BN - 1) / BN);
    gg.T[e] = p[e].T;
    gg.ws2[e] = FMT == kNV ? p[e].ws2 : 1.0f;
    gg.tile_begin[e] = blocks;
    blocks += tiles;
  }
  if (blocks == 0) return 0;
  hipLaunchKernelGGL((gemm_grouped_kernel<MODE, FMT, BM, BN, WGM, WGN, STAGES, BK>), dim3(blocks),
                     dim3(64 * WGM * WGN), 0, s, gg);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// The streamed dS: two resident workgroups per CU (the grid never exceeds the
// tile count, so every XCD's stretch of positions has a workgroup), each
// running about total / 512 tiles.
#define SQ_CFG_DS_STREAM 128, 128, 2, 4
template <int FMT, int BM, int BN, int WGM, int WGN>
static int launch_ds_stream(GemmGroup& gg, const ExpertProblem* p, int n, hipStream_t s) {
  using L = SmemLayout<kDs, BM, BN, 2, kBK, WGM * WGN>;
  static_assert(2 * L::kBytes <= 160 * 1024, "two workgroups per CU");
  gg.count = n;
  for (int e = 0; e < n; ++e) {
    gg.T[e] = p[e].T;
    gg.ws2[e] = 1.0f;
    gg.tile_begin[e] = 0;
  }
  const int64_t total = (int64_t)((gg.base.M + BM - 1) / BM) * ((gg.base.N + BN - 1) / BN) * n;
  if (total == 0) return 0;
  const int blocks = (int)(total < 2 * kCUs ? total : 2 * kCUs);
  hipLaunchKernelGGL((ds_stream_kernel<FMT, BM, BN, WGM, WGN>), dim3(blocks), dim3(64 * WGM * WGN), 0, s, gg);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Grouped products below the large tile: experts of a few hundred tokens or
// fewer pad their last token tile, so the MXFP4 register forward takes 64 x
// 256 tiles (64-token granularity, 8 waves of 64 x 32; the same flops per
// tile as 128 x 128): 128 experts of 64 tokens 167 -> 128 us, of 256 tokens
// 61 -> 59 us.  dX takes them only when experts average at most 96 tokens
// (at 64 tokens 184 -> 117 us; at 256, 72 -> 82 us, where 128 x 128 wins).
#define SQ_CFG_GROUPED_FWDC 64, 256, 1, 8, 4, 64
#define SQ_CFG_GROUPED_THIN 64, 256, 1, 8, 2, 64
// Experts of at least 2048 tokens whose 256 x 256 tiles would not fill the
// chip (the 8B step's k and v projections, 1024 x 4096 at 4096 tokens, as
// one grouped forward) take 128 x 256 tiles, 8 waves of 64 x 64, four stages:
// 77.3 -> 75.9 us for the pair.
#define SQ_CFG_GROUPED_FWDC_LONG 128, 256, 2, 4, 4, 64

// Grouped dX on 128 x 128 tiles: an expert whose last 128-token tile would
// hold 64 rows or fewer can send those rows to a second launch of 64 x 256
// tiles (the same per-element sums: every output row is computed alone), so
// that tile is not half padding.  Over the MoE layer's routed split (128
// experts, 256 rows on average) half the experts end that way: for the gate
// and up dX (I = 2048) 5120 tiles become 4096 and 512 of 64 x 256, and the
// product ran 214 -> 203 us.  The second launch is worth it only when it
// saves more than it costs: counted in rounds of two workgroups per CU, the
// 64 x 256 launch takes whole rounds (a partial round still lasts a tile) at
// about 1.15 times a 128 x 128 tile (the down dX, I = 768, would go from
// 1920 tiles to 1536 and 192: 175 -> 180 us, so it stays whole).  If the
// moved pointers do not fit the launch's 32-bit offsets, the experts run
// unsplit.
template <int FMT>
static int dx_split_tails(GemmGroup& gg, const ExpertProblem* p, int n, hipStream_t s) {
  const int64_t cols = (gg.base.I + 127) / 128, cols_thin = (gg.base.I + 255) / 256;
  int64_t all = 0, kept = 0, moved = 0;
  for (int e = 0; e < n; ++e) {
    const int t = p[e].T % 128;
    all += (int64_t)((p[e].T + 127) / 128) * cols;
    if (t > 0 && t <= 64) {
      kept += (int64_t)(p[e].T / 128) * cols;
      moved += cols_thin;
    } else {
      kept += (int64_t)((p[e].T + 127) / 128) * cols;
    }
  }
  const double slots = 2.0 * kCUs;
  if (moved == 0 || (double)kept / slots + 1.15 * (double)((moved + 2 * kCUs - 1) / (2 * kCUs)) >= (double)all / slots)
    return launch_grouped<kDx, FMT, SQ_CFG_SMALL>(gg, p, n, s);
  ExpertProblem whole[kGroupMax], tail[kGroupMax];
  int nw = 0, nt = 0;
  const size_t a_row = (size_t)gg.base.O * 2, out_row = (size_t)gg.base.I * (gg.base.out_bf16 ? 2 : 4);
  for (int e = 0; e < n; ++e) {
    const int t = p[e].T % 128;
    if (t == 0 || t > 64) {
      whole[nw++] = p[e];
      continue;
    }
    const int head = p[e].T - t;
    if (head > 0) {
      whole[nw] = p[e];
      whole[nw++].T = head;
    }
    tail[nt] = p[e];
    tail[nt].a = static_cast<const uint8_t*>(p[e].a) + (size_t)head * a_row;
    tail[nt].out = static_cast<uint8_t*>(p[e].out) + (size_t)head * out_row;
    tail[nt++].T = t;
  }
  GemmGroup gw = gg, gt = gg;
  if (nt == 0 || !set_experts(gw, whole, nw, false) || !set_experts(gt, tail, nt, false))
    return launch_grouped<kDx, FMT, SQ_CFG_SMALL>(gg, p, n, s);
  const int rc = nw > 0 ? launch_grouped<kDx, FMT, SQ_CFG_SMALL>(gw, whole, nw, s) : 0;
  if (rc != 0) return rc;
  return launch_grouped<kDx, FMT, SQ_CFG_GROUPED_THIN>(gt, tail, nt, s);
}

// The large tile when the experts' tiles fill the chip and an expert averages
// at least 512 tokens (rows of the forward and dX, the contraction of dS:
// shorter token sums leave a 256 x 256 dS tile a few stages between its
// prologue and epilogue, where two 128 x 128 workgroups per CU do better).
template <int MODE, int FMT, int BM, int BN, int... REST>
static int grouped_sized(GemmGroup& gg, const ExpertProblem* p, int n, hipStream_t s) {
  int64_t tokens = 0, big = 0;
  for (int e = 0; e < n; ++e) {
    tokens += p[e].T;
    const int M = MODE == kDs ? gg.base.M : p[e].T;
    big += (int64_t)((M + BM - 1) / BM) * ((gg.base.N + BN - 1) / BN);
  }
  const bool large = big >= kCUs && tokens >= (int64_t)512 * n;
  if (large) return launch_grouped<MODE, FMT, BM, BN, REST...>(gg, p, n, s);
  if constexpr (MODE == kFwdC) {
    if (tokens >= (int64_t)2048 * n) return launch_grouped<MODE, FMT, SQ_CFG_GROUPED_FWDC_LONG>(gg, p, n, s);
    return launch_grouped<MODE, FMT, SQ_CFG_GROUPED_FWDC>(gg, p, n, s);
  }
  else if constexpr (MODE == kDs) return launch_ds_stream<FMT, SQ_CFG_DS_STREAM>(gg, p, n, s);
  else if constexpr (MODE == kDx) {
    if (tokens <= (int64_t)96 * n) return launch_grouped<MODE, FMT, SQ_CFG_GROUPED_THIN>(gg, p, n, s);
    return dx_split_tails<FMT>(gg, p, n, s);
  } else return launch_grouped<MODE, FMT, SQ_CFG_SMALL>(gg, p, n, s);
}

template <int MODE>
static int run_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, int out_bf16, hipStream_t s) {
  GemmGroup gg{};
  gg.base.O = O;
  gg.base.I = I;
  gg.base.G = I / (fmt == kMX ? 32 : 16);
  gg.base.out_bf16 = out_bf16;
  gg.base.ksplit = 1;
  if (MODE == kFwdR) { gg.base.N = O; gg.base.K = I; }
  else if (MODE == kDx) { gg.base.N = I; gg.base.K = O; }
  else { gg.base.M = I; gg.base.N = O; }
  // Launch sets: from the first expert not yet launched, every later one
  // whose pointers keep each kind's span under 4 GiB, up to kGroupMax (the
  // experts of a stacked tensor, or of one allocator pool, share a set; an
  // expert's results do not depend on the set it runs in).
  const bool regs = MODE == kFwdR && fmt == kMX && regs_dequant_ok(gg.base.G, p, n);
  std::vector<uint8_t> done((size_t)n, 0);
  ExpertProblem set[kGroupMax];
  for (int first = 0; first < n;) {
    uintptr_t lo[4], hi[4];
    for (int k = 0; k < 4; ++k) { lo[k] = UINTPTR_MAX; hi[k] = 0; }
    int m = 0;
    for (int e = first; e < n && m < kGroupMax; ++e) {
      if (done[(size_t)e]) continue;
      const void* ptr[4] = {p[e].a, MODE == kDs ? p[e].b : static_cast<const void*>(p[e].scales), p[e].codes,
                            p[e].out};
      uintptr_t nlo[4], nhi[4];
      bool fits = true;
      for (int k = 0; k < 4; ++k) {
        const uintptr_t v = reinterpret_cast<uintptr_t>(ptr[k]);
        nlo[k] = v != 0 && v < lo[k] ? v : lo[k];
        nhi[k] = v != 0 && v > hi[k] ? v : hi[k];
        fits = fits && (nlo[k] == UINTPTR_MAX || nhi[k] - nlo[k] <= 0xFFFFFFFFu);
      }
      if (!fits) continue;
      for (int k = 0; k < 4; ++k) { lo[k] = nlo[k]; hi[k] = nhi[k]; }
      set[m++] = p[e];
      done[(size_t)e] = 1;
    }
    while (first < n && done[(size_t)first]) ++first;
    if (!set_experts(gg, set, m, MODE == kDs)) return -1;     // cannot happen: the set was chosen to fit
    int rc;
    if (regs)
      rc = grouped_sized<kFwdC, kMX, SQ_CFG_FWDC>(gg, set, m, s);
    else if (MODE == kFwdR)
      rc = fmt == kMX ? grouped_sized<kFwdR, kMX, SQ_CFG_FWD>(gg, set, m, s)
                      : grouped_sized<kFwdR, kNV, SQ_CFG_FWD>(gg, set, m, s);
    else if (MODE == kDx)
      rc = fmt == kMX ? grouped_sized<kDx, kMX, SQ_CFG_DX>(gg, set, m, s)
                      : grouped_sized<kDx, kNV, SQ_CFG_DX>(gg, set, m, s);
    else
      rc = fmt == kMX ? grouped_sized<kDs, kMX, SQ_CFG_DS>(gg, set, m, s)
                      : grouped_sized<kDs, kNV, SQ_CFG_DS>(gg, set, m, s);
    if (rc != 0) return rc;
  }
  return 0;
}

int gemm_fwd_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, int y_bf16, hipStream_t s) {
  return run_grouped<kFwdR>(fmt, O, I, n, p, y_bf16, s);
}
int gemm_dx_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, int dx_bf16, hipStream_t s) {
  return run_grouped<kDx>(fmt, O, I, n, p, dx_bf16, s);
}
int gemm_dscale_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, hipStream_t s) {
  return run_grouped<kDs>(fmt, O, I, n, p, 0, s);
}

// Split of the token sum for dS when the large tile leaves CUs idle: each of
// `splits` workgroups per tile reduces its own range of K stages into a
// partial [O, G] plane, and a second pass adds the planes in order.
struct DsPlan {
  int splits, ksteps_per;
};
static DsPlan ds_plan(int fmt, int T, int O, int I) {
  (void)fmt;
  constexpr int BM = 256, BN = 256, BK = 64;     // the SQ_CFG_DS tile
  const int64_t tiles = (int64_t)((I + BM - 1) / BM) * ((O + BN - 1) / BN);
  const int nk = (T + BK - 1) / BK;
  DsPlan p{1, nk};
  if (tiles >= kCUs || tiles == 0) return p;
  int splits = (int)(kCUs / tiles);
  splits = min(splits, min(nk / 4, 8));
  if (splits < 2) return p;
  p.splits = splits;
  p.ksteps_per = (nk + splits - 1) / splits;
  return p;
}

size_t gemm_dscale_workspace(int fmt, int T, int O, int I) {
  const DsPlan p = ds_plan(fmt, T, O, I);
  if (p.splits < 2) return 0;
  return (size_t)p.splits * O * (I / (fmt == kMX ? 32 : 16)) * sizeof(float);
}

// dS[i] = sum over s of part[s][i], s in increasing order.
__global__ __launch_bounds__(256) void ds_reduce_kernel(const float* __restrict__ part, float* __restrict__ dS,
                                                        int64_t n, int splits) {
  const int64_t i4 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (i4 >= n) return;
  float4 acc = *reinterpret_cast<const float4*>(part + i4);
  for (int sp = 1; sp < splits; ++sp) {
    const float4 v = *reinterpret_cast<const float4*>(part + (size_t)sp * n + i4);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  dS[i4] = acc.x; dS[i4 + 1] = acc.y; dS[i4 + 2] = acc.z; dS[i4 + 3] = acc.w;
}

static int gemm_dscale_ws(int fmt, int T, int O, int I, const void* X, const void* dY, const uint8_t* codes,
                          float* dS, void* workspace, hipStream_t s);

int gemm_dscale(int fmt, int T, int O, int I, const void* X, const void* dY,
                const uint8_t* codes, float* dS, void* workspace, hipStream_t s) {
  return gemm_dscale_ws(fmt, T, O, I, X, dY, codes, dS, workspace, s);
}

// ------------------------------------------------------------------ static scratch
// The split token sum of dS with its partial planes in a fixed device array
// instead of a caller workspace, for callers that cannot allocate.  Its size
// bounds every plan: a layer is split only when its 256 x 256 tiles number
// fewer than the CUs, into splits <= 256 / tiles ranges, so the partial planes
// hold splits * O * I / B fp32 values <= 256 * 65536 / B * 4 bytes, 4 MiB for
// B = 16.  Each device holds its own copy of the array until the process ends;
// its device address is looked up once per device.
static __device__ __align__(256) uint8_t scratch[kDscaleScratchBytes];
static_assert((size_t)kCUs * 256 * 256 / 16 * sizeof(float) <= kDscaleScratchBytes,
              "the static scratch holds the partial planes of every split plan");

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the current device (nullptr on a HIP error).
void* scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch[dev].store(p, std::memory_order_release);
  }
  return p;
}
}  // namespace

int gemm_dscale_static(int fmt, int T, int O, int I, const void* X, const void* dY, const uint8_t* codes, float* dS,
                       hipStream_t s) {
  if (gemm_dscale_workspace(fmt, T, O, I) > kDscaleScratchBytes) return -2;
  void* ws = scratch_ptr();
  if (!ws) return -1;
  return gemm_dscale_ws(fmt, T, O, I, X, dY, codes, dS, ws, s);
}

static int gemm_dscale_ws(int fmt, int T, int O, int I, const void* X, const void* dY, const uint8_t* codes,
                          float* dS, void* workspace, hipStream_t s) {
  GemmArgs g{};
  g.a = static_cast<const uint16_t*>(X);
  g.b = static_cast<const uint16_t*>(dY);
  g.codes = codes; g.out = dS;
  g.T = T; g.O = O; g.I = I; g.G = I / (fmt == kMX ? 32 : 16);
  g.M = I; g.N = O; g.K = T;
  g.ws2 = 1.0f;
  g.out_bf16 = 0;
  const DsPlan p = ds_plan(fmt, T, O, I);
  if (p.splits < 2) {
    g.ksplit = 1;
    return fmt == kMX ? launch_sized<kDs, kMX, SQ_CFG_DS>(g, s) : launch_sized<kDs, kNV, SQ_CFG_DS>(g, s);
  }
  g.ksplit = p.splits;
  g.ksteps_per = p.ksteps_per;
  g.out = workspace;
  const int rc = fmt == kMX ? launch_gemm<kDs, kMX, SQ_CFG_DS>(g, s) : launch_gemm<kDs, kNV, SQ_CFG_DS>(g, s);
  if (rc != 0) return rc;
  const int64_t n = (int64_t)O * g.G;                 // a multiple of 8: O % 8 == 0
  const int64_t blocks = (n / 4 + 255) / 256;
  hipLaunchKernelGGL(ds_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     static_cast<const float*>(workspace), dS, n, p.splits);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace sq
