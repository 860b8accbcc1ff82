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
#include "sq_rtn.h"
#include "sq_launch.h"

namespace sq {

// merge tuning knobs (build-time)

// ------------------------------------------------------------------ merge
// The planes of a launch are cut into spans: delta_span(fmt, small) scale bytes
// (delta mode: delta_steps(fmt, small) steps of 4 scales and a 16-byte fp32
// delta per lane) or copy_span(small) bytes (copy mode: copy_steps(small)
// steps of 16 bytes per lane).  Workgroup w takes spans w, w + grid,
// w + 2 grid, ...: at any moment the whole grid streams through one window of
// the planes, which keeps the DRAM accesses of all workgroups together (a
// workgroup walking a private region of its own streams markedly slower).
// Consecutive lanes touch consecutive 4-byte scale words and 16-byte delta
// words; delta and copy sources are read once, with streaming loads.  The
// plane pointers are restrict: a scale store cannot alias a later load.
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef sq_f32x4 f32x4_t;

// One delta span: delta_steps(FMT) steps of 4 scales per lane, all loads
// issued before any compute.  Scale bytes are written with streaming stores;
// NVFP4 planes (2x the bytes of MXFP4's, well past the 256 MB last-level
// cache between whole-model merges) also read them with streaming loads,
// which on MXFP4 planes measured slower.
template <int FMT, int FAST, bool SMALL>
__device__ __forceinline__ void merge_delta_span(uint8_t* __restrict__ sc, const float* __restrict__ dl, int64_t n,
                                                 int64_t off, const Ws2Div& ws2, int tid) {
  constexpr int kDeltaSteps = delta_steps(FMT, SMALL), kDeltaSpan = delta_span(FMT, SMALL);
  if (off + kDeltaSpan <= n) {
    uint32_t sv[kDeltaSteps];
    f32x4_t dv[kDeltaSteps];
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g) {
      const int64_t i = off + g * 1024 + tid * 4;
      if constexpr (FMT == kNV)
        sv[g] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(sc + i));
      else
        sv[g] = *reinterpret_cast<const uint32_t*>(sc + i);
      dv[g] = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(dl + i));
    }
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g) {
      const uint32_t v = sv[g];
      if constexpr (FMT == kNV)
        sv[g] = nv_merge_word<FAST>(v, dv[g], ws2);
      else
        sv[g] = merge_one_t<FMT>(v & 0xFFu, dv[g][0], ws2) | (merge_one_t<FMT>((v >> 8) & 0xFFu, dv[g][1], ws2) << 8) |
                (merge_one_t<FMT>((v >> 16) & 0xFFu, dv[g][2], ws2) << 16) |
                (merge_one_t<FMT>(v >> 24, dv[g][3], ws2) << 24);
    }
#pragma unroll
    for (int g = 0; g < kDeltaSteps; ++g)
      __builtin_nontemporal_store(sv[g], reinterpret_cast<uint32_t*>(sc + off + g * 1024 + tid * 4));
  } else {
    for (int64_t k = off + tid; k < n && k < off + kDeltaSpan; k += 256)
      sc[k] = (uint8_t)merge_one_t<FMT>(sc[k], dl[k], ws2);
  }
}

// One copy span: copy_steps(SMALL) steps of 16 bytes per lane, loads first.
template <bool SMALL>
__device__ __forceinline__ void merge_copy_span(uint8_t* __restrict__ sc, const uint8_t* __restrict__ sr, int64_t n,
                                                int64_t off, int tid) {
  constexpr int kCopySteps = copy_steps(SMALL), kCopySpan = copy_span(SMALL);
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

// KINDS: the plane kinds this instance handles (a launch whose planes are all
// of one kind gets an instance with that kind's code alone, and so that
// kind's register budget and occupancy).
template <int KINDS, bool SMALL>
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
    const float* __restrict__ dl = static_cast<const float*>(batch.aux[pi]);
    if ((KINDS & kMergeCopy) && batch.mode[pi] == 1) {
      merge_copy_span<SMALL>(sc, static_cast<const uint8_t*>(batch.aux[pi]), n, rel * copy_span(SMALL), tid);
    } else if ((KINDS & kMergeNvDelta) && (KINDS == kMergeNvDelta || batch.fmt[pi] == kNV)) {
      const Ws2Div w = make_ws2_div(batch.ws2[pi]);
      if (w.div.fast)
        merge_delta_span<kNV, 1, SMALL>(sc, dl, n, rel * delta_span(kNV, SMALL), w, tid);
      else
        merge_delta_span<kNV, 0, SMALL>(sc, dl, n, rel * delta_span(kNV, SMALL), w, tid);
    } else if (KINDS & kMergeMxDelta) {
      merge_delta_span<kMX, 0, SMALL>(sc, dl, n, rel * delta_span(kMX, SMALL), make_ws2_div(1.0f), tid);
    }
  }
}

int merge_launch(const MergeBatch& b, hipStream_t s) {
  if (b.spans <= 0) return 0;
  // Measured on the 8B model's planes (medians of interleaved runs): copies
  // stream best from 2048 workgroups, MXFP4 deltas from 4096, and NVFP4
  // deltas (16-step spans, a longer grid step per scale) from 16384.
  constexpr int64_t kNvGrid = 16384, kMxGrid = 4096;
  const int64_t cap = b.kinds == kMergeCopy ? 2048 : ((b.kinds & kMergeNvDelta) ? kNvGrid : kMxGrid);
  const dim3 grid((unsigned)(b.spans < cap ? b.spans : cap));
  if (b.small) {
    // few scales in all: one-step spans, one workgroup each
    const dim3 all((unsigned)b.spans);
    switch (b.kinds) {
      case kMergeCopy: hipLaunchKernelGGL((merge_kernel<kMergeCopy, true>), all, dim3(256), 0, s, b); break;
      case kMergeMxDelta: hipLaunchKernelGGL((merge_kernel<kMergeMxDelta, true>), all, dim3(256), 0, s, b); break;
      case kMergeNvDelta: hipLaunchKernelGGL((merge_kernel<kMergeNvDelta, true>), all, dim3(256), 0, s, b); break;
      default:
        hipLaunchKernelGGL((merge_kernel<kMergeCopy | kMergeMxDelta | kMergeNvDelta, true>), all, dim3(256), 0, s, b);
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }
  switch (b.kinds) {
    case kMergeCopy: hipLaunchKernelGGL((merge_kernel<kMergeCopy, false>), grid, dim3(256), 0, s, b); break;
    case kMergeMxDelta: hipLaunchKernelGGL((merge_kernel<kMergeMxDelta, false>), grid, dim3(256), 0, s, b); break;
    case kMergeNvDelta: hipLaunchKernelGGL((merge_kernel<kMergeNvDelta, false>), grid, dim3(256), 0, s, b); break;
    default:
      hipLaunchKernelGGL((merge_kernel<kMergeCopy | kMergeMxDelta | kMergeNvDelta, false>), grid, dim3(256), 0, s, b);
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// ------------------------------------------------------------------ RTN
// Each workgroup takes 256 rtn_chunks(FMT, RULE) chunks of one weight: a lane
// loads its chunks (c, c + 256, ...) before working on any, so that many
// 16-byte loads are in flight per lane.  (A grid-stride form with 2 to 8 chunks per lane in flight
// ran slower on the 8B model's weights: the per-chunk work is long enough
// that short-lived workgroups keep more loads in flight across the chip.)
// One launch covers up to kRtnPerLaunch weights, so a whole model takes a
// few launches instead of one per weight, each with its own ramp and tail.
template <int FMT, int RULE>
__global__ __launch_bounds__(256) void rtn_kernel(RtnBatch batch_arg) {
  (void)batch_arg;
  // read through the kernarg segment (constant address space): the
  // workgroup-uniform table stays in scalar registers
  const __attribute__((address_space(4))) RtnBatch& b =
      *(const __attribute__((address_space(4))) RtnBatch*)__builtin_amdgcn_kernarg_segment_ptr();
  const int wg = (int)blockIdx.x;
  int lo = 0, hi = b.count - 1;                 // the last weight whose spans start at or before wg
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b.span_begin[mid] <= wg) lo = mid;
    else hi = mid - 1;
  }
  const int p = lo;
  // a given ws2 is also the weight's ws2 output (one store, no launch of its own)
  if (b.ws2_out[p] != nullptr && wg == b.span_begin[p] && threadIdx.x == 0) *b.ws2_out[p] = b.ws2_val[p];
  const int64_t n_chunks = b.n_chunks[p];
  const uint16_t* __restrict__ W = b.w[p];
  uint8_t* codes = b.codes[p];
  uint8_t* scales = b.scales[p];
  constexpr int kRtnChunks = rtn_chunks(FMT, RULE);
  // NVFP4 nearest and toward zero: a lane takes whole 16-weight blocks (its
  // chunks 2 b and 2 b + 1 for blocks b = b0 + 256 u), so each block's scale
  // arithmetic runs once (rtn_block16_nv)
  constexpr bool kBlocks = FMT == kNV && (RULE == kRuleEven || RULE == kRuleAway || RULE == kRuleRtz);
  if constexpr (kBlocks) {
    static_assert(kRtnChunks % 2 == 0, "whole blocks per lane");
    const int64_t b0 = (int64_t)(wg - b.span_begin[p]) * (rtn_span(FMT, RULE) / 2) + threadIdx.x;
    uint4 v[kRtnChunks];
#pragma unroll
    for (int u = 0; u < kRtnChunks / 2; ++u) {
      const int64_t c = 2 * (b0 + 256 * u);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (c + h < n_chunks) {
          const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(W + 8 * (c + h)));
          v[2 * u + h] = make_uint4(t[0], t[1], t[2], t[3]);
        } else {
          v[2 * u + h] = make_uint4(0, 0, 0, 0);
        }
      }
    }
    const int64_t n_blocks = n_chunks / 2;
    const int64_t pack = (reinterpret_cast<uintptr_t>(scales) & 3) == 0 ? n_blocks / 4 * 4 : 0;
    const RcpDivisor wd = make_rcp_divisor(b.ws2_ptr[p] ? *b.ws2_ptr[p] : b.ws2_val[p]);
    // the block scale fp32(e4m3 * ws2) and its reciprocal for each of the 128
    // scale bytes, once per workgroup instead of once per block
    __shared__ float tab[256];
    if (threadIdx.x < 128) {
      const float e = __fmul_rn(e4m3_to_f32(threadIdx.x), wd.d);
      tab[2 * threadIdx.x] = e;
      tab[2 * threadIdx.x + 1] = __fdiv_rn(1.0f, e);
    }
    __syncthreads();
    const __attribute__((address_space(3))) float* tl = (const __attribute__((address_space(3))) float*)tab;
    if (wd.d >= 0x1p-55f && wd.d <= 0x1p55f) {
#pragma unroll
      for (int u = 0; u < kRtnChunks / 2; ++u) {
        const int64_t blk = b0 + 256 * u;
        rtn_block16_nv<RULE, 1>(v[2 * u], v[2 * u + 1], blk, blk < n_blocks, wd, tl, codes, scales, pack);
      }
    } else {
#pragma unroll
      for (int u = 0; u < kRtnChunks / 2; ++u) {
        const int64_t blk = b0 + 256 * u;
        rtn_block16_nv<RULE, -1>(v[2 * u], v[2 * u + 1], blk, blk < n_blocks, wd, tl, codes, scales, pack);
      }
    }
    return;
  }
  const int64_t c0 = (int64_t)(wg - b.span_begin[p]) * rtn_span(FMT, RULE) + threadIdx.x;
  uint4 v[kRtnChunks];
#pragma unroll
  for (int u = 0; u < kRtnChunks; ++u) {
    const int64_t c = c0 + 256 * u;
    // the weight is read once: streaming (non-temporal) loads
    if (c < n_chunks) {
      const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(W + 8 * c));
      v[u] = make_uint4(t[0], t[1], t[2], t[3]);
    } else {
      v[u] = make_uint4(0, 0, 0, 0);
    }
  }
  // scale bytes of whole groups of four blocks leave as 4-byte stores when
  // the plane is 4-byte aligned
  constexpr int kGroup = 4 * (ScaleOperand<FMT>::kBlock / 8);
  const int64_t pack = (reinterpret_cast<uintptr_t>(scales) & 3) == 0 ? n_chunks / kGroup * kGroup : 0;
  const float* ws2_ptr = b.ws2_ptr[p];
  const float ws2_val = b.ws2_val[p];
  const float* amax_t = b.amax_t[p];
  const uint64_t seed = b.seed[p];
  // the NVFP4 ws2 and its reciprocal, once for both chunks (a per-workgroup
  // table of the 128 effective scales' reciprocals timed no faster)
  constexpr bool kHoist = FMT == kNV && RULE != kRuleWholeTensor;
  RcpDivisor wd;
  if (kHoist) wd = make_rcp_divisor(ws2_ptr ? *ws2_ptr : ws2_val);
  // a ws2 in [2^-55, 2^55] (one test per weight, workgroup-uniform) lets
  // every quotient of the weight skip div_exact's range check
  if (kHoist && wd.d >= 0x1p-55f && wd.d <= 0x1p55f) {
#pragma unroll
    for (int u = 0; u < kRtnChunks; ++u) {
      const int64_t c = c0 + 256 * u;
      rtn_chunk<FMT, RULE, 1>(v[u], c, c < n_chunks, ws2_ptr, ws2_val, amax_t, seed, codes, scales, pack, &wd);
    }
    return;
  }
#pragma unroll
  for (int u = 0; u < kRtnChunks; ++u) {
    const int64_t c = c0 + 256 * u;
    rtn_chunk<FMT, RULE>(v[u], c, c < n_chunks, ws2_ptr, ws2_val, amax_t, seed, codes, scales, pack,
                         kHoist ? &wd : nullptr);
  }
}

// Tensor amax passes of up to kRtnPerLaunch weights per launch: the slots
// are zeroed, every weight's workgroups fold their maxima into its slot, and
// the slots are finished (ws2 from the amax, or a given value stored).
struct AmaxBatch {
  const uint16_t* w[kRtnPerLaunch];
  float* slot[kRtnPerLaunch];
  int64_t n_chunks[kRtnPerLaunch];
  int32_t wg_begin[kRtnPerLaunch + 1];   // workgroups [wg_begin[p], wg_begin[p + 1]) take weight p
  float val[kRtnPerLaunch];              // finishing: 0 = ws2 from the amax, else the value stored
  int32_t count;
};
static_assert(sizeof(AmaxBatch) <= 4096, "kernel arguments are limited to 4 KiB");

__global__ __launch_bounds__(64) void rtn_slots_zero(AmaxBatch b) {
  if ((int)threadIdx.x < b.count) *reinterpret_cast<uint32_t*>(b.slot[threadIdx.x]) = 0u;
}

// Tensor amax (as bf16 bits, in an fp32 slot) of each weight: 4 loads in
// flight per lane, one integer atomicMax per workgroup (a max of bit patterns
// is order-independent, so the result is deterministic).
__global__ __launch_bounds__(256) void rtn_amax(AmaxBatch batch_arg) {
  (void)batch_arg;
  const __attribute__((address_space(4))) AmaxBatch& b =
      *(const __attribute__((address_space(4))) AmaxBatch*)__builtin_amdgcn_kernarg_segment_ptr();
  const int wg = (int)blockIdx.x;
  int lo = 0, hi = b.count - 1;                 // the weight whose workgroups hold wg
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (b.wg_begin[mid] <= wg) lo = mid;
    else hi = mid - 1;
  }
  const uint16_t* __restrict__ W = b.w[lo];
  const int64_t n_chunks = b.n_chunks[lo];
  __shared__ uint32_t red[4];
  uint32_t am = 0;
  const int64_t stride = (int64_t)(b.wg_begin[lo + 1] - b.wg_begin[lo]) * 256;
  int64_t c = (int64_t)(wg - b.wg_begin[lo]) * 256 + threadIdx.x;
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
    atomicMax(reinterpret_cast<unsigned int*>(b.slot[lo]), max(max(red[0], red[1]), max(red[2], red[3])) << 16);
}

// ws2 = amax / 6 / 448 (1 for an all-zero weight) in place of the amax, or
// the given value
__global__ __launch_bounds__(64) void rtn_slots_finish(AmaxBatch b) {
  const int k = (int)threadIdx.x;
  if (k >= b.count) return;
  float* slot = b.slot[k];
  if (b.val[k] != 0.0f) {
    *slot = b.val[k];
    return;
  }
  float ws2 = __fdiv_rn(__fdiv_rn(*slot, 6.0f), 448.0f);
  if (ws2 == 0.0f) ws2 = 1.0f;
  *slot = ws2;
}

__global__ void rtn_ws2_store(float* slot, float v) { *slot = v; }

namespace {
template <int FMT, int RULE>
int rtn_batch(const RtnBatch& b, hipStream_t s) {
  if (b.spans <= 0) return 0;
  hipLaunchKernelGGL((rtn_kernel<FMT, RULE>), dim3((unsigned)b.spans), dim3(256), 0, s, b);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <int FMT>
int rtn_batch_rule(int rule, const RtnBatch& b, hipStream_t s) {
  switch (rule) {
    case kRuleEven: return rtn_batch<FMT, kRuleEven>(b, s);
    case kRuleAway: return rtn_batch<FMT, kRuleAway>(b, s);
    case kRuleRtz: return rtn_batch<FMT, kRuleRtz>(b, s);
    case kRuleStochastic: return rtn_batch<FMT, kRuleStochastic>(b, s);
    case kRuleWholeTensor: return rtn_batch<FMT, kRuleWholeTensor>(b, s);
    default: return -1;
  }
}

// Amax passes over the weights that need one, kRtnPerLaunch per launch set:
// zero the slots, fold each weight's amax into its slot, then (finish) turn
// the slots into ws2 or store the given values.
class AmaxPasses {
 public:
  AmaxPasses(bool finish, hipStream_t s) : finish_(finish), s_(s) {}
  int add(const uint16_t* w, int64_t n_chunks, float* slot, float val) {
    const int p = b_.count++;
    b_.w[p] = w;
    b_.slot[p] = slot;
    b_.n_chunks[p] = n_chunks;
    b_.val[p] = val;
    b_.wg_begin[p] = wgs_;
    const int64_t want = (n_chunks + 1023) / 1024;
    wgs_ += (int32_t)(want < 1024 ? (want > 0 ? want : 1) : 1024);
    b_.wg_begin[p + 1] = wgs_;
    return b_.count == kRtnPerLaunch ? flush() : 0;
  }
  int flush() {
    if (b_.count == 0) return 0;
    hipLaunchKernelGGL(rtn_slots_zero, dim3(1), dim3(64), 0, s_, b_);
    hipLaunchKernelGGL(rtn_amax, dim3((unsigned)wgs_), dim3(256), 0, s_, b_);
    if (finish_) hipLaunchKernelGGL(rtn_slots_finish, dim3(1), dim3(64), 0, s_, b_);
    b_ = AmaxBatch{};
    wgs_ = 0;
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }

 private:
  AmaxBatch b_{};
  int32_t wgs_ = 0;
  bool finish_;
  hipStream_t s_;
};

// Slots finished after the codes are written (whole-tensor rule), kRtnPerLaunch per launch.
class SlotFinish {
 public:
  explicit SlotFinish(hipStream_t s) : s_(s) {}
  int add(float* slot, float val) {
    const int p = b_.count++;
    b_.slot[p] = slot;
    b_.val[p] = val;
    return b_.count == kRtnPerLaunch ? flush() : 0;
  }
  int flush() {
    if (b_.count == 0) return 0;
    hipLaunchKernelGGL(rtn_slots_finish, dim3(1), dim3(64), 0, s_, b_);
    b_ = AmaxBatch{};
    return hipGetLastError() == hipSuccess ? 0 : -1;
  }

 private:
  AmaxBatch b_{};
  hipStream_t s_;
};
}  // namespace

int rtn_grouped_launch(int fmt, int rule, int n, const RtnItem* items, hipStream_t s) {
  const bool nv = fmt == kNV;
  // pre-passes: the tensor amax of every weight that needs one (whole-tensor
  // rule: ws2_out holds the amax while the codes are written; a recomputed
  // NVFP4 ws2: ws2_out receives the ws2), each into its own ws2_out slot
  {
    AmaxPasses pre(rule != kRuleWholeTensor, s);
    for (int k = 0; k < n; ++k) {
      const RtnItem& it = items[k];
      if (rule == kRuleWholeTensor || (nv && !(it.ws2_in > 0.0f)))
        if (pre.add(static_cast<const uint16_t*>(it.W), it.O * it.I / 8, it.ws2_out, 0.0f) != 0) return -1;
    }
    if (pre.flush() != 0) return -1;
  }
  RtnBatch batch{};
  int64_t spans = 0;
  auto flush = [&]() -> int {
    batch.spans = (int32_t)spans;
    const int rc = nv ? rtn_batch_rule<kNV>(rule, batch, s) : rtn_batch_rule<kMX>(rule, batch, s);
    batch = RtnBatch{};
    spans = 0;
    return rc;
  };
  for (int k = 0; k < n; ++k) {
    const RtnItem& it = items[k];
    const int64_t n_chunks = it.O * it.I / 8;
    if (n_chunks == 0) {
      // no workgroup of its own: a given ws2 reaches its slot by a launch
      if (nv && rule != kRuleWholeTensor && it.ws2_in > 0.0f && it.ws2_out)
        hipLaunchKernelGGL(rtn_ws2_store, dim3(1), dim3(1), 0, s, it.ws2_out, it.ws2_in);
      continue;
    }
    const int64_t span = rtn_span(fmt, rule);
    const int64_t c = (n_chunks + span - 1) / span;
    if (batch.count == kRtnPerLaunch || spans + c > INT32_MAX)
      if (flush() != 0) return -1;
    const int p = batch.count++;
    batch.w[p] = static_cast<const uint16_t*>(it.W);
    batch.codes[p] = it.codes;
    batch.scales[p] = it.scales;
    batch.n_chunks[p] = n_chunks;
    batch.seed[p] = it.seed;
    batch.span_begin[p] = (int32_t)spans;
    if (rule == kRuleWholeTensor) {
      batch.amax_t[p] = it.ws2_out;
      batch.ws2_val[p] = nv ? (it.ws2_in > 0.0f ? it.ws2_in : 0.0f) : 1.0f;
    } else if (nv) {
      batch.ws2_ptr[p] = it.ws2_in > 0.0f ? nullptr : it.ws2_out;
      batch.ws2_val[p] = it.ws2_in;
      batch.ws2_out[p] = it.ws2_in > 0.0f ? it.ws2_out : nullptr;
    } else {
      batch.ws2_val[p] = 1.0f;
    }
    spans += c;
  }
  if (batch.count > 0 && flush() != 0) return -1;
  if (rule == kRuleWholeTensor) {
    // then the ws2 used: recomputed from the amax (NVFP4 without ws2_in), else
    // ws2_in (NVFP4) or 1 (MXFP4)
    SlotFinish post(s);
    for (int k = 0; k < n; ++k) {
      const RtnItem& it = items[k];
      if (post.add(it.ws2_out, nv && !(it.ws2_in > 0.0f) ? 0.0f : (nv ? it.ws2_in : 1.0f)) != 0) return -1;
    }
    if (post.flush() != 0) return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s) {
  return rtn_rule_launch(fmt, O, I, W, ws2_in, tie == 1 ? kRuleAway : kRuleEven, 0, codes, scales, ws2_out, s);
}

int rtn_rule_launch(int fmt, int O, int I, const void* W, float ws2_in, int rule, uint64_t seed,
                    uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s) {
  const RtnItem it{O, I, W, codes, scales, ws2_out, ws2_in, seed};
  return rtn_grouped_launch(fmt, rule, 1, &it, s);
}

}  // namespace sq
