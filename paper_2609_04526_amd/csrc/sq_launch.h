// Internal launchers behind the C ABI (all arguments already validated).
// Each returns 0 on success and -1 when the HIP runtime reports an error.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sq {

int gemm_fwd(int fmt, int T, int O, int I, const void* X, const uint8_t* codes,
             const uint8_t* scales, float ws2, void* Y, int y_bf16, hipStream_t s);
int gemm_dx(int fmt, int T, int O, int I, const void* dY, const uint8_t* codes,
            const uint8_t* scales, float ws2, void* dX, int dx_bf16, hipStream_t s);
int gemm_dscale(int fmt, int T, int O, int I, const void* X, const void* dY,
                const uint8_t* codes, float* dS, void* workspace, hipStream_t s);
// Workspace bytes gemm_dscale needs (partial dS planes of a split token sum).
size_t gemm_dscale_workspace(int fmt, int T, int O, int I);
// gemm_dscale with the partial planes in the library's static device scratch
// (kDscaleScratchBytes per device); -2 if the plan would need more.
constexpr size_t kDscaleScratchBytes = size_t(4) << 20;
int gemm_dscale_static(int fmt, int T, int O, int I, const void* X, const void* dY,
                       const uint8_t* codes, float* dS, hipStream_t s);

// Planes of one merge launch, as arrays (kernel arguments are limited to
// 4 KiB; this layout fits 112 planes).  Plane p is cut into spans of
// delta_span(fmt, small) scales (delta mode) or copy_span(small) bytes (copy
// mode) and owns the spans [span_begin[p], span_begin[p+1]).
constexpr int kMergePlanesPerLaunch = 112;
enum MergeKind { kMergeCopy = 1, kMergeMxDelta = 2, kMergeNvDelta = 4 };
constexpr int kMergeDeltaStepsMx = 8, kMergeDeltaStepsNv = 16, kMergeCopySteps = 8;
// Steps of 4 scales (and a 16-byte fp32 delta) per lane in one delta span;
// NVFP4's longer grid step hides better behind more loads in flight.  A
// launch over few scales (below kMergeSmallScales in all) takes one-step
// spans instead, so that it still spreads over the CUs.
constexpr int64_t kMergeSmallScales = int64_t(1) << 24;
constexpr int delta_steps(int fmt, bool small = false) {
  return small ? 1 : (fmt == 1 ? kMergeDeltaStepsNv : kMergeDeltaStepsMx);
}
constexpr int delta_span(int fmt, bool small = false) { return 1024 * delta_steps(fmt, small); }   // 256 lanes x 4 scales per step
constexpr int copy_steps(bool small = false) { return small ? 1 : kMergeCopySteps; }
constexpr int copy_span(bool small = false) { return 4096 * copy_steps(small); }    // 256 lanes x 16 bytes per step
struct MergeBatch {
  uint8_t* scales[kMergePlanesPerLaunch];
  const void* aux[kMergePlanesPerLaunch];     // fp32 delta (delta mode) or source bytes (copy mode)
  int64_t n[kMergePlanesPerLaunch];
  int32_t span_begin[kMergePlanesPerLaunch];
  float ws2[kMergePlanesPerLaunch];
  uint8_t fmt[kMergePlanesPerLaunch];
  uint8_t mode[kMergePlanesPerLaunch];
  int32_t count;
  int32_t spans;                      // spans of all planes
  int32_t kinds;                      // planes present: kMergeCopy | kMergeMxDelta | kMergeNvDelta
  int32_t small;                      // one-step spans (the whole call covers few scales)
};
static_assert(sizeof(MergeBatch) <= 4096, "kernel argument budget");
int merge_launch(const MergeBatch& b, hipStream_t s);

// Grouped products over MoE experts that share O and I: each expert has its
// own tokens (T >= 0), activations, weights and output.  Up to kGroupMax
// experts per launch; the caller splits longer lists.
constexpr int kGroupMax = 128;
struct ExpertProblem {
  const void* a;            // fwd, ds: X [T, I]; dx: dY [T, O]
  const void* b;            // ds: dY [T, O]
  const uint8_t* codes;
  const uint8_t* scales;
  void* out;                // fwd: Y [T, O]; dx: dX [T, I]; ds: dS [O, G] fp32
  int T;
  float ws2;
};
int gemm_fwd_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, int y_bf16, hipStream_t s);
int gemm_dx_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, int dx_bf16, hipStream_t s);
int gemm_dscale_grouped(int fmt, int O, int I, int n, const ExpertProblem* p, hipStream_t s);

// One weight of a grouped re-quantisation (the arguments of one single call).
struct RtnItem {
  int64_t O, I;
  const void* W;
  uint8_t* codes;
  uint8_t* scales;
  float* ws2_out;
  float ws2_in;
  uint64_t seed;
};
// Weights of one re-quantisation launch (one format, one rule), as arrays
// within the 4 KiB kernel-argument limit.  Weight p owns the workgroups
// [span_begin[p], span_begin[p+1]), rtn_span(fmt, rule) chunks of 8 weights
// each.
constexpr int kRtnPerLaunch = 56;
// Chunks of 8 weights per lane: MXFP4 nearest-even (the lightest per-chunk
// work) streams best with two; NVFP4 nearest, away and toward zero take two
// whole 16-weight blocks per lane (nearest-even over 28 linears of the 8B
// shapes: 0.389 ms, against 0.44 ms with one block and with four, whose
// longer-lived waves leave fewer loads in flight); the others four.
constexpr int rtn_chunks(int fmt, int rule) {
  return (fmt == 0 && rule == 0) ? 2 : 4;
}
constexpr int rtn_span(int fmt, int rule) { return 256 * rtn_chunks(fmt, rule); }
struct RtnBatch {
  const uint16_t* w[kRtnPerLaunch];
  uint8_t* codes[kRtnPerLaunch];
  uint8_t* scales[kRtnPerLaunch];
  const float* ws2_ptr[kRtnPerLaunch];    // recomputed ws2 (NVFP4), else null
  const float* amax_t[kRtnPerLaunch];     // tensor amax (whole-tensor rule), else null
  int64_t n_chunks[kRtnPerLaunch];
  uint64_t seed[kRtnPerLaunch];
  int32_t span_begin[kRtnPerLaunch];
  float ws2_val[kRtnPerLaunch];
  float* ws2_out[kRtnPerLaunch];          // slot that receives ws2_val (the weight's first workgroup), or null
  int32_t count;
  int32_t spans;
};
static_assert(sizeof(RtnBatch) <= 4096, "kernel arguments are limited to 4 KiB");
// Re-quantises n weights under one rule (as rtn_rule_launch on each, in
// launches of up to kRtnPerLaunch weights); every weight that needs an amax
// slot has its own ws2_out.
int rtn_grouped_launch(int fmt, int rule, int n, const RtnItem* items, hipStream_t s);

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s);
// rule: 0 nearest-even, 1 nearest-away, 2 toward zero, 3 stochastic (Philox
// key `seed`), 4 whole-tensor scale (ws2_out required: the amax slot).
int rtn_rule_launch(int fmt, int O, int I, const void* W, float ws2_in, int rule, uint64_t seed,
                    uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s);

// QAT-LoRA weight-space STE: fused W_eff + nearest re-quantisation, and the
// factor gradients through the rank (lora_grads_workspace bytes of scratch).

// QAST low-rank scale step for E stacked experts (E = 1: one plane): on-grid
// scale bytes (+ clamp mask) and the factor gradients; qast_grads_workspace
// bytes of partial dA planes.  ws2: E per-expert scalars (NVFP4).
constexpr int kWs2TableMax = 256;
struct Ws2Table {
  float v[kWs2TableMax];
};
int qast_scales_launch(int fmt, int E, int O, int G, int r, const uint8_t* base, const void* B, const void* A,
                       float c, const float* ws2, uint8_t* out, uint8_t* mask, hipStream_t s);
size_t qast_grads_workspace(int E, int O, int G, int r);
int qast_grads_launch(int E, int O, int G, int r, const float* dS, const uint8_t* mask, const void* B, const void* A,
                      float c, float* dB, float* dA, void* workspace, hipStream_t s);

// QAT-LoRA weight-space STE: fused W_eff + nearest re-quantisation of E
// stacked experts (ws2: E per-expert scalars, NVFP4), and the factor
// gradients through the rank of E experts whose token rows are stacked
// expert-major (T: E token counts; lora_grads_batched_workspace bytes of
// scratch).  The single-weight forms are E = 1.
int qat_requant_launch(int fmt, int E, int O, int I, int r, const uint8_t* codes, const uint8_t* scales,
                       const float* ws2, const void* B, const void* A, float c, uint8_t* codes_out,
                       uint8_t* scales_out, hipStream_t s);
size_t lora_grads_workspace(int T, int O, int I, int r);
int lora_grads_launch(int T, int O, int I, int r, const void* X, const void* dY, const void* B, const void* A,
                      float c, float* dB, float* dA, void* workspace, hipStream_t s);
size_t lora_grads_batched_workspace(int E, const int64_t* T, int O, int I, int r);
int lora_grads_batched_launch(int E, const int64_t* T, int O, int I, int r, const void* X, const void* dY,
                              const void* B, const void* A, float c, float* dB, float* dA, void* workspace,
                              hipStream_t s);

// Rollback and byte audit (sq_audit.hip).
int applied_launch(int fmt, int64_t n, const uint8_t* before, const uint8_t* after, float* applied, hipStream_t s);
int rollback_launch(int fmt, int64_t n, uint8_t* scales, const float* applied, hipStream_t s);
int byte_diff_launch(int64_t n, const uint8_t* a, const uint8_t* b, uint64_t* counts, hipStream_t s);

}  // namespace sq
