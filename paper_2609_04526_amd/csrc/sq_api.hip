// C ABI of libscaleqlora (declared in include/scaleqlora.h): host-side
// argument validation, then one or a few launches on the caller's stream.
// Nothing here allocates device memory or synchronises.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "../../include/scaleqlora.h"
#include "sq_launch.h"

#define SQ_EXPORT extern "C" __attribute__((visibility("default")))

static_assert(SQ_DSCALE_SCRATCH_BYTES == sq::kDscaleScratchBytes, "header and library agree on the scratch size");

namespace {

constexpr int64_t kDimMax = (int64_t(1) << 31) - 1;

int block_of(int fmt) { return fmt == SQ_MXFP4 ? 32 : 16; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// The GEMM kernels address each operand through one buffer resource with a
// 32-bit byte range (offsets from 2^31 up read as zeros), so every operand
// must stay below 2 GiB.
constexpr int64_t kOperandBytesMax = (int64_t(1) << 31) - 16;

int check_layer(int fmt, int64_t T, int64_t O, int64_t I) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  if (T < 0 || O < 1 || I < 1 || T > kDimMax || O > kDimMax || I > kDimMax) return SQ_ERR_SHAPE;
  if (O % 8 != 0 || I % block_of(fmt) != 0) return SQ_ERR_SHAPE;
  if (T * I * 2 > kOperandBytesMax || T * O * 2 > kOperandBytesMax || O * I / 2 > kOperandBytesMax)
    return SQ_ERR_SHAPE;
  return SQ_OK;
}

bool ws2_ok(float ws2) { return isfinite(ws2) && ws2 > 0.0f; }

int check_gemm(int fmt, int64_t T, int64_t O, int64_t I, const void* act, const uint8_t* codes,
               const uint8_t* scales, float ws2, const void* out, int out_dtype) {
  int st = check_layer(fmt, T, O, I);
  if (st != SQ_OK) return st;
  if (out_dtype != SQ_OUT_F32 && out_dtype != SQ_OUT_BF16) return SQ_ERR_ARG;
  if (!codes || !scales) return SQ_ERR_ARG;
  if (T > 0 && (!act || !out)) return SQ_ERR_ARG;
  if (fmt == SQ_NVFP4 && !ws2_ok(ws2)) return SQ_ERR_ARG;
  if (!aligned(act, 16) || !aligned(out, 16) || !aligned(codes, 4)) return SQ_ERR_ALIGN;
  return SQ_OK;
}

int hip_status(int rc) { return rc == 0 ? SQ_OK : SQ_ERR_HIP; }

int check_merge_plane(int fmt, int64_t n, const uint8_t* scales, const float* delta, const uint8_t* src,
                      float ws2, int mode) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  if (mode != SQ_MERGE_DELTA && mode != SQ_MERGE_COPY) return SQ_ERR_ARG;
  if (n < 0) return SQ_ERR_SHAPE;
  if (n == 0) return SQ_OK;
  if (!scales) return SQ_ERR_ARG;
  if (mode == SQ_MERGE_DELTA) {
    if (!delta) return SQ_ERR_ARG;
    if (fmt == SQ_NVFP4 && !ws2_ok(ws2)) return SQ_ERR_ARG;
    if (!aligned(delta, 16)) return SQ_ERR_ALIGN;
  } else {
    if (!src) return SQ_ERR_ARG;
    if (!aligned(src, 16)) return SQ_ERR_ALIGN;
  }
  if (!aligned(scales, 16)) return SQ_ERR_ALIGN;
  return SQ_OK;
}

int run_merge(int n_desc, const sq_merge_desc* d, hipStream_t s) {
  int64_t total = 0;
  for (int k = 0; k < n_desc; ++k) total += d[k].n;
  const bool small = total < sq::kMergeSmallScales;
  sq::MergeBatch batch{};
  batch.small = small;
  int64_t spans = 0;
  for (int k = 0; k < n_desc; ++k) {
    if (d[k].n == 0) continue;
    const int64_t unit = d[k].mode == SQ_MERGE_COPY ? sq::copy_span(small) : sq::delta_span(d[k].fmt, small);
    const int64_t c = (d[k].n + unit - 1) / unit;
    if (batch.count == sq::kMergePlanesPerLaunch || spans + c > INT32_MAX) {
      batch.spans = (int32_t)spans;
      if (sq::merge_launch(batch, s) != 0) return SQ_ERR_HIP;
      batch = sq::MergeBatch{};
      batch.small = small;
      spans = 0;
    }
    const int p = batch.count++;
    batch.scales[p] = d[k].scales;
    batch.aux[p] = d[k].mode == SQ_MERGE_DELTA ? static_cast<const void*>(d[k].delta)
                                               : static_cast<const void*>(d[k].src);
    batch.n[p] = d[k].n;
    batch.span_begin[p] = (int32_t)spans;
    batch.ws2[p] = d[k].ws2;
    batch.fmt[p] = (uint8_t)d[k].fmt;
    batch.mode[p] = (uint8_t)d[k].mode;
    batch.kinds |= d[k].mode == SQ_MERGE_COPY ? sq::kMergeCopy
                                              : (d[k].fmt == SQ_NVFP4 ? sq::kMergeNvDelta : sq::kMergeMxDelta);
    spans += c;
  }
  batch.spans = (int32_t)spans;
  if (batch.count > 0 && sq::merge_launch(batch, s) != 0) return SQ_ERR_HIP;
  return SQ_OK;
}

}  // namespace

SQ_EXPORT int sq_fwd(int fmt, int64_t T, int64_t O, int64_t I, const void* X, const uint8_t* codes,
                     const uint8_t* scales, float ws2, void* Y, int y_dtype, void* stream) {
  int st = check_gemm(fmt, T, O, I, X, codes, scales, ws2, Y, y_dtype);
  if (st != SQ_OK) return st;
  if (T == 0) return SQ_OK;
  return hip_status(sq::gemm_fwd(fmt, (int)T, (int)O, (int)I, X, codes, scales, ws2, Y,
                                 y_dtype == SQ_OUT_BF16, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_bwd_dx(int fmt, int64_t T, int64_t O, int64_t I, const void* dY, const uint8_t* codes,
                        const uint8_t* scales, float ws2, void* dX, int dx_dtype, void* stream) {
  int st = check_gemm(fmt, T, O, I, dY, codes, scales, ws2, dX, dx_dtype);
  if (st != SQ_OK) return st;
  if (T == 0) return SQ_OK;
  return hip_status(sq::gemm_dx(fmt, (int)T, (int)O, (int)I, dY, codes, scales, ws2, dX,
                                dx_dtype == SQ_OUT_BF16, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT size_t sq_bwd_dscale_workspace(int fmt, int64_t T, int64_t O, int64_t I) {
  if (check_layer(fmt, T, O, I) != SQ_OK) return 0;
  return sq::gemm_dscale_workspace(fmt, (int)T, (int)O, (int)I);
}

SQ_EXPORT int sq_bwd_dscale(int fmt, int64_t T, int64_t O, int64_t I, const void* X, const void* dY,
                            const uint8_t* codes, float* dS, void* workspace, size_t workspace_bytes,
                            void* stream) {
  int st = check_layer(fmt, T, O, I);
  if (st != SQ_OK) return st;
  if (!codes || !dS) return SQ_ERR_ARG;
  if (T > 0 && (!X || !dY)) return SQ_ERR_ARG;
  if (!aligned(X, 16) || !aligned(dY, 16) || !aligned(codes, 4) || !aligned(dS, 4)) return SQ_ERR_ALIGN;
  const size_t need = sq_bwd_dscale_workspace(fmt, T, O, I);
  if (need > 0 && (!workspace || workspace_bytes < need)) return SQ_ERR_WORKSPACE;
  if (need > 0 && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  return hip_status(sq::gemm_dscale(fmt, (int)T, (int)O, (int)I, X, dY, codes, dS, workspace,
                                    static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_bwd_dscale_noalloc(int fmt, int64_t T, int64_t O, int64_t I, const void* X, const void* dY,
                                    const uint8_t* codes, float* dS, void* stream) {
  int st = check_layer(fmt, T, O, I);
  if (st != SQ_OK) return st;
  if (!codes || !dS) return SQ_ERR_ARG;
  if (T > 0 && (!X || !dY)) return SQ_ERR_ARG;
  if (!aligned(X, 16) || !aligned(dY, 16) || !aligned(codes, 4) || !aligned(dS, 4)) return SQ_ERR_ALIGN;
  if (sq_bwd_dscale_workspace(fmt, T, O, I) > SQ_DSCALE_SCRATCH_BYTES) return SQ_ERR_WORKSPACE;
  const int rc = sq::gemm_dscale_static(fmt, (int)T, (int)O, (int)I, X, dY, codes, dS,
                                        static_cast<hipStream_t>(stream));
  return rc == -2 ? SQ_ERR_WORKSPACE : hip_status(rc);
}

SQ_EXPORT int sq_merge_scales(int fmt, int64_t n, uint8_t* scales, const float* delta, const uint8_t* src,
                              float ws2, int mode, void* stream) {
  int st = check_merge_plane(fmt, n, scales, delta, src, ws2, mode);
  if (st != SQ_OK) return st;
  sq_merge_desc d{};
  d.n = n; d.scales = scales; d.delta = delta; d.src = src; d.ws2 = ws2; d.fmt = fmt; d.mode = mode;
  return run_merge(1, &d, static_cast<hipStream_t>(stream));
}

SQ_EXPORT int sq_merge_scales_grouped(int n_desc, const sq_merge_desc* descs, void* stream) {
  if (n_desc < 0 || (n_desc > 0 && !descs)) return SQ_ERR_ARG;
  for (int k = 0; k < n_desc; ++k) {
    const sq_merge_desc& d = descs[k];
    if (d.reserved != 0) return SQ_ERR_ARG;
    int st = check_merge_plane(d.fmt, d.n, d.scales, d.delta, d.src, d.ws2, d.mode);
    if (st != SQ_OK) return st;
  }
  return run_merge(n_desc, descs, static_cast<hipStream_t>(stream));
}

namespace {
enum GroupedKind { kGroupedFwd, kGroupedDx, kGroupedDs };

int run_grouped(GroupedKind kind, int fmt, int64_t O, int64_t I, int n, const sq_expert_desc* d, int out_dtype,
                hipStream_t s) {
  int st = check_layer(fmt, 0, O, I);
  if (st != SQ_OK) return st;
  if (n < 0 || (n > 0 && !d)) return SQ_ERR_ARG;
  if (kind != kGroupedDs && out_dtype != SQ_OUT_F32 && out_dtype != SQ_OUT_BF16) return SQ_ERR_ARG;
  for (int e = 0; e < n; ++e) {
    const sq_expert_desc& x = d[e];
    if (x.reserved != 0) return SQ_ERR_ARG;
    st = check_layer(fmt, x.T, O, I);
    if (st != SQ_OK) return st;
    if (!x.codes) return SQ_ERR_ARG;
    if (!aligned(x.codes, 4)) return SQ_ERR_ALIGN;
    if (kind == kGroupedDs) {
      if (!x.out || (x.T > 0 && (!x.act || !x.act2))) return SQ_ERR_ARG;
      if (!aligned(x.act, 16) || !aligned(x.act2, 16) || !aligned(x.out, 4)) return SQ_ERR_ALIGN;
    } else {
      if (!x.scales || (x.T > 0 && (!x.act || !x.out))) return SQ_ERR_ARG;
      if (fmt == SQ_NVFP4 && !ws2_ok(x.ws2)) return SQ_ERR_ARG;
      if (!aligned(x.act, 16) || !aligned(x.out, 16)) return SQ_ERR_ALIGN;
    }
  }
  // one table entry per expert that has work (the forward and dX skip empty experts)
  sq::ExpertProblem p[sq::kGroupMax];
  int m = 0;
  auto flush = [&]() -> int {
    if (m == 0) return 0;
    int rc;
    if (kind == kGroupedFwd) rc = sq::gemm_fwd_grouped(fmt, (int)O, (int)I, m, p, out_dtype == SQ_OUT_BF16, s);
    else if (kind == kGroupedDx) rc = sq::gemm_dx_grouped(fmt, (int)O, (int)I, m, p, out_dtype == SQ_OUT_BF16, s);
    else rc = sq::gemm_dscale_grouped(fmt, (int)O, (int)I, m, p, s);
    m = 0;
    return rc;
  };
  for (int e = 0; e < n; ++e) {
    const sq_expert_desc& x = d[e];
    if (kind != kGroupedDs && x.T == 0) continue;
    p[m].a = x.act;
    p[m].b = x.act2;
    p[m].codes = x.codes;
    p[m].scales = x.scales;
    p[m].out = x.out;
    p[m].T = (int)x.T;
    p[m].ws2 = fmt == SQ_NVFP4 ? x.ws2 : 1.0f;
    if (++m == sq::kGroupMax && flush() != 0) return SQ_ERR_HIP;
  }
  return flush() == 0 ? SQ_OK : SQ_ERR_HIP;
}
}  // namespace

SQ_EXPORT int sq_fwd_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs,
                             int y_dtype, void* stream) {
  return run_grouped(kGroupedFwd, fmt, O, I, n_experts, descs, y_dtype, static_cast<hipStream_t>(stream));
}

SQ_EXPORT int sq_bwd_dx_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs,
                                int dx_dtype, void* stream) {
  return run_grouped(kGroupedDx, fmt, O, I, n_experts, descs, dx_dtype, static_cast<hipStream_t>(stream));
}

SQ_EXPORT int sq_bwd_dscale_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs,
                                    void* stream) {
  return run_grouped(kGroupedDs, fmt, O, I, n_experts, descs, SQ_OUT_F32, static_cast<hipStream_t>(stream));
}

SQ_EXPORT int rtn_quantize(int fmt, int64_t O, int64_t I, const void* W, float ws2_in, int tie,
                           uint8_t* codes_out, uint8_t* scales_out, float* ws2_out, void* stream) {
  int st = check_layer(fmt, 0, O, I);
  if (st != SQ_OK) return st;
  if (tie != SQ_TIE_EVEN && tie != SQ_TIE_AWAY) return SQ_ERR_ARG;
  if (!W || !codes_out || !scales_out) return SQ_ERR_ARG;
  if (fmt == SQ_NVFP4) {
    if (!(ws2_in > 0.0f) && !ws2_out) return SQ_ERR_ARG;     // recomputing needs the slot
    if (ws2_in > 0.0f && !isfinite(ws2_in)) return SQ_ERR_ARG;
    if (ws2_out && !aligned(ws2_out, 4)) return SQ_ERR_ALIGN;
  }
  if (!aligned(W, 16) || !aligned(codes_out, 4)) return SQ_ERR_ALIGN;
  return hip_status(sq::rtn_launch(fmt, (int)O, (int)I, W, ws2_in, tie, codes_out, scales_out,
                                   fmt == SQ_NVFP4 ? ws2_out : nullptr, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int rtn_quantize_rule(int fmt, int64_t O, int64_t I, const void* W, float ws2_in, int rule,
                                uint64_t seed, uint8_t* codes_out, uint8_t* scales_out, float* ws2_out,
                                void* stream) {
  int st = check_layer(fmt, 0, O, I);
  if (st != SQ_OK) return st;
  if (rule < SQ_RULE_NEAREST_EVEN || rule > SQ_RULE_WHOLE_TENSOR) return SQ_ERR_ARG;
  if (!W || !codes_out || !scales_out) return SQ_ERR_ARG;
  if (ws2_in > 0.0f && !isfinite(ws2_in)) return SQ_ERR_ARG;
  const bool slot = rule == SQ_RULE_WHOLE_TENSOR || (fmt == SQ_NVFP4 && !(ws2_in > 0.0f));
  if (slot && !ws2_out) return SQ_ERR_ARG;                   // the amax slot
  if (ws2_out && !aligned(ws2_out, 4)) return SQ_ERR_ALIGN;
  if (!aligned(W, 16) || !aligned(codes_out, 4)) return SQ_ERR_ALIGN;
  float* out = (fmt == SQ_NVFP4 || rule == SQ_RULE_WHOLE_TENSOR) ? ws2_out : nullptr;
  return hip_status(sq::rtn_rule_launch(fmt, (int)O, (int)I, W, fmt == SQ_NVFP4 ? ws2_in : 0.0f, rule, seed,
                                        codes_out, scales_out, out, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int rtn_quantize_grouped(int fmt, int rule, int n, const sq_rtn_desc* descs, void* stream) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  if (rule < SQ_RULE_NEAREST_EVEN || rule > SQ_RULE_WHOLE_TENSOR) return SQ_ERR_ARG;
  if (n < 0 || (n > 0 && !descs)) return SQ_ERR_ARG;
  std::vector<sq::RtnItem> items((size_t)n);
  std::vector<const float*> slots;
  for (int k = 0; k < n; ++k) {
    const sq_rtn_desc& d = descs[k];
    int st = check_layer(fmt, 0, d.O, d.I);
    if (st != SQ_OK) return st;
    if (d.reserved != 0) return SQ_ERR_ARG;
    if (!d.W || !d.codes_out || !d.scales_out) return SQ_ERR_ARG;
    if (d.ws2_in > 0.0f && !isfinite(d.ws2_in)) return SQ_ERR_ARG;
    const bool slot = rule == SQ_RULE_WHOLE_TENSOR || (fmt == SQ_NVFP4 && !(d.ws2_in > 0.0f));
    if (slot && !d.ws2_out) return SQ_ERR_ARG;
    if (d.ws2_out && !aligned(d.ws2_out, 4)) return SQ_ERR_ALIGN;
    if (!aligned(d.W, 16) || !aligned(d.codes_out, 4)) return SQ_ERR_ALIGN;
    if (slot) slots.push_back(d.ws2_out);
    float* out = (fmt == SQ_NVFP4 || rule == SQ_RULE_WHOLE_TENSOR) ? d.ws2_out : nullptr;
    items[(size_t)k] = sq::RtnItem{d.O, d.I, d.W, d.codes_out, d.scales_out, out,
                                   fmt == SQ_NVFP4 ? d.ws2_in : 0.0f, d.seed};
  }
  std::sort(slots.begin(), slots.end());
  if (std::adjacent_find(slots.begin(), slots.end()) != slots.end()) return SQ_ERR_ARG;   // a shared amax slot
  if (n == 0) return SQ_OK;
  return hip_status(sq::rtn_grouped_launch(fmt, rule, n, items.data(), static_cast<hipStream_t>(stream)));
}

namespace {
constexpr int kQastRankMax = 64;

int check_qast_plane(int64_t O, int64_t G, int r, int64_t E = 1) {
  if (E < 1 || E > 65535) return SQ_ERR_SHAPE;
  if (O < 1 || G < 1 || O > kDimMax || G > kDimMax || E * O * G > kDimMax) return SQ_ERR_SHAPE;
  if (E * O * r > kDimMax || E * r * G > kDimMax) return SQ_ERR_SHAPE;
  if (r < 1 || r > kQastRankMax) return SQ_ERR_SHAPE;
  return SQ_OK;
}

int qast_scales_checked(int fmt, int64_t E, int64_t O, int64_t G, int r, const uint8_t* base_scales, const void* B,
                        const void* A, float alpha_over_r, const float* ws2, uint8_t* scales_out,
                        uint8_t* clamp_mask_out, void* stream) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  int st = check_qast_plane(O, G, r, E);
  if (st != SQ_OK) return st;
  if (!base_scales || !B || !A || !scales_out) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (fmt == SQ_NVFP4) {
    if (!ws2) return SQ_ERR_ARG;
    for (int64_t e = 0; e < E; ++e)
      if (!ws2_ok(ws2[e])) return SQ_ERR_ARG;
  }
  if (!aligned(B, 2) || !aligned(A, 2)) return SQ_ERR_ALIGN;
  return hip_status(sq::qast_scales_launch(fmt, (int)E, (int)O, (int)G, r, base_scales, B, A, alpha_over_r, ws2,
                                           scales_out, clamp_mask_out, static_cast<hipStream_t>(stream)));
}

int qast_grads_checked(int64_t E, int64_t O, int64_t G, int r, const float* dS, const uint8_t* clamp_mask,
                       const void* B, const void* A, float alpha_over_r, float* dB, float* dA, void* workspace,
                       size_t workspace_bytes, void* stream) {
  int st = check_qast_plane(O, G, r, E);
  if (st != SQ_OK) return st;
  if (!dS || !B || !A || !dB || !dA) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (!aligned(dS, 4) || !aligned(B, 2) || !aligned(A, 2) || !aligned(dB, 4) || !aligned(dA, 4))
    return SQ_ERR_ALIGN;
  const size_t need = sq::qast_grads_workspace((int)E, (int)O, (int)G, r);
  if (!workspace || workspace_bytes < need) return SQ_ERR_WORKSPACE;
  if (!aligned(workspace, 4)) return SQ_ERR_ALIGN;
  return hip_status(sq::qast_grads_launch((int)E, (int)O, (int)G, r, dS, clamp_mask, B, A, alpha_over_r, dB, dA,
                                          workspace, static_cast<hipStream_t>(stream)));
}
}  // namespace

SQ_EXPORT int sq_qast_scales(int fmt, int64_t O, int64_t G, int r, const uint8_t* base_scales, const void* B,
                             const void* A, float alpha_over_r, float ws2, uint8_t* scales_out,
                             uint8_t* clamp_mask_out, void* stream) {
  return qast_scales_checked(fmt, 1, O, G, r, base_scales, B, A, alpha_over_r, &ws2, scales_out, clamp_mask_out,
                             stream);
}

SQ_EXPORT int sq_qast_scales_batched(int fmt, int64_t E, int64_t O, int64_t G, int r, const uint8_t* base_scales,
                                     const void* B, const void* A, float alpha_over_r, const float* ws2,
                                     uint8_t* scales_out, uint8_t* clamp_mask_out, void* stream) {
  return qast_scales_checked(fmt, E, O, G, r, base_scales, B, A, alpha_over_r, ws2, scales_out, clamp_mask_out,
                             stream);
}

SQ_EXPORT size_t sq_qast_factor_grads_workspace(int64_t O, int64_t G, int r) {
  if (check_qast_plane(O, G, r) != SQ_OK) return 0;
  return sq::qast_grads_workspace(1, (int)O, (int)G, r);
}

SQ_EXPORT size_t sq_qast_factor_grads_batched_workspace(int64_t E, int64_t O, int64_t G, int r) {
  if (check_qast_plane(O, G, r, E) != SQ_OK) return 0;
  return sq::qast_grads_workspace((int)E, (int)O, (int)G, r);
}

SQ_EXPORT int sq_qast_factor_grads(int64_t O, int64_t G, int r, const float* dS, const uint8_t* clamp_mask,
                                   const void* B, const void* A, float alpha_over_r, float* dB, float* dA,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  return qast_grads_checked(1, O, G, r, dS, clamp_mask, B, A, alpha_over_r, dB, dA, workspace, workspace_bytes,
                            stream);
}

SQ_EXPORT int sq_qast_factor_grads_batched(int64_t E, int64_t O, int64_t G, int r, const float* dS,
                                           const uint8_t* clamp_mask, const void* B, const void* A,
                                           float alpha_over_r, float* dB, float* dA, void* workspace,
                                           size_t workspace_bytes, void* stream) {
  return qast_grads_checked(E, O, G, r, dS, clamp_mask, B, A, alpha_over_r, dB, dA, workspace, workspace_bytes,
                            stream);
}

namespace {
constexpr int kLoraRankMax = 64;
constexpr int64_t kRequantRowsMax = int64_t(65535) * 16;     // grid.y of the fused re-quantiser
constexpr int64_t kLoraTokensMax = int64_t(65535) * 128;     // grid.y of the token-chunk kernel

int check_lora_dims(int64_t T, int64_t O, int64_t I, int r) {
  if (T < 0 || T > kLoraTokensMax || O < 1 || I < 1 || O > kDimMax || I > kDimMax) return SQ_ERR_SHAPE;
  if (O % 8 != 0 || I % 8 != 0) return SQ_ERR_SHAPE;
  if (T * I * 2 > kOperandBytesMax || T * O * 2 > kOperandBytesMax) return SQ_ERR_SHAPE;
  if (r < 1 || r > kLoraRankMax) return SQ_ERR_SHAPE;
  return SQ_OK;
}
}  // namespace

SQ_EXPORT int sq_qat_requant(int fmt, int64_t O, int64_t I, int r, const uint8_t* codes, const uint8_t* scales,
                             float ws2, const void* B, const void* A, float alpha_over_r, uint8_t* codes_out,
                             uint8_t* scales_out, void* stream) {
  int st = check_layer(fmt, 0, O, I);
  if (st != SQ_OK) return st;
  if (r < 1 || r > kLoraRankMax || O > kRequantRowsMax) return SQ_ERR_SHAPE;
  if (!codes || !scales || !B || !A || !codes_out || !scales_out) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (fmt == SQ_NVFP4 && !ws2_ok(ws2)) return SQ_ERR_ARG;
  if (!aligned(codes, 4) || !aligned(codes_out, 4) || !aligned(A, 16) || !aligned(B, 2)) return SQ_ERR_ALIGN;
  const float w = fmt == SQ_NVFP4 ? ws2 : 1.0f;
  return hip_status(sq::qat_requant_launch(fmt, 1, (int)O, (int)I, r, codes, scales, &w, B, A, alpha_over_r,
                                           codes_out, scales_out, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_qat_requant_batched(int fmt, int64_t E, int64_t O, int64_t I, int r, const uint8_t* codes,
                                     const uint8_t* scales, const float* ws2, const void* B, const void* A,
                                     float alpha_over_r, uint8_t* codes_out, uint8_t* scales_out, void* stream) {
  int st = check_layer(fmt, 0, O, I);
  if (st != SQ_OK) return st;
  if (E < 1 || E > 65535 || r < 1 || r > kLoraRankMax || O > kRequantRowsMax) return SQ_ERR_SHAPE;
  if (E * O * I / 2 > kDimMax || E * O * r > kDimMax || E * r * I > kDimMax) return SQ_ERR_SHAPE;
  if (!codes || !scales || !B || !A || !codes_out || !scales_out) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (fmt == SQ_NVFP4) {
    if (!ws2) return SQ_ERR_ARG;
    for (int64_t e = 0; e < E; ++e)
      if (!ws2_ok(ws2[e])) return SQ_ERR_ARG;
  }
  if (!aligned(codes, 4) || !aligned(codes_out, 4) || !aligned(A, 16) || !aligned(B, 2)) return SQ_ERR_ALIGN;
  return hip_status(sq::qat_requant_launch(fmt, (int)E, (int)O, (int)I, r, codes, scales, ws2, B, A, alpha_over_r,
                                           codes_out, scales_out, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT size_t sq_lora_grads_workspace(int64_t T, int64_t O, int64_t I, int r) {
  if (check_lora_dims(T, O, I, r) != SQ_OK) return 0;
  return sq::lora_grads_workspace((int)T, (int)O, (int)I, r);
}

SQ_EXPORT int sq_lora_grads(int64_t T, int64_t O, int64_t I, int r, const void* X, const void* dY, const void* B,
                            const void* A, float alpha_over_r, float* dB, float* dA, void* workspace,
                            size_t workspace_bytes, void* stream) {
  int st = check_lora_dims(T, O, I, r);
  if (st != SQ_OK) return st;
  if (!B || !A || !dB || !dA || (T > 0 && (!X || !dY))) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (!aligned(X, 16) || !aligned(dY, 16) || !aligned(A, 16) || !aligned(B, 2) || !aligned(dB, 4) ||
      !aligned(dA, 4))
    return SQ_ERR_ALIGN;
  const size_t need = sq::lora_grads_workspace((int)T, (int)O, (int)I, r);
  if (need > 0 && (!workspace || workspace_bytes < need)) return SQ_ERR_WORKSPACE;
  if (need > 0 && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  return hip_status(sq::lora_grads_launch((int)T, (int)O, (int)I, r, X, dY, B, A, alpha_over_r, dB, dA, workspace,
                                          static_cast<hipStream_t>(stream)));
}

namespace {
int check_lora_batch(int64_t E, const int64_t* T, int64_t O, int64_t I, int r) {
  if (E < 1 || E > 65535 || !T) return E < 1 || E > 65535 ? SQ_ERR_SHAPE : SQ_ERR_ARG;
  int64_t total = 0;
  for (int64_t e = 0; e < E; ++e) {
    int st = check_lora_dims(T[e], O, I, r);
    if (st != SQ_OK) return st;
    total += T[e];
  }
  if (total * I * 2 > kOperandBytesMax || total * O * 2 > kOperandBytesMax) return SQ_ERR_SHAPE;
  if (E * O * r > kDimMax || E * r * I > kDimMax) return SQ_ERR_SHAPE;
  return SQ_OK;
}
}  // namespace

SQ_EXPORT size_t sq_lora_grads_batched_workspace(int64_t E, const int64_t* T, int64_t O, int64_t I, int r) {
  if (check_lora_batch(E, T, O, I, r) != SQ_OK) return 0;
  return sq::lora_grads_batched_workspace((int)E, T, (int)O, (int)I, r);
}

SQ_EXPORT int sq_lora_grads_batched(int64_t E, const int64_t* T, int64_t O, int64_t I, int r, const void* X,
                                    const void* dY, const void* B, const void* A, float alpha_over_r, float* dB,
                                    float* dA, void* workspace, size_t workspace_bytes, void* stream) {
  int st = check_lora_batch(E, T, O, I, r);
  if (st != SQ_OK) return st;
  int64_t total = 0;
  for (int64_t e = 0; e < E; ++e) total += T[e];
  if (!B || !A || !dB || !dA || (total > 0 && (!X || !dY))) return SQ_ERR_ARG;
  if (!isfinite(alpha_over_r)) return SQ_ERR_ARG;
  if (!aligned(X, 16) || !aligned(dY, 16) || !aligned(A, 16) || !aligned(B, 2) || !aligned(dB, 4) ||
      !aligned(dA, 4))
    return SQ_ERR_ALIGN;
  const size_t need = sq::lora_grads_batched_workspace((int)E, T, (int)O, (int)I, r);
  if (need > 0 && (!workspace || workspace_bytes < need)) return SQ_ERR_WORKSPACE;
  if (need > 0 && !aligned(workspace, 16)) return SQ_ERR_ALIGN;
  return hip_status(sq::lora_grads_batched_launch((int)E, T, (int)O, (int)I, r, X, dY, B, A, alpha_over_r, dB, dA,
                                                  workspace, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_scale_applied_delta(int fmt, int64_t n, const uint8_t* before, const uint8_t* after, float* applied,
                                     void* stream) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  if (n < 0) return SQ_ERR_SHAPE;
  if (n == 0) return SQ_OK;
  if (!before || !after || !applied) return SQ_ERR_ARG;
  if (!aligned(before, 16) || !aligned(after, 16) || !aligned(applied, 16)) return SQ_ERR_ALIGN;
  return hip_status(sq::applied_launch(fmt, n, before, after, applied, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_scale_rollback(int fmt, int64_t n, uint8_t* scales, const float* applied, void* stream) {
  if (fmt != SQ_MXFP4 && fmt != SQ_NVFP4) return SQ_ERR_FORMAT;
  if (n < 0) return SQ_ERR_SHAPE;
  if (n == 0) return SQ_OK;
  if (!scales || !applied) return SQ_ERR_ARG;
  if (!aligned(scales, 16) || !aligned(applied, 16)) return SQ_ERR_ALIGN;
  return hip_status(sq::rollback_launch(fmt, n, scales, applied, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT int sq_byte_diff(int64_t n, const uint8_t* a, const uint8_t* b, uint64_t* counts, void* stream) {
  if (n < 0) return SQ_ERR_SHAPE;
  if (!counts) return SQ_ERR_ARG;
  if (n == 0) return SQ_OK;
  if (!a || !b) return SQ_ERR_ARG;
  if (!aligned(a, 16) || !aligned(b, 16) || !aligned(counts, 8)) return SQ_ERR_ALIGN;
  return hip_status(sq::byte_diff_launch(n, a, b, counts, static_cast<hipStream_t>(stream)));
}

SQ_EXPORT const char* sq_status_str(int status) {
  switch (status) {
    case SQ_OK: return "SQ_OK";
    case SQ_ERR_ARG: return "SQ_ERR_ARG: invalid argument";
    case SQ_ERR_SHAPE: return "SQ_ERR_SHAPE: invalid shape";
    case SQ_ERR_ALIGN: return "SQ_ERR_ALIGN: misaligned pointer";
    case SQ_ERR_FORMAT: return "SQ_ERR_FORMAT: unknown format";
    case SQ_ERR_WORKSPACE: return "SQ_ERR_WORKSPACE: workspace too small";
    case SQ_ERR_HIP: return "SQ_ERR_HIP: HIP runtime error";
    case SQ_ERR_UNIMPLEMENTED: return "SQ_ERR_UNIMPLEMENTED";
    default: return "unknown status";
  }
}

SQ_EXPORT int sq_abi_version(void) { return SQ_ABI_VERSION; }
