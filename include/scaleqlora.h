/*
 * scaleqlora.h -- C ABI of the Scale-QLoRA frozen-code FP4 linear layer for
 * AMD Instinct MI355X (gfx950).
 *
 * The layer stores a weight as a frozen plane of 4-bit E2M1 codes and a plane
 * of per-block scale bytes (paper, Section 2, "Native FP4 microscaling
 * storage"):
 *
 *     W[o,i] = code[o,i] * eff[o, i / B]
 *
 *   MXFP4 (SQ_MXFP4): B = 32, one E8M0 byte per block, eff = 2^(byte-127).
 *   NVFP4 (SQ_NVFP4): B = 16, one E4M3 byte per block times one fp32
 *                     per-tensor scalar ws2, eff = e4m3(byte) * ws2.
 *
 * The only trainable field is the block scale (Section 3, "Scale-QLoRA
 * forward" and "QAST makes merge exact by construction").  This library
 * provides the layer's forward, its two backward products (dX and the
 * per-block scale gradient dS), the scale-plane merge / swap, and the
 * round-to-nearest re-quantiser that the naive weight-space merge uses.
 *
 * Conventions shared by every entry point
 * ----------------------------------------
 * Shapes    T tokens, O output features, I input features, G = I / B blocks.
 * Layouts   all row-major, densely packed, no strides:
 *             X   bf16  [T, I]        dY  bf16  [T, O]
 *             Y         [T, O]        dX        [T, I]
 *             codes uint8 [O, I/2]    two codes per byte, the LOW nibble holds
 *                                     the even column i, the high nibble i+1;
 *                                     nibble = sign(bit 3) | exponent(2) |
 *                                     mantissa(1), values +-{0,.5,1,1.5,2,3,4,6}
 *             scales uint8 [O, G]     E8M0 (MX) or E4M3 "fn" (NV) bytes
 *             dS  fp32  [O, G]
 * Pointers  every data pointer is a DEVICE pointer (memory of the current HIP
 *           device); the caller allocates and owns every buffer.  No entry point
 *           allocates device memory.  Inputs are never written.
 * Streams   `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *           Every call only enqueues work on it and returns; nothing is
 *           synchronised.  Calls are reentrant and thread-safe.
 * Shapes    T >= 0; O >= 1, O % 8 == 0; I >= 1, I % B == 0.  T == 0 is legal:
 *           Y and dX are empty and dS is written as zeros.  Every dimension
 *           stays below 2^31, and X, dY and the code plane each stay below
 *           2 GiB (T*I*2, T*O*2 and O*I/2 bytes).
 * Alignment X, dY, Y, dX: 16 bytes.  codes: 4 bytes.  dS: 4 bytes.
 *           Merge scale planes, deltas and sources: 16 bytes.
 * Errors    arguments are checked on the host before anything is enqueued; a
 *           violation returns a negative sq_status and enqueues nothing.  A
 *           failed launch returns SQ_ERR_HIP.  Data values are never checked:
 *           NaN inputs and NaN scale bytes (E8M0 0xFF, E4M3 0x7F/0xFF)
 *           propagate to the outputs.
 */
#ifndef SCALEQLORA_H
#define SCALEQLORA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SQ_ABI_VERSION 1

/* Status codes returned by every int-valued entry point. */
typedef enum {
  SQ_OK = 0,
  SQ_ERR_ARG = -1,           /* NULL pointer, unknown enum value, bad scalar */
  SQ_ERR_SHAPE = -2,         /* dimension out of range or not a multiple */
  SQ_ERR_ALIGN = -3,         /* pointer misaligned for the layout above */
  SQ_ERR_FORMAT = -4,        /* unknown sq_format */
  SQ_ERR_WORKSPACE = -5,     /* workspace missing or too small */
  SQ_ERR_HIP = -6,           /* the HIP runtime reported an error */
  SQ_ERR_UNIMPLEMENTED = -7
} sq_status;

typedef enum { SQ_MXFP4 = 0, SQ_NVFP4 = 1 } sq_format;
typedef enum { SQ_OUT_F32 = 0, SQ_OUT_BF16 = 1 } sq_out_dtype;
typedef enum { SQ_TIE_EVEN = 0, SQ_TIE_AWAY = 1 } sq_tie;
typedef enum { SQ_MERGE_DELTA = 0, SQ_MERGE_COPY = 1 } sq_merge_mode;
typedef enum {
  SQ_RULE_NEAREST_EVEN = 0,  /* = rtn_quantize with SQ_TIE_EVEN */
  SQ_RULE_NEAREST_AWAY = 1,  /* = rtn_quantize with SQ_TIE_AWAY */
  SQ_RULE_RTZ = 2,           /* codes toward zero, per-block scales */
  SQ_RULE_STOCHASTIC = 3,    /* codes by stochastic rounding, per-block scales */
  SQ_RULE_WHOLE_TENSOR = 4   /* one scale from the tensor amax, nearest-even codes */
} sq_rule;

/*
 * Forward, Y = X W^T (paper Section 2 storage equation; Section 3,
 * "Scale-QLoRA forward": y = x W'^T).
 *
 * X bf16 [T, I]; codes [O, I/2]; scales [O, G]; ws2 the NVFP4 per-tensor
 * scalar (ignored for MXFP4; for NVFP4 it must be finite and > 0).
 * Y [T, O] is written in y_dtype (SQ_OUT_F32 or SQ_OUT_BF16, round to nearest
 * even).  The dequantised weight code * scale is formed exactly in bf16 on
 * chip and the contraction accumulates in fp32 on the bf16 matrix cores; for
 * NVFP4 ws2 is applied once to the fp32 accumulator.  Results are
 * deterministic.  The order in which the fp32 sums of one 64-deep K stage are
 * taken depends on the path: MXFP4 with codes 16-byte and scales 8-byte
 * aligned and I % 256 == 0 dequantises in registers (a lane takes 32
 * consecutive k), other
 * calls dequantise through LDS, so the two can differ in the last bits.
 */
int sq_fwd(int fmt, int64_t T, int64_t O, int64_t I,
           const void* X, const uint8_t* codes, const uint8_t* scales, float ws2,
           void* Y, int y_dtype, void* stream);

/*
 * Input gradient, dX = dY W.  With the codes frozen, the gradient reaching the
 * layer input passes through the same on-grid weight the forward used
 * (Section 3, QAST forward with the straight-through estimator: the forward
 * runs on the on-grid scale).
 *
 * dY bf16 [T, O]; codes, scales, ws2 as for sq_fwd; dX [T, I] in dx_dtype.
 */
int sq_bwd_dx(int fmt, int64_t T, int64_t O, int64_t I,
              const void* dY, const uint8_t* codes, const uint8_t* scales, float ws2,
              void* dX, int dx_dtype, void* stream);

/*
 * Per-block scale gradient (the gradient Section 3's scale adapter receives
 * through eff_scale', by the chain rule through W = code * eff):
 *
 *     dS[o,b] = sum_{j in block b} code[o,j] * sum_t dY[t,o] * X[t,j]
 *
 * X bf16 [T, I]; dY bf16 [T, O]; codes [O, I/2]; dS fp32 [O, G], fully
 * overwritten.  dS is the gradient with respect to the effective fp32 scale
 * eff (for NVFP4 the gradient with respect to the E4M3 value is dS * ws2), so
 * this call takes no scale plane.  The dW tile is produced on the matrix cores
 * and reduced against the codes on chip; no [O, I] tensor is written.
 * Deterministic: the same inputs give bitwise identical dS.
 * workspace / workspace_bytes: device scratch of at least
 * sq_bwd_dscale_workspace(fmt, T, O, I) bytes, 16-byte aligned (NULL / 0
 * when that is 0); its contents on entry do not matter and are overwritten.
 * A missing or short workspace returns SQ_ERR_WORKSPACE.
 */
int sq_bwd_dscale(int fmt, int64_t T, int64_t O, int64_t I,
                  const void* X, const void* dY, const uint8_t* codes, float* dS,
                  void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes sq_bwd_dscale needs for this shape (0 = none).  It is
 * nonzero when the layer has too few 256 x 256 output tiles to occupy every
 * compute unit and enough tokens to split: the token sum then runs as S
 * ranges (2 <= S <= 8) whose partial dS planes (S * O * G fp32) are added in
 * a fixed order.  Returns 0 for invalid arguments as well; sq_bwd_dscale
 * then reports the error. */
size_t sq_bwd_dscale_workspace(int fmt, int64_t T, int64_t O, int64_t I);

/*
 * sq_bwd_dscale without a workspace, for callers that cannot allocate device
 * memory: code being captured into a HIP graph, tight serving and training
 * loops, harnesses that forbid allocation.  It computes exactly what
 * sq_bwd_dscale computes (same kernels, same summation order, bitwise equal
 * dS) and allocates nothing: when the token sum is split, the partial dS
 * planes live in a static device array of the library, SQ_DSCALE_SCRATCH_BYTES
 * per device (every shape's plan fits in it; a larger need would return
 * SQ_ERR_WORKSPACE).  The array is shared by every call on a device and keeps
 * the last call's partial planes; calls that overlap on one device (on
 * different streams, or from different threads without ordering) race on it
 * and must be serialised by the caller.  Arguments and errors otherwise as
 * sq_bwd_dscale.
 */
#define SQ_DSCALE_SCRATCH_BYTES ((size_t)4 << 20)
int sq_bwd_dscale_noalloc(int fmt, int64_t T, int64_t O, int64_t I,
                          const void* X, const void* dY, const uint8_t* codes, float* dS, void* stream);

/*
 * Scale-plane merge or swap, in place, over n scale bytes (Section 3, "QAST
 * makes merge exact by construction": the merge writes the on-grid scale byte
 * training used and copies the codes; stability recipe items (ii)-(iii): the
 * NVFP4 ceiling clamp min(eff, 448*ws2) runs on the same path; Appendix B,
 * "Payoff 2": a hot swap overwrites the scale bytes and leaves codes
 * untouched).  No code plane is taken, so no code byte can change.
 *
 * mode SQ_MERGE_DELTA: delta fp32 [n] is an update of the effective scale.
 *   NVFP4: e = fp32(e4m3(b) * ws2); e2 = fp32(e + delta); e2 = min(e2,
 *          fp32(448 * ws2)); q = fp32(e2 / ws2); b' = E4M3 nearest-even,
 *          saturating at 448.
 *   MXFP4: e2 = fp32(2^(b-127) + delta); b' = E8M0 of 2^round(log2 e2),
 *          nearest in the log domain (exponent clamped to [-127, 127];
 *          e2 <= 0 gives 0x00; NaN gives 0xFF).
 *   Every step is one correctly rounded fp32 operation (no fused multiply-add).
 *   src is ignored.
 * mode SQ_MERGE_COPY: scales[k] = src[k] (delta and ws2 ignored).
 * scales, delta, src: device, 16-byte aligned; n >= 0.
 */
int sq_merge_scales(int fmt, int64_t n, uint8_t* scales, const float* delta,
                    const uint8_t* src, float ws2, int mode, void* stream);

/* One scale plane of a grouped merge. */
typedef struct sq_merge_desc {
  int64_t n;                /* scale bytes in this plane */
  uint8_t* scales;          /* device, in place, 16-byte aligned */
  const float* delta;       /* device, SQ_MERGE_DELTA */
  const uint8_t* src;       /* device, SQ_MERGE_COPY */
  float ws2;                /* NVFP4 per-tensor scalar */
  int32_t fmt;              /* sq_format */
  int32_t mode;             /* sq_merge_mode */
  int32_t reserved;         /* must be 0 */
} sq_merge_desc;

/*
 * sq_merge_scales over many planes in as few launches as possible (a whole
 * model's scale planes, Appendix B "Payoff 2": swapping the served task writes
 * only the scale plane of every target linear).  descs is a HOST array of
 * n_desc descriptors, each validated like a sq_merge_scales call; planes must
 * not overlap.  The descriptors are read during the call only.
 */
int sq_merge_scales_grouped(int n_desc, const sq_merge_desc* descs, void* stream);

/*
 * Grouped products over the experts of an MoE layer (Section 3, MoE path: the
 * expert weights are stacked and every expert's scale adapter is applied in
 * one batched pass): experts share O and I (and the format) and each has its
 * own routed tokens, activations, weights and outputs.  Each expert computes
 * exactly what the single-product entry point computes for it (sq_fwd,
 * sq_bwd_dx, sq_bwd_dscale), with the same accumulation order per output
 * element (the MXFP4 forward dequantises in registers when every expert's
 * codes are 16-byte and scales 8-byte aligned and I % 256 == 0, as sq_fwd
 * does for one); the whole list runs in one launch per 128 experts (fewer
 * when one kind of pointer of those experts spans 4 GiB or more), and
 * sq_bwd_dx_grouped may run the rows of experts' short last token tiles in a
 * second launch of its own.
 *
 *   act     sq_fwd_grouped, sq_bwd_dscale_grouped: X_e bf16 [T_e, I];
 *           sq_bwd_dx_grouped: dY_e bf16 [T_e, O]  (16-byte aligned)
 *   act2    sq_bwd_dscale_grouped: dY_e bf16 [T_e, O] (16-byte aligned);
 *           otherwise ignored
 *   codes   expert e's codes [O, I/2] (4-byte aligned)
 *   scales  expert e's scale bytes [O, G] (sq_fwd_grouped, sq_bwd_dx_grouped)
 *   out     Y_e [T_e, O] / dX_e [T_e, I] in the given dtype (16-byte aligned),
 *           or dS_e fp32 [O, G] (4-byte aligned; all zeros when T_e = 0)
 *   T       tokens routed to expert e, 0 <= T_e (pointers that only serve
 *           tokens may be NULL when T_e = 0)
 *   ws2     expert e's NVFP4 per-tensor scalar (finite, > 0; ignored for
 *           MXFP4 and by sq_bwd_dscale_grouped)
 *   reserved must be 0
 * n_experts >= 0; descs is read during the call only.
 */
typedef struct {
  const void* act;
  const void* act2;
  const uint8_t* codes;
  const uint8_t* scales;
  void* out;
  int64_t T;
  float ws2;
  int32_t reserved;
} sq_expert_desc;

int sq_fwd_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs, int y_dtype,
                   void* stream);
int sq_bwd_dx_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs, int dx_dtype,
                      void* stream);
int sq_bwd_dscale_grouped(int fmt, int64_t O, int64_t I, int n_experts, const sq_expert_desc* descs, void* stream);

/*
 * Round-to-nearest re-quantisation of a bf16 weight [O, I] into codes and
 * scales, the naive merge W' = requant(dequant(W) + (alpha/r) BA) (Section 2,
 * "The naive re-quantized merge is the failure mode").
 *
 *   MXFP4: per block k = ceil(log2(fp32(amax / 6))) (the shipping rule, with
 *          the mantissa masked off; Appendix "Calibrated PTQ on a Sparse MoE"),
 *          clamped to [-127, 127], all-zero block -> k = -127; byte k + 127;
 *          q = w / 2^k.
 *   NVFP4: per-tensor ws2 = ws2_in when ws2_in > 0, else recomputed as
 *          fp32(fp32(amax_tensor / 6) / 448) (1 for an all-zero tensor); per
 *          block byte = E4M3 nearest-even of fp32(fp32(amax / 6) / ws2) (the
 *          amax/6 nearest rule; Appendix "Why the Naive Merge Returns the
 *          Base"); se = fp32(e4m3(byte) * ws2); q = fp32(w / se) (0 if se = 0).
 *   Codes: |q| to the nearest E2M1 magnitude with ties per `tie` (SQ_TIE_EVEN:
 *          even mantissa; SQ_TIE_AWAY: away from zero), saturating at 6; the
 *          sign bit is the sign of w, also for a zero magnitude; a NaN q codes
 *          as magnitude 0.
 *
 * W bf16 [O, I]; codes_out [O, I/2]; scales_out [O, G]; ws2_out: device fp32
 * scalar receiving the ws2 used (NVFP4; may be NULL for MXFP4 or when ws2_in
 * > 0).  Recomputing ws2 needs ws2_out (it holds the tensor amax in between).
 */
int rtn_quantize(int fmt, int64_t O, int64_t I, const void* W, float ws2_in, int tie,
                 uint8_t* codes_out, uint8_t* scales_out, float* ws2_out, void* stream);

/*
 * Re-quantisation of a bf16 weight under a serving-side rule, the out-of-family
 * deploy quantisers of the robustness sweep (Appendix B, threat model (a) and
 * the deployment-quantizer sweep: truncation, stochastic rounding and a
 * whole-tensor scale alongside the nearest rules).
 *
 *   SQ_RULE_NEAREST_EVEN / _AWAY: exactly rtn_quantize with that tie rule.
 *   SQ_RULE_RTZ: scales as rtn_quantize; each code magnitude is the largest
 *          E2M1 magnitude not above min(|q|, 6).
 *   SQ_RULE_STOCHASTIC: scales as rtn_quantize; with lo the truncated
 *          magnitude and hi the next one (hi = lo at 6), the code takes hi iff
 *          u_e < (min(|q|, 6) - lo) / (hi - lo), where u_e for element
 *          e = o*I + i is word e % 4 of Philox4x64-10 at counter (e / 4, 0, 0,
 *          0) and key (seed, 0), its top 24 bits times 2^-24.  On-grid values
 *          never move.
 *   SQ_RULE_WHOLE_TENSOR: every block takes the scale rtn_quantize would give
 *          a block whose amax is the tensor amax (for NVFP4, ws2 fixed or
 *          recomputed as in rtn_quantize); codes nearest-even.
 *   A NaN q codes as magnitude 0 and the sign bit is the sign of w (all rules).
 *
 * Arguments as rtn_quantize.  ws2_out (device fp32 scalar, 4-byte aligned) is
 * required for SQ_RULE_WHOLE_TENSOR (it holds the tensor amax during the call
 * and the ws2 used at the end, 1 for MXFP4) and wherever rtn_quantize needs it.
 * seed is used by SQ_RULE_STOCHASTIC only.
 */
int rtn_quantize_rule(int fmt, int64_t O, int64_t I, const void* W, float ws2_in, int rule, uint64_t seed,
                      uint8_t* codes_out, uint8_t* scales_out, float* ws2_out, void* stream);

/* One weight of a grouped re-quantisation: the per-weight arguments of
 * rtn_quantize_rule. */
typedef struct sq_rtn_desc {
  int64_t O, I;             /* weight shape [O, I] */
  const void* W;            /* device bf16 [O, I], 16-byte aligned */
  uint8_t* codes_out;       /* device [O, I/2], 4-byte aligned */
  uint8_t* scales_out;      /* device [O, I/B] */
  float* ws2_out;           /* device fp32 scalar, 4-byte aligned, or NULL (as rtn_quantize_rule) */
  float ws2_in;             /* NVFP4 per-tensor ws2 (> 0), or <= 0 to recompute */
  int32_t reserved;         /* must be 0 */
  uint64_t seed;            /* Philox key of SQ_RULE_STOCHASTIC */
} sq_rtn_desc;

/*
 * rtn_quantize_rule over many weights of one format under one rule (the
 * naive merge re-quantises every linear of the model, Section 2): each
 * weight's codes, scales and ws2_out are exactly those of its own
 * rtn_quantize_rule call, and the weights share launches (up to 56 per
 * launch) instead of taking one each.  descs is a HOST array of n
 * descriptors, read during the call only, each validated like a
 * rtn_quantize_rule call; outputs must not overlap one another or any W, and
 * a weight that needs its ws2_out slot (whole-tensor rule, or NVFP4 with
 * ws2_in <= 0) must not share it with another weight (SQ_ERR_ARG).
 */
int rtn_quantize_grouped(int fmt, int rule, int n, const sq_rtn_desc* descs, void* stream);

/*
 * QAST low-rank scale step (Section 3, "Scale-QLoRA forward": Delta_S =
 * (alpha/r) B A with A block-level, eff' = eff + Delta_S; "QAST makes merge
 * exact by construction": the forward uses round_grid(eff'); stability recipe
 * (ii)-(iii): the NVFP4 ceiling clamp, on the same grid-and-clamp path as the
 * merge).
 *
 * sq_qast_scales writes the on-grid scale bytes the QAST forward computes with
 * (pass them as `scales` to sq_fwd / sq_bwd_dx):
 *   Delta_S[o,g] = fp32(alpha_over_r * S[o,g]), S[o,g] = sum over k = 0..r-1 in
 *                  increasing order of B[o,k] A[k,g], fp32, each product exact;
 *   scales_out   = the SQ_MERGE_DELTA update of base_scales by Delta_S (the
 *                  same function the merge runs, bit for bit);
 *   clamp_mask_out[o,g] = 0 where the NVFP4 ceiling min(eff', 448 ws2) bound,
 *                  else 1 (always 1 for MXFP4); may be NULL.
 * O, G >= 1 with O*G < 2^31; 1 <= r <= 64.  base_scales, scales_out,
 * clamp_mask_out: device uint8 [O, G] (scales_out may equal base_scales);
 * B: device bf16 [O, r]; A: device bf16 [r, G]; alpha_over_r finite; ws2 as
 * for sq_fwd (ignored for MXFP4).
 */
int sq_qast_scales(int fmt, int64_t O, int64_t G, int r, const uint8_t* base_scales, const void* B,
                   const void* A, float alpha_over_r, float ws2, uint8_t* scales_out,
                   uint8_t* clamp_mask_out, void* stream);

/*
 * Gradients of the low-rank factors from the scale gradient dS (sq_bwd_dscale)
 * through the straight-through estimator and the clamp:
 *   dB = alpha_over_r (dS * m) A^T   fp32 [O, r]
 *   dA = alpha_over_r B^T (dS * m)   fp32 [r, G]
 * m = clamp_mask (NULL: all 1).  Accumulation is fp32 in a fixed order, so the
 * results are deterministic.  workspace: device scratch of at least
 * sq_qast_factor_grads_workspace(O, G, r) bytes (partial dA planes), 4-byte
 * aligned, contents irrelevant.
 */
size_t sq_qast_factor_grads_workspace(int64_t O, int64_t G, int r);
int sq_qast_factor_grads(int64_t O, int64_t G, int r, const float* dS, const uint8_t* clamp_mask,
                         const void* B, const void* A, float alpha_over_r, float* dB, float* dA,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * The QAST step for the E experts of an MoE layer in the same launches
 * (Section 3, MoE path: every expert's Delta_S in one batched pass).  The
 * experts are stacked: base_scales, scales_out, clamp_mask_out, dS [E, O, G];
 * B [E, O, r]; A [E, r, G]; dB fp32 [E, O, r]; dA fp32 [E, r, G].  Expert e
 * computes exactly what sq_qast_scales / sq_qast_factor_grads compute for its
 * planes.  ws2: host array of E per-expert NVFP4 scalars (read during the
 * call; ignored and may be NULL for MXFP4).  1 <= E <= 65535 and
 * E*O*G, E*O*r, E*r*G < 2^31; workspace: at least
 * sq_qast_factor_grads_batched_workspace(E, O, G, r) bytes.
 */
int sq_qast_scales_batched(int fmt, int64_t E, int64_t O, int64_t G, int r, const uint8_t* base_scales,
                           const void* B, const void* A, float alpha_over_r, const float* ws2, uint8_t* scales_out,
                           uint8_t* clamp_mask_out, void* stream);
size_t sq_qast_factor_grads_batched_workspace(int64_t E, int64_t O, int64_t G, int r);
int sq_qast_factor_grads_batched(int64_t E, int64_t O, int64_t G, int r, const float* dS, const uint8_t* clamp_mask,
                                 const void* B, const void* A, float alpha_over_r, float* dB, float* dA,
                                 void* workspace, size_t workspace_bytes, void* stream);

/*
 * QAT-LoRA weight-space STE comparator (Section 2 related work, "Merge-aware
 * weight-space": W <- W + (quantize(W) - W).detach() on W = W_base + (alpha/r)
 * B A; Appendix "Training cost per step").  The fake-quantised forward weight
 * is a (codes, scales) pair on the native grid, so sq_fwd and sq_bwd_dx run on
 * the output of sq_qat_requant directly.
 *
 * sq_qat_requant: one fused pass writing the nearest-rule re-quantisation of
 *   W_eff[o,i] = bf16(fp32(base[o,i] + fp32(alpha_over_r * S[o,i])))
 *   base[o,i]  = fp32(code[o,i] * eff[o, i/B]), eff as sq_fwd (NVFP4: fp32
 *                e4m3(byte) * ws2);
 *   S[o,i]     = sum over k = 0..r-1 in increasing order of B[o,k] A[k,i],
 *                fp32, each product exact;
 * with bf16 rounding to nearest even (NaN -> +NaN).  The codes and scales are
 * exactly what rtn_quantize(fmt, W_eff, SQ_TIE_EVEN, ws2) writes (NVFP4 keeps
 * the given ws2).  codes, scales: the base [O, I/2], [O, G]; B bf16 [O, r];
 * A bf16 [r, I] (16-byte aligned); 1 <= r <= 64; O <= 1048560; alpha_over_r
 * finite; codes_out, scales_out must not overlap the inputs.
 *
 * sq_lora_grads: the factor gradients through the straight-through estimator,
 *   dB = alpha_over_r dY^T X A^T   fp32 [O, r]
 *   dA = alpha_over_r B^T dY^T X   fp32 [r, I]
 * computed through the rank (P = X A^T and Q = dY B first), without forming
 * dY^T X; fp32 accumulation in a fixed order (deterministic).  X bf16 [T, I],
 * dY bf16 [T, O] (16-byte aligned), B bf16 [O, r], A bf16 [r, I] (16-byte
 * aligned); 0 <= T <= 8388480 (T = 0 writes zeros); O, I multiples of 8;
 * 1 <= r <= 64.  workspace: device scratch of at least
 * sq_lora_grads_workspace(T, O, I, r) bytes, 16-byte aligned, contents
 * irrelevant (0 bytes when T = 0; 0 is also returned for invalid sizes).
 */
int sq_qat_requant(int fmt, int64_t O, int64_t I, int r, const uint8_t* codes, const uint8_t* scales, float ws2,
                   const void* B, const void* A, float alpha_over_r, uint8_t* codes_out, uint8_t* scales_out,
                   void* stream);
size_t sq_lora_grads_workspace(int64_t T, int64_t O, int64_t I, int r);
int sq_lora_grads(int64_t T, int64_t O, int64_t I, int r, const void* X, const void* dY, const void* B,
                  const void* A, float alpha_over_r, float* dB, float* dA, void* workspace, size_t workspace_bytes,
                  void* stream);

/*
 * The QAT-LoRA comparator over the E experts of an MoE layer (Section 3, MoE
 * path, with the weight-space adapter in place of the scale adapter; Appendix
 * "Training cost per step": the MoE comparison).  Expert e computes exactly
 * what the single call computes for its weight, bit for bit.
 *
 * sq_qat_requant_batched: E stacked experts: codes [E, O, I/2], scales
 *   [E, O, G], B bf16 [E, O, r], A bf16 [E, r, I], codes_out, scales_out as
 *   codes, scales; ws2: host array of E per-expert NVFP4 scalars (read during
 *   the call; ignored and may be NULL for MXFP4).  1 <= E <= 65535, E*O*I/2,
 *   E*O*r and E*r*I below 2^31; otherwise as sq_qat_requant.
 * sq_lora_grads_batched: T is a host array of E token counts (T_e >= 0, read
 *   during the call).  X bf16 [sum T_e, I] and dY bf16 [sum T_e, O] hold the
 *   experts' routed token rows one expert after another (the rows of expert
 *   e start after those of experts 0 .. e-1); B bf16 [E, O, r], A bf16
 *   [E, r, I]; dB fp32 [E, O, r], dA fp32 [E, r, I] (an expert without tokens
 *   gets zeros).  workspace: at least sq_lora_grads_batched_workspace bytes
 *   (the sum of each expert's sq_lora_grads_workspace), 16-byte aligned.
 *   Otherwise as sq_lora_grads.
 */
int sq_qat_requant_batched(int fmt, int64_t E, int64_t O, int64_t I, int r, const uint8_t* codes,
                           const uint8_t* scales, const float* ws2, const void* B, const void* A, float alpha_over_r,
                           uint8_t* codes_out, uint8_t* scales_out, void* stream);
size_t sq_lora_grads_batched_workspace(int64_t E, const int64_t* T, int64_t O, int64_t I, int r);
int sq_lora_grads_batched(int64_t E, const int64_t* T, int64_t O, int64_t I, int r, const void* X, const void* dY,
                          const void* B, const void* A, float alpha_over_r, float* dB, float* dA, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * Merge rollback (Appendix B, "Payoff 3: invertible merges and rollback"): a
 * merged scale plane plus the on-grid delta the merge applied restores the
 * base plane byte for byte, with no retained base.  The delta lives in the
 * stored field's value domain: the E4M3 value for NVFP4 (ws2 stays out), the
 * effective scale 2^(b-127) for MXFP4.
 *
 * sq_scale_applied_delta: applied[i] = value(after[i]) - value(before[i]),
 *   one fp32 subtraction (exact when the two values are within 24 binades,
 *   which covers every pair of finite E4M3 bytes).
 * sq_scale_rollback: scales[i] = encode(value(scales[i]) - applied[i]), in
 *   place, with the merge's encoders (E4M3 nearest-even saturating; E8M0
 *   log-nearest).
 * before, after, scales: device uint8 [n]; applied: device fp32 [n]; all
 * 16-byte aligned; n >= 0.
 */
int sq_scale_applied_delta(int fmt, int64_t n, const uint8_t* before, const uint8_t* after, float* applied,
                           void* stream);
int sq_scale_rollback(int fmt, int64_t n, uint8_t* scales, const float* applied, void* stream);

/*
 * Byte audit (Appendix B, "Payoff 5: verifiability and provenance"): with codes
 * frozen a scale-merged artifact may differ from its base only in the scale
 * plane.  Adds to counts[0] the number of bytes i with a[i] != b[i] and to
 * counts[1] the number of differing 4-bit nibbles (E2M1 codes for a code
 * plane).  a, b: device uint8 [n], 16-byte aligned; counts: device uint64 [2],
 * 8-byte aligned, accumulated (the caller zeroes it), exact and
 * order-independent.
 */
int sq_byte_diff(int64_t n, const uint8_t* a, const uint8_t* b, uint64_t* counts, void* stream);

/* Human-readable name of a status code (static storage). */
const char* sq_status_str(int status);

/* SQ_ABI_VERSION of the built library. */
int sq_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SCALEQLORA_H */
