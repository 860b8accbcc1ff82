"""Oracle for the QAT-LoRA weight-space STE step (test infrastructure only).

The merge-aware weight-space baseline the paper measures Scale-QLoRA against
(§2 related work, "Merge-aware weight-space"; App. "Training cost per step"):
ordinary LoRA on the weight, W = W_base + (alpha/r) B A with B [O, r] and
A [r, I], trained on the native grid through a straight-through estimator.
The forward computes with quantize(W); the backward treats quantize as the
identity, so the gradient reaching W is the dense dW = dY^T X and, by the
chain rule through W, dB = (alpha/r) dW A^T and dA = (alpha/r) B^T dW.

quantize() is the per-block nearest rule of rtn.quantize with ties to even
(the training STE's rule); for NVFP4 the per-tensor ws2 stays at the base's.

Readings (the paper fixes no precision for W):
* the rank-r term S[o, i] adds B[o, k] A[k, i] for k = 0 .. r-1 in fp32,
  rounding after each addition (every product of bf16 factors is exact in
  fp32), then Delta = fp32(alpha/r * S) -- the same order qast.delta_s uses;
* the base weight is the fp32 value code * eff with eff the fp32 effective
  scale (exact for MXFP4; for NVFP4 eff = fp32(e4m3 * ws2), then one rounding
  of the product);
* W_eff = bf16(fp32(base + Delta)), rounded to nearest even: the weight is a
  bf16 tensor, as the bf16 training the paper runs keeps it.
"""

import numpy as np

from . import codec, linear, qast, rtn


def _f32(x) -> np.ndarray:
    if hasattr(x, "float"):
        x = x.float().cpu().numpy()
    return np.asarray(x, dtype=np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> nearest-even bf16 value (as fp32); NaN stays NaN, overflow goes to inf."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32)
    return np.where(nan, np.float32(np.nan), out)


def base_weight_f32(fmt: str, codes_packed: np.ndarray, scale_bytes: np.ndarray, ws2: float = 1.0) -> np.ndarray:
    """fp32 code * eff, eff the fp32 effective scale of each block."""
    c = linear.code_values(codes_packed).astype(np.float32)
    eff = codec.effective_scales(fmt, scale_bytes, ws2).astype(np.float32)
    return c * np.repeat(eff, codec.BLOCK[fmt], axis=1)


def effective_weight(fmt: str, codes_packed, scale_bytes, ws2, B, A, alpha_over_r: float) -> np.ndarray:
    """W_eff [O, I] as bf16 values (fp32 array)."""
    base = base_weight_f32(fmt, codes_packed, scale_bytes, ws2)
    delta = qast.delta_s(B, A, alpha_over_r)              # fp32 [O, I], k in increasing order
    return bf16_round(base + delta)


def requant(fmt: str, codes_packed, scale_bytes, ws2, B, A, alpha_over_r: float):
    """The fake-quantised forward weight as (codes, scale bytes): the fake-quantised
    weight equals linear.dequant(fmt, codes, scales, ws2) exactly."""
    W = effective_weight(fmt, codes_packed, scale_bytes, ws2, B, A, alpha_over_r)
    codes, sbytes, _ = rtn.quantize(fmt, W, rtn.TIE_EVEN, ws2 if fmt == codec.NV else None)
    return codes, sbytes


def lora_grads(X, dY, B, A, alpha_over_r: float):
    """(dB [O, r], dA [r, I]) in fp64 through the STE: dW = dY^T X materialised."""
    X64, dY64 = _f32(X).astype(np.float64), _f32(dY).astype(np.float64)
    B64, A64 = _f32(B).astype(np.float64), _f32(A).astype(np.float64)
    dW = dY64.T @ X64
    c = float(np.float32(alpha_over_r))
    return c * (dW @ A64.T), c * (B64.T @ dW)


def lora_grads_sampled(X, dY, B, A, alpha_over_r: float, rows, cols):
    """dB[rows, :] and dA[:, cols] in fp64, each from its own rows / columns of
    dW = dY^T X: dB[o, :] = c dW[o, :] A^T, dA[:, i] = c B^T dW[:, i]."""
    X64, dY64 = _f32(X).astype(np.float64), _f32(dY).astype(np.float64)
    B64, A64 = _f32(B).astype(np.float64), _f32(A).astype(np.float64)
    c = float(np.float32(alpha_over_r))
    dW_rows = dY64[:, rows].T @ X64                       # [len(rows), I]
    dW_cols = dY64.T @ X64[:, cols]                       # [O, len(cols)]
    return c * (dW_rows @ A64.T), c * (B64.T @ dW_cols)
