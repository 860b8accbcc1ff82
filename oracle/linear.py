"""Oracle for the frozen-code linear layer: dequant, forward, dX, dS (test infrastructure only).

Paper §2 ("Native FP4 microscaling storage"): W[o,i] = code[o,i] * eff_scale[o, g(i)],
g(i) = i // block.  Paper §3 ("Scale-QLoRA forward"): the layer computes
y = x W'^T with W' built from the frozen codes and the (adapted) block scales.

Backward.  With the codes frozen, the only trainable field is eff_scale.  By the
chain rule through W[o,i] = code[o,i] * eff[o, g(i)]:
    dX = dY W,
    dW[o,j] = sum_t dY[t,o] X[t,j],
    dS[o,b] = dL/d eff[o,b] = sum_{j in block b} code[o,j] * dW[o,j].
dS is the gradient with respect to the effective fp32 scale (for NVFP4 the
gradient with respect to the E4M3 value is dS * ws2).  It does not read the
scale field.

Every contraction is a float64 matmul on exact values: the inputs X, dY are
bf16 (exact in fp64) and every dequantised weight code*scale is exact in fp64.
"""

import numpy as np

from . import codec


def code_values(codes_packed: np.ndarray) -> np.ndarray:
    """[O, I/2] packed codes -> [O, I] fp64 E2M1 values."""
    return codec.E2M1_TABLE[codec.unpack_nibbles(codes_packed)]


def dequant(fmt: str, codes_packed: np.ndarray, scale_bytes: np.ndarray, ws2: float = 1.0) -> np.ndarray:
    """W[o,i] = code[o,i] * eff[o, i // block] in fp64."""
    c = code_values(codes_packed)
    eff = codec.effective_scales(fmt, scale_bytes, ws2)
    block = codec.BLOCK[fmt]
    O, I = c.shape
    if eff.shape != (O, I // block):
        raise ValueError(f"scale plane {eff.shape} does not match codes {c.shape} / block {block}")
    return c * np.repeat(eff, block, axis=1)


def forward(X: np.ndarray, W: np.ndarray) -> np.ndarray:
    """Y = X W^T, X [T, I], W [O, I] -> [T, O]."""
    return np.asarray(X, np.float64) @ np.asarray(W, np.float64).T


def backward_dx(dY: np.ndarray, W: np.ndarray) -> np.ndarray:
    """dX = dY W, dY [T, O], W [O, I] -> [T, I]."""
    return np.asarray(dY, np.float64) @ np.asarray(W, np.float64)


def backward_dscale(fmt: str, X: np.ndarray, dY: np.ndarray, codes_packed: np.ndarray) -> np.ndarray:
    """dS[o,b] = sum_{j in block b} code[o,j] * (dY^T X)[o,j]  -> [O, G] fp64."""
    dW = np.asarray(dY, np.float64).T @ np.asarray(X, np.float64)      # [O, I]
    c = code_values(codes_packed)
    block = codec.BLOCK[fmt]
    O, I = c.shape
    return (c * dW).reshape(O, I // block, block).sum(axis=2)
