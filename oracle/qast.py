"""Oracle for one QAST low-rank scale step (test infrastructure only).

Paper §3, "Scale-QLoRA forward": the adapter is a rank-r correction of the
per-block scales, Delta_S = (B A)(alpha/r) with B [O, r] and A [r, G] (A is
block-level: one column per scale block), eff' = eff + Delta_S, and the
layer computes with W'[o, i] = code[o, i] * eff'[o, i / B].  The scale
arithmetic is fp32.

§3, "QAST makes merge exact by construction": the forward rounds eff' onto
the deployment grid (round_grid) and uses that on-grid value, while the
straight-through estimator passes the gradient to eff' unchanged.  Stability
recipe item (ii): NVFP4 clamps eff' at 448 * ws2 before rounding; item
(iii): the merge reuses the identical grid-and-clamp path.  Here the scale
bytes the forward uses are therefore exactly merge.merge_delta(base, Delta_S).

Gradients: the clamp is on the differentiable path (the paper: a plain STE
leaks gradient above the ceiling), so the gradient reaching eff' is dS where
the clamp did not bind and 0 where it did (at equality it passes, as a min
does).  Then, by the chain rule through Delta_S = c B A with c = alpha/r:
    dB = c (dS * m) A^T        [O, r]
    dA = c B^T (dS * m)        [r, G]
dS is the gradient with respect to the effective scale (linear.backward_dscale).

Reading (the paper gives no summation order): Delta_S adds the r rank-one
terms B[o, k] A[k, g] for k = 0 .. r-1 in fp32, rounding after each addition,
then multiplies once by fp32(alpha/r).  With bf16 factors every product is
exact in fp32, so this fixes Delta_S bit for bit.
"""

import numpy as np

from . import codec, merge


def _bf16_values(x) -> np.ndarray:
    """Values of bf16 factors as fp32 (torch tensors or arrays already holding them)."""
    if hasattr(x, "float"):
        x = x.float().cpu().numpy()
    return np.asarray(x, dtype=np.float32)


def delta_s(B, A, alpha_over_r: float) -> np.ndarray:
    """Delta_S [O, G] in fp32: sum over k in increasing order, then times alpha/r."""
    b = _bf16_values(B)
    a = _bf16_values(A)
    if b.ndim != 2 or a.ndim != 2 or b.shape[1] != a.shape[0]:
        raise ValueError("B must be [O, r] and A [r, G]")
    acc = np.zeros((b.shape[0], a.shape[1]), dtype=np.float32)
    for k in range(b.shape[1]):
        acc = acc + b[:, k:k + 1] * a[k:k + 1, :]          # product exact, one rounding per add
    return acc * np.float32(alpha_over_r)


def clamp_mask(fmt: str, base_bytes: np.ndarray, dS_: np.ndarray, ws2: float = 1.0) -> np.ndarray:
    """1 where the gradient passes the NVFP4 ceiling clamp (eff' <= 448 ws2), else 0.

    MXFP4 has no ceiling clamp on its path: every entry passes.  NaN eff'
    compares false against the ceiling and passes, like the min keeps it."""
    b = np.asarray(base_bytes, dtype=np.uint8)
    if fmt == codec.MX:
        return np.ones(b.shape, dtype=np.uint8)
    w = np.float32(ws2)
    e = codec.E4M3_TABLE[b].astype(np.float32) * w
    e2 = e + np.asarray(dS_, dtype=np.float32)
    cap = np.float32(codec.E4M3_MAX) * w
    return np.where(e2 > cap, 0, 1).astype(np.uint8)


def qast_scales(fmt: str, base_bytes: np.ndarray, B, A, alpha_over_r: float, ws2: float = 1.0):
    """On-grid scale bytes the QAST forward uses, and the clamp mask for the backward."""
    d = delta_s(B, A, alpha_over_r)
    return merge.merge_delta(fmt, base_bytes, d, ws2), clamp_mask(fmt, base_bytes, d, ws2)


def factor_grads(dS: np.ndarray, mask: np.ndarray, B, A, alpha_over_r: float):
    """dB [O, r] and dA [r, G] in fp64 from the scale gradient dS [O, G]."""
    g = np.asarray(dS, dtype=np.float64) * np.asarray(mask, dtype=np.float64)
    b = _bf16_values(B).astype(np.float64)
    a = _bf16_values(A).astype(np.float64)
    c = float(np.float32(alpha_over_r))
    return c * (g @ a.T), c * (b.T @ g)
