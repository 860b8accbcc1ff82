"""Oracle for the scale-plane merge and swap (test infrastructure only).

Paper §3, "QAST makes merge exact by construction": training rounds the adapted
effective scale onto the deployment grid in every forward pass, with
round_grid(s) = e4m3(s / ws2) * ws2 for NVFP4 and 2**round(log2 s) for MXFP4,
so the merge writes exactly that on-grid scale byte and copies the codes.
Stability recipe items (ii)-(iii): NVFP4 clamps the scale at 448 * ws2 in the
forward and the merge must reuse the identical grid-and-clamp path, or
ceiling-hitting scales turn into NaN.  App. B.2 ("Payoff 2"): a hot swap
overwrites the scale bytes and leaves the codes untouched.

The merge reads and writes scale bytes only; nothing here takes a code plane.
Each step below is one correctly rounded fp32 operation (numpy float32).
"""

import numpy as np

from . import codec


def merge_delta(fmt: str, scale_bytes: np.ndarray, delta: np.ndarray, ws2: float = 1.0) -> np.ndarray:
    """New scale bytes for eff' = eff + delta rounded onto the grid.

    NVFP4:  e  = f32(dec_e4m3(b) * ws2)
            e2 = f32(e + delta)
            e2 = min(e2, f32(448 * ws2))          (clamp; NaN propagates)
            q  = f32(e2 / ws2)
            b' = e4m3 nearest-even, saturating
    MXFP4:  e2 = f32(2**(b-127) + delta)
            b' = e8m0 of 2**round(log2 e2)
    """
    b = np.asarray(scale_bytes, dtype=np.uint8)
    d = np.asarray(delta, dtype=np.float32)
    if b.shape != d.shape:
        raise ValueError("delta must match the scale plane")
    if fmt == codec.NV:
        w = np.float32(ws2)
        dec = codec.E4M3_TABLE[b].astype(np.float32)              # exact
        e = dec * w
        e2 = e + d
        cap = np.float32(codec.E4M3_MAX) * w
        e2 = np.where(e2 > cap, cap, e2)                           # NaN compares false: kept
        q = e2 / w
        return codec.e4m3_encode(q)
    if fmt == codec.MX:
        dec = codec.E8M0_TABLE[b].astype(np.float32)              # exact, incl. 2**-127
        e2 = dec + d
        return codec.e8m0_encode_log(e2)
    raise ValueError(fmt)


def merge_copy(scale_bytes: np.ndarray, src: np.ndarray) -> np.ndarray:
    """Swap: the scale plane becomes src, byte for byte."""
    src = np.asarray(src, dtype=np.uint8)
    if np.asarray(scale_bytes).shape != src.shape:
        raise ValueError("src must match the scale plane")
    return src.copy()

