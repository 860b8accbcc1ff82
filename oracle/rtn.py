"""Oracle for round-to-nearest re-quantisation of a bf16 weight (test infrastructure only).

This is the naive merge the paper argues against (§2, "The naive re-quantized
merge is the failure mode": W' = requant(dequant(W) + (alpha/r) BA)), kept as
the baseline that rewrites every code.

Scale selection:
* MXFP4: k = ceil(log2(amax/6)), the shipping rule the paper adopts as its RTN
  baseline (App. "Calibrated PTQ on a sparse MoE", first paragraph: ceil of
  log2(absmax/6) with the mantissa masked off).  Exponents clamp to [-127, 127];
  an all-zero block takes k = -127.
* NVFP4: the amax/6 nearest-rounding rule (App. "Why the naive merge returns the
  base", premise (iii)): byte = e4m3_nearest(amax/6/ws2).  ws2 is held at the
  given value, or recomputed from the tensor as fp32(fp32(amax/6)/448) (the
  per-tensor-scalar conventions of App. B threat model (a)); an all-zero
  tensor recomputes to ws2 = 1.

Codes: q = w / eff_scale, magnitude rounded to the nearest E2M1 value with the
chosen tie rule (ties to the even mantissa, or half away from zero, App. B
threat model (a): tools differ in tie-breaking), saturating at 6; the sign bit
is the sign of w, also when the magnitude rounds to 0.  A NaN q codes as
magnitude 0.

Deploy-rule variants (App. "Deployment-quantizer sweep" / threat model: rules
a serving-side quantiser may apply to a continuous merged tensor), in
quantize_rule: round toward zero (the largest E2M1 magnitude not above |q|),
stochastic rounding (|q| goes up to the next magnitude with probability equal
to its fractional position between the two neighbours, drawn from Philox4x64-10
with the uniform of element e = o*I + i taken as described in philox.py), and
whole-tensor scaling (one scale for the whole tensor from the tensor amax, by
the same scale rule, with nearest-even codes).  On-grid values are fixed points
of truncation and of stochastic rounding, as they are of nearest rounding.
"""

import numpy as np

from . import codec, philox

TIE_EVEN = "even"
TIE_AWAY = "away"
RULE_RTZ = "rtz"
RULE_STOCHASTIC = "stochastic"
RULE_WHOLE_TENSOR = "whole_tensor"
_GRID = codec.E2M1_TABLE[:8]          # 0, .5, 1, 1.5, 2, 3, 4, 6 (magnitude index order)


def e2m1_round_magnitude(q: np.ndarray, tie: str) -> np.ndarray:
    """|q| (fp32) -> E2M1 magnitude index 0..7, nearest with the given tie rule."""
    a = np.abs(np.asarray(q, dtype=np.float32).astype(np.float64))
    nan = np.isnan(a)
    a = np.where(nan, 0.0, np.minimum(a, 6.0))
    hi = np.minimum(np.searchsorted(_GRID, a, side="right"), 7)
    lo = np.maximum(hi - 1, 0)
    d_lo = a - _GRID[lo]
    d_hi = _GRID[hi] - a
    if tie == TIE_EVEN:
        tie_pick = np.where(lo % 2 == 0, lo, hi)
    elif tie == TIE_AWAY:
        tie_pick = hi
    else:
        raise ValueError(tie)
    idx = np.where(d_lo < d_hi, lo, np.where(d_hi < d_lo, hi, tie_pick))
    idx = np.where(a >= 6.0, 7, idx)
    return np.where(nan, 0, idx).astype(np.uint8)


def ceil_log2(x: np.ndarray) -> np.ndarray:
    """Exact ceil(log2 x) for positive finite fp32 x."""
    f, e = np.frexp(np.asarray(x, dtype=np.float32).astype(np.float64))   # x = f * 2**e
    return np.where(f == 0.5, e - 1, e)


def recompute_ws2(W: np.ndarray) -> np.float32:
    amax = np.float32(np.max(np.abs(np.asarray(W, np.float32)))) if np.asarray(W).size else np.float32(0)
    ws2 = (amax / np.float32(6.0)) / np.float32(codec.E4M3_MAX)
    return np.float32(1.0) if ws2 == 0 else np.float32(ws2)


def quantize(fmt: str, W: np.ndarray, tie: str = TIE_EVEN, ws2=None):
    """W: [O, I] values exactly representable in bf16 (given as fp32/fp64).

    Returns (codes_packed [O, I/2] uint8, scale_bytes [O, G] uint8, ws2 fp32)."""
    W = np.asarray(W, dtype=np.float32)
    O, I = W.shape
    block = codec.BLOCK[fmt]
    G = I // block
    Wb = W.reshape(O, G, block)
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        amax = np.max(np.abs(Wb), axis=2)                              # exact
        if fmt == codec.MX:
            x = amax / np.float32(6.0)
            pos = np.isfinite(x) & (x > 0)
            k = np.where(pos, ceil_log2(np.where(pos, x, 1.0)), -127)
            k = np.where(np.isposinf(x), 127, k)
            k = np.clip(k, -127, 127)
            sbytes = np.where(np.isnan(x), 0xFF, k + 127).astype(np.uint8)
            eff = codec.E8M0_TABLE[sbytes]                              # fp64, exact power of two
            q = (Wb.astype(np.float64) / eff[:, :, None]).astype(np.float32)   # exact
            out_ws2 = np.float32(1.0)
        elif fmt == codec.NV:
            out_ws2 = recompute_ws2(W) if ws2 is None else np.float32(ws2)
            x = (amax / np.float32(6.0)) / out_ws2
            sbytes = codec.e4m3_encode(x)
            se = codec.E4M3_TABLE[sbytes].astype(np.float32) * out_ws2  # fp32 product
            q = np.where(se[:, :, None] == 0, np.float32(0.0), Wb / se[:, :, None])
        else:
            raise ValueError(fmt)
    mag = e2m1_round_magnitude(q, tie)
    sign = np.signbit(Wb).astype(np.uint8) << 3
    nib = (mag | sign).reshape(O, I)
    return codec.pack_nibbles(nib), sbytes.reshape(O, G), np.float32(out_ws2)


def e2m1_round_rule(q: np.ndarray, rule: str, u: np.ndarray = None) -> np.ndarray:
    """|q| (fp32) -> E2M1 magnitude index 0..7 under RTZ or stochastic rounding
    (u: fp32 uniforms in [0, 1) of q's shape).  Saturates at 6; NaN -> 0."""
    a = np.abs(np.asarray(q, dtype=np.float32).astype(np.float64))
    nan = np.isnan(a)
    a = np.where(nan, 0.0, np.minimum(a, 6.0))
    lo = np.searchsorted(_GRID, a, side="right") - 1            # largest magnitude <= a
    if rule == RULE_RTZ:
        idx = lo
    elif rule == RULE_STOCHASTIC:
        hi = np.minimum(lo + 1, 7)
        gap = _GRID[hi] - _GRID[lo]
        frac = np.where(gap > 0, (a - _GRID[lo]) / np.where(gap > 0, gap, 1.0), 0.0)   # exact
        idx = np.where(np.asarray(u, dtype=np.float64) < frac, hi, lo)
    else:
        raise ValueError(rule)
    return np.where(nan, 0, idx).astype(np.uint8)


def quantize_rule(fmt: str, W: np.ndarray, rule: str, ws2=None, seed: int = 0, row0: int = 0):
    """quantize() under a deploy rule: "even" / "away" (nearest, per-block scales),
    "rtz", "stochastic" (per-block scales, other code rounding) or "whole_tensor"
    (one scale for the tensor, nearest-even codes).  Same returns as quantize().
    row0: W holds rows row0 .. of a larger tensor of the same width, so the
    stochastic rule's element index starts at row0 * I."""
    if rule in (TIE_EVEN, TIE_AWAY):
        return quantize(fmt, W, rule, ws2)
    W = np.asarray(W, dtype=np.float32)
    O, I = W.shape
    block = codec.BLOCK[fmt]
    G = I // block
    if rule == RULE_WHOLE_TENSOR:
        amax_t = np.float32(np.max(np.abs(W))) if W.size else np.float32(0)
        tiled = np.zeros((O, G, block), np.float32)
        tiled[:, :, 0] = amax_t                                   # every block sees the tensor amax
        _, sbytes, out_ws2 = quantize(fmt, tiled.reshape(O, I), TIE_EVEN,
                                      ws2 if ws2 is not None else (recompute_ws2(W) if fmt == codec.NV else None))
        eff = codec.effective_scales(fmt, sbytes, out_ws2).astype(np.float32)
        Wb = W.reshape(O, G, block)
        with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
            if fmt == codec.MX:
                q = (Wb.astype(np.float64) / eff[:, :, None].astype(np.float64)).astype(np.float32)
            else:
                q = np.where(eff[:, :, None] == 0, np.float32(0.0), Wb / eff[:, :, None])
        mag = e2m1_round_magnitude(q, TIE_EVEN)
    else:
        codes, sbytes, out_ws2 = quantize(fmt, W, TIE_EVEN, ws2)
        eff = codec.effective_scales(fmt, sbytes, out_ws2).astype(np.float32)
        Wb = W.reshape(O, G, block)
        with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
            if fmt == codec.MX:
                q = (Wb.astype(np.float64) / eff[:, :, None].astype(np.float64)).astype(np.float32)
            else:
                q = np.where(eff[:, :, None] == 0, np.float32(0.0), Wb / eff[:, :, None])
        u = philox.uniforms24(O * I, seed, row0 * I).reshape(O, G, block) if rule == RULE_STOCHASTIC else None
        mag = e2m1_round_rule(q, rule, u)
    sign = np.signbit(W.reshape(O, G, block)).astype(np.uint8) << 3
    nib = (mag | sign).reshape(O, I)
    return codec.pack_nibbles(nib), sbytes.reshape(O, G), np.float32(out_ws2)
