"""Oracle codecs for the native FP4 microscaling formats (test infrastructure only).

Paper §2, "Native FP4 microscaling storage":
* a weight is W[o,i] = code[o,i] * eff_scale[o, i // block];
* code is a 4-bit E2M1 value in +-{0, 0.5, 1, 1.5, 2, 3, 4, 6};
* NVFP4 (block 16): eff_scale = E4M3 byte value (max 448) * fp32 per-tensor ws2;
* MXFP4 (block 32): eff_scale = E8M0 byte, a power of two with no mantissa.

Bit-level readings where the paper gives values but not layouts (listed as
readings in the design notes): E2M1 is sign | 2 exponent bits (bias 1) | 1
mantissa bit; E8M0 is 2**(byte-127) with 0xFF = NaN; E4M3 is sign | 4
exponent bits (bias 7, with subnormals) | 3 mantissa bits, 0x7F/0xFF = NaN,
no infinities (the "fn" variant whose maximum is the 448 the paper states).
"""

import math

import numpy as np

MX = "mx"
NV = "nv"
BLOCK = {MX: 32, NV: 16}
E4M3_MAX = 448.0


# ---------------------------------------------------------------- E2M1 codes
def e2m1_value(nibble: int) -> float:
    """Value of a 4-bit E2M1 code from its bit fields."""
    sign = (nibble >> 3) & 1
    exp = (nibble >> 1) & 3
    man = nibble & 1
    if exp == 0:                       # subnormal: 0 or 0.5
        mag = man * 0.5
    else:                              # normal: 2^(exp-1) * (1 + man/2)
        mag = 2.0 ** (exp - 1) * (1.0 + man / 2.0)
    return -mag if sign else mag


E2M1_TABLE = np.array([e2m1_value(n) for n in range(16)], dtype=np.float64)


def unpack_nibbles(packed: np.ndarray) -> np.ndarray:
    """[R, C/2] uint8 -> [R, C] code indices.  Low nibble holds the even column."""
    packed = np.asarray(packed, dtype=np.uint8)
    out = np.empty(packed.shape[:-1] + (packed.shape[-1] * 2,), dtype=np.uint8)
    out[..., 0::2] = packed & 0x0F
    out[..., 1::2] = packed >> 4
    return out


def pack_nibbles(nibbles: np.ndarray) -> np.ndarray:
    """[R, C] code indices (0..15) -> [R, C/2] uint8, low nibble = even column."""
    nibbles = np.asarray(nibbles, dtype=np.uint8)
    return (nibbles[..., 0::2] & 0x0F) | ((nibbles[..., 1::2] & 0x0F) << 4)


# ---------------------------------------------------------------- E8M0 scales
def e8m0_value(byte: int) -> float:
    """2**(byte-127); 0xFF is NaN."""
    if byte == 0xFF:
        return math.nan
    return math.ldexp(1.0, byte - 127)


E8M0_TABLE = np.array([e8m0_value(b) for b in range(256)], dtype=np.float64)


# ---------------------------------------------------------------- E4M3 scales
def e4m3_value(byte: int) -> float:
    sign = (byte >> 7) & 1
    exp = (byte >> 3) & 0xF
    man = byte & 7
    if exp == 0xF and man == 7:
        return math.nan
    if exp == 0:
        mag = man / 8.0 * 2.0 ** -6
    else:
        mag = (1.0 + man / 8.0) * 2.0 ** (exp - 7)
    return -mag if sign else mag


E4M3_TABLE = np.array([e4m3_value(b) for b in range(256)], dtype=np.float64)
# bytes 0x00..0x7E are the non-negative finite values in increasing order
_E4M3_POS = E4M3_TABLE[:0x7F].copy()


def e4m3_encode(x) -> np.ndarray:
    """Round fp32 values to the nearest E4M3 value, ties to the even mantissa,
    saturating at +-448 (the paper's clamp keeps merged scales finite; a
    non-saturating cast would turn them into NaN).  NaN encodes as 0x7F.

    Exact: every candidate grid value and every fp32 input is exact in fp64,
    and so are the two distances compared."""
    v = np.asarray(x, dtype=np.float32).astype(np.float64)
    a = np.abs(v)
    nan = np.isnan(v)
    a_safe = np.where(nan, 0.0, np.minimum(a, E4M3_MAX))
    hi = np.searchsorted(_E4M3_POS, a_safe, side="right")      # first grid value > a
    hi = np.minimum(hi, len(_E4M3_POS) - 1)
    lo = np.maximum(hi - 1, 0)                                   # grid value <= a
    d_lo = a_safe - _E4M3_POS[lo]
    d_hi = _E4M3_POS[hi] - a_safe
    tie_pick = np.where(lo % 2 == 0, lo, hi)                     # tie: even mantissa
    code = np.where(d_lo < d_hi, lo, np.where(d_hi < d_lo, hi, tie_pick))
    code = np.where(a_safe >= E4M3_MAX, 0x7E, code)              # saturate
    sign = np.where(np.signbit(v), 0x80, 0)
    out = np.where(nan, 0x7F, code | sign)
    return out.astype(np.uint8)


def e8m0_encode_log(x) -> np.ndarray:
    """round_grid for MXFP4: 2**round(log2 s), nearest in the log domain.

    For s = m * 2**k with m in [1, 2) the rounded exponent is k+1 iff
    log2 m > 1/2, i.e. iff m*m > 2.  m has at most 24 significant bits, so
    m*m is exact in fp64 and a tie (m = sqrt 2) cannot occur.  Exponents are
    clamped to the representable [-127, 127].  Readings: s <= 0 encodes as
    0x00 (the smallest scale), +inf as 0xFE, NaN as 0xFF."""
    v = np.asarray(x, dtype=np.float32).astype(np.float64)
    pos = np.isfinite(v) & (v > 0)
    f, e = np.frexp(np.where(pos, v, 1.0))                     # v = f * 2**e, f in [0.5, 1)
    m = 2.0 * f                                                  # v = m * 2**(e-1), m in [1, 2)
    k = (e - 1) + (m * m > 2.0)
    k = np.clip(k, -127, 127)
    out = np.where(pos, k + 127, 0)
    out = np.where(np.isposinf(v), 0xFE, out)
    out = np.where(np.isnan(v), 0xFF, out)
    return out.astype(np.uint8)


def effective_scales(fmt: str, scale_bytes: np.ndarray, ws2: float = 1.0) -> np.ndarray:
    """Per-block effective scale in fp64: E8M0 value (MX) or E4M3 value * ws2 (NV).
    The NV product of a <=4-significant-bit value and an fp32 is exact in fp64."""
    scale_bytes = np.asarray(scale_bytes, dtype=np.uint8)
    if fmt == MX:
        return E8M0_TABLE[scale_bytes]
    if fmt == NV:
        return E4M3_TABLE[scale_bytes] * float(np.float32(ws2))
    raise ValueError(fmt)
