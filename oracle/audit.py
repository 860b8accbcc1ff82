"""Oracle for merge rollback and the byte audit (test infrastructure only).

Appendix B, "Payoff 3: invertible merges and rollback": a scale merge is
undone by subtracting the on-grid scale delta the merge applied (not the raw
training delta, which leaves some bytes off), and the base comes back byte for
byte with no retained base checkpoint.  "Payoff 5: verifiability": with codes
frozen, a merged artifact differs from its base only in the scale plane, so a
byte comparison audits it.

The applied delta is taken in the value domain of the stored field: for NVFP4
the E4M3 value e4m3(b') - e4m3(b) (the per-tensor ws2 is the same on both
sides and stays out of it), for MXFP4 the effective scale 2^(b'-127) -
2^(b-127).  Both differences are exact in fp32 whenever the two values are
within 24 binades (E4M3 values carry 4 significant bits and span 2^-9 .. 448;
powers of two need one bit each), so rollback re-encodes the exact base value.
"""

import numpy as np

from . import codec


def _values(fmt: str, b: np.ndarray) -> np.ndarray:
    b = np.asarray(b, dtype=np.uint8)
    if fmt == codec.NV:
        return codec.E4M3_TABLE[b]
    if fmt == codec.MX:
        return codec.E8M0_TABLE[b]
    raise ValueError(fmt)


def applied_delta(fmt: str, before: np.ndarray, after: np.ndarray) -> np.ndarray:
    """fp32 on-grid delta value(after) - value(before), one fp32 subtraction (both
    values are fp32-representable; NaN where either byte is NaN)."""
    return _values(fmt, after).astype(np.float32) - _values(fmt, before).astype(np.float32)


def rollback(fmt: str, merged: np.ndarray, applied: np.ndarray) -> np.ndarray:
    """Bytes of value(merged) - applied, re-encoded on the grid (one fp32 subtraction)."""
    v = _values(fmt, merged).astype(np.float32) - np.asarray(applied, dtype=np.float32)
    if fmt == codec.NV:
        return codec.e4m3_encode(v)
    return codec.e8m0_encode_log(v)


def diff_counts(a: np.ndarray, b: np.ndarray):
    """(differing bytes, differing 4-bit nibbles) between two byte planes."""
    a = np.asarray(a, dtype=np.uint8).reshape(-1)
    b = np.asarray(b, dtype=np.uint8).reshape(-1)
    x = a ^ b
    return int(np.count_nonzero(x)), int(np.count_nonzero(x & 0x0F) + np.count_nonzero(x & 0xF0))
