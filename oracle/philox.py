"""Philox4x64-10 counter-based generator (test infrastructure only).

Written from its published definition (Salmon, Moraes, Dror, Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC 2011): a 4 x 64-bit counter and a
2 x 64-bit key; ten rounds, each taking the two 128-bit products of the
multipliers with counter words 0 and 2 and recombining their halves with the
other words and the key; the key is bumped by two Weyl constants between
rounds.  The stochastic re-quantisation rule draws its uniforms from it, so
that the GPU path and this oracle see the same random numbers.
"""

import numpy as np

M0 = 0xD2E7470EE14C6C93
M1 = 0xCA5A826395121157
W0 = 0x9E3779B97F4A7C15          # golden ratio
W1 = 0xBB67AE8584CAA73B          # sqrt(3) - 1
_MASK32 = np.uint64(0xFFFFFFFF)


def _mulhilo(a: np.ndarray, m: int):
    """(high, low) 64-bit halves of the 128-bit products a * m, elementwise (uint64)."""
    a = np.asarray(a, dtype=np.uint64)
    m0, m1 = np.uint64(m & 0xFFFFFFFF), np.uint64(m >> 32)
    a0, a1 = a & _MASK32, a >> np.uint64(32)
    p00, p01, p10, p11 = a0 * m0, a0 * m1, a1 * m0, a1 * m1      # each < 2^64
    mid = (p00 >> np.uint64(32)) + (p01 & _MASK32) + (p10 & _MASK32)
    hi = p11 + (p01 >> np.uint64(32)) + (p10 >> np.uint64(32)) + (mid >> np.uint64(32))
    lo = (mid << np.uint64(32)) | (p00 & _MASK32)
    return hi, lo


def philox4x64_10(c0, c1, c2, c3, k0: int, k1: int):
    """The four output words for counters (c0, c1, c2, c3) (arrays of uint64) and key (k0, k1)."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint64) for c in (c0, c1, c2, c3))
    k0 = np.uint64(k0 & 0xFFFFFFFFFFFFFFFF)
    k1 = np.uint64(k1 & 0xFFFFFFFFFFFFFFFF)
    with np.errstate(over="ignore"):
        for r in range(10):
            if r:
                k0 = k0 + np.uint64(W0)
                k1 = k1 + np.uint64(W1)
            hi0, lo0 = _mulhilo(c0, M0)
            hi1, lo1 = _mulhilo(c2, M1)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return c0, c1, c2, c3


def uniforms24(n: int, seed: int, start: int = 0) -> np.ndarray:
    """u_e for e = start .. start+n-1: counter (e // 4, 0, 0, 0), key (seed, 0),
    output word e % 4, its top 24 bits times 2^-24 (exact in fp32; u in [0, 1))."""
    e = np.arange(start, start + n, dtype=np.uint64)
    z = np.zeros_like(e)
    words = philox4x64_10(e >> np.uint64(2), z, z, z, seed, 0)
    w = np.choose((e & np.uint64(3)).astype(np.int64), words)
    return ((w >> np.uint64(40)).astype(np.float64) * 2.0 ** -24).astype(np.float32)
