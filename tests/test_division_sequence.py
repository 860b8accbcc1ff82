"""The reciprocal division sequence the kernels use (q0 = fp32(x r) with
r = fp32(1/d), then two corrections q + fp32(x - d q) r, each a fused
multiply-add), emulated exactly on the CPU and compared with true division.
It must give fp32(a / 6) for every positive finite bf16 a >= 2^-120 (the
re-quantisers' block amax / 6) and fp32(x / ws2) for quotients at or above
2^-26 with ws2 in [2^-64, 2^64] (merge and re-quantiser ws2 steps)."""

from fractions import Fraction

import numpy as np


def rn32(x: Fraction) -> float:
    """Round a rational to the nearest fp32 (ties to even), subnormals included."""
    if x == 0:
        return 0.0
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    if Fraction(2) ** (e + 1) <= a:
        e += 1
    assert e <= 127, "past the fp32 range"
    e = max(e, -126)                      # subnormals share the smallest normal's ulp
    m = a / Fraction(2) ** (e - 23)
    f = m.numerator // m.denominator
    rem = m - f
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and f % 2 == 1):
        f += 1
    return sign * float(f * Fraction(2) ** (e - 23))


def fma(a, b, c):
    return rn32(Fraction(float(a)) * Fraction(float(b)) + Fraction(float(c)))


def div_seq(x, d):
    x, d = np.float32(x), np.float32(d)
    r = np.float32(1.0) / d
    q0 = np.float32(x * r)
    q1 = fma(fma(-q0, d, x), r, q0)
    return np.float32(fma(fma(-q1, d, x), r, q1))


def test_amax_over_six_all_bf16():
    bits = np.arange(0, 0x7F80, dtype=np.uint32) << 16
    vals = bits.view(np.float32)
    vals = vals[vals >= np.float32(2.0 ** -120)]
    assert vals.size == 31744
    six = np.float32(6.0)
    for a in vals:
        assert div_seq(a, six) == np.float32(a / six), a


def test_ws2_quotients_near_e4m3_midpoints():
    """Quotients within a few ulps of E4M3 values and of the midpoints between
    them (where a wrong last bit would change the encoded byte)."""
    g = np.random.default_rng(7)
    pos = []
    for e in range(-6, 9):
        for m in range(8):
            pos.append((1 + m / 8) * 2.0 ** e)
    pos += [m / 8 * 2.0 ** -6 for m in range(1, 8)]
    pos = np.unique(np.array(pos))
    targets = np.concatenate([pos, (pos[:-1] + pos[1:]) / 2])
    for ws2 in (np.float32(1 / 448), np.float32(0.0123), np.float32(2.0 ** -60), np.float32(5.5e17)):
        for t in g.choice(targets, 40, replace=False):
            for k in range(-4, 5):
                q = np.float32(t * (1 + k * 2.0 ** -23))
                x = np.float32(np.float64(q) * np.float64(ws2))
                assert div_seq(x, ws2) == np.float32(x / ws2), (ws2, x)
