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


def e4m3_values():
    """Every positive finite E4M3 ("fn") value."""
    vals = [m / 8 * 2.0 ** -6 for m in range(1, 8)]
    vals += [(1 + m / 8) * 2.0 ** e for e in range(-6, 9) for m in range(8)]
    return np.array([v for v in vals if v <= 448.0])


def bf16(x):
    """Round fp32 values to bf16 (nearest even), as float32."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32)


def element_quotient(w, d):
    """The NVFP4 re-quantiser's per-weight quotient for a block whose scale d
    is nonzero and whose |w| / d stays below 2^100: the two corrected
    products of div_seq, with the sign of w copied onto the result."""
    return np.float32(np.copysign(div_seq(w, d), np.float32(w)))


def test_rtn_element_quotient_is_the_rounded_quotient():
    """fp32(w / eff) for bf16 weights w (zeros, subnormal and normal bf16,
    values next to every E2M1 decision point) and block scales
    eff = fp32(e4m3 * ws2): equal bit for bit, signed zeros included, where
    the quotient is at or above 2^-26; below, both are smaller than 0.25 with
    the sign of w, so the E2M1 code (a signed zero) is the same."""
    g = np.random.default_rng(11)
    e4 = e4m3_values()
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    vals = np.concatenate([mids, [0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]])
    checked = 0
    for ws2 in (np.float32(1 / 448), np.float32(3.0517578e-05), np.float32(0.0123), np.float32(2.0 ** -55),
                np.float32(2.0 ** 55)):
        for s in g.choice(e4, 24, replace=False):
            eff = np.float32(np.float32(s) * ws2)
            ws = [np.float32(0.0), np.float32(-0.0), np.float32(2.0 ** -133), -np.float32(2.0 ** -130)]
            for v in g.choice(vals, 6, replace=False):
                for k in range(-3, 4):
                    ws.append(bf16(np.float32(v * float(eff) * (1 + k * 2.0 ** -8))))
                    ws.append(-bf16(np.float32(v * float(eff) * (1 + k * 2.0 ** -9))))
            for w in ws:
                w = np.float32(w)
                if not np.isfinite(w) or abs(float(w)) > 2.0 ** 100 * float(eff):
                    continue
                got = element_quotient(w, eff)
                ref = rn32(Fraction(float(w)) / Fraction(float(eff)))
                ref = np.float32(np.copysign(ref, w)) if ref == 0 else np.float32(ref)
                if abs(float(ref)) >= 2.0 ** -26:
                    assert got.view(np.uint32) == ref.view(np.uint32), (ws2, eff, w, got, ref)
                else:
                    assert abs(float(got)) < 0.25 and np.signbit(got) == np.signbit(w), (eff, w, got)
                checked += 1
    assert checked > 3000


def hard_quotients(n, seed, within=2.0 ** -21):
    """bf16 weights w and fp32 block scales d whose quotient w / d lies within
    `within` ulp of a midpoint between two fp32 values (where a quotient off
    by a fraction of an ulp rounds the wrong way), found among n random
    pairs in float64 (53 bits resolve the distance to 2^-29 ulp)."""
    g = np.random.default_rng(seed)
    out = []
    for _ in range(n // 4_000_000):
        m = 4_000_000
        w = (128 + g.integers(0, 128, m)).astype(np.float64) * 2.0 ** (g.integers(-8, 8, m) - 7)
        d = g.uniform(1.0, 2.0, m).astype(np.float32).astype(np.float64) * 2.0 ** g.integers(-10, 10, m)
        x = w / d
        e = np.floor(np.log2(x))
        t = x / 2.0 ** (e - 23)
        dist = np.abs(t - np.floor(t) - 0.5)
        for i in np.nonzero(dist < within)[0]:
            out.append((np.float32(w[i]) * (1 if g.integers(0, 2) else -1), np.float32(d[i])))
    return out


def test_rtn_element_quotient_hard_cases():
    """Quotients within 2^-21 ulp of an fp32 rounding midpoint, the cases a
    quotient that is merely faithful can round the wrong way: the element
    form still gives fp32(w / d) bit for bit."""
    cases = hard_quotients(16_000_000, 13)
    assert len(cases) >= 6
    naive_wrong = 0
    for w, d in cases:
        ref = np.float32(rn32(Fraction(float(w)) / Fraction(float(d))))
        assert element_quotient(w, d).view(np.uint32) == ref.view(np.uint32), (w, d)
        naive_wrong += np.float32(np.float32(w) * np.float32(np.float32(1.0) / d)) != ref
    # the cases are hard: the plain product with the reciprocal misrounds some
    assert naive_wrong >= 2


def product_window_flag(q0):
    """The NVFP4 re-quantiser's test on a block's product quotients: a bit
    pattern within 3 of a multiple of 2^21 (a value whose significand has at
    most two fraction bits)."""
    b = np.asarray(q0, np.float32).view(np.uint32).astype(np.uint64)
    return ((b + 3) % (1 << 21)) < 7


def test_rtn_product_quotient_window():
    """Where the product quotient q0 = fp32(w fp32(1/d)) lies more than 3 float
    steps from every value whose significand has at most two fraction bits,
    its E2M1 code under each rule (nearest even, nearest away, toward zero)
    is that of fp32(w / d).  Quotients are aimed at every rounding boundary
    and grid point of E2M1 (0.25 .. 6) from both sides, with bf16 weights of
    both signs and fp32 divisors over a wide exponent range; the window is
    needed (some codes of q0 differ from the exact quotient's) and catches
    every such case."""
    from oracle import rtn
    g = np.random.default_rng(29)
    targets = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    n = 2_000_000
    w = bf16((g.uniform(1.0, 2.0, n) * 2.0 ** g.integers(-30, 30, n)).astype(np.float32))
    w = np.where(g.integers(0, 2, n) == 1, -w, w).astype(np.float32)
    v = g.choice(targets, n) * (1.0 + g.integers(-12, 13, n) * 2.0 ** -24)
    d = (np.abs(w).astype(np.float64) / v).astype(np.float32)
    r = (np.float32(1.0) / d).astype(np.float32)
    q0 = (w * r).astype(np.float32)
    qx = (w / d).astype(np.float32)
    flag = product_window_flag(q0)
    differ = np.zeros(n, bool)
    for rule in ("even", "away", "rtz"):
        if rule == "rtz":
            c0, cx = rtn.e2m1_round_rule(q0, rule), rtn.e2m1_round_rule(qx, rule)
        else:
            c0, cx = rtn.e2m1_round_magnitude(q0, rule), rtn.e2m1_round_magnitude(qx, rule)
        differ |= c0 != cx
    assert np.array_equal(np.signbit(q0), np.signbit(qx))
    # the bound the window rests on: q0 within 3 float steps of fp32(w / d),
    # here and over unaimed pairs (any divisor significand, quotients across
    # many binades)
    steps = np.abs(q0.view(np.uint32).astype(np.int64) - qx.view(np.uint32).astype(np.int64))
    assert steps.max() <= 3
    w2 = bf16((g.uniform(1.0, 2.0, n) * 2.0 ** g.integers(-20, 20, n)).astype(np.float32))
    d2 = (g.uniform(1.0, 2.0, n) * 2.0 ** g.integers(-20, 20, n)).astype(np.float32)
    q2 = (w2 * (np.float32(1.0) / d2).astype(np.float32)).astype(np.float32)
    x2 = (w2 / d2).astype(np.float32)
    assert np.abs(q2.view(np.uint32).astype(np.int64) - x2.view(np.uint32).astype(np.int64)).max() <= 3
    assert differ.sum() > 100
    assert not np.any(differ & ~flag), np.nonzero(differ & ~flag)[0][:5]
    # on quotients spread evenly the window is rare
    u = (g.uniform(0.0, 8.0, n)).astype(np.float32)
    assert product_window_flag(u).mean() < 1e-5
