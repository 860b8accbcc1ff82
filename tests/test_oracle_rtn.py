"""Pins for the oracle's round-to-nearest re-quantisation (CPU only).

Pinned against: the paper's worked two-element block (midpoint distances and the
optimal competitor over power-of-two scales), brute-force nearest-on-grid search,
the ceil-log2 scale rule restated as "smallest k with 6*2**k >= amax", and the
Delta=0 control (re-quantising an on-grid weight moves no block and no code)."""

import numpy as np
import pytest

from conftest import read_golden
from oracle import codec, linear, rtn
from paper_2609_04526_amd import inputs


def test_tie_rules_at_midpoints():
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0], np.float32)
    grid = codec.E2M1_TABLE[:8]
    even = grid[rtn.e2m1_round_magnitude(mids, rtn.TIE_EVEN)]
    away = grid[rtn.e2m1_round_magnitude(mids, rtn.TIE_AWAY)]
    assert even.tolist() == [0, 1, 1, 2, 2, 4, 4]
    assert away.tolist() == [0.5, 1, 1.5, 2, 3, 4, 6]


def test_worked_voronoi_block():
    rows, _ = read_golden("voronoi_block.txt")
    W = np.array(rows["codes"])
    D = np.array(rows["delta"])
    grid = codec.E2M1_TABLE[:8]
    mids = (grid[:-1] + grid[1:]) / 2
    dist = [min(abs(w - m) for m in mids) for w in W]
    assert np.allclose(dist, rows["midpoint_distance"])
    T = (W + D).astype(np.float32)
    base_cost = float(np.sum((T - W) ** 2))
    assert round(base_cost, 5) == rows["base_cost"][0]
    # at a fixed scale the cost-minimising codes are the coordinatewise rounding of T/s
    best = None
    for k in range(-6, 7):
        s = 2.0 ** k
        idx = rtn.e2m1_round_magnitude((T / s).astype(np.float32), rtn.TIE_EVEN)
        Q = grid[idx] * np.sign(T) * s
        if np.array_equal(Q, W):
            continue                      # the base itself is excluded from the competitor set
        cost = float(np.sum((T - Q) ** 2))
        if best is None or cost < best[0]:
            best = (cost, s, grid[idx])
    assert round(best[0], 5) == rows["best_cost"][0]
    assert best[1] == rows["best_scale"][0]
    assert best[2].tolist() == rows["best_codes"]


@pytest.mark.parametrize("tie", [rtn.TIE_EVEN, rtn.TIE_AWAY])
def test_e2m1_rounding_matches_brute_force(tie):
    g = np.random.default_rng(9)
    q = np.concatenate([g.uniform(0, 8, 5000), np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])]).astype(np.float32)
    out = rtn.e2m1_round_magnitude(q, tie)
    grid = codec.E2M1_TABLE[:8]
    for n, v in enumerate(q.astype(np.float64)):
        d = np.abs(grid - min(v, 6.0))
        c = np.flatnonzero(d == d.min())
        if len(c) == 1:
            ref = c[0]
        else:
            ref = c[1] if tie == rtn.TIE_AWAY else [x for x in c if x % 2 == 0][0]
        assert out[n] == ref


def test_mx_scale_rule_is_smallest_covering_exponent():
    g = np.random.default_rng(10)
    W = (g.standard_normal((8, 64)) * np.exp2(g.integers(-12, 4, size=(8, 1)))).astype(np.float32)
    W = W.astype(np.float32)
    codes, sb, _ = rtn.quantize("mx", W)
    amax = np.abs(W.reshape(8, 2, 32)).max(axis=2).astype(np.float64)
    for o in range(8):
        for b in range(2):
            x = float(np.float32(np.float32(amax[o, b]) / np.float32(6)))
            k = next(k for k in range(-127, 128) if 2.0 ** k >= x)
            assert sb[o, b] == k + 127
    # every rescaled weight then fits the E2M1 range
    q = W.reshape(8, 2, 32) / np.ldexp(1.0, sb.astype(int) - 127)[:, :, None]
    assert np.abs(q).max() <= 6.0


def test_mx_delta_zero_is_fixed_point():
    """An on-grid MX weight whose every block holds a +-6 code re-quantises to itself."""
    O, I = 16, 128
    codes = inputs.codes_uniform(1101, O, I)
    nib = codec.unpack_nibbles(codes)
    nib[:, ::32] = 7                       # +6 in every block
    codes = codec.pack_nibbles(nib)
    sb = inputs.e8m0_uniform_exponents(1102, O, I // 32, -8, -3)
    W = linear.dequant("mx", codes, sb).astype(np.float32)
    for tie in (rtn.TIE_EVEN, rtn.TIE_AWAY):
        c2, s2, _ = rtn.quantize("mx", W, tie)
        assert np.array_equal(s2, sb)
        assert np.array_equal(c2, codes)


def test_nv_delta_zero_is_fixed_point_with_power_of_two_ws2():
    O, I = 16, 64
    codes = inputs.codes_uniform(1103, O, I)
    nib = codec.unpack_nibbles(codes)
    nib[:, ::16] = 15                      # -6 in every block
    codes = codec.pack_nibbles(nib)
    sb = inputs.e4m3_abs_normal(1104, O, I // 16)
    sb[sb == 0] = 0x38                     # no zero scales (a zero block has no fixed point)
    ws2 = np.float32(2.0 ** -9)
    W = linear.dequant("nv", codes, sb, float(ws2)).astype(np.float32)
    c2, s2, w2 = rtn.quantize("nv", W, rtn.TIE_EVEN, ws2)
    assert w2 == ws2
    assert np.array_equal(s2, sb)
    assert np.array_equal(c2, codes)


def test_nv_recomputed_ws2_and_scale_rule():
    g = np.random.default_rng(12)
    W = g.standard_normal((8, 64)).astype(np.float32)
    codes, sb, ws2 = rtn.quantize("nv", W)
    amax = np.float32(np.abs(W).max())
    assert ws2 == np.float32(np.float32(amax / np.float32(6)) / np.float32(448))
    # the largest block hits the E4M3 ceiling exactly
    assert sb.max() == 0x7E
    blk = np.abs(W.reshape(8, 4, 16)).max(axis=2)
    for o in range(8):
        for b in range(4):
            x = np.float32(np.float32(blk[o, b] / np.float32(6)) / ws2)
            cand = [(abs(float(x) - codec.e4m3_value(c)), c) for c in range(0x7F)]
            m = min(cand)[0]
            ok = [c for d, c in cand if d == m]
            assert sb[o, b] in ok


def test_sign_bit_kept_on_zero_codes():
    W = np.zeros((1, 32), np.float32)
    W[0, 1] = -0.0
    W[0, 2] = -1e-6
    W[0, 3] = 6.0
    codes, _, _ = rtn.quantize("mx", W)
    nib = codec.unpack_nibbles(codes)[0]
    assert nib[1] == 8 and nib[2] == 8 and nib[0] == 0 and nib[3] == 7
