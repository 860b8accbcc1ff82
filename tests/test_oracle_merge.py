"""Pins for the oracle's scale merge / swap (CPU only).

Pinned against: the paper's Delta=0 control (re-quantising an un-adapted plane moves
no block), the exact +-1 exponent step (2**a +- 2**b is exact in fp32), the NVFP4
ceiling clamp (without it the cast yields NaN, stability recipe item (iii)), exact
rollback with the applied on-grid delta (App. B "Payoff 3"), and brute-force
nearest-on-grid searches written independently of the encoders."""

import math

import numpy as np
import pytest
import torch

from oracle import codec, merge
from paper_2609_04526_amd import inputs

FINITE_MX = np.arange(0, 255, dtype=np.uint8)
FINITE_NV = np.array([b for b in range(0x7F)], dtype=np.uint8)


@pytest.mark.parametrize("ws2", [1.0 / 448.0, 2.0 ** -8, 0.3712, 1.0])
def test_delta_zero_is_identity_nv(ws2):
    out = merge.merge_delta("nv", FINITE_NV, np.zeros(FINITE_NV.shape, np.float32), ws2)
    assert np.array_equal(out, FINITE_NV)


def test_delta_zero_is_identity_mx():
    out = merge.merge_delta("mx", FINITE_MX, np.zeros(FINITE_MX.shape, np.float32))
    assert np.array_equal(out, FINITE_MX)


def test_mx_exponent_step_reproduced_exactly():
    sb = inputs.e8m0_uniform_exponents(1001, 256, 16, -8, -3)
    d = inputs.e8m0_step_delta(1009, sb, 0.10)
    out = merge.merge_delta("mx", sb, d)
    moved = d != 0
    assert moved.sum() == round(0.1 * sb.size)
    up = d > 0
    assert np.array_equal(out[moved & up], sb[moved & up] + 1)
    assert np.array_equal(out[moved & ~up], sb[moved & ~up] - 1)
    assert np.array_equal(out[~moved], sb[~moved])


def test_nv_clamp_prevents_nan():
    ws2 = np.float32(1.0 / 448.0)
    sb = np.array([0x7E, 0x70, 0x40], dtype=np.uint8)
    eff = codec.E4M3_TABLE[sb] * float(ws2)
    d = (2 * 448 * float(ws2) - eff).astype(np.float32)         # push every block to 2x the ceiling
    out = merge.merge_delta("nv", sb, d, ws2)
    assert np.all(out == 0x7E)
    # without the clamp a non-saturating cast of the grid value is NaN
    q = (eff.astype(np.float32) + d) / ws2
    assert np.all(np.isnan(torch.from_numpy(q.astype(np.float32)).to(torch.float8_e4m3fn).float().numpy()))


def test_mx_rounding_matches_brute_force_log_nearest():
    g = np.random.default_rng(5)
    sb = g.integers(100, 140, size=4000).astype(np.uint8)
    d = (g.standard_normal(4000) * np.ldexp(1.0, sb.astype(int) - 127) * 1.5).astype(np.float32)
    out = merge.merge_delta("mx", sb, d)
    e2 = (np.ldexp(1.0, sb.astype(int) - 127).astype(np.float32) + d).astype(np.float64)
    for n in range(sb.size):
        if e2[n] <= 0:
            assert out[n] == 0
            continue
        l2 = math.log2(e2[n])
        if abs(l2 - math.floor(l2) - 0.5) < 1e-9:
            continue
        best = min(range(-127, 128), key=lambda k: abs(l2 - k))
        assert out[n] == best + 127


def test_nv_rounding_matches_brute_force_grid_search():
    ws2 = np.float32(1.0 / 448.0)
    g = np.random.default_rng(6)
    sb = g.integers(0, 0x7F, size=3000).astype(np.uint8)
    eff = (codec.E4M3_TABLE[sb] * float(ws2)).astype(np.float32)
    d = (g.standard_normal(3000) * 0.3 * np.maximum(eff, 1e-3 * float(ws2))).astype(np.float32)
    out = merge.merge_delta("nv", sb, d, ws2)
    grid = [(b, codec.e4m3_value(b)) for b in range(0x7F)]
    e = (codec.E4M3_TABLE[sb].astype(np.float32) * ws2)
    e2 = (e + d)
    e2 = np.minimum(e2, np.float32(448) * ws2)
    q = (e2 / ws2).astype(np.float64)
    for n in range(sb.size):
        a = abs(q[n])
        dist = [(abs(a - v), b) for b, v in grid]
        m = min(x for x, _ in dist)
        cands = [b for x, b in dist if x == m]
        b = cands[0] if len(cands) == 1 else [c for c in cands if c % 2 == 0][0]
        if q[n] < 0 or (q[n] == 0 and math.copysign(1, q[n]) < 0):
            b |= 0x80
        assert out[n] == b, (n, q[n])


def test_rollback_with_applied_on_grid_delta_is_exact():
    sb = inputs.e8m0_normal_exponents(1002, 64, 128, -6, 1.5)
    d = inputs.relative_jitter(1003, np.ldexp(1.0, sb.astype(int) - 127), 0.8)
    merged = merge.merge_delta("mx", sb, d)
    applied = (np.ldexp(1.0, merged.astype(int) - 127) - np.ldexp(1.0, sb.astype(int) - 127)).astype(np.float32)
    # the difference of two powers of two this close is exact in fp32
    assert np.array_equal(applied.astype(np.float64),
                          np.ldexp(1.0, merged.astype(int) - 127) - np.ldexp(1.0, sb.astype(int) - 127))
    back = merge.merge_delta("mx", merged, -applied)
    assert np.array_equal(back, sb)
    assert (merged != sb).any()


def test_copy_mode_and_idempotence():
    sb = inputs.e4m3_abs_normal(1004, 32, 64)
    src = inputs.e4m3_abs_normal(1005, 32, 64)
    out = merge.merge_copy(sb, src)
    assert np.array_equal(out, src)
    assert np.array_equal(merge.merge_copy(out, src), src)
    ws2 = np.float32(1 / 448)
    once = merge.merge_delta("nv", sb, inputs.relative_jitter(1006, codec.E4M3_TABLE[sb] * float(ws2), 0.3), ws2)
    again = merge.merge_delta("nv", once, np.zeros(once.shape, np.float32), ws2)
    assert np.array_equal(once, again)


def test_nan_bytes_propagate():
    assert merge.merge_delta("mx", np.array([0xFF], np.uint8), np.zeros(1, np.float32))[0] == 0xFF
    assert merge.merge_delta("nv", np.array([0x7F], np.uint8), np.zeros(1, np.float32), 1.0)[0] == 0x7F
