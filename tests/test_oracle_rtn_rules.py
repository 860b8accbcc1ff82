"""Pins for the oracle's deploy-rule re-quantisers and its Philox generator (CPU only).

Pinned against: numpy's own Philox4x64-10 bit generator (an independent
implementation; numpy advances the counter before each block), brute-force
truncation on the E2M1 grid, the fixed-point property the paper states for
truncation and stochastic rounding (an exactly representable value does not
move), unbiasedness of stochastic rounding, the extreme uniforms (0 rounds up,
just below 1 rounds down), and the whole-tensor scale rule written directly."""

import numpy as np
import pytest

from oracle import codec, philox, rtn

GRID = codec.E2M1_TABLE[:8]


@pytest.mark.parametrize("key", [0, 5, 0xDEADBEEFCAFEF00D])
def test_philox_matches_numpy(key):
    bg = np.random.Philox(key=np.array([key, 0], dtype=np.uint64), counter=np.zeros(4, dtype=np.uint64))
    ref = bg.random_raw(4 * 6)
    c = np.arange(1, 7, dtype=np.uint64)
    z = np.zeros_like(c)
    words = philox.philox4x64_10(c, z, z, z, key, 0)
    got = np.stack(words, axis=1).reshape(-1)
    assert np.array_equal(got, ref)


def test_uniforms_window_is_a_slice():
    full = philox.uniforms24(1000, 21)
    assert np.array_equal(philox.uniforms24(301, 21, start=599), full[599:900])


def test_uniforms_are_24_bit_and_uniform():
    u = philox.uniforms24(1 << 16, 11)
    assert u.dtype == np.float32 and np.all(u >= 0) and np.all(u < 1)
    assert np.all((u.astype(np.float64) * 2 ** 24) % 1 == 0)
    assert abs(float(u.mean()) - 0.5) < 0.01
    assert not np.array_equal(u, philox.uniforms24(1 << 16, 12))


def test_rtz_brute_force_and_fixed_points():
    g = np.random.default_rng(3)
    q = np.concatenate([g.uniform(-8, 8, 20000), GRID, -GRID, [np.nan]]).astype(np.float32)
    idx = rtn.e2m1_round_rule(q, rtn.RULE_RTZ)
    for x, i in zip(q.tolist(), idx.tolist()):
        if x != x:
            assert i == 0
            continue
        a = min(abs(x), 6.0)
        assert i == max(k for k in range(8) if GRID[k] <= a)
    on = rtn.e2m1_round_rule(GRID.astype(np.float32), rtn.RULE_RTZ)
    assert np.array_equal(on, np.arange(8))


def test_stochastic_fixed_points_extremes_and_mean():
    on = np.tile(GRID, 100).astype(np.float32)
    for u in (np.zeros(on.size), np.full(on.size, 1 - 2 ** -24), np.random.default_rng(1).random(on.size)):
        assert np.array_equal(rtn.e2m1_round_rule(on, rtn.RULE_STOCHASTIC, u.astype(np.float32)),
                              np.tile(np.arange(8), 100))
    q = np.full(4, 2.5, np.float32)                               # halfway between 2 and 3
    assert np.array_equal(rtn.e2m1_round_rule(q, rtn.RULE_STOCHASTIC, np.zeros(4, np.float32)), [5] * 4)
    assert np.array_equal(rtn.e2m1_round_rule(q, rtn.RULE_STOCHASTIC, np.full(4, 0.999, np.float32)), [4] * 4)
    # unbiased: the mean rounded value approaches |q|
    n = 200000
    for x in (0.3, 1.1, 2.7, 4.9):
        u = philox.uniforms24(n, 7)
        idx = rtn.e2m1_round_rule(np.full(n, x, np.float32), rtn.RULE_STOCHASTIC, u)
        lo = GRID[np.searchsorted(GRID, x, side="right") - 1]
        hi = GRID[np.searchsorted(GRID, x, side="right")]
        sd = (hi - lo) * 0.5 / np.sqrt(n)
        assert abs(float(GRID[idx].mean()) - x) < 5 * sd


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_code_rules_keep_the_block_scales(fmt):
    """RTZ and stochastic only round codes: the scale bytes equal the nearest rule's."""
    W = (np.random.default_rng(4).standard_normal((16, 128)) * 0.02).astype(np.float32)
    W = np.asarray(np.float32(W).view(np.uint32) & 0xFFFF0000, np.uint32).view(np.float32)   # bf16 values
    _, s0, w0 = rtn.quantize(fmt, W, rtn.TIE_EVEN)
    for rule in (rtn.RULE_RTZ, rtn.RULE_STOCHASTIC):
        _, s, w = rtn.quantize_rule(fmt, W, rule, seed=9)
        assert np.array_equal(s, s0) and w == w0


def test_whole_tensor_rule_direct():
    W = (np.random.default_rng(5).standard_normal((8, 96)) * 0.05).astype(np.float32)
    W = np.asarray(W.view(np.uint32) & 0xFFFF0000, np.uint32).view(np.float32)
    c, s, _ = rtn.quantize_rule("mx", W, rtn.RULE_WHOLE_TENSOR)
    amax = float(np.max(np.abs(W)))
    k = int(np.ceil(np.log2(np.float32(amax / np.float32(6.0)))))
    assert np.all(s == k + 127)
    q = W / np.float32(2.0 ** k)
    mag = rtn.e2m1_round_magnitude(q, rtn.TIE_EVEN)
    nib = mag | (np.signbit(W).astype(np.uint8) << 3)
    assert np.array_equal(c, codec.pack_nibbles(nib))
    cn, sn, wn = rtn.quantize_rule("nv", W, rtn.RULE_WHOLE_TENSOR)
    assert np.all(sn == sn[0, 0])
    assert sn[0, 0] == codec.e4m3_encode(np.float32(np.float32(amax) / np.float32(6.0)) / wn)


def test_row_offset_matches_the_whole_tensor():
    W = (np.random.default_rng(6).standard_normal((12, 64)) * 0.1).astype(np.float32)
    W = np.asarray(W.view(np.uint32) & 0xFFFF0000, np.uint32).view(np.float32)
    c, s, _ = rtn.quantize_rule("mx", W, rtn.RULE_STOCHASTIC, seed=8)
    c7, s7, _ = rtn.quantize_rule("mx", W[7:9], rtn.RULE_STOCHASTIC, seed=8, row0=7)
    assert np.array_equal(c7, c[7:9]) and np.array_equal(s7, s[7:9])
