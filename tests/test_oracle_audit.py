"""Pins for the oracle's rollback and byte audit (CPU only).

Pinned against: exhaustive rollback over every pair of finite E4M3 bytes and
every pair of E8M0 bytes within 24 binades (the exactness argument), the
paper's observation that subtracting the raw training delta instead of the
applied one leaves some bytes off while the applied delta restores all of them
(App. B "Payoff 3"), and brute-force byte / nibble counts."""

import numpy as np

from oracle import audit, codec, merge
from paper_2609_04526_amd import inputs


def test_nv_rollback_exhaustive_pairs():
    finite = np.array([b for b in range(256) if (b & 0x7F) != 0x7F], dtype=np.uint8)
    before = np.repeat(finite, finite.size)
    after = np.tile(finite, finite.size)
    d = audit.applied_delta("nv", before, after)
    # exact: the fp32 difference equals the fp64 one
    assert np.array_equal(d.astype(np.float64), codec.E4M3_TABLE[after] - codec.E4M3_TABLE[before])
    back = audit.rollback("nv", after, d)
    # -0 and +0 hold the same value; every other byte comes back exactly
    same = (back == before) | ((back & 0x7F) == 0) & ((before & 0x7F) == 0)
    assert np.all(same)


def test_mx_rollback_within_24_binades():
    b = np.arange(0, 255, dtype=np.uint8)
    before = np.repeat(b, b.size)
    after = np.tile(b, b.size)
    near = np.abs(before.astype(int) - after.astype(int)) <= 24
    d = audit.applied_delta("mx", before[near], after[near])
    assert np.array_equal(d.astype(np.float64),
                          codec.E8M0_TABLE[after[near]] - codec.E8M0_TABLE[before[near]])
    assert np.array_equal(audit.rollback("mx", after[near], d), before[near])


def test_applied_delta_restores_where_the_raw_delta_does_not():
    """The paper's subtlety: rolling back with the raw training delta leaves bytes off."""
    O, G = 256, 256
    base = inputs.e4m3_abs_normal(301, O, G)
    ws2 = float(np.float32(1.0 / 448.0))
    eff = codec.effective_scales("nv", base, ws2)
    raw = (inputs.rng(302).standard_normal((O, G)) * 0.05 * eff).astype(np.float32)
    merged = merge.merge_delta("nv", base, raw, ws2)
    applied = audit.applied_delta("nv", base, merged)
    assert np.array_equal(audit.rollback("nv", merged, applied), base)
    # the raw delta, converted to the E4M3 value domain, does not undo the rounding
    raw_v = (raw / np.float32(ws2)).astype(np.float32)
    wrong = audit.rollback("nv", merged, raw_v)
    assert np.count_nonzero(wrong != base) > 0
    assert np.count_nonzero(merged != base) > 0


def test_diff_counts_brute_force():
    g = np.random.default_rng(5)
    a = g.integers(0, 256, size=3001).astype(np.uint8)
    b = a.copy()
    idx = g.choice(a.size, 200, replace=False)
    b[idx] ^= g.integers(1, 256, size=200).astype(np.uint8)
    nb = sum(1 for x, y in zip(a.tolist(), b.tolist()) if x != y)
    nn = sum(((x ^ y) & 15 != 0) + ((x ^ y) >> 4 != 0) for x, y in zip(a.tolist(), b.tolist()))
    assert audit.diff_counts(a, b) == (nb, nn)
    assert audit.diff_counts(a, a) == (0, 0)
