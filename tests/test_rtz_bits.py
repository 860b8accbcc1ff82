"""The re-quantiser's round-toward-zero code from the quotient's bits
(e2m1_rtz_code in csrc/sq_rtn.h: bits 22..30 give b = 254 + 2e + f1, the
magnitude index is min(max(b - 252, 0), 7), or 1 for b = 252, and the sign
bit comes from q), emulated on the CPU and compared with the oracle's
toward-zero rounding over every positive and negative fp32 pattern of a
bf16 value, every fp32 value next to each E2M1 grid point, and random fp32
values over the whole exponent range (NaN excluded: the kernel fixes NaN
blocks up separately)."""

import numpy as np

from oracle import rtn


def rtz_code(q):
    u = np.asarray(q, np.float32).view(np.uint32).astype(np.int64)
    b = (u >> 22) & 0x1FF
    m = np.minimum(np.maximum(b - 252, 0), 7) | (b == 252).astype(np.int64)
    return (m | ((u >> 28) & 8)).astype(np.uint8)


def oracle_code(q):
    q = np.asarray(q, np.float32)
    return (rtn.e2m1_round_rule(q, "rtz") | (np.signbit(q).astype(np.uint8) << 3)).astype(np.uint8)


def test_rtz_code_from_bits():
    bf = (np.arange(0, 0x10000, dtype=np.uint32) << 16).view(np.float32)
    grid = np.array([0.5, 1, 1.5, 2, 3, 4, 6, 0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5, 8, 12], np.float32)
    steps = np.arange(-64, 65, dtype=np.int64)
    near = (grid.view(np.uint32).astype(np.int64)[:, None] + steps[None, :]).ravel().astype(np.uint32).view(np.float32)
    g = np.random.default_rng(5)
    rnd = g.integers(0, 1 << 32, 2_000_000, dtype=np.uint64).astype(np.uint32).view(np.float32)
    q = np.concatenate([bf, near, -near, rnd, np.float32([0.0, -0.0, np.inf, -np.inf])])
    q = q[~np.isnan(q)]
    assert np.array_equal(rtz_code(q), oracle_code(q))
