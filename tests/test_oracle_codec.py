"""Pins for the oracle's element codecs (CPU only).

Each check ties the oracle to something other than itself: the value tables the
paper prints, torch's own float8 decoders, exhaustive enumeration, and two
independent exact rounding methods."""

import math

import numpy as np
import pytest
import torch

from conftest import read_golden
from oracle import codec


def test_e2m1_value_set_matches_paper():
    _, bare = read_golden("e2m1_values.txt")
    paper = sorted(bare[0])
    mags = sorted(set(abs(v) for v in codec.E2M1_TABLE))
    assert mags == paper
    # sign bit: nibble n+8 is the negative of nibble n
    for n in range(8):
        assert codec.E2M1_TABLE[n + 8] == -codec.E2M1_TABLE[n]
        assert codec.E2M1_TABLE[n] >= 0
    # magnitude increases with the 3-bit index (the order the RTN grid relies on)
    assert all(np.diff(codec.E2M1_TABLE[:8]) > 0)


def test_nibble_pack_roundtrip_and_order():
    nib = np.arange(16, dtype=np.uint8).reshape(2, 8)
    packed = codec.pack_nibbles(nib)
    assert packed[0, 0] == (0 | (1 << 4))          # low nibble = even column
    assert np.array_equal(codec.unpack_nibbles(packed), nib)


def test_e4m3_decode_matches_torch_all_bytes():
    t = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ours = codec.E4M3_TABLE
    assert np.array_equal(np.isnan(t), np.isnan(ours))
    ok = ~np.isnan(t)
    assert np.array_equal(t[ok], ours[ok])


def test_e4m3_grid_count_and_max_match_paper():
    rows, _ = read_golden("formats.txt")
    finite = codec.E4M3_TABLE[np.isfinite(codec.E4M3_TABLE)]
    assert len(set(v for v in finite if v > 0)) == int(rows["e4m3_positive_finite"][0])
    assert finite.max() == rows["e4m3_max"][0]
    assert codec.BLOCK["nv"] == int(rows["nv_block"][0])
    assert codec.BLOCK["mx"] == int(rows["mx_block"][0])


def test_e8m0_decode_matches_torch_all_bytes():
    dt = getattr(torch, "float8_e8m0fnu", None)
    if dt is None:
        pytest.skip("torch lacks float8_e8m0fnu")
    t = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(dt).to(torch.float64).numpy()
    ours = codec.E8M0_TABLE
    assert np.array_equal(np.isnan(t), np.isnan(ours))
    ok = ~np.isnan(t)
    assert np.array_equal(t[ok], ours[ok])


def _e4m3_sweep():
    pos = codec.E4M3_TABLE[:0x7F]
    mids = (pos[:-1] + pos[1:]) / 2
    mids32 = mids.astype(np.float32)
    below = np.nextafter(mids32, np.float32(0))
    above = np.nextafter(mids32, np.float32(np.inf))
    rnd = np.random.default_rng(7).uniform(0, 463, size=20000).astype(np.float32)
    tiny = np.random.default_rng(8).uniform(0, 2.0 ** -6, size=5000).astype(np.float32)
    x = np.concatenate([pos.astype(np.float32), mids32, below, above, rnd, tiny])
    return np.concatenate([x, -x])


def test_e4m3_encoder_matches_torch_cast_in_range():
    # torch's cast is round-to-nearest-even and non-saturating; below 464 it cannot overflow.
    x = _e4m3_sweep()
    x = x[np.abs(x) < 464]
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codec.e4m3_encode(x), t)


def test_e4m3_encoder_saturates_where_cast_gives_nan():
    x = np.array([465.0, 500.0, 1e6, np.inf], dtype=np.float32)
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float32).numpy()
    assert np.all(np.isnan(t))                   # the NaN the paper's clamp prevents
    assert np.all(codec.e4m3_encode(x) == 0x7E)  # saturating: 448
    assert np.all(codec.e4m3_encode(-x) == 0xFE)
    assert codec.e4m3_encode(np.array([np.nan], np.float32))[0] == 0x7F


def test_e4m3_encoder_fixed_points():
    b = np.array([i for i in range(256) if i not in (0x7F, 0xFF)], dtype=np.uint8)
    assert np.array_equal(codec.e4m3_encode(codec.E4M3_TABLE[b].astype(np.float32)), b)


def test_e8m0_encoder_fixed_points():
    k = np.arange(-127, 128)
    x = np.ldexp(1.0, k).astype(np.float32)          # 2**-127 is an fp32 subnormal, still exact
    assert np.array_equal(codec.e8m0_encode_log(x), (k + 127).astype(np.uint8))


def test_e8m0_encoder_matches_fp64_log2_away_from_midpoints():
    g = np.random.default_rng(3)
    x = np.exp2(g.uniform(-120, 120, size=50000)).astype(np.float32)
    l2 = np.log2(x.astype(np.float64))
    frac = l2 - np.floor(l2)
    keep = np.abs(frac - 0.5) > 1e-9
    ref = np.clip(np.rint(l2[keep]), -127, 127) + 127
    assert np.array_equal(codec.e8m0_encode_log(x[keep]), ref.astype(np.uint8))


def test_e8m0_encoder_two_exact_methods_agree():
    """Method A (the oracle): m*m > 2 in fp64.  Method B: the fp32 mantissa field
    compared with the first field value above sqrt(2): fp32(sqrt 2) = 0x3FB504F3 is
    below sqrt 2, so the threshold is field >= 0x3504F4."""
    g = np.random.default_rng(11)
    fields = np.concatenate([
        np.arange(0x3504F4 - 4096, 0x3504F4 + 4096, dtype=np.uint32),
        g.integers(0, 1 << 23, size=50000, dtype=np.uint32),
    ])
    exps = g.integers(1, 250, size=fields.size, dtype=np.uint32)    # normal fp32 exponents
    bits = (exps << 23) | fields
    x = bits.view(np.float32)
    k = exps.astype(np.int64) - 127 + (fields >= 0x3504F4)
    ref = (np.clip(k, -127, 127) + 127).astype(np.uint8)
    assert np.array_equal(codec.e8m0_encode_log(x), ref)
    # the threshold itself, checked against sqrt(2) in exact integer arithmetic:
    # m = 1 + field/2^23 > sqrt 2  <=>  (2^23 + field)^2 > 2 * 2^46
    assert (2 ** 23 + 0x3504F4) ** 2 > 2 * 2 ** 46 > (2 ** 23 + 0x3504F3) ** 2


def test_e8m0_encoder_special_values():
    x = np.array([0.0, -1.0, np.inf, np.nan, 1e-45, 3.0e38], dtype=np.float32)
    out = codec.e8m0_encode_log(x)
    assert list(out) == [0x00, 0x00, 0xFE, 0xFF, 0x00, 0xFE]
    # linear-domain rounding would send 1.45 up (nearest of 1 and 2); the log rule keeps it at 1
    assert codec.e8m0_encode_log(np.array([1.40, 1.45, 1.5], np.float32)).tolist() == [127, 128, 128]
    assert codec.e8m0_encode_log(np.array([1.414], np.float32))[0] == 127
