"""Pins for the oracle's dequant / forward / dX / dS (CPU only).

The paper prints no tensor values for the layer, so the oracle is pinned by
(1) brute force from the storage equation on tiny layers, written with its own
nibble extraction and scale decoding, (2) finite differences of a scalar loss
with respect to every block scale (Y is linear in the scales, so central
differences are exact up to fp64 rounding), and (3) the exact homogeneity
identity sum(eff * dS) = <dY, Y> = <X, dX> (Euler's relation for a function
linear in eff, and the adjoint relation between forward and dX)."""

import numpy as np
import pytest

from conftest import read_golden
from oracle import codec, linear
from paper_2609_04526_amd import inputs


def _paper_e2m1():
    _, bare = read_golden("e2m1_values.txt")
    mags = bare[0]                     # ascending magnitudes, index = low 3 bits
    return [m for m in mags] + [-m for m in mags]


def _brute_weight(fmt, codes, sbytes, ws2):
    """W from the storage equation with independent decoding (pure Python)."""
    e2m1 = _paper_e2m1()
    O, half = codes.shape
    I = 2 * half
    block = 32 if fmt == "mx" else 16
    W = [[0.0] * I for _ in range(O)]
    for o in range(O):
        for i in range(I):
            byte = int(codes[o][i // 2])
            nib = byte % 16 if i % 2 == 0 else byte // 16
            sb = int(sbytes[o][i // block])
            if fmt == "mx":
                s = 2.0 ** (sb - 127)
            else:
                sign = -1.0 if sb >= 128 else 1.0
                e, m = (sb // 8) % 16, sb % 8
                s = sign * (m / 8 * 2.0 ** -6 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)) * ws2
            W[o][i] = e2m1[nib] * s
    return W


def _tiny(fmt, T, O, I, seed):
    G = I // (32 if fmt == "mx" else 16)
    X = inputs.bf16_normal(seed, (T, I)).double().numpy()
    dY = inputs.bf16_normal(seed + 1, (T, O)).double().numpy()
    codes = inputs.codes_uniform(seed + 2, O, I)
    if fmt == "mx":
        sb = inputs.e8m0_uniform_exponents(seed + 3, O, G, -8, -3)
        ws2 = 1.0
    else:
        sb = inputs.e4m3_abs_normal(seed + 3, O, G)
        ws2 = float(np.float32(1.0 / 448.0))
    return X, dY, codes, sb, ws2


@pytest.mark.parametrize("fmt,T,O,I", [("mx", 3, 5, 64), ("nv", 4, 3, 48), ("mx", 1, 1, 32)])
def test_brute_force_tiny(fmt, T, O, I):
    X, dY, codes, sb, ws2 = _tiny(fmt, T, O, I, 100)
    Wb = _brute_weight(fmt, codes, sb, ws2)
    W = linear.dequant(fmt, codes, sb, ws2)
    assert np.array_equal(W, np.array(Wb))
    Y = linear.forward(X, W)
    dX = linear.backward_dx(dY, W)
    dS = linear.backward_dscale(fmt, X, dY, codes)
    block = 32 if fmt == "mx" else 16
    e2m1 = _paper_e2m1()
    for t in range(T):
        for o in range(O):
            ref = sum(X[t][i] * Wb[o][i] for i in range(I))
            assert Y[t, o] == pytest.approx(ref, rel=1e-12, abs=1e-14)
        for i in range(I):
            ref = sum(dY[t][o] * Wb[o][i] for o in range(O))
            assert dX[t, i] == pytest.approx(ref, rel=1e-12, abs=1e-14)
    for o in range(O):
        for b in range(I // block):
            ref = 0.0
            for j in range(b * block, (b + 1) * block):
                byte = int(codes[o][j // 2])
                nib = byte % 16 if j % 2 == 0 else byte // 16
                ref += e2m1[nib] * sum(dY[t][o] * X[t][j] for t in range(T))
            assert dS[o, b] == pytest.approx(ref, rel=1e-12, abs=1e-13)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_dscale_equals_finite_differences(fmt):
    T, O, I = 6, 4, 64
    X, dY, codes, sb, ws2 = _tiny(fmt, T, O, I, 200)
    block = codec.BLOCK[fmt]
    c = linear.code_values(codes)
    eff = codec.effective_scales(fmt, sb, ws2)

    def loss(e):
        W = c * np.repeat(e, block, axis=1)
        return float(np.sum(dY * (X @ W.T)))     # L = <dY, Y>, so dL/dY = dY

    dS = linear.backward_dscale(fmt, X, dY, codes)
    for o in range(O):
        for b in range(I // block):
            h = 0.25 * abs(eff[o, b]) + 1e-3
            ep, em = eff.copy(), eff.copy()
            ep[o, b] += h
            em[o, b] -= h
            fd = (loss(ep) - loss(em)) / (2 * h)
            assert fd == pytest.approx(dS[o, b], rel=1e-9, abs=1e-9)
    if fmt == "nv":
        # gradient w.r.t. the E4M3 value v (eff = v * ws2) is dS * ws2
        v = codec.E4M3_TABLE[sb]
        o, b, h = 1, 2, 0.01
        vp, vm = v.copy(), v.copy()
        vp[o, b] += h
        vm[o, b] -= h
        fd = (loss(vp * ws2) - loss(vm * ws2)) / (2 * h)
        assert fd == pytest.approx(dS[o, b] * ws2, rel=1e-9)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_homogeneity_identity(fmt):
    T, O, I = 37, 24, 96
    X, dY, codes, sb, ws2 = _tiny(fmt, T, O, I, 300)
    W = linear.dequant(fmt, codes, sb, ws2)
    Y = linear.forward(X, W)
    dX = linear.backward_dx(dY, W)
    dS = linear.backward_dscale(fmt, X, dY, codes)
    eff = codec.effective_scales(fmt, sb, ws2)
    a = float(np.sum(eff * dS))
    b = float(np.sum(dY * Y))
    c = float(np.sum(X * dX))
    assert a == pytest.approx(b, rel=1e-11)
    assert c == pytest.approx(b, rel=1e-11)


def test_dscale_reads_no_scales_and_is_blockwise():
    """dS must not change when the scale bytes change, and must follow the codes
    block by block: zeroing one block's codes zeroes exactly that dS entry."""
    T, O, I = 5, 3, 64
    X, dY, codes, sb, _ = _tiny("mx", T, O, I, 400)
    dS = linear.backward_dscale("mx", X, dY, codes)
    codes2 = codes.copy()
    codes2[1, 16:32] = 0                     # row 1, columns 32..63 = block 1
    dS2 = linear.backward_dscale("mx", X, dY, codes2)
    assert dS2[1, 1] == 0.0
    mask = np.ones_like(dS, dtype=bool)
    mask[1, 1] = False
    assert np.array_equal(dS[mask], dS2[mask])


def test_llama8b_shape_table_matches_paper_sizes():
    rows, _ = read_golden("llama8b_sizes.txt")
    L = inputs.LLAMA8B_LAYERS
    shapes = inputs.LLAMA8B_LAYER
    assert L * len(shapes) == rows["linears"][0]
    scale_pr = L * sum(o + i // 16 for _, o, i in shapes)
    qlora_pr = L * sum(o + i for _, o, i in shapes)
    assert round(scale_pr / 1e6, 3) == rows["scale_params_per_rank_millions"][0]
    assert round(qlora_pr / 1e6, 3) == rows["qlora_params_per_rank_millions"][0]
    weights = L * sum(o * i for _, o, i in shapes)
    assert weights // 2 == rows["code_plane_mib"][0] * 2 ** 20
    assert weights // 16 == rows["nv_scale_plane_mib"][0] * 2 ** 20
